"""Power of the output-law statistic that the bf16 GPU rollouts are held to
(law_util.chi2_against_law at the tiny V 64, T 4 model, Sec. 3.1, Eq. 2).

On the oracle's own rollouts (bf16-rounded weights, fp32 arithmetic) the
statistic passes, and each mistake planted in the acceptance rule (Sec. 4.2,
Eq. 5) fails it by a wide margin, at a quarter of the GPU tests' draws."""
import numpy as np
import pytest

import oracle
import synth
from tests import law_util as lu

N = 16384


@pytest.fixture(scope="module")
def om():
    shape, blob = lu.law_model()
    return shape, oracle.Model(shape, synth.bf16_rounded_blob(shape, blob))


def _run(om, case, sync=False, debug=0):
    shape, m = om
    c = lu.CASES[case]
    k = len(c["prefix"])
    law, _, _ = lu.exact_law(m, shape, 1, c["prefix"], c["top_k"], c["tau"], c["cfg"])
    pre = np.zeros((N, shape.T), dtype=np.int32)
    pre[:, :k] = c["prefix"]
    b = synth.Batch(pre, np.full(N, k, dtype=np.int32), np.full(N, 1, dtype=np.int32),
                    np.full(N, c["tau"], dtype=np.float32))
    oracle.set_debug(debug)
    try:
        r = m.rollout(b, W=c["W"], H=c["H"], top_k=c["top_k"], cfg_scale=c["cfg"], seed=4242,
                      exec_mode=1, sync=sync)
    finally:
        oracle.set_debug(0)
    return r, law, k, shape.vocab


@pytest.mark.parametrize("case,sync", [("full_vocab_cfg", False), ("top3", False),
                                       ("top3", True)])
def test_oracle_rollouts_pass_the_law_statistic(om, case, sync):
    r, law, k, V = _run(om, case, sync)
    pv, cells = lu.chi2_against_law(r["tokens"], k, law, V)
    assert pv > 1e-3 and cells >= 50, (pv, cells)
    assert r["counts"].max() > 1 and r["rejected"] > 0
    assert lu.waited(r["counts"]) == sync


@pytest.mark.parametrize("case", ["full_vocab_cfg", "top3"])
@pytest.mark.parametrize("flag", [oracle.DEBUG_RESIDUAL_DROPS_Q, oracle.DEBUG_INVERTED_RATIO])
def test_planted_acceptance_mistakes_fail_the_law_statistic(om, case, flag):
    r, law, k, V = _run(om, case, debug=flag)
    try:
        pv, _ = lu.chi2_against_law(r["tokens"], k, law, V)
    except AssertionError:   # a draw outside the support
        pv = 0.0
    assert pv < 1e-6, pv


def test_exact_law_is_a_distribution_with_the_expected_support(om):
    shape, m = om
    for case, size in [("full_vocab_cfg", 64 ** 2), ("top3", 3 ** 4)]:
        c = lu.CASES[case]
        law, contexts, gap = lu.exact_law(m, shape, 1, c["prefix"], c["top_k"], c["tau"], c["cfg"])
        assert len(law) == size
        assert abs(sum(law.values()) - 1.0) < 1e-5
        # one context per internal node of the walk (two under guidance)
        inner = sum(len(law) ** (j / (shape.T - len(c["prefix"]))) for j in range(shape.T - len(c["prefix"])))
        assert len(contexts) == round(inner) * (2 if c["cfg"] else 1)
        assert (gap == np.inf) == (c["top_k"] == 0)
