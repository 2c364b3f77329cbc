"""Output law of bf16 rollouts (Sec. 3.1, Eq. 2; Sec. 4.2, Eq. 5).

With the probabilistic acceptance test, speculative Jacobi decoding leaves each
sequence distributed as token-by-token sampling from the model's transformed
distribution (temperature, top-k, guidance). bf16 rollouts cannot be matched
with the fp32 oracle token for token, so these tests check that law instead.

* 65536 images of a tiny bf16 model (V 64, T 4, lm_head bias) share one class
  and one prefix.
  Their independent Philox streams make them independent draws.
* The counts of their generated suffixes go into a chi-square test against the
  exact joint law. The oracle computes that law by walking every suffix in the
  support (bf16-rounded weights, fp32 arithmetic).
* Cells with fewer than 5 expected draws are pooled. A suffix outside the
  oracle's support fails outright.
* The GPU's token-by-token mode (VERIFY_AR) is held to the same law as a control.
* The test's power comes from the same statistic on the oracle: mistakes planted
  in the oracle's acceptance rule fail it there (test_oracle_law_power.py).

Preconditions, asserted: the GPU forward agrees with the oracle at every
context of the walk, and the top-k margin at those contexts is far wider than
that disagreement, so the two sides truncate to the same support."""
import numpy as np
import pytest

import oracle
import synth
from tests import gpu_util as gu
from tests import law_util as lu

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

N_IMAGES = 65536
PVALUE_FLOOR = 1e-3


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import paper_2608_18183_amd as P
    P.load_library()
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")


def P():
    import paper_2608_18183_amd
    return paper_2608_18183_amd


@pytest.fixture(scope="module")
def model():
    shape, blob = lu.law_model()
    om = oracle.Model(shape, gu.bf16_rounded_blob(shape, blob))
    return shape, om, gu.make_ctx(shape, "bf16", blob)


def _forward_agreement(ctx, om, shape, contexts):
    """Max-abs difference of the GPU and oracle logits at the walk's contexts
    (the row that predicts the next token)."""
    toks = np.zeros((len(contexts), shape.T), dtype=np.int32)
    for i, (_, seq) in enumerate(contexts):
        toks[i, :len(seq)] = seq
    lens = [len(seq) for _, seq in contexts]
    labels = [c for c, _ in contexts]
    got = ctx.hbsjd_forward(torch.from_numpy(toks).cuda(), lens, labels).cpu().numpy()
    ref = np.concatenate(om.forward_batch(labels, [seq for _, seq in contexts]))
    last = np.cumsum(np.asarray(lens) + 1) - 1
    return float(np.abs(got[last].astype(np.float64) - ref[last]).max())


@pytest.mark.parametrize("case,progress,verify",
                         [("full_vocab_cfg", "independent", "prob"),
                          ("top3", "sync", "prob"),
                          ("full_vocab_cfg", "independent", "ar"),
                          ("top3", "independent", "prob"),
                          ("top3", "independent", "ar")])
def test_bf16_rollout_law_matches_exact_law(model, case, progress, verify):
    shape, om, ctx = model
    c = lu.CASES[case]
    cls, k = 1, len(c["prefix"])
    law, contexts, gap = lu.exact_law(om, shape, cls, c["prefix"], c["top_k"], c["tau"], c["cfg"])
    assert abs(sum(law.values()) - 1.0) < 1e-5
    err = _forward_agreement(ctx, om, shape, contexts)
    assert err < 1e-2, err
    if c["top_k"]:
        # a guided logit moves by at most (|1 - s| + |s|) err
        assert gap > 2 * (abs(1 - c["cfg"]) + abs(c["cfg"])) * err, (gap, err)

    prefix = np.zeros((N_IMAGES, shape.T), dtype=np.int32)
    prefix[:, :k] = c["prefix"]
    batch = synth.Batch(prefix, np.full(N_IMAGES, k, dtype=np.int32),
                        np.full(N_IMAGES, cls, dtype=np.int32),
                        np.full(N_IMAGES, c["tau"], dtype=np.float32))
    out = ctx.hbsjd_rollout(
        gu.device_batch(batch), batch.prefix_len, batch.labels, batch.temperature, c["W"],
        history=c["H"], top_k=c["top_k"], cfg_scale=c["cfg"], seed=4242,
        verify_mode=P().VERIFY_AR if verify == "ar" else P().VERIFY_PROB,
        progress=P().PROGRESS_SYNC if progress == "sync" else P().PROGRESS_INDEPENDENT)
    tok = out["tokens"].cpu().numpy()
    assert np.array_equal(tok[:, :k], prefix[:, :k])
    pv, cells = lu.chi2_against_law(tok, k, law, shape.vocab)
    assert cells >= 50, cells
    assert pv > PVALUE_FLOOR, (pv, cells)
    if verify == "prob":
        # the rollout really speculated: rounds committed several tokens and
        # drafts were rejected
        cnt = out["counts"].cpu().numpy()
        assert cnt.max() > 1 and out["rejected"] > 0
        if progress == "sync":
            assert lu.waited(cnt)   # images waited at the shared boundary at position 3
