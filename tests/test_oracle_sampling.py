"""Pins of the oracle's sampling pieces: Philox against rocRAND, the pinned sum
against exact summation, the inverse CDF against float64 searchsorted, the
transform against float64 softmax, and the verification rule (Sec. 4.2, Eq. 5)
against the speculative-sampling lemma (accept probability sum_v min(p, q);
output distributed as p)."""
import math
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest
from scipy import stats

import oracle
from tests import np_reference as npr

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def rocrand_probe():
    src = os.path.join(HERE, "rocrand_philox_probe.cpp")
    if shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include/rocrand"):
        pytest.skip("rocRAND headers not available")
    d = tempfile.mkdtemp()
    exe = os.path.join(d, "probe")
    subprocess.check_call(["g++", "-O1", "-std=c++17", "-I/opt/rocm/include",
                           "-D__HIP_PLATFORM_AMD__", src, "-o", exe])
    yield exe
    shutil.rmtree(d, ignore_errors=True)


def test_philox_matches_rocrand(rocrand_probe):
    rng = np.random.default_rng(0)
    # rocRAND reaches the second counter word through a 64-bit offset, so t < 2^30 here
    pairs = [(0, 0), (1, 0), (0, 1), (255, 576), (2**31, 7), (2**32 - 1, 2**30 - 1)]
    pairs += [(int(b), int(t) >> 2) for b, t in rng.integers(0, 2**32, size=(20, 2),
                                                           dtype=np.uint64)]
    for seed in [0, 1000, 0xDEADBEEFCAFEF00D, 2**64 - 1]:
        args = [rocrand_probe, str(seed)] + [str(x) for bt in pairs for x in bt]
        lines = subprocess.check_output(args, text=True).strip().splitlines()
        for (b, t), line in zip(pairs, lines):
            ref = [int(x) for x in line.split()]
            got = oracle.philox(seed, [b, t, 0, 0]).tolist()
            assert got == ref, (seed, b, t)


def test_uniforms_are_uniform_and_independent():
    n = 4000
    u = np.array([oracle.uniforms(1234, b % 50, b // 50) for b in range(n)], dtype=np.float64)
    assert u.min() >= 0.0 and u.max() <= 1.0 - 2.0**-24
    # 24-bit grid
    assert np.all(np.floor(u * 2**24) == u * 2**24)
    for c in range(3):
        assert stats.kstest(u[:, c], "uniform").pvalue > 1e-3
    cc = np.corrcoef(u.T)
    assert np.all(np.abs(cc[np.triu_indices(3, 1)]) < 0.06)


@pytest.mark.parametrize("n", [1, 4, 63, 64, 65, 256, 16384, 1000])
def test_pinned_sum_error_bound(n):
    rng = np.random.default_rng(n)
    w = rng.random(n).astype(np.float32)
    s = float(oracle.pinned_sum(w))
    exact = math.fsum(w.astype(np.float64))
    bound = (64 + n // 64 + 2) * 2.0**-24 * float(np.sum(np.abs(w.astype(np.float64))))
    assert abs(s - exact) <= bound
    # integers with an exact fp32 total are summed exactly in any association
    wi = rng.integers(0, 100, size=n).astype(np.float32)
    assert float(oracle.pinned_sum(wi)) == float(np.sum(wi.astype(np.int64)))


def test_inv_cdf_matches_float64_search():
    rng = np.random.default_rng(1)
    checked = 0
    for trial in range(300):
        n = int(rng.integers(1, 400))
        w = rng.random(n).astype(np.float32)
        w[rng.random(n) < 0.3] = 0.0
        if not np.any(w > 0):
            continue
        u = np.float32(rng.random())
        c = np.cumsum(w.astype(np.float64))
        target = float(u) * c[-1]
        # skip targets that sit within rounding distance of a boundary
        if np.min(np.abs(c - target)) < 1e-5 * c[-1]:
            continue
        ref = int(np.searchsorted(c, target, side="right"))
        got = oracle.inv_cdf(w, u)
        assert got == ref, (trial, got, ref)
        assert w[got] > 0
        checked += 1
    assert checked > 200


def test_inv_cdf_edge_cases():
    w = np.array([0, 0, 0.5, 0, 0.25, 0], dtype=np.float32)
    assert oracle.inv_cdf(w, 0.0) == 2
    assert oracle.inv_cdf(w, 1.0 - 2**-24) == 4
    assert oracle.inv_cdf(np.array([0, 0, 3.0], dtype=np.float32), 0.999) == 2
    assert oracle.inv_cdf(np.zeros(5, dtype=np.float32), 0.5) == -1
    # the largest positive entry when rounding leaves u * total at the total
    assert oracle.inv_cdf(np.array([1e-30, 1.0, 0.0], dtype=np.float32), 1.0 - 2**-24) == 1


def test_inv_cdf_frequencies():
    rng = np.random.default_rng(2)
    w = np.array([0.1, 0.0, 0.4, 0.2, 0.3], dtype=np.float32)
    us = rng.random(20000).astype(np.float32)
    counts = np.bincount([oracle.inv_cdf(w, u) for u in us], minlength=5)
    assert counts[1] == 0
    keep = w > 0
    w64 = w[keep].astype(np.float64)
    assert stats.chisquare(counts[keep], 20000 * w64 / w64.sum()).pvalue > 1e-3


@pytest.mark.parametrize("V,tau,k", [(256, 1.0, 0), (1000, 0.7, 50), (16384, 1.0, 2000),
                                     (16384, 0.3, 2000), (16384, 1.5, 1000), (64, 2.0, 64),
                                     (64, 1.0, 1)])
def test_transform_matches_float64_softmax(V, tau, k):
    rng = np.random.default_rng(V + k)
    l = (rng.standard_normal(V) * 3).astype(np.float32)
    p = oracle.transform(l, tau, k).astype(np.float64)
    ref = npr.softmax_topk(l, tau, k)
    assert np.max(np.abs(p - ref)) <= 1e-6
    assert abs(p.sum() - 1.0) <= 1e-5
    if 0 < k < V:
        assert np.count_nonzero(p) == k
        assert set(np.nonzero(p)[0]) == set(np.argsort(-l, kind="stable")[:k])


def test_transform_top_k_keeps_ties_and_large_k_is_off():
    l = np.array([1.0, 3.0, 2.0, 2.0, 2.0, 0.5], dtype=np.float32)
    p = oracle.transform(l, 1.0, 2)        # the 2nd largest value 2.0 is tied three ways
    assert np.count_nonzero(p) == 4 and p[0] == 0 and p[5] == 0
    full = oracle.transform(l, 1.0, 0)
    assert np.array_equal(oracle.transform(l, 1.0, 6), full)
    assert np.array_equal(oracle.transform(l, 1.0, 100), full)
    assert np.all(full > 0)


def test_cfg_combine():
    rng = np.random.default_rng(3)
    lc, lu = rng.standard_normal(100).astype(np.float32), rng.standard_normal(100).astype(np.float32)
    # s = 1 is the conditional branch up to the rounding of (l_c - l_u)
    assert np.max(np.abs(oracle.cfg_combine(lc, lu, 1.0) - lc)) <= 4 * 2.0**-24 * 8
    assert np.array_equal(oracle.cfg_combine(lc, lu, 0.0), lu)
    ref = lu.astype(np.float64) + 2.0 * (lc.astype(np.float64) - lu)
    assert np.max(np.abs(oracle.cfg_combine(lc, lu, 2.0) - ref)) < 1e-5


def _lemma_run(p, q, n, seed):
    """n independent single-draft verifications of z ~ q against p."""
    rng = np.random.default_rng(seed)
    V = p.size
    q64 = q.astype(np.float64)
    z = rng.choice(V, size=n, p=q64 / q64.sum())
    P = np.broadcast_to(p, (n, 1, V))
    Q = np.broadcast_to(q, (n, 1, V))
    ua = rng.random((n, 1)).astype(np.float32)
    ur = rng.random(n).astype(np.float32)
    counts, toks = oracle.verify_probs(P, Q, z[:, None], ua, ur)
    accepted = toks[:, 0] == z
    return counts, toks[:, 0], accepted, z


def _rand_dist(rng, V, zeros=0):
    x = rng.random(V) ** 3
    if zeros:
        x[rng.choice(V, zeros, replace=False)] = 0
    return (x / x.sum()).astype(np.float32)


def test_verify_accept_probability_closed_form():
    rng = np.random.default_rng(4)
    for trial in range(3):
        p, q = _rand_dist(rng, 8, zeros=2), _rand_dist(rng, 8, zeros=1)
        n = 40000
        counts, toks, acc, z = _lemma_run(p, q, n, trial)
        assert np.all(counts == 1)
        pa = float(np.minimum(p, q).sum())          # 1 - TV(p, q)
        sigma = math.sqrt(pa * (1 - pa) / n)
        # acceptance is decided by the ratio test, measure it from the uniforms' side
        assert abs(acc.mean() - pa) < 5 * sigma + 1e-3


def _output_pvalue(p, toks):
    V = p.size
    obs = np.bincount(toks, minlength=V)
    keep = p > 0
    p64 = p[keep].astype(np.float64)
    exp = len(toks) * p64 / p64.sum()
    extra = obs[~keep].sum()
    if extra:
        return 0.0
    return stats.chisquare(obs[keep], exp).pvalue


def test_verify_output_is_distributed_as_p():
    rng = np.random.default_rng(5)
    for trial in range(3):
        p, q = _rand_dist(rng, 6, zeros=1), _rand_dist(rng, 6, zeros=1)
        _, toks, _, _ = _lemma_run(p, q, 60000, 10 + trial)
        assert _output_pvalue(p, toks) > 1e-4


def test_verify_point_mass_proposal():
    """A history draft has q = delta_z: accepted with probability p(z), else a
    draw from p with z removed."""
    rng = np.random.default_rng(6)
    p = _rand_dist(rng, 7)
    zt = 3
    q = np.zeros(7, dtype=np.float32)
    q[zt] = 1.0
    n = 40000
    counts, toks, acc, z = _lemma_run(p, q, n, 7)
    assert np.all(z == zt)
    sigma = math.sqrt(p[zt] * (1 - p[zt]) / n)
    assert abs(acc.mean() - p[zt]) < 5 * sigma
    assert _output_pvalue(p, toks) > 1e-4


@pytest.mark.parametrize("flag", [oracle.DEBUG_RESIDUAL_DROPS_Q, oracle.DEBUG_INVERTED_RATIO])
def test_planted_verify_mistakes_are_caught(flag):
    rng = np.random.default_rng(5)
    p, q = _rand_dist(rng, 6, zeros=1), _rand_dist(rng, 6, zeros=1)
    oracle.set_debug(flag)
    try:
        _, toks, _, _ = _lemma_run(p, q, 60000, 10)
    finally:
        oracle.set_debug(0)
    assert _output_pvalue(p, toks) < 1e-6


def test_verify_deterministic_cases():
    rng = np.random.default_rng(8)
    B, W, V = 5, 4, 50
    p = np.stack([[_rand_dist(rng, V) for _ in range(W)] for _ in range(B)])
    drafts = rng.integers(0, V, size=(B, W)).astype(np.int32)
    for b in range(B):
        for j in range(W):
            if p[b, j, drafts[b, j]] == 0:
                p[b, j, drafts[b, j]] = 0.01
    ua = rng.random((B, W)).astype(np.float32)
    ur = rng.random(B).astype(np.float32)
    # q == p: every draft accepted, all W committed
    counts, toks = oracle.verify_probs(p, p, drafts, ua, ur)
    assert np.all(counts == W) and np.array_equal(toks, drafts)
    # q = delta at a token p gives zero mass: rejected at once, replacement from p
    q = np.zeros_like(p)
    p2 = p.copy()
    for b in range(B):
        for j in range(W):
            q[b, j, drafts[b, j]] = 1.0
        p2[b, 0, drafts[b, 0]] = 0.0
    counts, toks = oracle.verify_probs(p2, q, drafts, ua, ur)
    assert np.all(counts == 1)
    for b in range(B):
        assert toks[b, 0] != drafts[b, 0] and p2[b, 0, toks[b, 0]] > 0
        assert np.all(toks[b, 1:] == -1)
