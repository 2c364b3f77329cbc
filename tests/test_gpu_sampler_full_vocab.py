"""GPU parity of the sampling side at the workloads' full vocabulary (V = 16384):
the distribution transform (CFG, temperature, top-k with ties kept, softmax;
Sec. 4.2, where verification runs on full-vocabulary target and proposal rows
and, with guidance, on the fused guided logits) element by element against the
oracle, the replacement draw's underflow fallback (Eq. 5's residual [p - q]_+
all zero in fp32), and fp32 rollouts at V = 16384 with top-k 2000 and 1000,
per-image temperatures 0.3 / 1.5, an lm_head bias N(0, 4^2) and CFG 2.0, token-
and count-identical to the oracle.

Bars: the kept set of each row, the argmax and every draw are decisions and are
compared exactly (the kept set against its definition on the fp32 y = l / tau,
the draw against the oracle's inverse CDF run on the GPU's own p row, so both
take it on the same fp32 values); p itself differs from the oracle only through
the exponential's last-bit rounding (each side's own expf), so it is compared
to 2e-6 relative, or to 2^-126 absolute where exp underflows below fp32's
normal range."""
import zlib

import numpy as np
import pytest

import oracle
import synth
from tests import gpu_util as gu

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

V = 16384


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import paper_2608_18183_amd as P
    P.load_library()
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")


def P():
    import paper_2608_18183_amd
    return paper_2608_18183_amd


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _rows(rng, n, kind):
    """Logits rows of one kind: 'stress' (N(0, 1) plus a shared N(0, 4^2) bias,
    the stress workload's lm_head), 'flat' (N(0, 0.3): near-uniform),
    'cluster' (3000 distinct values 6 + k 2^-19, k < 20000: a span of 0.038,
    a few of the top-k search's 1024 bins over the row's range, each holding
    far more entries than the search ranks at once, so it narrows its range),
    'ties' (3000 entries exactly equal at the top), 'const' (every entry
    equal)."""
    bias = np.random.default_rng(99).normal(0, 4.0, V)
    x = rng.normal(0, 1, (n, V))
    if kind == "stress":
        x = x + bias
    elif kind == "flat":
        x = 0.3 * x
    elif kind == "cluster":
        for r in range(n):
            idx = rng.choice(V, 3000, replace=False)
            x[r, idx] = 6.0 + rng.choice(20000, 3000, replace=False) * 2.0 ** -19
    elif kind == "ties":
        for r in range(n):
            idx = rng.choice(V, 3000, replace=False)
            x[r, idx] = 6.0
    elif kind == "const":
        x[:] = 1.25
    return x.astype(np.float32)


def _oracle_rows(lg, tau, top_k, cfg_scale):
    n = lg.shape[0]
    p = np.empty((n, V), dtype=np.float32)
    am = np.empty(n, dtype=np.int64)
    for r in range(n):
        g = oracle.cfg_combine(lg[r, 0], lg[r, 1], cfg_scale) if lg.shape[1] == 2 else lg[r, 0]
        am[r] = oracle.argmax(g)
        p[r] = oracle.transform(g, float(tau[r]), top_k)
    return p, am


@pytest.mark.parametrize("kind,top_k,cfg", [("stress", 2000, 0.0), ("stress", 1000, 2.0),
                                            ("flat", 2000, 0.0), ("flat", 0, 2.0),
                                            ("cluster", 2000, 0.0), ("ties", 2000, 0.0),
                                            ("ties", 3500, 2.0), ("const", 1000, 0.0),
                                            ("stress", 1, 0.0), ("stress", V - 1, 0.0)])
def test_transform_rows_match_oracle(kind, top_k, cfg):
    rng = np.random.default_rng(zlib.crc32(f"{kind} {top_k} {cfg}".encode()))
    n = 96
    ncfg = 2 if cfg else 1
    lg = np.stack([_rows(rng, n, kind) for _ in range(ncfg)], axis=1)   # [n, cfg, V]
    if kind == "ties" and cfg:
        lg[:, 1] = lg[:, 0]          # guided = conditional: the ties survive the combine
    tau = np.where(np.arange(n) % 2 == 0, 0.3, 1.5).astype(np.float32)
    pos = rng.integers(1, 600, n).astype(np.int32)
    seed = 4321
    gp, ga, gd = P().hbsjd_transform_rows(_dev(lg if cfg else lg[:, 0]), _dev(tau), _dev(pos),
                                          top_k=top_k, cfg_scale=cfg, seed=seed)
    gp, ga, gd = gp.cpu().numpy(), ga.cpu().numpy(), gd.cpu().numpy()
    rp, ra = _oracle_rows(lg, tau, top_k, cfg)
    # the kept set by its definition: y >= the top_k-th largest y, ties kept
    g = lg[:, 0] if not cfg else np.stack([oracle.cfg_combine(lg[r, 0], lg[r, 1], cfg)
                                           for r in range(n)])
    y = g / tau[:, None]
    kept = np.ones_like(y, dtype=bool)
    if 0 < top_k < V:
        kept = y >= -np.sort(-y, axis=1)[:, top_k - 1:top_k]
    assert not np.any((gp > 0) & ~kept) and not np.any((rp > 0) & ~kept)
    # every kept entry is positive unless exp underflows below fp32's normal
    # range, where each side's exp may round or flush differently
    normal = np.float32(2.0 ** -126)
    assert np.all(gp[kept & (rp >= normal)] > 0)
    if 0 < top_k < V and kind not in ("ties", "const"):
        assert np.all(kept.sum(1) == top_k)
    if kind == "ties":
        assert np.all(kept.sum(1) == max(top_k, 3000))
    np.testing.assert_allclose(gp, rp, rtol=2e-6, atol=normal)
    assert np.array_equal(ga, ra)
    same = 0
    for r in range(n):
        u = oracle.uniforms(seed, r, int(pos[r]))[0]
        assert gd[r] == oracle.inv_cdf(gp[r], u), r
        same += gd[r] == oracle.inv_cdf(rp[r], u)
    assert same >= n - 1


def test_transform_rows_argument_errors():
    lg = torch.zeros((4, 2, 64), dtype=torch.float32, device="cuda")
    tau = torch.ones(4, dtype=torch.float32, device="cuda")
    pos = torch.ones(4, dtype=torch.int32, device="cuda")
    for kw, bad in [(dict(top_k=-1), lg), (dict(), lg[:, :, :62].contiguous())]:
        with pytest.raises(P().HbsjdError) as ei:
            P().hbsjd_transform_rows(bad, tau, pos, **kw)
        assert ei.value.code == "EINVAL"
    nan = lg.clone()
    nan[2, 0, 5] = float("nan")
    with pytest.raises(P().HbsjdError) as ei:
        P().hbsjd_transform_rows(nan, tau, pos, cfg_scale=2.0)
    assert ei.value.code == "EINVAL"


def test_verify_residual_underflow_falls_back_to_p():
    """A rejected draft whose proposal covers p everywhere (q = p, with q(z)
    one ulp above p(z)): [p - q]_+ is zero in fp32, so the replacement is drawn
    from p (reading 7). Also rows at V = 16384 with q = p elsewhere and a
    point-mass proposal: the same code as the rollout's verification."""
    rng = np.random.default_rng(7)
    B, W = 24, 3
    p = rng.random((B, W, V)).astype(np.float32) ** 3
    p /= p.sum(-1, keepdims=True)
    drafts = rng.integers(0, V, (B, W)).astype(np.int32)
    q = p.copy()
    ua = np.zeros((B, W), dtype=np.float32)
    top = np.float32(1.0 - 2.0 ** -24)          # the largest u: any P/Q < 1 rejects
    for b in range(B):
        z = drafts[b, 1]
        q[b, 1, z] = np.nextafter(p[b, 1, z], np.float32(1.0))
        if b % 2:
            ua[b, 1] = top                      # rejected with an all-zero residual
        elif b % 4 == 0:                        # draft 3 has a point-mass proposal
            q[b, 2] = 0
            q[b, 2, drafts[b, 2]] = 1.0
            ua[b, 2] = top
    ur = rng.random(B).astype(np.float32)
    rc, rt = oracle.verify_probs(p, q, drafts, ua, ur)
    gc, gt = P().hbsjd_verify_probs(_dev(p), _dev(q), _dev(drafts), _dev(ua), _dev(ur))
    assert np.array_equal(gc.cpu().numpy(), rc)
    assert np.array_equal(gt.cpu().numpy(), rt)
    assert (rc[1::2] == 2).all() and (rc[::2] == 3).all(), rc
    for b in range(1, B, 2):                    # the underflow fallback was taken
        assert rt[b, 1] == oracle.inv_cdf(p[b, 1], ur[b])
    for b in range(0, B, 4):                    # the point-mass residual removes z
        assert rt[b, 2] != drafts[b, 2]


# ------------------------------------------------------------------ fp32 rollouts at V = 16384


def _full_vocab_workload(B=8):
    shape = synth.ModelShape(2, 64, 1, 128, V, 10, 8, has_lm_bias=True)
    return synth.Workload("fullvocab", shape, "f32", B, 8, 24, 2000, 2.0, bias_std=4.0,
                          prefix_lo=0, prefix_hi=32, temperature="alt0.3/1.5")


@pytest.mark.parametrize("top_k,cfg,W", [(2000, 2.0, 8), (1000, 2.0, 6), (2000, 0.0, 12)])
def test_rollout_f32_full_vocab_equals_oracle(top_k, cfg, W):
    wl = _full_vocab_workload()
    shape = wl.model
    blob = synth.make_weights(shape, 0, std=wl.weight_std, bias_std=wl.bias_std)
    om = oracle.Model(shape, blob)
    batch = synth.make_batch(wl, 1)
    batch.prefix_len[3] = shape.T - 2
    ctx = gu.make_ctx(shape, "f32", blob)
    g = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                          batch.temperature, W, history=wl.history, top_k=top_k,
                          cfg_scale=cfg, seed=2024, exec_mode=P().EXEC_AUTO, gamma=3)
    o = om.rollout(batch, W=W, H=wl.history, top_k=top_k, cfg_scale=cfg, seed=2024,
                   exec_mode=2, gamma=3)
    assert np.array_equal(g["tokens"].cpu().numpy(), o["tokens"])
    assert np.array_equal(g["counts"].cpu().numpy(), o["counts"])
    assert g["verified"] == o["verified"] and g["rejected"] == o["rejected"]
    assert o["rejected"] > 0
