"""GPU parity: the HIP path, called through the C ABI, against the oracle on the
same seeded inputs.

Bars: bit-exact for the RNG, the verification kernel on identical fp32 rows and
uniforms, and the fp32-mode rollout tokens; 3e-2 max-abs / 1e-2 mean-abs for
the logits of a bf16 model (fp16 operands and activations on the GPU) against
the fp32 oracle run on the same bf16-rounded weights."""
import numpy as np
import pytest

import oracle
import synth
from tests import gpu_util as gu

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import paper_2608_18183_amd as P
    P.load_library()
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")


def P():
    import paper_2608_18183_amd
    return paper_2608_18183_amd


# ------------------------------------------------------------------ RNG


def test_philox_matches_oracle():
    rng = np.random.default_rng(0)
    bt = rng.integers(0, 2**31, size=(5000, 2)).astype(np.int32)
    bt[:10] = [[0, 0], [1, 0], [0, 1], [255, 576], [2**31 - 1, 2**31 - 1], [3, 7], [31, 63],
               [100, 1], [0, 575], [4095, 600]]
    for seed in [0, 1000, 0xDEADBEEFCAFEF00D]:
        got = P().hbsjd_philox(seed, torch.from_numpy(bt).cuda()).cpu().numpy().view(np.uint32)
        for i in range(0, 5000, 37):
            ref = oracle.philox(seed, [int(bt[i, 0]), int(bt[i, 1]), 0, 0])
            assert np.array_equal(got[i], ref), (seed, i)


# ------------------------------------------------------------------ verify kernel


def _rand_rows(rng, B, W, V, zero_frac):
    x = rng.random((B, W, V)) ** 4
    x[rng.random((B, W, V)) < zero_frac] = 0.0
    x[..., 0] += 1e-3
    x /= x.sum(-1, keepdims=True)
    return x.astype(np.float32)


@pytest.mark.parametrize("B,W,V,zf", [(64, 8, 256, 0.3), (32, 16, 16384, 0.8), (16, 4, 4, 0.0),
                                      (8, 33, 1000, 0.5), (128, 1, 64, 0.0)])
def test_verify_probs_bit_exact(B, W, V, zf):
    rng = np.random.default_rng(V + W)
    p = _rand_rows(rng, B, W, V, zf)
    q = _rand_rows(rng, B, W, V, zf)
    # some drafts are history drafts with a point-mass proposal, some have q == p
    drafts = np.zeros((B, W), dtype=np.int32)
    for b in range(B):
        for j in range(W):
            kind = (b + j) % 5
            if kind == 0:
                q[b, j] = 0
                drafts[b, j] = rng.integers(0, V)
                q[b, j, drafts[b, j]] = 1.0
            else:
                if kind == 1:
                    q[b, j] = p[b, j]
                qq = q[b, j].astype(np.float64)
                drafts[b, j] = rng.choice(V, p=qq / qq.sum())
    ua = rng.random((B, W)).astype(np.float32)
    ur = rng.random(B).astype(np.float32)
    rc, rt = oracle.verify_probs(p, q, drafts, ua, ur)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    gc, gt = P().hbsjd_verify_probs(T(p), T(q), T(drafts), T(ua), T(ur))
    assert np.array_equal(gc.cpu().numpy(), rc)
    assert np.array_equal(gt.cpu().numpy(), rt)
    assert rc.min() >= 1 and rc.max() <= W


# ------------------------------------------------------------------ forward


def test_forward_f32_tiny_matches_oracle(tiny):
    w, blob, om = tiny
    shape = w.model
    ctx = gu.make_ctx(shape, "f32", blob)
    rng = np.random.default_rng(3)
    lens = [0, 1, 17, 63, 64]
    labels = [0, 3, 9, 10, 5]          # 10 is the null class
    toks = rng.integers(0, shape.vocab, size=(len(lens), shape.T)).astype(np.int32)
    got = ctx.hbsjd_forward(torch.from_numpy(toks).cuda(), lens, labels).cpu().numpy()
    ref = om.forward_batch(labels, [toks[i, :n] for i, n in enumerate(lens)])
    ref = np.concatenate(ref)
    assert got.shape == ref.shape
    err = np.abs(got - ref)
    assert err.max() < 1e-4, err.max()


def _bf16_forward_case(name, lens, seed, atol_max=3e-2, atol_mean=1e-2):
    wl = synth.WORKLOADS[name]
    shape = wl.model
    blob = synth.make_weights(shape, 0, std=wl.weight_std, bias_std=wl.bias_std)
    ctx = gu.make_ctx(shape, "bf16", blob)
    om = oracle.Model(shape, gu.bf16_rounded_blob(shape, blob))
    rng = np.random.default_rng(seed)
    toks = rng.integers(0, shape.vocab, size=(len(lens), shape.T)).astype(np.int32)
    labels = rng.integers(0, shape.n_classes + 1, size=len(lens)).astype(np.int32)
    got = ctx.hbsjd_forward(torch.from_numpy(toks).cuda(), lens, labels).cpu().numpy()
    ref = np.concatenate(om.forward_batch(labels, [toks[i, :n] for i, n in enumerate(lens)]))
    err = np.abs(got.astype(np.float64) - ref)
    print(name, "max", err.max(), "mean", err.mean(), "logit scale", np.abs(ref).max())
    assert err.max() <= atol_max and err.mean() <= atol_mean, (err.max(), err.mean())


def test_forward_bf16_llamagen_b_matches_oracle():
    _bf16_forward_case("llamagen_b", [0, 7, 130], 1)


def test_forward_bf16_stress_shape_with_bias_matches_oracle():
    _bf16_forward_case("stress_b", [200, 3], 2)


def test_forward_bf16_llamagen_xl_matches_oracle():
    _bf16_forward_case("llamagen_xl_cfg", [40, 0, 90], 3)


@pytest.mark.parametrize("n_seq", [12, 44])
def test_forward_bf16_many_rows_matches_oracle(n_seq):
    """Forwards of ~3000 and ~11000 rows: enough tiles that the O and W2
    projections run without a K split, on the 64x64 tile and then on the
    128x128 one (and the other GEMMs on their large-launch variants); sampled
    sequences against the oracle."""
    wl = synth.WORKLOADS["llamagen_b"]
    shape = wl.model
    blob = synth.make_weights(shape, 0, std=wl.weight_std)
    ctx = gu.make_ctx(shape, "bf16", blob)
    rng = np.random.default_rng(21)
    lens = np.full(n_seq, shape.T - 1, dtype=np.int32)
    lens[0], lens[5] = 3, 200
    toks = rng.integers(0, shape.vocab, size=(len(lens), shape.T)).astype(np.int32)
    labels = rng.integers(0, shape.n_classes + 1, size=len(lens)).astype(np.int32)
    got = ctx.hbsjd_forward(torch.from_numpy(toks).cuda(), lens.tolist(), labels).cpu().numpy()
    row0 = np.concatenate([[0], np.cumsum(lens + 1)])
    assert got.shape == (row0[-1], shape.vocab)
    om = oracle.Model(shape, gu.bf16_rounded_blob(shape, blob))
    pick = [0, 5, n_seq - 1]
    ref = om.forward_batch(labels[pick], [toks[i, :lens[i]] for i in pick])
    for i, r in zip(pick, ref):
        err = np.abs(got[row0[i]:row0[i + 1]].astype(np.float64) - r)
        assert err.max() <= 3e-2 and err.mean() <= 1e-2, (i, err.max(), err.mean())


@pytest.mark.parametrize("d,f", [(64, 64), (128, 320), (192, 256)])
def test_forward_bf16_short_contractions_match_oracle(d, f):
    """Contractions of 1 to 5 64-deep K steps (K = d, f): fewer steps than the
    GEMM keeps in flight, exactly as many, and a few more."""
    shape = synth.small_shape(n_layers=2, d_model=d, n_heads=d // 64, mlp_hidden=f, vocab=1024,
                              n_classes=10, grid=8)
    blob = synth.make_weights(shape, 0, std=0.03)
    ctx = gu.make_ctx(shape, "bf16", blob)
    om = oracle.Model(shape, gu.bf16_rounded_blob(shape, blob))
    rng = np.random.default_rng(d)
    lens = [0, 5, 40, 63, 17]
    toks = rng.integers(0, shape.vocab, size=(len(lens), shape.T)).astype(np.int32)
    labels = rng.integers(0, shape.n_classes + 1, size=len(lens)).astype(np.int32)
    got = ctx.hbsjd_forward(torch.from_numpy(toks).cuda(), lens, labels).cpu().numpy()
    ref = np.concatenate(om.forward_batch(labels, [toks[i, :n] for i, n in enumerate(lens)]))
    err = np.abs(got.astype(np.float64) - ref)
    assert err.max() <= 3e-2 and err.mean() <= 1e-2, (err.max(), err.mean())


# ------------------------------------------------------------------ rollouts


def _run_both(w, blob, om, batch, seed, W, mode, gamma=2, top_k=0, greedy=False, H=24,
              dtype="f32", cfg=0.0):
    ctx = gu.make_ctx(w.model, dtype, blob)
    g = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                          batch.temperature, W, history=H, top_k=top_k, cfg_scale=cfg, seed=seed,
                          verify_mode=P().VERIFY_GREEDY if greedy else P().VERIFY_PROB,
                          exec_mode=mode, gamma=gamma)
    o = om.rollout(batch, W=W, H=H, top_k=top_k, cfg_scale=cfg, seed=seed, greedy=greedy,
                   exec_mode={P().EXEC_FULL: 0, P().EXEC_COMPACT: 1, P().EXEC_AUTO: 2}[mode],
                   gamma=gamma)
    return g, o


@pytest.mark.parametrize("seed", [1000, 1001, 1002])
@pytest.mark.parametrize("mode", ["full", "compact", "auto"])
def test_rollout_f32_tiny_equals_oracle(tiny, seed, mode):
    w, blob, om = tiny
    batch = synth.make_batch(w, 1)
    m = {"full": P().EXEC_FULL, "compact": P().EXEC_COMPACT, "auto": P().EXEC_AUTO}[mode]
    g, o = _run_both(w, blob, om, batch, seed, w.window, m)
    assert np.array_equal(g["tokens"].cpu().numpy(), o["tokens"])
    assert g["rounds"] == o["rounds"]
    assert np.array_equal(g["counts"].cpu().numpy(), o["counts"])
    assert np.array_equal(g["active"], o["active"])
    assert g["verified"] == o["verified"] and g["rejected"] == o["rejected"]


@pytest.mark.parametrize("W,top_k,greedy,H", [(1, 0, False, 24), (16, 0, False, 24),
                                               (4, 20, False, 3), (8, 0, True, 24),
                                               (3, 5, False, 1)])
def test_rollout_f32_tiny_variants_equal_oracle(tiny, W, top_k, greedy, H):
    w, blob, om = tiny
    batch = synth.make_batch(w, 7)
    batch.prefix_len[2] = w.model.T        # one image with nothing to generate
    batch.temperature[:] = [1.0, 0.7, 1.3, 2.0]
    g, o = _run_both(w, blob, om, batch, 55, W, P().EXEC_AUTO, top_k=top_k, greedy=greedy, H=H)
    assert np.array_equal(g["tokens"].cpu().numpy(), o["tokens"])
    assert np.array_equal(g["counts"].cpu().numpy(), o["counts"])


def test_rollout_f32_cfg_equals_oracle():
    shape = synth.small_shape(n_layers=2, d_model=32, n_heads=2, mlp_hidden=48, vocab=64,
                              n_classes=4, grid=4)
    blob = synth.make_weights(shape, 3, std=0.2)
    om = oracle.Model(shape, blob)
    w = synth.Workload("t", shape, "f32", 6, 3, 2, 7, 2.0, prefix_lo=0, prefix_hi=9)
    batch = synth.make_batch(w, 5)
    g, o = _run_both(w, blob, om, batch, 77, 3, P().EXEC_AUTO, top_k=7, H=2, cfg=2.0)
    assert np.array_equal(g["tokens"].cpu().numpy(), o["tokens"])
    assert np.array_equal(g["counts"].cpu().numpy(), o["counts"])


@pytest.mark.parametrize("case", ["single_image", "all_complete", "window_past_end"])
def test_rollout_f32_edge_cases_equal_oracle(tiny, case):
    """Degenerate batches against the oracle: one image; every image already
    complete (no round runs); a window far longer than what is left."""
    w, blob, om = tiny
    T = w.model.T
    if case == "single_image":
        batch = synth.make_batch(w, 4, batch=1)
        W = w.window
    elif case == "all_complete":
        batch = synth.make_batch(w, 5)
        batch.prefix_len[:] = T
        W = w.window
    else:
        batch = synth.make_batch(w, 6)
        batch.prefix_len[:] = [T - 1, T - 3, T - 2, 0]
        W = 40
    g, o = _run_both(w, blob, om, batch, 321, W, P().EXEC_AUTO)
    assert np.array_equal(g["tokens"].cpu().numpy(), o["tokens"])
    assert g["rounds"] == o["rounds"]
    assert np.array_equal(g["counts"].cpu().numpy(), o["counts"])
    if case == "all_complete":
        assert g["rounds"] == 0
        assert np.array_equal(g["tokens"].cpu().numpy(), batch.prefix_tokens)


def test_rollout_bf16_full_equals_compact_and_counts_are_bounded():
    wl = synth.WORKLOADS["llamagen_b"]
    shape = wl.model
    blob = synth.make_weights(shape, 0)
    batch = synth.make_batch(wl, 1, batch=8)
    batch.prefix_len[3] = shape.T - 5
    outs = []
    ctx = gu.make_ctx(shape, "bf16", blob)
    for mode in [P().EXEC_FULL, P().EXEC_COMPACT, P().EXEC_AUTO]:
        outs.append(ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                                      batch.temperature, wl.window, top_k=wl.top_k, seed=1000,
                                      exec_mode=mode, gamma=4))
    t0 = outs[0]["tokens"].cpu().numpy()
    for o in outs[1:]:
        assert np.array_equal(o["tokens"].cpu().numpy(), t0)
        assert np.array_equal(o["counts"].cpu().numpy(), outs[0]["counts"].cpu().numpy())
    c = outs[0]["counts"].cpu().numpy()
    T = shape.T
    for b in range(8):
        k = int(batch.prefix_len[b])
        assert c[:, b].sum() == T - k
        assert np.array_equal(t0[b, :k], batch.prefix_tokens[b, :k])
        n = k
        for x in c[:, b]:
            if n < T:
                assert 1 <= x <= min(wl.window, T - n)
            else:
                assert x == 0
            n += x
    assert (t0 >= 0).all() and (t0 < shape.vocab).all()


def test_rollout_bf16_full_equals_compact_across_kernel_choices():
    """With 192 images of the B model a Full round has 3264 rows, enough for
    the wide GEMM kernel on QKV, W1|W3 and the lm_head, while Compact rounds
    size their kernels for the active images only (the host's row bound), so
    the two modes run different kernels as images finish (prefix lengths
    spread over the grid). Tokens and counts must still agree bit for bit,
    with AUTO switching between the two at gamma = 96."""
    wl = synth.WORKLOADS["llamagen_b"]
    shape = wl.model
    blob = synth.make_weights(shape, 0)
    batch = synth.make_batch(wl, 7, batch=192)
    batch.prefix_len[:] = np.linspace(0, shape.T - 2, 192).astype(batch.prefix_len.dtype)
    ctx = gu.make_ctx(shape, "bf16", blob)
    outs = [ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                              batch.temperature, wl.window, top_k=wl.top_k, seed=1003,
                              exec_mode=mode, gamma=96)
            for mode in (P().EXEC_FULL, P().EXEC_COMPACT, P().EXEC_AUTO)]
    t0 = outs[0]["tokens"].cpu().numpy()
    for o in outs[1:]:
        assert np.array_equal(o["tokens"].cpu().numpy(), t0)
        assert np.array_equal(o["counts"].cpu().numpy(), outs[0]["counts"].cpu().numpy())
    assert outs[0]["rounds"] > 10


@pytest.mark.parametrize("kernel", ["seq", "split"])
def test_forward_bf16_each_attention_kernel_matches_oracle(kernel, monkeypatch):
    """Two of the attention kernels (causal attention of each sequence's rows
    over its own paged cache, Sec. 4.2): one wavefront walking a block's key
    tiles in order, and four wavefronts splitting them and merging. A launch
    takes one by its capacity; HBSJD_ATTN_KERNEL forces either on every
    launch. Both
    meet the forward bar against the oracle on ragged prefill segments (1 to
    256 rows: one to eight 32-row query blocks)."""
    monkeypatch.setenv("HBSJD_ATTN_KERNEL", kernel)
    _bf16_forward_case("llamagen_b", [40, 0, 90, 255, 17], 11)


def test_forward_bf16_query_split_attention_matches_oracle(monkeypatch):
    """The attention kernel of the rounds (segments of at most 64 rows: four
    wavefronts take 16 query rows each and share the key tiles through LDS),
    forced on every launch it fits, meets the forward bar against the oracle
    on ragged segments of 1 to 64 rows."""
    monkeypatch.setenv("HBSJD_ATTN_KERNEL", "qs")
    _bf16_forward_case("llamagen_b", [40, 0, 63, 16, 17, 5], 12)


@pytest.mark.parametrize("W", [8, 16, 32, 63])
def test_rollout_bf16_query_split_attention_equals_sequential(W, monkeypatch):
    """The query-split attention kernel computes every row with the sequential
    kernel's arithmetic, so a rollout forced onto it (every round; the
    prefill's long segments take the sequential kernel) gives the
    same tokens and counts as one forced onto the sequential kernel, in Full
    and Compact rounds alike (Sec. 4.3), at windows of 9 to 64 rows."""
    wl = synth.WORKLOADS["llamagen_b"]
    shape = wl.model
    blob = synth.make_weights(shape, 0)
    batch = synth.make_batch(wl, 1, batch=8)
    batch.prefix_len[3] = shape.T - 5
    outs = {}
    for kernel in ["seq", "qs"]:
        monkeypatch.setenv("HBSJD_ATTN_KERNEL", kernel)
        ctx = gu.make_ctx(shape, "bf16", blob)
        for mode in [P().EXEC_FULL, P().EXEC_COMPACT]:
            o = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                                  batch.temperature, W, top_k=wl.top_k, seed=1000,
                                  exec_mode=mode, gamma=4)
            outs[kernel, mode] = (o["tokens"].cpu().numpy(), o["counts"].cpu().numpy())
        del ctx
    monkeypatch.delenv("HBSJD_ATTN_KERNEL", raising=False)
    ref = outs["seq", P().EXEC_FULL]
    for key, (tok, cnt) in outs.items():
        assert np.array_equal(tok, ref[0]), key
        assert np.array_equal(cnt, ref[1]), key


@pytest.mark.parametrize("W", [8, 16, 32])
def test_rollout_bf16_full_equals_compact_sequential_attention(W, monkeypatch):
    """Full and Compact rounds (Sec. 4.3) give identical tokens with the
    sequential attention kernel on every launch, at windows of 9, 17 and 33
    rows (one, two and three 16-row query groups per block)."""
    monkeypatch.setenv("HBSJD_ATTN_KERNEL", "seq")
    wl = synth.WORKLOADS["llamagen_b"]
    shape = wl.model
    blob = synth.make_weights(shape, 0)
    batch = synth.make_batch(wl, 1, batch=8)
    batch.prefix_len[3] = shape.T - 5
    ctx = gu.make_ctx(shape, "bf16", blob)
    outs = [ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                              batch.temperature, W, top_k=wl.top_k, seed=1000, exec_mode=mode,
                              gamma=4)
            for mode in [P().EXEC_FULL, P().EXEC_COMPACT]]
    t0 = outs[0]["tokens"].cpu().numpy()
    assert np.array_equal(outs[1]["tokens"].cpu().numpy(), t0)
    assert np.array_equal(outs[1]["counts"].cpu().numpy(), outs[0]["counts"].cpu().numpy())
    c = outs[0]["counts"].cpu().numpy()
    for b in range(8):
        assert c[:, b].sum() == shape.T - int(batch.prefix_len[b])


# ------------------------------------------------------------------ cached-AR baseline


def _ar_counts_ok(counts, prefix_len, T):
    """One token per round while an image is active, nothing after."""
    for b, k in enumerate(prefix_len):
        col = counts[:, b]
        assert col.sum() == T - k
        assert (col[:T - k] == 1).all() and (col[T - k:] == 0).all()


@pytest.mark.parametrize("greedy,top_k", [(False, 0), (False, 20), (True, 0)])
def test_rollout_ar_f32_tiny_equals_oracle_ar(tiny, greedy, top_k):
    w, blob, om = tiny
    batch = synth.make_batch(w, 3)
    batch.prefix_len[1] = 0                 # the class token starts the sequence
    batch.prefix_len[2] = w.model.T         # nothing to generate
    batch.temperature[:] = [1.0, 0.6, 1.4, 1.9]
    ctx = gu.make_ctx(w.model, "f32", blob)
    g = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                          batch.temperature, 1, top_k=top_k, seed=321,
                          verify_mode=P().VERIFY_AR_GREEDY if greedy else P().VERIFY_AR)
    ref = om.rollout_ar(batch, top_k=top_k, seed=321, greedy=greedy)
    assert np.array_equal(g["tokens"].cpu().numpy(), ref)
    T = w.model.T
    assert g["rounds"] == int(np.max(T - batch.prefix_len))
    _ar_counts_ok(g["counts"].cpu().numpy(), batch.prefix_len, T)
    assert g["rejected"] == 0


def test_rollout_ar_f32_cfg_equals_oracle_ar():
    shape = synth.small_shape(n_layers=2, d_model=32, n_heads=2, mlp_hidden=48, vocab=64,
                              n_classes=4, grid=4)
    blob = synth.make_weights(shape, 3, std=0.2)
    om = oracle.Model(shape, blob)
    w = synth.Workload("t", shape, "f32", 6, 3, 2, 7, 2.0, prefix_lo=0, prefix_hi=9)
    batch = synth.make_batch(w, 5)
    ctx = gu.make_ctx(shape, "f32", blob)
    g = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                          batch.temperature, 1, top_k=7, cfg_scale=2.0, seed=78,
                          verify_mode=P().VERIFY_AR)
    ref = om.rollout_ar(batch, top_k=7, cfg_scale=2.0, seed=78)
    assert np.array_equal(g["tokens"].cpu().numpy(), ref)


def test_rollout_ar_bf16_equals_sjd_window_1():
    # W = 1 SJD accepts every draft (its proposal is the same row recomputed),
    # so it reproduces the AR baseline token for token on the GPU as well, as
    # long as the row at position k_b (SJD prefill, first AR round) sees the
    # same K split of O and W2 in both launches: 4 parts at these prefixes
    wl = synth.WORKLOADS["llamagen_b"]
    shape = wl.model
    blob = synth.make_weights(shape, 0)
    batch = synth.make_batch(wl, 2, batch=4)
    batch.prefix_len[:] = [shape.T - 40, 0, shape.T - 17, shape.T - 64]
    ctx = gu.make_ctx(shape, "bf16", blob)
    ar = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                           batch.temperature, 1, top_k=wl.top_k, seed=4242,
                           verify_mode=P().VERIFY_AR)
    sj = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                           batch.temperature, 1, top_k=wl.top_k, seed=4242)
    a, s = ar["tokens"].cpu().numpy(), sj["tokens"].cpu().numpy()
    assert np.array_equal(a, s)
    assert sj["rejected"] == 0
    _ar_counts_ok(ar["counts"].cpu().numpy(), batch.prefix_len, shape.T)
    assert (a >= 0).all() and (a < shape.vocab).all()


# ------------------------------------------------------------------ batch-synchronous windows


@pytest.mark.parametrize("W,top_k,greedy,H,mode", [(4, 0, False, 24, "auto"), (3, 5, False, 2, "full"),
                                                    (4, 0, True, 24, "compact"),
                                                    (9, 20, False, 3, "auto"), (1, 0, False, 24, "full")])
def test_rollout_sync_f32_tiny_equals_oracle(tiny, W, top_k, greedy, H, mode):
    """The Batch-Synchronous SJD ablation (Sec. 4.1, Table 2) against the
    oracle's shared-window schedule: tokens, per-round counts (0 while an image
    waits at a boundary), rounds and statistics."""
    w, blob, om = tiny
    batch = synth.make_batch(w, 3)
    batch.prefix_len[1] = 60                 # finishes early
    m = {"full": P().EXEC_FULL, "compact": P().EXEC_COMPACT, "auto": P().EXEC_AUTO}[mode]
    ctx = gu.make_ctx(w.model, "f32", blob)
    g = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                          batch.temperature, W, history=H, top_k=top_k, seed=77,
                          verify_mode=P().VERIFY_GREEDY if greedy else P().VERIFY_PROB,
                          exec_mode=m, gamma=2, progress=P().PROGRESS_SYNC)
    o = om.rollout(batch, W=W, H=H, top_k=top_k, seed=77, greedy=greedy,
                   exec_mode={P().EXEC_FULL: 0, P().EXEC_COMPACT: 1, P().EXEC_AUTO: 2}[m],
                   gamma=2, sync=True)
    assert np.array_equal(g["tokens"].cpu().numpy(), o["tokens"])
    assert g["rounds"] == o["rounds"]
    assert np.array_equal(g["counts"].cpu().numpy(), o["counts"])
    assert np.array_equal(g["active"], o["active"])
    assert g["verified"] == o["verified"] and g["rejected"] == o["rejected"]
    assert g["image_rounds"] == o["image_rounds"]


def test_rollout_sync_f32_cfg_equals_oracle():
    shape = synth.small_shape(n_layers=2, d_model=32, n_heads=2, mlp_hidden=48, vocab=64,
                              n_classes=4, grid=4)
    blob = synth.make_weights(shape, 3, std=0.2)
    om = oracle.Model(shape, blob)
    w = synth.Workload("t", shape, "f32", 6, 3, 2, 7, 2.0, prefix_lo=0, prefix_hi=9)
    batch = synth.make_batch(w, 5)
    ctx = gu.make_ctx(shape, "f32", blob)
    g = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                          batch.temperature, 3, history=2, top_k=7, cfg_scale=2.0, seed=78,
                          exec_mode=P().EXEC_AUTO, gamma=2, progress=P().PROGRESS_SYNC)
    o = om.rollout(batch, W=3, H=2, top_k=7, cfg_scale=2.0, seed=78, exec_mode=2, gamma=2,
                   sync=True)
    assert np.array_equal(g["tokens"].cpu().numpy(), o["tokens"])
    assert np.array_equal(g["counts"].cpu().numpy(), o["counts"])


def test_rollout_sync_bf16_schedule_and_modes():
    from tests.test_oracle_rollout import replay_sync_schedule
    wl = synth.WORKLOADS["llamagen_b"]
    shape = wl.model
    blob = synth.make_weights(shape, 0)
    batch = synth.make_batch(wl, 1, batch=8)
    batch.prefix_len[3] = shape.T - 5
    ctx = gu.make_ctx(shape, "bf16", blob)
    outs = [ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                              batch.temperature, wl.window, top_k=wl.top_k, seed=1000,
                              exec_mode=mode, gamma=4, progress=P().PROGRESS_SYNC)
            for mode in [P().EXEC_FULL, P().EXEC_COMPACT, P().EXEC_AUTO]]
    t0 = outs[0]["tokens"].cpu().numpy()
    c0 = outs[0]["counts"].cpu().numpy()
    for o in outs[1:]:
        assert np.array_equal(o["tokens"].cpu().numpy(), t0)
        assert np.array_equal(o["counts"].cpu().numpy(), c0)
    n = replay_sync_schedule(c0, batch.prefix_len, shape.T, wl.window)
    assert (n == shape.T).all()
    for b in range(8):
        k = int(batch.prefix_len[b])
        assert np.array_equal(t0[b, :k], batch.prefix_tokens[b, :k])
    assert (t0 >= 0).all() and (t0 < shape.vocab).all()
    assert (c0 == 0).any() and outs[0]["image_rounds"] == int((c0 > 0).sum())


# ------------------------------------------------------------------ round API and errors


def _cfg_case():
    shape = synth.small_shape(n_layers=2, d_model=32, n_heads=2, mlp_hidden=48, vocab=64,
                              n_classes=4, grid=4)
    blob = synth.make_weights(shape, 3, std=0.2)
    w = synth.Workload("t", shape, "f32", 6, 3, 2, 7, 2.0, prefix_lo=0, prefix_hi=9)
    return w, blob, oracle.Model(shape, blob), synth.make_batch(w, 5)


# (W, H, top_k, cfg, greedy, sync); the tiny workload unless cfg is set
ROUND_CASES = {
    "tiny": (4, 24, 0, 0.0, False, False),
    "tiny_h3": (6, 3, 20, 0.0, False, False),
    "tiny_sync": (4, 2, 0, 0.0, False, True),
    "tiny_greedy": (5, 4, 0, 0.0, True, False),
    "cfg_topk": (3, 2, 7, 2.0, False, False),
}


@pytest.mark.parametrize("name", sorted(ROUND_CASES))
def test_round_state_equals_oracle_windows(tiny, name):
    """Round by round through the C ABI (hbsjd_rollout_begin, hbsjd_round,
    hbsjd_get_state) against the oracle's recorded windows: after the prefill
    and after every round the GPU's cursors, drafts and proposal
    probabilities q(z) equal the oracle's (Sec. 4.2: reused predictions, then
    history tokens at offset H). Drafts and counts are compared exactly; q(z)
    of a reused draft is a probability computed by each side's own fp32
    forward and softmax, compared to 2e-4 relative (the fp32 forward bar of
    1e-4 on the logits moves a probability by at most about twice that at
    temperature >= 0.7), and 1 exactly for history drafts and greedy mode.
    Rounds alternate between Full and Compact."""
    W, H, top_k, cfg, greedy, sync = ROUND_CASES[name]
    if cfg:
        w, blob, om, batch = _cfg_case()
    else:
        w, blob, om = tiny
        batch = synth.make_batch(w, 1)
        batch.temperature[:] = [1.0, 0.7, 1.3, 2.0]
        batch.prefix_len[2] = 60
    ref = om.rollout(batch, W=W, H=H, top_k=top_k, cfg_scale=cfg, seed=1000, greedy=greedy,
                     sync=sync, trace=True)
    ctx = gu.make_ctx(w.model, "f32", blob)
    kw = dict(history=H, top_k=top_k, cfg_scale=cfg, seed=1000,
              verify_mode=P().VERIFY_GREEDY if greedy else P().VERIFY_PROB,
              progress=P().PROGRESS_SYNC if sync else P().PROGRESS_INDEPENDENT)
    ctx.hbsjd_rollout_begin(gu.device_batch(batch), batch.prefix_len, batch.labels,
                            batch.temperature, W, **kw)

    def same_state(i, st):
        d, q = ref["trace_drafts"][i], ref["trace_q"][i]
        assert np.array_equal(st["drafts"], d), (i, st["drafts"].tolist(), d.tolist())
        hist = (q == 1.0) | (d < 0)
        assert np.array_equal(st["q_token_prob"][hist], q[hist]), i
        np.testing.assert_allclose(st["q_token_prob"][~hist], q[~hist], rtol=2e-4, atol=0)

    st = ctx.hbsjd_get_state()
    assert np.array_equal(st["cursors"], batch.prefix_len)
    same_state(0, st)
    cursors = st["cursors"].copy()
    r = 0
    while True:
        mode = [P().EXEC_FULL, P().EXEC_COMPACT][r % 2]
        counts, active = ctx.hbsjd_round(mode)
        assert np.array_equal(counts, ref["counts"][r]), r
        cursors += counts
        st = ctx.hbsjd_get_state()
        assert np.array_equal(st["cursors"], cursors)
        same_state(r + 1, st)
        r += 1
        if active == 0:
            break
    assert r == ref["rounds"]
    assert np.array_equal(st["tokens"], ref["tokens"])


def test_graph_replays_equal_eager_launches(monkeypatch):
    """Rounds run as captured HIP graphs replayed every round (and across
    rollouts), one pair per kernel plan of the round's products; a context
    created with HBSJD_NO_GRAPHS=1 launches the same kernels eagerly. Several
    rollouts, alternated between the two contexts so eager work and
    synchronisations sit between the replays, must agree bit for bit in tokens
    and per-round counts."""
    wl = synth.WORKLOADS["llamagen_b"]
    shape = wl.model
    blob = synth.make_weights(shape, 0)
    batch = synth.make_batch(wl, 3, batch=8)
    batch.prefix_len[2] = shape.T - 3
    graph = gu.make_ctx(shape, "bf16", blob)
    monkeypatch.setenv("HBSJD_NO_GRAPHS", "1")
    eager = gu.make_ctx(shape, "bf16", blob)
    monkeypatch.delenv("HBSJD_NO_GRAPHS")
    for seed, mode, prog in [(1000, P().EXEC_AUTO, P().PROGRESS_INDEPENDENT),
                             (1001, P().EXEC_FULL, P().PROGRESS_INDEPENDENT),
                             (1002, P().EXEC_AUTO, P().PROGRESS_SYNC),
                             (1000, P().EXEC_COMPACT, P().PROGRESS_INDEPENDENT)]:
        outs = [c.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                                batch.temperature, wl.window, top_k=wl.top_k, seed=seed,
                                exec_mode=mode, gamma=4, progress=prog) for c in (graph, eager)]
        assert np.array_equal(outs[0]["tokens"].cpu().numpy(), outs[1]["tokens"].cpu().numpy())
        assert np.array_equal(outs[0]["counts"].cpu().numpy(), outs[1]["counts"].cpu().numpy())
        assert outs[0]["rounds"] == outs[1]["rounds"] and outs[0]["rounds"] > 2


def test_graph_replays_follow_the_row_bound(monkeypatch):
    """With 192 images of the B model a full round has 3264 rows, enough for
    the wide GEMM kernel, and the products switch to smaller tiles as images
    finish (prefix lengths spread over the grid), so the graph context
    captures a pair per kernel plan while the eager one picks per round.
    Tokens and counts must agree bit for bit."""
    wl = synth.WORKLOADS["llamagen_b"]
    shape = wl.model
    blob = synth.make_weights(shape, 0)
    batch = synth.make_batch(wl, 5, batch=192)
    batch.prefix_len[:] = np.linspace(0, shape.T - 2, 192).astype(batch.prefix_len.dtype)
    graph = gu.make_ctx(shape, "bf16", blob)
    monkeypatch.setenv("HBSJD_NO_GRAPHS", "1")
    eager = gu.make_ctx(shape, "bf16", blob)
    monkeypatch.delenv("HBSJD_NO_GRAPHS")
    for seed, mode in [(1000, P().EXEC_COMPACT), (1001, P().EXEC_AUTO)]:
        outs = [c.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                                batch.temperature, wl.window, top_k=wl.top_k, seed=seed,
                                exec_mode=mode, gamma=96) for c in (graph, eager)]
        assert np.array_equal(outs[0]["tokens"].cpu().numpy(), outs[1]["tokens"].cpu().numpy())
        assert np.array_equal(outs[0]["counts"].cpu().numpy(), outs[1]["counts"].cpu().numpy())
        assert outs[0]["rounds"] == outs[1]["rounds"] and outs[0]["rounds"] > 10


def test_argument_errors(tiny):
    w, blob, _ = tiny
    ctx = gu.make_ctx(w.model, "f32", blob)
    batch = synth.make_batch(w, 1)
    dev = gu.device_batch(batch)
    E = P().HbsjdError

    def call(**kw):
        args = dict(prefix_len=batch.prefix_len, class_labels=batch.labels,
                    temperature=batch.temperature, window=4)
        args.update(kw)
        return ctx.hbsjd_rollout(dev, **args)

    bad = [dict(window=0), dict(history=0), dict(top_k=-1), dict(max_rounds=3),
           dict(prefix_len=np.array([0, 0, 0, 65])), dict(class_labels=np.array([0, 0, 0, 10])),
           dict(temperature=np.array([1, 1, 0, 1.0])),
           dict(temperature=np.array([1, 1, np.nan, 1.0])), dict(progress=2),
           dict(progress=-1), dict(exec_mode=3), dict(verify_mode=4)]
    for kw in bad:
        with pytest.raises(E) as ei:
            call(**kw)
        assert ei.value.code == "EINVAL", kw
    bad_tok = batch.prefix_tokens.copy()
    bad_tok[0, 0] = w.model.vocab
    batch.prefix_len[0] = max(1, batch.prefix_len[0])
    with pytest.raises(E) as ei:
        ctx.hbsjd_rollout(torch.from_numpy(bad_tok).cuda(), batch.prefix_len, batch.labels,
                          batch.temperature, 4)
    assert ei.value.code == "EINVAL"
    # the context still works after EINVAL
    call()
    fresh = gu.make_ctx(w.model, "f32", blob)
    with pytest.raises(E) as ei:
        fresh.hbsjd_round(P().EXEC_AUTO)
    assert ei.value.code == "ESTATE"
    small = gu.make_ctx(w.model, "f32", blob, max_kv_bytes=1024)
    with pytest.raises(E) as ei:
        small.hbsjd_rollout(dev, batch.prefix_len, batch.labels, batch.temperature, 4)
    assert ei.value.code == "ENOMEM"


# ------------------------------------------------------------------ gamma calibration


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_calibrate_gamma_drives_auto_mode(tiny, dtype):
    if dtype == "f32":
        w, blob, _ = tiny
        shape, B, W = w.model, 4, w.window
    else:
        wl = synth.WORKLOADS["llamagen_b"]
        shape, B, W = wl.model, 8, wl.window
        blob = synth.make_weights(shape, 0)
        w = synth.Workload("b8", shape, "bf16", B, W, 24, 0, 0.0, prefix_lo=0, prefix_hi=128)
    ctx = gu.make_ctx(shape, dtype, blob)
    g = ctx.hbsjd_calibrate_gamma(B, W)
    assert 0 <= g <= B
    with pytest.raises(P().HbsjdError):
        ctx.hbsjd_round()                    # the synthetic state is not a rollout
    batch = synth.make_batch(w, 9, batch=B)
    batch.prefix_len[0] = shape.T - 2        # finishes early, so A shrinks
    out = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                            batch.temperature, W, seed=5, exec_mode=P().EXEC_AUTO, gamma=-1)
    for a, m in zip(out["active"], out["mode"]):
        assert m == (0 if a > g else 1)      # Eq. 6 with the calibrated threshold
    ref = ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                            batch.temperature, W, seed=5, exec_mode=P().EXEC_FULL)
    assert np.array_equal(out["tokens"].cpu().numpy(), ref["tokens"].cpu().numpy())


# ------------------------------------------------------------------ kernel timing


def test_profile_sampling_brackets_one_launch_in_every(tiny):
    """Per-class timing brackets one launch in `every` of each timed class and
    changes no result."""
    w, blob, _ = tiny
    ctx = gu.make_ctx(w.model, "f32", blob)
    batch = synth.make_batch(w, 3)

    def run():
        return ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                                 batch.temperature, w.window, history=w.history, seed=5)

    base = run()["tokens"].cpu().numpy()
    counts = {}
    for every in (1, 3):
        ctx.hbsjd_profile_sample(every)
        ctx.hbsjd_profile_start(["qkv", "verify"])
        out = run()
        prof = ctx.hbsjd_profile_read()
        ctx.hbsjd_profile_start(())
        assert np.array_equal(out["tokens"].cpu().numpy(), base)
        assert prof["qkv"][0] > 0 and prof["verify"][0] > 0
        assert prof["attn"] == (0.0, 0)
        counts[every] = (prof["qkv"][1], prof["verify"][1])
    ctx.hbsjd_profile_sample(1)
    for n1, n3 in zip(counts[1], counts[3]):
        assert n1 > 3 and -(-n1 // 3) - 1 <= n3 <= -(-n1 // 3), counts
    for bad in (0, -2):
        with pytest.raises(P().HbsjdError) as ei:
            ctx.hbsjd_profile_sample(bad)
        assert ei.value.code == "EINVAL"


# ------------------------------------------------------------------ GEMM kernel choice


@pytest.mark.parametrize("name", ["stress_b", "llamagen_xl_cfg"])
def test_gemm_kernel_choice_does_not_change_results(monkeypatch, name):
    """Every projection may run on the wide kernel (tiles of 256, 192 or 128 rows
    by 256 columns) or on the 128 x 128 / 64 x 64 one, chosen per launch from
    the rows present; Full and Compact
    rounds (Sec. 4.3) process the same row in launches of different sizes, so
    the kernels must agree bit for bit. Forward logits of the same sequences
    with every launch forced onto one kernel (HBSJD_GEMM_TILE: the wide kernel
    at its chosen tile height, at 256, 192 or 128 rows, or at 256 rows with a
    last round of 128-row halves; or the small-tile kernel) and chosen per
    launch must be identical, at a row count where the choice varies."""
    wl = synth.WORKLOADS[name]
    shape = wl.model
    blob = synth.make_weights(shape, 0, std=wl.weight_std, bias_std=wl.bias_std)
    rng = np.random.default_rng(5)
    n = 12 if shape.T > 300 else 24
    lens = np.full(n, shape.T - 1, dtype=np.int32)
    lens[1] = 17
    toks = rng.integers(0, shape.vocab, size=(n, shape.T)).astype(np.int32)
    labels = rng.integers(0, shape.n_classes + 1, size=n).astype(np.int32)
    outs = {}
    for force in ["wide", "wide256", "wide256h", "wide192", "wide128", "small", ""]:
        if force:
            monkeypatch.setenv("HBSJD_GEMM_TILE", force)
        else:
            monkeypatch.delenv("HBSJD_GEMM_TILE", raising=False)
        ctx = gu.make_ctx(shape, "bf16", blob)
        outs[force] = ctx.hbsjd_forward(torch.from_numpy(toks).cuda(), lens.tolist(),
                                        labels).cpu().numpy()
        del ctx
    monkeypatch.delenv("HBSJD_GEMM_TILE", raising=False)
    for force, out in outs.items():
        assert np.array_equal(out.view(np.uint32), outs["small"].view(np.uint32)), force
