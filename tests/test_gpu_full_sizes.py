"""GPU rollouts at the workloads' full sizes, in the launch configuration
bench.py times (AUTO execution with the calibrated gamma, the workload's W, H,
top-k, guidance and temperatures). bf16 tokens cannot be compared with the
fp32 oracle one for one, so these check what holds at any size:
  * every round commits 1..min(W, T - n) tokens and the counts sum to T - k;
  * prefixes are kept and every token is in the vocabulary;
  * Full, Compact and AUTO execution give the same tokens (Sec. 4.3);
and, on sampled sequences of the rollout (B, stress, L and XL shapes), that the
oracle's logits match the GPU forward (3e-2 max-abs / 1e-2 mean-abs) and every
generated token lies in the oracle's top-k support (with a 5% margin for
rounding at the edge)."""
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


def _setup(name):
    wl = synth.WORKLOADS[name]
    shape = wl.model
    blob = synth.make_weights(shape, 0, std=wl.weight_std, bias_std=wl.bias_std)
    batch = synth.make_batch(wl, 1)
    ctx = gu.make_ctx(shape, "bf16", blob)
    return wl, shape, blob, batch, ctx


def _rollout(ctx, wl, batch, seed, mode, gamma=-1, progress=0):
    return ctx.hbsjd_rollout(gu.device_batch(batch), batch.prefix_len, batch.labels,
                             batch.temperature, wl.window, history=wl.history, top_k=wl.top_k,
                             cfg_scale=wl.cfg_scale, seed=seed, exec_mode=mode, gamma=gamma,
                             progress=progress)


def _check_invariants(out, batch, wl, T, V):
    tok = out["tokens"].cpu().numpy()
    cnt = out["counts"].cpu().numpy()
    for b, k in enumerate(batch.prefix_len):
        k = int(k)
        assert np.array_equal(tok[b, :k], batch.prefix_tokens[b, :k])
        assert cnt[:, b].sum() == T - k
        n = k
        for x in cnt[:, b]:
            if n < T:
                assert 1 <= x <= min(wl.window, T - n), (b, n, x)
            else:
                assert x == 0
            n += x
    assert (tok >= 0).all() and (tok < V).all()
    return tok


@pytest.mark.parametrize("name", ["llamagen_b", "stress_b"])
def test_full_size_rollout_invariants_and_modes(name):
    wl, shape, blob, batch, ctx = _setup(name)
    g = ctx.hbsjd_calibrate_gamma(wl.batch, wl.window)
    assert 0 <= g <= wl.batch
    auto = _rollout(ctx, wl, batch, 1000, P().EXEC_AUTO)
    t_auto = _check_invariants(auto, batch, wl, shape.T, shape.vocab)
    for a, m in zip(auto["active"], auto["mode"]):
        assert m == (0 if a > g else 1)
    for mode in [P().EXEC_FULL, P().EXEC_COMPACT]:
        o = _rollout(ctx, wl, batch, 1000, mode)
        assert np.array_equal(o["tokens"].cpu().numpy(), t_auto)
        assert np.array_equal(o["counts"].cpu().numpy(), auto["counts"].cpu().numpy())
    # mean committed per round stays within the window
    mean = auto["verified"] / max(auto["image_rounds"], 1)
    assert 1.0 <= mean <= wl.window


@pytest.mark.parametrize("name", ["llamagen_b", "stress_b"])
def test_full_size_rollout_samples_match_oracle(name):
    wl, shape, blob, batch, ctx = _setup(name)
    ctx.hbsjd_calibrate_gamma(wl.batch, wl.window)
    out = _rollout(ctx, wl, batch, 1001, P().EXEC_AUTO)
    tok = _check_invariants(out, batch, wl, shape.T, shape.vocab)
    # two sampled images: the shortest and the longest prefix
    pick = [int(np.argmin(batch.prefix_len)), int(np.argmax(batch.prefix_len))]
    T = shape.T
    seqs = [tok[b, :T - 1] for b in pick]
    labels = [int(batch.labels[b]) for b in pick]
    om = oracle.Model(shape, gu.bf16_rounded_blob(shape, blob))
    ref = om.forward_batch(labels, seqs)
    dev = np.zeros((len(pick), T), dtype=np.int32)   # [n_seqs][T], the entry's layout
    for j, sq in enumerate(seqs):
        dev[j, :T - 1] = sq
    got = ctx.hbsjd_forward(torch.from_numpy(dev).cuda(), [T - 1] * len(pick),
                            labels).cpu().numpy()
    got = got.reshape(len(pick), T, shape.vocab)
    for j, b in enumerate(pick):
        err = np.abs(got[j].astype(np.float64) - ref[j])
        assert err.max() <= 3e-2 and err.mean() <= 1e-2, (b, err.max(), err.mean())
        # row t - 1 predicts position t; generated positions are k+1..T
        k = int(batch.prefix_len[b])
        y = ref[j][k:T] / float(batch.temperature[b])
        drawn = tok[b, k:T]
        rank = (y > y[np.arange(len(drawn)), drawn][:, None]).sum(axis=1) + 1
        assert rank.max() <= int(wl.top_k * 1.05), (b, rank.max())


def test_full_size_l_shape_forward_and_rollout():
    wl, shape, blob, batch, ctx = _setup("llamagen_l")
    # forward parity on sampled sequences of the full shape
    om = oracle.Model(shape, gu.bf16_rounded_blob(shape, blob))
    rng = np.random.default_rng(11)
    lens = [0, 37, 96]
    labels = rng.integers(0, shape.n_classes, size=len(lens)).astype(np.int32)
    toks = rng.integers(0, shape.vocab, size=(len(lens), shape.T)).astype(np.int32)
    got = ctx.hbsjd_forward(torch.from_numpy(toks).cuda(), lens, labels).cpu().numpy()
    ref = np.concatenate(om.forward_batch(labels, [toks[i, :n] for i, n in enumerate(lens)]))
    err = np.abs(got.astype(np.float64) - ref)
    assert err.max() <= 3e-2 and err.mean() <= 1e-2, (err.max(), err.mean())
    ctx.hbsjd_calibrate_gamma(wl.batch, wl.window)
    out = _rollout(ctx, wl, batch, 1000, P().EXEC_AUTO)
    tok = _check_invariants(out, batch, wl, shape.T, shape.vocab)
    # the image with the shortest prefix: every token it generated lies in the
    # oracle's top-k support of its completed sequence (the batch's prefill
    # and rounds all feed its cache)
    b = int(np.argmin(batch.prefix_len))
    k = int(batch.prefix_len[b])
    ref = om.forward_batch([int(batch.labels[b])], [tok[b, :shape.T - 1]])[0]
    y = ref[k:shape.T]
    drawn = tok[b, k:shape.T]
    rank = (y > y[np.arange(len(drawn)), drawn][:, None]).sum(axis=1) + 1
    assert rank.max() <= int(wl.top_k * 1.05), (b, rank.max())


def test_full_size_xl_cfg_rollout_invariants_and_samples():
    """The XL workload with guidance (256 verifier row sets of W + 1 rows):
    invariants, AUTO = Compact, and on the image with the shortest prefix the
    oracle's conditional and null-class logits of its first 96 generated
    positions against the GPU forward (3e-2 / 1e-2), with every token it drew
    inside the top-k support of the oracle's guided logits (Sec. 4.2: CFG
    branches verify on the fused guided logits)."""
    wl, shape, blob, batch, ctx = _setup("llamagen_xl_cfg")
    ctx.hbsjd_calibrate_gamma(wl.batch, wl.window)
    out = _rollout(ctx, wl, batch, 1000, P().EXEC_AUTO)
    tok = _check_invariants(out, batch, wl, shape.T, shape.vocab)
    comp = _rollout(ctx, wl, batch, 1000, P().EXEC_COMPACT)
    assert np.array_equal(comp["tokens"].cpu().numpy(), tok)
    b = int(np.argmin(batch.prefix_len))
    k = int(batch.prefix_len[b])
    n = min(shape.T - 1, k + 96)                 # positions 0..n: predictions of 1..n+1
    labels = [int(batch.labels[b]), shape.n_classes]
    om = oracle.Model(shape, gu.bf16_rounded_blob(shape, blob))
    ref = om.forward_batch(labels, [tok[b, :n], tok[b, :n]])
    dev = np.zeros((2, shape.T), dtype=np.int32)
    dev[:, :n] = tok[b, :n]
    got = ctx.hbsjd_forward(torch.from_numpy(dev).cuda(), [n, n], labels).cpu().numpy()
    got = got.reshape(2, n + 1, shape.vocab)
    for j in range(2):
        err = np.abs(got[j].astype(np.float64) - ref[j])
        assert err.max() <= 3e-2 and err.mean() <= 1e-2, (j, err.max(), err.mean())
    lc, lu = ref[0][k:n + 1], ref[1][k:n + 1]
    y = (lu + wl.cfg_scale * (lc - lu)) / float(batch.temperature[b])
    drawn = tok[b, k:n + 1]
    rank = (y > y[np.arange(len(drawn)), drawn][:, None]).sum(axis=1) + 1
    assert rank.max() <= int(wl.top_k * 1.05), (b, rank.max())


def test_full_size_sync_schedule():
    """The Batch-Synchronous ablation at the B workload's full size: the
    shared-window schedule holds and it needs at least as many rounds as the
    longest suffix needs windows."""
    from tests.test_oracle_rollout import replay_sync_schedule
    wl, shape, blob, batch, ctx = _setup("llamagen_b")
    out = _rollout(ctx, wl, batch, 1000, P().EXEC_AUTO, gamma=wl.batch, progress=P().PROGRESS_SYNC)
    c = out["counts"].cpu().numpy()
    n = replay_sync_schedule(c, batch.prefix_len, shape.T, wl.window)
    assert (n == shape.T).all()
    tok = out["tokens"].cpu().numpy()
    for b, k in enumerate(batch.prefix_len):
        assert np.array_equal(tok[b, :k], batch.prefix_tokens[b, :k])
    assert (tok >= 0).all() and (tok < shape.vocab).all()
    L = shape.T - batch.prefix_len
    assert out["rounds"] >= int(np.ceil(L.max() / wl.window))
