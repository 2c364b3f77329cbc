"""Whole-algorithm pins of the oracle's batched SJD rollout (Sec. 4.2-4.3):
special cases that reduce to token-by-token sampling, exact invariants, and a
chi-square test of the suffix distribution against brute-force enumeration of
the AR joint (Eq. 1-2)."""
import itertools

import numpy as np
import pytest
from scipy import stats

import oracle
import synth


def _batch(w, seed=1, B=None):
    return synth.make_batch(w, seed, batch=B)


@pytest.mark.parametrize("seed", [1000, 1001, 1002])
def test_window_one_is_token_by_token_sampling(tiny, seed):
    w, _, om = tiny
    b = _batch(w)
    r = om.rollout(b, W=1, seed=seed)
    ar = om.rollout_ar(b, seed=seed)
    assert np.array_equal(r["tokens"], ar)
    assert r["rejected"] == 0


def test_window_one_matches_ar_with_top_k_temperature_and_cfg():
    shape = synth.small_shape(n_layers=2, d_model=32, n_heads=2, mlp_hidden=48, vocab=40,
                              n_classes=4, grid=4)
    om = oracle.Model(shape, synth.make_weights(shape, 3, std=0.2))
    w = synth.Workload("t", shape, "f32", 6, 1, 3, 7, 2.0, prefix_lo=0, prefix_hi=9)
    b = _batch(w, 5)
    b.temperature[:] = [0.5, 0.9, 1.0, 1.3, 2.0, 0.7]
    r = om.rollout(b, W=1, H=3, top_k=7, cfg_scale=2.0, seed=77)
    ar = om.rollout_ar(b, top_k=7, cfg_scale=2.0, seed=77)
    assert np.array_equal(r["tokens"], ar)


@pytest.mark.parametrize("W,H", [(1, 24), (4, 24), (16, 24), (4, 1), (16, 3)])
def test_greedy_sjd_equals_greedy_ar(tiny, W, H):
    w, _, om = tiny
    b = _batch(w, 2)
    r = om.rollout(b, W=W, H=H, seed=5, greedy=True)
    ar = om.rollout_ar(b, seed=5, greedy=True)
    assert np.array_equal(r["tokens"], ar)


@pytest.mark.parametrize("W", [2, 4, 9])
def test_full_compact_auto_identical(tiny, W):
    w, _, om = tiny
    b = _batch(w, 3)
    b.prefix_len[1] = 60             # finishes early, so the modes differ physically
    runs = [om.rollout(b, W=W, seed=11, exec_mode=0),
            om.rollout(b, W=W, seed=11, exec_mode=1),
            om.rollout(b, W=W, seed=11, exec_mode=2, gamma=2)]
    for r in runs[1:]:
        assert np.array_equal(r["tokens"], runs[0]["tokens"])
        assert np.array_equal(r["counts"], runs[0]["counts"])
    auto = runs[2]
    assert np.array_equal(auto["mode"], np.where(auto["active"] > 2, 0, 1))
    assert np.all(runs[0]["mode"] == 0) and np.all(runs[1]["mode"] == 1)


@pytest.mark.parametrize("W", [1, 3, 4, 16])
def test_counts_bounds_and_bookkeeping(tiny, W):
    w, _, om = tiny
    b = _batch(w, 4)
    b.prefix_len[2] = w.model.T      # nothing to generate
    r = om.rollout(b, W=W, seed=21)
    T = w.model.T
    counts = r["counts"]
    for i in range(len(b.prefix_len)):
        k = int(b.prefix_len[i])
        c = counts[:, i]
        assert c.sum() == T - k
        n = k
        for x in c:
            if n >= T:
                assert x == 0
            else:
                assert 1 <= x <= min(W, T - n)
            n += x
        assert np.array_equal(r["tokens"][i, :k], b.prefix_tokens[i, :k])
    assert r["rounds"] <= T - int(b.prefix_len.min())
    assert counts[:, 2].sum() == 0
    assert r["active"][0] == int(np.sum(b.prefix_len < T))


def test_images_are_independent(tiny):
    w, _, om = tiny
    b = _batch(w, 6)
    r1 = om.rollout(b, W=4, seed=9)
    b2 = _batch(w, 6)
    b2.prefix_len[3] = 2
    b2.prefix_tokens[3] = (b2.prefix_tokens[3] + 1) % w.model.vocab
    b2.labels[3] = (b2.labels[3] + 1) % w.model.n_classes
    r2 = om.rollout(b2, W=4, seed=9)
    assert np.array_equal(r1["tokens"][:3], r2["tokens"][:3])
    assert np.array_equal(r1["counts"][:, :3].sum(0), r2["counts"][:, :3].sum(0))


# ------------------------------------------------------------------ batch-synchronous windows


def replay_sync_schedule(counts, prefix_len, T, W):
    """Replays per-round counts against the shared-window rule (Sec. 4.1,
    Fig. 2a): image b's window w ends at min(k_b + (w+1) W, T); the batch moves
    to window w+1 only when every active image has reached the end of window w;
    until then an image at its boundary commits nothing. Returns the final
    cursors."""
    n = np.asarray(prefix_len, dtype=np.int64).copy()
    e = np.minimum(n + W, T)
    for c in counts:
        act = n < T
        if not np.any(act & (n < e)):
            e = np.minimum(e + W, T)
        for b in range(len(n)):
            if not act[b]:
                assert c[b] == 0
            elif n[b] < e[b]:
                assert 1 <= c[b] <= min(W, e[b] - n[b]), (b, n[b], e[b], c[b])
            else:
                assert c[b] == 0, (b, n[b], e[b], c[b])
        n += c
    return n


@pytest.mark.parametrize("W,H", [(1, 24), (3, 24), (4, 2), (16, 3)])
def test_sync_greedy_equals_greedy_ar(tiny, W, H):
    w, _, om = tiny
    b = _batch(w, 2)
    r = om.rollout(b, W=W, H=H, seed=5, greedy=True, sync=True)
    ar = om.rollout_ar(b, seed=5, greedy=True)
    assert np.array_equal(r["tokens"], ar)
    assert np.array_equal(replay_sync_schedule(r["counts"], b.prefix_len, w.model.T, W),
                          np.full(len(b.prefix_len), w.model.T))


def test_sync_greedy_with_cfg_equals_greedy_ar():
    shape = synth.small_shape(n_layers=2, d_model=32, n_heads=2, mlp_hidden=48, vocab=40,
                              n_classes=4, grid=4)
    om = oracle.Model(shape, synth.make_weights(shape, 3, std=0.2))
    w = synth.Workload("t", shape, "f32", 6, 3, 2, 7, 2.0, prefix_lo=0, prefix_hi=9)
    b = _batch(w, 5)
    r = om.rollout(b, W=3, H=2, top_k=7, cfg_scale=2.0, seed=77, greedy=True, sync=True)
    ar = om.rollout_ar(b, top_k=7, cfg_scale=2.0, seed=77, greedy=True)
    assert np.array_equal(r["tokens"], ar)
    replay_sync_schedule(r["counts"], b.prefix_len, shape.T, 3)


@pytest.mark.parametrize("seed", [1000, 1001])
def test_sync_window_one_is_token_by_token_sampling(tiny, seed):
    w, _, om = tiny
    b = _batch(w)
    r = om.rollout(b, W=1, seed=seed, sync=True)
    assert np.array_equal(r["tokens"], om.rollout_ar(b, seed=seed))


def test_sync_single_window_is_independent_progress(tiny):
    """When one window spans every suffix (W >= T - k_b) no boundary falls
    before T, so the synchronous schedule is the independent one."""
    w, _, om = tiny
    b = _batch(w, 7)
    T = w.model.T
    b.prefix_len[:] = np.maximum(b.prefix_len, T - 16)
    ind = om.rollout(b, W=16, seed=31)
    syn = om.rollout(b, W=16, seed=31, sync=True)
    assert np.array_equal(ind["tokens"], syn["tokens"])
    assert np.array_equal(ind["counts"], syn["counts"])


@pytest.mark.parametrize("W", [2, 4, 9])
def test_sync_schedule_full_compact_and_waiting(tiny, W):
    w, _, om = tiny
    b = _batch(w, 3)
    b.prefix_len[1] = 60
    T = w.model.T
    runs = [om.rollout(b, W=W, seed=11, exec_mode=m, gamma=2, sync=True) for m in (0, 1, 2)]
    for r in runs[1:]:
        assert np.array_equal(r["tokens"], runs[0]["tokens"])
        assert np.array_equal(r["counts"], runs[0]["counts"])
    r = runs[0]
    n = replay_sync_schedule(r["counts"], b.prefix_len, T, W)
    assert np.array_equal(n, np.full(len(b.prefix_len), T))
    for i in range(len(b.prefix_len)):
        assert np.array_equal(r["tokens"][i, :b.prefix_len[i]], b.prefix_tokens[i, :b.prefix_len[i]])
    assert r["rounds"] <= T - int(b.prefix_len.min())
    assert (r["counts"] == 0).any()
    assert r["image_rounds"] == int((r["counts"] > 0).sum())
    ind = om.rollout(b, W=W, seed=11)
    assert r["rounds"] >= max(int(np.ceil((T - k) / W)) for k in b.prefix_len)
    assert ind["verified"] == r["verified"] == int((T - b.prefix_len).sum())


# ------------------------------------------------------------------ chi-square


def _tiny_peaky():
    shape = synth.small_shape(n_layers=2, d_model=16, n_heads=2, mlp_hidden=32, vocab=4,
                              n_classes=3, grid=2)
    blob = synth.make_weights(shape, 11, std=1.0)
    return shape, blob, oracle.Model(shape, blob)


def _exact_joint(om, shape, cls, top_k, tau, cfg):
    """Probability of each of the V^T suffixes under token-by-token sampling."""
    V, T = shape.vocab, shape.T
    out = np.zeros(V ** T)
    for idx, seq in enumerate(itertools.product(range(V), repeat=T)):
        lg = om.forward_seq(cls, seq[:-1]).astype(np.float32)
        if cfg:
            lu = om.forward_seq(shape.n_classes, seq[:-1]).astype(np.float32)
        pr = 1.0
        for t in range(T):
            l = oracle.cfg_combine(lg[t], lu[t], cfg) if cfg else lg[t]
            pr *= float(oracle.transform(l, tau, top_k)[seq[t]].astype(np.float64))
        out[idx] = pr
    return out / out.sum()


def _chi2_pvalue(om, shape, W, H, top_k, tau, cfg, n=20000, seed=123, sync=False):
    V, T = shape.vocab, shape.T
    cls = 1
    probs = _exact_joint(om, shape, cls, top_k, tau, cfg)
    b = synth.Batch(np.zeros((n, T), dtype=np.int32), np.zeros(n, dtype=np.int32),
                    np.full(n, cls, dtype=np.int32), np.full(n, tau, dtype=np.float32))
    r = om.rollout(b, W=W, H=H, top_k=top_k, cfg_scale=cfg, seed=seed, exec_mode=1, sync=sync)
    idx = np.zeros(n, dtype=np.int64)
    for t in range(T):
        idx = idx * V + r["tokens"][:, t]
    obs = np.bincount(idx, minlength=V ** T).astype(np.float64)
    exp = probs * n
    if np.any(obs[exp == 0] > 0):
        return 0.0, r
    big = exp >= 5
    o = np.append(obs[big], obs[~big].sum())
    e = np.append(exp[big], exp[~big].sum())
    if e[-1] == 0:
        o, e = o[:-1], e[:-1]
    return stats.chisquare(o, e * o.sum() / e.sum()).pvalue, r


@pytest.mark.slow
@pytest.mark.parametrize("W,H,top_k,tau,cfg", [(2, 24, 0, 1.0, 0.0), (3, 2, 0, 1.0, 0.0),
                                                (3, 1, 2, 1.0, 0.0), (2, 2, 0, 0.7, 2.0),
                                                (4, 1, 3, 1.3, 0.0)])
def test_sjd_suffix_distribution_matches_brute_force(W, H, top_k, tau, cfg):
    shape, _, om = _tiny_peaky()
    pv, r = _chi2_pvalue(om, shape, W, H, top_k, tau, cfg)
    assert pv > 1e-3, pv
    # the rollout really speculated: some rounds committed more than one token
    assert r["counts"].max() > 1 and r["rejected"] > 0


@pytest.mark.slow
@pytest.mark.parametrize("W,H,top_k,tau,cfg", [(2, 24, 0, 1.0, 0.0), (3, 1, 2, 1.0, 0.0),
                                                (2, 2, 0, 0.7, 2.0)])
def test_sync_suffix_distribution_matches_brute_force(W, H, top_k, tau, cfg):
    """Batch-synchronous windows change which drafts are verified when, not the
    law of the output: 20000 images share every window boundary, so most of
    them wait (and re-draw their first draft) at each boundary."""
    shape, _, om = _tiny_peaky()
    pv, r = _chi2_pvalue(om, shape, W, H, top_k, tau, cfg, sync=True)
    assert pv > 1e-3, pv
    assert r["counts"].max() > 1 and r["rejected"] > 0
    assert (r["counts"] == 0).any()      # waiting image-rounds happened


@pytest.mark.slow
@pytest.mark.parametrize("flag", [oracle.DEBUG_RESIDUAL_DROPS_Q, oracle.DEBUG_INVERTED_RATIO])
def test_planted_mistakes_fail_the_distribution_test(flag):
    shape, _, om = _tiny_peaky()
    oracle.set_debug(flag)
    try:
        pv, _ = _chi2_pvalue(om, shape, 3, 2, 0, 1.0, 0.0)
    finally:
        oracle.set_debug(0)
    assert pv < 1e-6, pv
