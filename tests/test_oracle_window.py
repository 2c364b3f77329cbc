"""Pins of the window refresh (Sec. 4.2, "Independent rollout states"): after the
prefill and after every round, positions covered by the round's rows get a
reused prediction and the rest get the history token at offset H, taken from the
committed tokens followed by the drafts already set (one position back when
pos - H < 1).

The expected windows below were worked out by hand, not by running any code.
They use a student whose argmax is one fixed token c = 31 at every position
(an lm_head bias of 50 on c against N(0, 0.02) weights): under greedy
verification (Eq. 4) every reused prediction is c and every committed token
after the prefix is c, so each window is determined by the prefix x_t = t, by
W and H, and by the rule itself. A history token therefore shows up as a small
prefix number at a fixed place in the window, and shifting the offset or the
reused row by one position changes that place.
"""
import numpy as np
import pytest

import oracle
import synth

C = 31   # the student's fixed argmax


@pytest.fixture(scope="module")
def fixed_argmax_model():
    shape = synth.small_shape(n_layers=1, d_model=16, n_heads=2, mlp_hidden=32, vocab=32,
                              n_classes=3, grid=5, has_lm_bias=True)
    blob = synth.make_weights(shape, 11, std=0.02, bias_std=0.0)
    synth.split_blob(shape, blob)["b_lm"][C] = 50.0
    return shape, oracle.Model(shape, blob)


def _batch(shape, prefix_lens):
    B = len(prefix_lens)
    toks = np.zeros((B, shape.T), dtype=np.int32)
    toks[:] = np.arange(1, shape.T + 1, dtype=np.int32)    # x_t = t
    return synth.Batch(toks, np.array(prefix_lens, dtype=np.int32),
                       np.zeros(B, dtype=np.int32), np.ones(B, dtype=np.float32))


def _run(model, prefix_lens, W, H, sync=False):
    shape, om = model
    b = _batch(shape, prefix_lens)
    return om.rollout(b, W=W, H=H, seed=3, greedy=True, sync=sync, trace=True)


# T = 25; the comments list the window's positions and where each draft comes from


def _case_independent_k10_w4_h6():
    return dict(prefix_lens=[10], W=4, H=6, counts=[[2], [4], [4], [4], [1]], windows=[
        # after the prefill: 11 reused; 12, 13, 14 <- S[6], S[7], S[8]
        [[C, 6, 7, 8]],
        # round 1 commits c at 11 and c at 12 (the draft 6 is rejected); rows
        # predicted 11..15, so 13..15 are reused; 16 <- S[10] = 10
        [[C, C, C, 10]],
        # round 2 commits 13..16 (10 rejected); 17 reused; 18..20 <- S[12..14] = c
        [[C, C, C, C]],
        [[C, C, C, C]],
        # round 4 reaches 24: one position left, reused
        [[C, -1, -1, -1]],
        [[-1, -1, -1, -1]],
    ])


def _case_independent_k10_w6_h3():
    # the history source lies among the drafts already set: 14 <- S[11] (the
    # reused draft), 15 <- S[12], 16 <- S[13] (history drafts themselves)
    return dict(prefix_lens=[10], W=6, H=3, counts=None, windows=[[[C, 9, 10, C, 9, 10]]])


def _case_fallback_k2_w4_h5():
    return dict(prefix_lens=[2], W=4, H=5, counts=None, windows=[
        # 3 reused; 4 and 5 have pos - H < 1, so they take S[pos - 1] = c; 6 <- S[1] = 1
        [[C, C, C, 1]],
        # round 1 commits 3..6 (the draft 1 is rejected); 7 reused; 8..10 <- S[3..5] = c
        [[C, C, C, C]],
    ])


CASES = {"k10_w4_h6": _case_independent_k10_w4_h6, "k10_w6_h3": _case_independent_k10_w6_h3,
         "fallback_k2_w4_h5": _case_fallback_k2_w4_h5}


def _check(model, case, sync=False):
    r = _run(model, case["prefix_lens"], case["W"], case["H"], sync=sync)
    tr = r["trace_drafts"]
    for i, want in enumerate(case["windows"]):
        assert np.array_equal(tr[i], np.array(want)), (i, tr[i].tolist(), want)
    if case["counts"] is not None:
        assert np.array_equal(r["counts"], np.array(case["counts"])), r["counts"].tolist()
    # greedy proposals are deterministic: q(z) = 1 wherever a draft exists
    assert np.array_equal(r["trace_q"], np.where(tr >= 0, 1.0, 0.0).astype(np.float32))
    return r


@pytest.mark.parametrize("name", sorted(CASES))
def test_window_refresh_matches_hand_derived_windows(fixed_argmax_model, name):
    _check(fixed_argmax_model, CASES[name]())


def test_batch_synchronous_windows_match_hand_derivation(fixed_argmax_model):
    """Shared window boundaries (Sec. 4.1, Fig. 2a; reading: window w of image b
    ends at min(k_b + (w+1) W, T)) on two images, k = 10 and k = 3, W = 4,
    H = 6: image 1 reaches its first boundary in round 1 and waits (count 0)
    while image 0 finishes its window; then both move on."""
    case = dict(prefix_lens=[10, 3], W=4, H=6, counts=[[2, 4], [2, 0], [2, 2], [2, 2], [4, 4],
                                                       [3, 4], [0, 4], [0, 2]], windows=[
        # image 0: 11 reused, 12..14 <- S[6..8]; image 1: 4 reused, 5 and 6
        # fall back to S[4], S[5] (c), 7 <- S[1] = 1
        [[C, 6, 7, 8], [C, C, C, 1]],
        # image 0 commits 11, 12 (6 rejected): 13..15 reused, 16 <- S[10] = 10;
        # image 1 commits 4..7 and sits at its boundary 7: 8 reused, 9 <- S[3] = 3,
        # 10, 11 <- S[4], S[5] = c
        [[C, C, C, 10], [C, 3, C, C]],
        # image 0 verifies up to its boundary 14 (two drafts, both accepted): 15
        # reused, 16 <- S[10] = 10, 17, 18 <- c; image 1 waits and redraws its
        # window from row 0 alone: the same window
        [[C, 10, C, C], [C, 3, C, C]],
    ])
    _check(fixed_argmax_model, case, sync=True)


@pytest.mark.parametrize("flag", [oracle.DEBUG_HISTORY_SHIFT, oracle.DEBUG_REUSE_SHIFT])
def test_planted_window_mistakes_fail_the_pins(fixed_argmax_model, flag):
    """A history offset one position off, or a reused prediction taken from the
    neighbouring row, must fail every hand-derived window."""
    oracle.set_debug(flag)
    try:
        failed = 0
        for name in sorted(CASES):
            try:
                _check(fixed_argmax_model, CASES[name]())
            except AssertionError:
                failed += 1
        assert failed == len(CASES)
    finally:
        oracle.set_debug(0)


def test_trace_q_of_probabilistic_windows(tiny):
    """Probabilistic mode (Eq. 5): a reused draft's recorded proposal
    probability is its row's p(z) > 0, and a history draft's is 1 (point
    mass). The first window position is always a reused prediction, and every
    complete image's window is empty."""
    w, _, om = tiny
    b = synth.make_batch(w, 1)
    r = om.rollout(b, W=4, H=24, seed=1000, trace=True)
    d, q = r["trace_drafts"], r["trace_q"]
    assert np.all(q[d < 0] == 0) and np.all(q[d >= 0] > 0) and np.all(q <= 1)
    first = d[:, :, 0]
    assert np.all(q[:, :, 0][first >= 0] < 1)     # no point mass at the first position
    n = np.array(b.prefix_len, dtype=np.int64)
    T = w.model.T
    for i, c in enumerate(r["counts"]):
        n = n + c
        assert np.all(d[i + 1][n >= T] == -1)
