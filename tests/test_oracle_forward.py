"""Pins of the oracle's decoder (the student p_theta of Sec. 3.1, Eq. 1) against
an independent float64 numpy composition, plus RoPE invariants."""
import numpy as np
import pytest

import oracle
import synth
from tests import np_reference as npr


def _check_forward(shape, blob, seed, n):
    rng = np.random.default_rng(seed)
    om = oracle.Model(shape, blob)
    toks = rng.integers(0, shape.vocab, size=n)
    cls = int(rng.integers(0, shape.n_classes + 1))   # includes the null class
    got = om.forward_seq(cls, toks).astype(np.float64)
    ref = npr.forward(shape, blob, cls, toks)
    return np.max(np.abs(got - ref)), np.max(np.abs(ref))


@pytest.mark.parametrize("n", [0, 1, 17, 64])
def test_forward_matches_float64_tiny(tiny, n):
    w, blob, _ = tiny
    err, scale = _check_forward(w.model, blob, n, n)
    assert err <= 2e-5 * max(1.0, scale), (err, scale)


def test_forward_matches_float64_with_bias_and_other_shape():
    shape = synth.small_shape(n_layers=3, d_model=48, n_heads=3, mlp_hidden=40, vocab=37,
                              n_classes=5, grid=5, has_lm_bias=True)
    blob = synth.make_weights(shape, 7, std=0.3, bias_std=1.0)
    err, scale = _check_forward(shape, blob, 3, shape.T)
    assert err <= 2e-5 * max(1.0, scale), (err, scale)


def test_planted_rope_sign_mistake_is_caught(tiny):
    w, blob, _ = tiny
    oracle.set_debug(oracle.DEBUG_ROPE_SIGN)
    try:
        err, scale = _check_forward(w.model, blob, 1, 30)
    finally:
        oracle.set_debug(0)
    assert err > 1e-3 * max(1.0, scale)


def test_rope_relative_shift_invariance():
    """q.k after 2D RoPE depends only on the grid offset between the two positions."""
    shape = synth.small_shape(d_model=64, n_heads=1, grid=8)
    om = oracle.Model(shape, synth.make_weights(shape, 0))
    rng = np.random.default_rng(0)
    q, k = rng.standard_normal(64).astype(np.float32), rng.standard_normal(64).astype(np.float32)
    G = shape.grid

    def pos(r, c):
        return 1 + r * G + c

    base = float(np.dot(om.rope(q, pos(1, 2)), om.rope(k, pos(3, 5))))
    for dr, dc in [(1, 0), (0, 2), (3, 1), (4, 2)]:
        other = float(np.dot(om.rope(q, pos(1 + dr, 2 + dc)), om.rope(k, pos(3 + dr, 5 + dc))))
        assert abs(other - base) <= 1e-4 * (1 + abs(base))
    # a different offset gives a different product
    assert abs(float(np.dot(om.rope(q, pos(1, 2)), om.rope(k, pos(4, 5)))) - base) > 1e-3


def test_rope_position_zero_identity_and_norm():
    shape = synth.small_shape(d_model=32, n_heads=2, grid=4)
    om = oracle.Model(shape, synth.make_weights(shape, 0))
    u = np.random.default_rng(1).standard_normal(16).astype(np.float32)
    assert np.array_equal(om.rope(u, 0), u)
    for s in [1, 5, 16, 20]:
        r = om.rope(u, s)
        assert abs(np.linalg.norm(r) - np.linalg.norm(u)) < 1e-5
    assert np.array_equal(om.rope(u, 16), om.rope(u, 19))   # clamped past T
    # position 1 is grid cell (0, 0): no rotation either
    assert np.allclose(om.rope(u, 1), u, atol=0)
