"""Pins of the oracle's teacher-scoring objective (Sec. 3.1, Eq. 3): the
bidirectional KL against scipy's relative entropy and the two-outcome closed
form, its invariants, and the per-position alignment of the sequence score
against one-sequence-at-a-time forwards."""
import numpy as np
import pytest
from scipy import stats

import oracle
import synth


def _softmax(l):
    e = np.exp(l - l.max())
    return e / e.sum()


def test_bikl_matches_scipy_relative_entropy():
    rng = np.random.default_rng(0)
    for V in [2, 7, 256, 4096]:
        ls, lt = rng.normal(0, 2, size=(2, V))
        p, q = _softmax(ls), _softmax(lt)
        ref = 0.5 * stats.entropy(p, q) + 0.5 * stats.entropy(q, p)
        assert oracle.bikl(ls, lt) == pytest.approx(ref, rel=1e-10, abs=1e-14)


def test_bikl_two_outcome_closed_form():
    for a, b in [(0.3, -1.2), (4.0, 0.0), (-2.5, 2.5)]:
        p = 1.0 / (1.0 + np.exp(-a))         # softmax([a, 0]) of the first entry
        q = 1.0 / (1.0 + np.exp(-b))
        kl_pq = p * np.log(p / q) + (1 - p) * np.log((1 - p) / (1 - q))
        kl_qp = q * np.log(q / p) + (1 - q) * np.log((1 - q) / (1 - p))
        got = oracle.bikl([a, 0.0], [b, 0.0])
        assert got == pytest.approx(0.5 * (kl_pq + kl_qp), rel=1e-12)
        # the two-outcome biKL is also (p - q)(logit p - logit q) / 2
        assert got == pytest.approx(0.5 * (p - q) * (a - b), rel=1e-12)


def test_bikl_invariants():
    rng = np.random.default_rng(1)
    ls, lt = rng.normal(0, 1, size=(2, 5, 300))
    d = oracle.bikl(ls, lt)
    assert d.shape == (5,) and (d > 0).all()
    assert np.allclose(d, oracle.bikl(lt, ls), rtol=1e-12)              # symmetric
    shift = rng.normal(0, 5, size=(5, 1))
    assert np.allclose(d, oracle.bikl(ls + shift, lt - 2 * shift), rtol=1e-9)
    assert np.all(oracle.bikl(ls, ls) == 0.0)
    # extra mass on one entry moves the divergence away from zero smoothly
    small = oracle.bikl(ls[0], ls[0] + 1e-3 * (np.arange(300) == 4))
    assert 0 < small < 1e-6


def _teacher_student():
    shape = synth.small_shape(n_layers=2, d_model=32, n_heads=2, mlp_hidden=48, vocab=64,
                              n_classes=4, grid=4)
    s = oracle.Model(shape, synth.make_weights(shape, 3, std=0.3))
    t = oracle.Model(shape, synth.make_weights(shape, 4, std=0.3))
    return shape, s, t


def test_score_alignment_against_single_sequence_forwards():
    shape, s, t = _teacher_student()
    T = shape.T
    rng = np.random.default_rng(5)
    tok = rng.integers(0, shape.vocab, size=(3, T)).astype(np.int32)
    k = np.array([0, 9, T], dtype=np.int32)
    lab = np.array([1, 3, 0], dtype=np.int32)
    per, loss = oracle.score_bikl(s, t, tok, k, lab)
    for b in range(3):
        for pos in range(1, T + 1):
            if pos <= k[b]:
                assert per[b, pos - 1] == 0.0
                continue
            # the distribution of x_pos given [class, x_1..x_{pos-1}] only
            ls = s.forward_seq(lab[b], tok[b, :pos - 1])[-1]
            lt = t.forward_seq(lab[b], tok[b, :pos - 1])[-1]
            assert per[b, pos - 1] == pytest.approx(float(oracle.bikl(ls, lt)), rel=1e-9)
    assert loss[0] == pytest.approx(per[0].mean())
    assert loss[1] == pytest.approx(per[1, 9:].mean())
    assert loss[2] == 0.0


def test_score_of_a_model_against_itself_is_zero():
    shape, s, _ = _teacher_student()
    tok = np.random.default_rng(6).integers(0, shape.vocab, size=(2, shape.T)).astype(np.int32)
    per, loss = oracle.score_bikl(s, s, tok, np.array([3, 0]), np.array([0, 2]))
    assert np.all(per == 0.0) and np.all(loss == 0.0)
