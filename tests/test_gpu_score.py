"""GPU teacher scoring (Sec. 3.1, Eq. 3) through the C ABI against the oracle:
the per-row bidirectional-KL kernel on seeded logits rows, and the whole
scoring call (two forwards + the kernel + the per-image mean) on a tiny fp32
student/teacher pair and on the B student with an L-architecture teacher in
bf16."""
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


@pytest.mark.parametrize("rows,V,scale", [(33, 256, 2.0), (7, 1000, 0.5), (300, 16384, 3.0),
                                          (5, 4, 1.0), (2, 16380, 8.0)])
def test_bikl_rows_matches_oracle(rows, V, scale):
    rng = np.random.default_rng(rows * 7 + V)
    ls = rng.normal(0, scale, size=(rows, V)).astype(np.float32)
    lt = (ls + rng.normal(0, scale, size=(rows, V))).astype(np.float32)
    lt[0] = ls[0]                                    # identical rows: exactly 0
    lt[1] = ls[1] + np.float32(3.0)                  # shifted rows: the same distribution
    got = P().hbsjd_bikl_rows(torch.from_numpy(ls).cuda(), torch.from_numpy(lt).cuda())
    got = got.cpu().numpy().astype(np.float64)
    ref = oracle.bikl(ls, lt)
    # fp32 sums of V terms each below max|ls - lt|: relative 1e-4 plus a floor
    tol = 1e-4 * np.abs(ref) + 2e-6 * (1 + np.abs(ls - lt).max(axis=1))
    assert np.all(np.abs(got - ref) <= tol), np.max(np.abs(got - ref) / tol)
    assert got[0] == 0.0
    assert abs(got[1]) <= 1e-5


def _tokens(rng, B, shape):
    return rng.integers(0, shape.vocab, size=(B, shape.T)).astype(np.int32)


def test_score_f32_tiny_matches_oracle():
    shape = synth.WORKLOADS["tiny"].model
    sb = synth.make_weights(shape, 0, std=0.2)
    tb = synth.make_weights(shape, 9, std=0.2)
    rng = np.random.default_rng(3)
    B = 5
    tok = _tokens(rng, B, shape)
    k = np.array([0, 17, shape.T, shape.T - 1, 40], dtype=np.int32)
    lab = rng.integers(0, shape.n_classes, size=B).astype(np.int32)
    s, t = gu.make_ctx(shape, "f32", sb), gu.make_ctx(shape, "f32", tb)
    per, loss = s.hbsjd_score_bikl(t, torch.from_numpy(tok).cuda(), k, lab)
    per, loss = per.cpu().numpy().astype(np.float64), loss.cpu().numpy().astype(np.float64)
    rper, rloss = oracle.score_bikl(oracle.Model(shape, sb), oracle.Model(shape, tb), tok, k, lab)
    assert np.allclose(per, rper, rtol=2e-4, atol=2e-6)
    assert np.allclose(loss, rloss, rtol=2e-4, atol=2e-6)
    assert np.all(per[2] == 0) and loss[2] == 0
    assert np.all(per[1, :17] == 0)
    # the same model on both sides scores zero everywhere
    s2 = gu.make_ctx(shape, "f32", sb)
    per0, loss0 = s.hbsjd_score_bikl(s2, torch.from_numpy(tok).cuda(), k, lab)
    assert torch.all(per0 == 0) and torch.all(loss0 == 0)


def _bf16_tol(ls, lt, eps=3e-2):
    """bf16 forwards carry logit errors of at most eps = 3e-2 (the forward bar).
    Moving both logits rows by at most eps moves D = (E_p[d] - E_q[d]) / 2,
    d = ls - lt, by at most 2 eps + eps (1 + eps) range(d): |d' - d| <= 2 eps,
    and each softmax moves by at most e^{2 eps} - 1 in total variation, which
    against d costs half that times d's range. That bound is the tolerance."""
    d = np.asarray(ls, np.float64) - np.asarray(lt, np.float64)
    return 2 * eps + eps * (1 + eps) * (d.max(axis=-1) - d.min(axis=-1))


def test_score_bf16_small_pair_matches_oracle():
    sshape = synth.small_shape(n_layers=2, d_model=128, n_heads=2, mlp_hidden=256, vocab=1024,
                               n_classes=10, grid=8)
    tshape = synth.small_shape(n_layers=3, d_model=192, n_heads=3, mlp_hidden=320, vocab=1024,
                               n_classes=10, grid=8)
    sb = synth.make_weights(sshape, 0, std=0.05)
    tb = synth.make_weights(tshape, 1, std=0.05)
    rng = np.random.default_rng(4)
    B = 6
    tok = _tokens(rng, B, sshape)
    k = np.array([0, 1, 30, sshape.T - 1, sshape.T, 12], dtype=np.int32)
    lab = rng.integers(0, 10, size=B).astype(np.int32)
    s, t = gu.make_ctx(sshape, "bf16", sb), gu.make_ctx(tshape, "bf16", tb)
    per, loss = s.hbsjd_score_bikl(t, torch.from_numpy(tok).cuda(), k, lab)
    per, loss = per.cpu().numpy().astype(np.float64), loss.cpu().numpy().astype(np.float64)
    so = oracle.Model(sshape, gu.bf16_rounded_blob(sshape, sb))
    to = oracle.Model(tshape, gu.bf16_rounded_blob(tshape, tb))
    rper, rloss = oracle.score_bikl(so, to, tok, k, lab)
    seqs = [tok[b, :sshape.T - 1] for b in range(B)]
    ls, lt = so.forward_batch(lab, seqs), to.forward_batch(lab, seqs)
    T = sshape.T
    for b in range(B):
        assert np.all(per[b, :k[b]] == 0)
        if k[b] == T:
            assert loss[b] == 0
            continue
        tol = _bf16_tol(ls[b][k[b]:T], lt[b][k[b]:T])
        err = np.abs(per[b, k[b]:] - rper[b, k[b]:])
        assert np.all(err <= tol), (b, (err / tol).max())
        assert abs(loss[b] - rloss[b]) <= tol.mean()
        assert loss[b] == pytest.approx(per[b, k[b]:].mean(), rel=1e-5)


def test_score_full_size_b_student_l_teacher():
    """The B student against an L-architecture teacher at the full 16x16 grid:
    a few early positions the oracle computes one at a time, the symmetry of
    the divergence (swapping the two models gives the same values up to fp32
    rounding), and the per-image mean."""
    wl = synth.WORKLOADS["llamagen_b"]
    sshape = wl.model
    tshape = synth.teacher_shape(sshape)
    sb = synth.make_weights(sshape, 0)
    tb = synth.make_weights(tshape, 5)
    rng = np.random.default_rng(8)
    B = wl.batch
    tok = torch.from_numpy(_tokens(rng, B, sshape)).cuda()
    k = synth.make_batch(wl, 1).prefix_len.astype(np.int32)
    k[0], k[1] = 2, sshape.T
    lab = rng.integers(0, sshape.n_classes, size=B).astype(np.int32)
    s, t = gu.make_ctx(sshape, "bf16", sb), gu.make_ctx(tshape, "bf16", tb)
    per, loss = s.hbsjd_score_bikl(t, tok, k, lab)
    per2, loss2 = t.hbsjd_score_bikl(s, tok, k, lab)
    torch.testing.assert_close(per2, per, rtol=1e-6, atol=1e-7)
    torch.testing.assert_close(loss2, loss, rtol=1e-6, atol=1e-7)
    per, loss = per.cpu().numpy().astype(np.float64), loss.cpu().numpy().astype(np.float64)
    T = sshape.T
    for b in range(B):
        assert np.all(per[b, :k[b]] == 0)
        if k[b] < T:
            assert np.all(per[b, k[b]:] >= -1e-6)
            assert loss[b] == pytest.approx(per[b, k[b]:].mean(), rel=1e-5)
    assert loss[1] == 0
    so = oracle.Model(sshape, gu.bf16_rounded_blob(sshape, sb))
    to = oracle.Model(tshape, gu.bf16_rounded_blob(tshape, tb))
    x = tok[0].cpu().numpy()
    for pos in [3, 4, 12]:
        ls = so.forward_seq(lab[0], x[:pos - 1])[-1]
        lt = to.forward_seq(lab[0], x[:pos - 1])[-1]
        ref = float(oracle.bikl(ls, lt))
        assert abs(per[0, pos - 1] - ref) <= _bf16_tol(ls, lt), (pos, per[0, pos - 1], ref)


def test_score_argument_errors():
    shape = synth.WORKLOADS["tiny"].model
    other = synth.small_shape(n_layers=1, d_model=64, n_heads=4, mlp_hidden=64, vocab=128,
                              n_classes=10, grid=8)
    s = gu.make_ctx(shape, "f32", synth.make_weights(shape, 0))
    t = gu.make_ctx(other, "f32", synth.make_weights(other, 1))
    tok = torch.zeros((2, shape.T), dtype=torch.int32, device="cuda")
    with pytest.raises(P().HbsjdError, match="EINVAL"):
        s.hbsjd_score_bikl(t, tok, [0, 0], [0, 0])          # vocabularies differ
    with pytest.raises(P().HbsjdError, match="EINVAL"):
        s.hbsjd_score_bikl(s, tok, [0, 0], [0, 0])          # one context twice
    t2 = gu.make_ctx(shape, "f32", synth.make_weights(shape, 1))
    with pytest.raises(P().HbsjdError, match="EINVAL"):
        s.hbsjd_score_bikl(t2, tok, [0, shape.T + 1], [0, 0])
    bad = tok.clone()
    bad[1, 5] = shape.vocab
    with pytest.raises(P().HbsjdError, match="EINVAL"):
        s.hbsjd_score_bikl(t2, bad, [0, 0], [0, 0])
    per, loss = s.hbsjd_score_bikl(t2, tok, [shape.T, shape.T], [0, 1])
    assert torch.all(per == 0) and torch.all(loss == 0)
