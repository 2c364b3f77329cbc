"""The entry point that allocates nothing: hbsjd_transform_rows_noalloc, called
through the C ABI, gives the same outputs as hbsjd_transform_rows (the same
kernels on the same inputs, so bit for bit) on two calls in a row, the second
with fewer rows than the first, so the second runs on the workspace the first
left behind; and it rejects more rows than its fixed workspace holds."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

V = 16384


def P():
    import paper_2608_18183_amd
    return paper_2608_18183_amd


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    P().load_library()
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")


def _inputs(rows, cfg, seed):
    rng = np.random.default_rng(seed)
    lg = rng.normal(0, 2.0, (rows, 2 if cfg else 1, V)).astype(np.float32)
    tau = np.where(np.arange(rows) % 2 == 0, 0.3, 1.5).astype(np.float32)
    pos = rng.integers(0, 600, rows).astype(np.int32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return dev(lg if cfg else lg[:, 0]), dev(tau), dev(pos)


@pytest.mark.parametrize("cfg", [0.0, 2.0])
def test_noalloc_equals_allocating_entry_on_two_calls(cfg):
    for i, rows in enumerate([700, 37]):
        lg, tau, pos = _inputs(rows, cfg, 100 + i)
        want = P().hbsjd_transform_rows(lg, tau, pos, top_k=1000, cfg_scale=cfg, seed=77 + i)
        out = (torch.full((rows, V), -7.0, dtype=torch.float32, device="cuda"),
               torch.full((rows,), -7, dtype=torch.int32, device="cuda"),
               torch.full((rows,), -7, dtype=torch.int32, device="cuda"))
        got = P().hbsjd_transform_rows(lg, tau, pos, top_k=1000, cfg_scale=cfg, seed=77 + i,
                                       out=out, noalloc=True)
        torch.cuda.synchronize()
        for g, w in zip(got, want):
            assert torch.equal(g, w), (rows, cfg)
        assert int((got[2] < 0).sum()) == 0


def test_noalloc_rejects_rows_beyond_its_workspace():
    rows = 65537
    lg = torch.zeros((rows, 4), dtype=torch.float32, device="cuda")
    tau = torch.ones(rows, dtype=torch.float32, device="cuda")
    pos = torch.ones(rows, dtype=torch.int32, device="cuda")
    with pytest.raises(P().HbsjdError) as ei:
        P().hbsjd_transform_rows(lg, tau, pos, noalloc=True)
    assert ei.value.code == "EINVAL"
    # the largest size it takes still works
    rows = 65536
    got = P().hbsjd_transform_rows(lg[:rows], tau[:rows], pos[:rows], noalloc=True)
    want = P().hbsjd_transform_rows(lg[:rows], tau[:rows], pos[:rows])
    for g, w in zip(got, want):
        assert torch.equal(g, w)
