"""The MFMA calibration entry (a measurement aid): it runs to completion on
every CU, leaves its sink untouched and rejects bad arguments."""
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def test_mfma_probe_runs_and_checks_arguments():
    import paper_2608_18183_amd as P
    P.load_library()
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible GPU")
    sink = torch.full((256,), 7.0, dtype=torch.float32, device="cuda")
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    P.hbsjd_mfma_probe(cus, 64, sink)
    torch.cuda.synchronize()
    assert bool((sink == 7.0).all())
    for wg, it in [(0, 64), (cus, 0), (-1, 5)]:
        with pytest.raises(P.HbsjdError) as ei:
            P.hbsjd_mfma_probe(wg, it, sink)
        assert ei.value.code == "EINVAL"
    with pytest.raises(ValueError):
        P.hbsjd_mfma_probe(cus, 64, sink[:16])
