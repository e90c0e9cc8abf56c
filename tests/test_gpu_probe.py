"""The MFMA throughput probe (a measurement helper of the library) runs and
leaves finite values in its sink; bench.py divides kernel rates by what it
measures."""
import pytest

torch = pytest.importorskip("torch")

from paper_2605_15684_amd import _lib


@pytest.mark.gpu
def test_probe_runs():
    sink = torch.full((8 * 256,), float("nan"), dtype=torch.float32, device="cuda")
    st = _lib.probe_mfma(8, 50, sink.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert torch.isfinite(sink).all()
