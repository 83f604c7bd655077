"""The measured-ceiling kernels (a benchmark aid beside the hook step) run
and leave their sinks alone."""
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def test_read_and_mfma_ceilings_run():
    from paper_2607_22595_amd import ceiling
    buf = torch.arange(1 << 20, dtype=torch.int32, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    assert ceiling.read(buf, sink) == 4 << 20
    fsink = torch.zeros(1, dtype=torch.float32, device="cuda")
    flops = ceiling.mfma(10, fsink)
    torch.cuda.synchronize()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    assert flops == cus * 4 * 8 * 10 * 2 * 32 * 32 * 16
    assert int(sink.item()) == 0 and float(fsink.item()) == 0.0
    with pytest.raises(ValueError):
        ceiling.read(buf.cpu(), sink)
