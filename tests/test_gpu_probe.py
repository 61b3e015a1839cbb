"""The matrix-core rate probe (mla_probe_mfma_bf16, a diagnostic the benchmark
sets its measured rates against): it runs on the device, reports the flop of its
launch, leaves its sink untouched, and measures a rate between a fraction of the
data sheet's dense bf16 figure and that figure itself."""
import pytest
import torch

pytestmark = pytest.mark.gpu


def test_probe_rate_is_physical():
    from paper_2609_07008_amd import mla
    stream = torch.cuda.current_stream()
    sink = torch.zeros(4, dtype=torch.float32, device="cuda")
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    flop = mla.probe_mfma_bf16(100, sink, stream=stream)
    assert flop == 2 * n_cu * 4 * 4 * 100 * 32768.0
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    flop = mla.probe_mfma_bf16(2000, sink, stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    tflops = flop / (e0.elapsed_time(e1) / 1e3) / 1e12
    print(f"probe: {n_cu} CUs, {tflops:.1f} TFLOP/s dense bf16", flush=True)
    assert 500.0 < tflops <= 2500.0 * 1.02
    assert torch.count_nonzero(sink).item() == 0
