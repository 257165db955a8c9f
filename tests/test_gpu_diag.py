"""The MFMA-rate diagnostic (tla_mfma_rate) runs on the device, writes a
finite value per thread, and a short timed run reports a rate below the
datasheet peak (it measures the peak's attainable side, not parity)."""
import pytest
import torch

import paper_2609_36529_amd as tla

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [0, 1])
def test_mfma_rate_runs(shape):
    sink = torch.full((256 * 256,), float("nan"), dtype=torch.float32, device="cuda")
    flop = tla.mfma_rate(shape, 256, 200, sink)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    flop = tla.mfma_rate(shape, 256, 200, sink)
    b.record()
    torch.cuda.synchronize()
    assert torch.isfinite(sink).all()
    tflops = flop / (a.elapsed_time(b) * 1e-3) / 1e12
    print(f"mfma shape {shape}: {tflops:.0f} TFLOP/s", flush=True)
    assert 0 < tflops < 2600
