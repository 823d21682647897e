"""GPU check of the matrix-core rate probe (a measurement helper of the benchmark)."""
import pytest
import torch

from paper_2606_29758_amd import pspo

pytestmark = pytest.mark.gpu

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16, published


def test_mfma_loop_rate_is_physical():
    """The probe runs and its rate lies below the published dense bf16 peak (it cannot
    exceed it) and well above zero (the loop really runs on every CU)."""
    assert torch.cuda.is_available()
    iters, blocks = 4096, 1024
    out = pspo.mfma_loop(iters, blocks)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record(stream)
    pspo.mfma_loop(iters, blocks, out)
    e.record(stream)
    torch.cuda.synchronize()
    tf = blocks * 4.0 * iters * 16 * 16384 / (s.elapsed_time(e) * 1e-3) / 1e12
    assert 0.2 * PEAK_BF16_TFLOPS < tf <= PEAK_BF16_TFLOPS, tf
    assert torch.isfinite(out).all()
