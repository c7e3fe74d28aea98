"""The MFMA-rate probe (device characterisation, not part of the method)
runs through the C ABI and leaves finite values in its sink."""
import pytest


@pytest.mark.gpu
def test_probe_mfma_runs(gpu_lib):
    import torch
    from paper_2607_15650_amd import api
    n_wg, iters = 8, 64
    sink = torch.full((n_wg * 256,), float("nan"), dtype=torch.float32, device="cuda")
    flops = api.probe_mfma_bf16(n_wg, iters, sink)
    torch.cuda.synchronize()
    assert flops == n_wg * 4 * iters * 4 * 32768
    assert bool(torch.isfinite(sink).all())
    assert float(sink.abs().sum()) > 0.0
