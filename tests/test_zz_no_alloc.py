"""The allocation-free weights call (ditango_contrib_noalloc) through the C
ABI against ditango_contrib with a caller workspace: the same kernels and
reduction order, so the weights must be equal bit for bit (and match the
float64 oracle).  Two calls in a row, the second with fewer rows and fewer
partitions, so that the fixed scratch still holds the first call's partial
sums where the second does not write."""
import ctypes

import numpy as np
import pytest

import oracle

from helpers import max_abs

pytestmark = pytest.mark.gpu


def _case(rng, P, B, H, q_len):
    lses = (rng.standard_normal((P, B, H, q_len)) * 2).astype(np.float32)
    lses[P - 1] -= 3.0
    lses[0, 0, 0, : min(50, q_len)] = -np.inf
    _, ml = oracle.merge([np.zeros((B, q_len, H, 1))] * P, [l.astype(np.float64) for l in lses])
    return lses, ml.astype(np.float32)


def test_contrib_noalloc_matches_workspace_call_twice():
    import torch
    from paper_2607_15650_amd import _lib
    L = _lib.lib()
    rng = np.random.default_rng(77)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    # the second call is smaller: fewer rows and fewer partitions
    for (P, B, H, q_len) in [(8, 2, 40, 9450), (5, 1, 3, 1001)]:
        lses, ml = _case(rng, P, B, H, q_len)
        print(f"contrib_noalloc P={P} B={B} H={H} q_len={q_len}", flush=True)
        ls = torch.from_numpy(lses).cuda()
        lo = torch.from_numpy(ml).cuda()
        wp_a = torch.full((P,), float("nan"), device="cuda")
        wp_b = torch.full((P,), float("nan"), device="cuda")
        wr_a = torch.full((B, H, q_len, P), float("nan"), device="cuda")
        wr_b = torch.full((B, H, q_len, P), float("nan"), device="cuda")
        need = L.ditango_contrib_workspace_bytes(B, H, q_len, P)
        assert 0 < need <= _lib.CONTRIB_SCRATCH_BYTES
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        st = L.ditango_contrib(ls.data_ptr(), lo.data_ptr(), P, B, H, q_len, wr_a.data_ptr(), wp_a.data_ptr(),
                               ws.data_ptr(), stream)
        assert st == 0
        st = L.ditango_contrib_noalloc(ls.data_ptr(), lo.data_ptr(), P, B, H, q_len, wr_b.data_ptr(),
                                       wp_b.data_ptr(), stream)
        assert st == 0
        # without per-row weights too
        wp_c = torch.full((P,), float("nan"), device="cuda")
        st = L.ditango_contrib_noalloc(ls.data_ptr(), lo.data_ptr(), P, B, H, q_len, None, wp_c.data_ptr(), stream)
        assert st == 0
        torch.cuda.synchronize()
        assert torch.equal(wp_a, wp_b) and torch.equal(wp_a, wp_c)
        assert torch.equal(wr_a, wr_b)
        W, wbar = oracle.contrib([l.astype(np.float64) for l in lses], ml.astype(np.float64))
        assert max_abs(wp_b.cpu().numpy(), wbar) <= 1e-6
        assert max_abs(wr_b.cpu().numpy(), W) <= 1e-6
    # beyond the scratch: rejected, nothing launched
    assert L.ditango_contrib_noalloc(ls.data_ptr(), lo.data_ptr(), 64, 4, 64, 9450, None, wp_b.data_ptr(),
                                     stream) == 2
