"""Shared helpers of the GPU parity tests: seeded inputs onto the GPU, the HIP
path through the C ABI, and the oracle on the same inputs."""
from __future__ import annotations

import numpy as np

import fixtures
from fixtures import bf16_bits, bf16_round

TOL = {
    # bf16 inputs with float32 accumulation: OUT max-abs, LSE max-abs
    "bf16": {"out": 1e-2, "lse": 2e-3, "w": 1e-3},
    # float32 inputs
    "f32": {"out": 1e-5, "lse": 1e-5, "w": 1e-6},
}


def exact_inputs(x: np.ndarray, dtype: str) -> np.ndarray:
    """The values the kernels see, as float64 for the oracle."""
    return (bf16_round(x) if dtype == "bf16" else x.astype(np.float32)).astype(np.float64)


def to_gpu(x: np.ndarray, dtype: str):
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(bf16_bits(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.cuda()


def torch_dtype(dtype: str):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def new_state_cache(P, B, q_len, H, D, dtype, fill=None):
    import torch
    out = torch.empty((P, B, q_len, H, D), dtype=torch_dtype(dtype), device="cuda")
    lse = torch.empty((P, B, H, q_len), dtype=torch.float32, device="cuda")
    if fill is not None:
        out.view(torch.int16 if dtype == "bf16" else torch.int32).fill_(fill)
        lse.view(torch.int32).fill_(fill)
    return out, lse


def max_abs(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    both_inf = np.isneginf(a) & np.isneginf(b)
    with np.errstate(invalid="ignore"):
        d = np.where(both_inf, 0.0, np.abs(a - b))
    return float(np.nanmax(d)) if d.size else 0.0


def per_head(fn, H: int, workers: int = 0):
    """fn(h) for every head h, in a thread pool; heads are independent in
    every oracle function, so the results are those of one call over all
    heads.  NumPy's matrix products and exponentials release the GIL; BLAS
    runs one thread per task."""
    import concurrent.futures as cf
    import os
    from threadpoolctl import threadpool_limits
    n = workers or max(1, min(H, len(os.sched_getaffinity(0)), 16))
    with threadpool_limits(1), cf.ThreadPoolExecutor(n) as ex:
        return list(ex.map(fn, range(H)))
