"""Python binding of the C ABI: torch tensors in, raw pointers and the current
HIP stream out.  Argument marshalling only; every step runs in the HIP kernels
of libditango.so.

Layouts (all tensors contiguous, on the same GPU):
  q            [B, q_len, H, D]            bf16 or float32
  k, v         [B, S, H, D]                same dtype as q
  out_states   [P, B, q_len, H, D]         same dtype as q (the state cache)
  lse_states   [P, B, H, q_len]            float32
  out          [B, q_len, H, D]            bf16 or float32
  lse          [B, H, q_len]               float32
"""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import torch

from . import _lib

_DT = {torch.float32: _lib.F32, torch.bfloat16: _lib.BF16}


def _dtype(t: torch.Tensor) -> int:
    try:
        return _DT[t.dtype]
    except KeyError:
        raise TypeError(f"unsupported dtype {t.dtype}; use torch.bfloat16 or torch.float32") from None


def _dev(*ts: torch.Tensor) -> None:
    dev = None
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("all tensors must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("all tensors must be contiguous")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError("all tensors must be on one device")
    # the kernels are enqueued on the current device's current stream
    if dev is not None and dev.index != torch.cuda.current_device():
        raise ValueError("tensors must be on the current device (torch.cuda.set_device)")


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def attn_workspace_bytes(dtype: torch.dtype, B: int, H: int, D: int, q_len: int,
                         offsets: Sequence[int], select: Sequence[int]) -> int:
    """Workspace bytes attn_partition_states uses for this launch on the
    current device (ditango_attn_workspace_bytes): 256 for the queue counters
    that balance the launch over the XCDs, plus the partial states of the
    tail split when a split shortens the last round; 0 for float32 inputs."""
    P = len(offsets) - 1
    offs = (ctypes.c_int64 * (P + 1))(*[int(x) for x in offsets])
    sel = (ctypes.c_uint8 * P)(*[1 if s else 0 for s in select])
    return int(_lib.lib().ditango_attn_workspace_bytes(_DT[dtype], B, H, D, q_len, offs, P, sel))


def attn_partition_states(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                          offsets: Sequence[int], select: Sequence[int], scale: float,
                          out_states: torch.Tensor, lse_states: torch.Tensor,
                          workspace: Optional[torch.Tensor] = None) -> None:
    """Fresh states of the selected partitions into their slots
    (ditango_attn_partition_states).  Unselected slots are left untouched.
    ``out_states`` is in the input dtype, or float32 for bf16 inputs
    (ditango_attn_partition_states_ex: states at full precision).  With a
    ``workspace`` (uint8, 256-byte aligned; ditango_attn_partition_states_ws)
    the last tasks are claimed from queue counters in its first 256 bytes,
    and with attn_workspace_bytes(...) bytes the last round is split over
    key ranges as well."""
    _dev(q, k, v, out_states, lse_states, workspace)
    B, q_len, H, D = q.shape
    P = len(offsets) - 1
    if len(select) != P:
        raise ValueError("select must have one entry per partition")
    if k.shape != v.shape or k.shape[0] != B or k.shape[2] != H or k.shape[3] != D:
        raise ValueError("k/v shape mismatch")
    if k.shape[1] != offsets[-1]:
        raise ValueError("offsets[-1] must equal the key/value sequence length")
    if tuple(out_states.shape) != (P, B, q_len, H, D):
        raise ValueError("out_states must be [P, B, q_len, H, D]")
    if out_states.dtype != q.dtype and not (q.dtype == torch.bfloat16 and out_states.dtype == torch.float32):
        raise ValueError("out_states must be in the input dtype, or float32 for bf16 inputs")
    if tuple(lse_states.shape) != (P, B, H, q_len) or lse_states.dtype != torch.float32:
        raise ValueError("lse_states must be float32 [P, B, H, q_len]")
    if k.dtype != q.dtype or v.dtype != q.dtype:
        raise ValueError("q, k, v must share a dtype")
    offs = (ctypes.c_int64 * (P + 1))(*[int(x) for x in offsets])
    sel = (ctypes.c_uint8 * P)(*[1 if s else 0 for s in select])
    if workspace is not None:
        st = _lib.lib().ditango_attn_partition_states_ws(
            q.data_ptr(), k.data_ptr(), v.data_ptr(), _dtype(q), B, H, D, q_len,
            offs, P, sel, float(scale), out_states.data_ptr(), _dtype(out_states), lse_states.data_ptr(),
            workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream())
        _lib.check("ditango_attn_partition_states_ws", st)
    elif out_states.dtype == q.dtype:
        st = _lib.lib().ditango_attn_partition_states(
            q.data_ptr(), k.data_ptr(), v.data_ptr(), _dtype(q), B, H, D, q_len,
            offs, P, sel, float(scale), out_states.data_ptr(), lse_states.data_ptr(), _stream())
        _lib.check("ditango_attn_partition_states", st)
    else:
        st = _lib.lib().ditango_attn_partition_states_ex(
            q.data_ptr(), k.data_ptr(), v.data_ptr(), _dtype(q), B, H, D, q_len,
            offs, P, sel, float(scale), out_states.data_ptr(), _dtype(out_states), lse_states.data_ptr(),
            _stream())
        _lib.check("ditango_attn_partition_states_ex", st)


def merge_states(out_states: torch.Tensor, lse_states: torch.Tensor, out: torch.Tensor,
                 lse_out: Optional[torch.Tensor] = None, slots: Optional[Sequence[int]] = None) -> None:
    """Composition of the listed slots (default: all) into ``out``/``lse_out``
    (ditango_merge_states)."""
    _dev(out_states, lse_states, out, lse_out)
    P, B, q_len, H, D = out_states.shape
    if tuple(lse_states.shape) != (P, B, H, q_len) or lse_states.dtype != torch.float32:
        raise ValueError("lse_states must be float32 [P, B, H, q_len]")
    if tuple(out.shape) != (B, q_len, H, D):
        raise ValueError("out must be [B, q_len, H, D]")
    if lse_out is not None and (tuple(lse_out.shape) != (B, H, q_len) or lse_out.dtype != torch.float32):
        raise ValueError("lse_out must be float32 [B, H, q_len]")
    if slots is None:
        sl, n = None, P
    else:
        n = len(slots)
        sl = (ctypes.c_int32 * n)(*[int(s) for s in slots])
    st = _lib.lib().ditango_merge_states(
        out_states.data_ptr(), lse_states.data_ptr(), _dtype(out_states), P, sl, n,
        B, H, D, q_len, out.data_ptr(), _dtype(out),
        lse_out.data_ptr() if lse_out is not None else None, _stream())
    _lib.check("ditango_merge_states", st)


def contrib_workspace_bytes(B: int, H: int, q_len: int, P: int) -> int:
    return int(_lib.lib().ditango_contrib_workspace_bytes(B, H, q_len, P))


def contrib(lse_states: torch.Tensor, lse_out: torch.Tensor, w_part: torch.Tensor,
            workspace: torch.Tensor, w_rows: Optional[torch.Tensor] = None) -> None:
    """Per-row and per-partition contribution weights (ditango_contrib)."""
    _dev(lse_states, lse_out, w_part, workspace, w_rows)
    P, B, H, q_len = lse_states.shape
    if lse_states.dtype != torch.float32 or lse_out.dtype != torch.float32:
        raise ValueError("lse_states and lse_out must be float32")
    if tuple(lse_out.shape) != (B, H, q_len):
        raise ValueError("lse_out must be [B, H, q_len]")
    if tuple(w_part.shape) != (P,) or w_part.dtype != torch.float32:
        raise ValueError("w_part must be float32 [P]")
    if w_rows is not None and (tuple(w_rows.shape) != (B, H, q_len, P) or w_rows.dtype != torch.float32):
        raise ValueError("w_rows must be float32 [B, H, q_len, P]")
    need = contrib_workspace_bytes(B, H, q_len, P)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace too small: need {need} bytes")
    st = _lib.lib().ditango_contrib(
        lse_states.data_ptr(), lse_out.data_ptr(), P, B, H, q_len,
        w_rows.data_ptr() if w_rows is not None else None, w_part.data_ptr(),
        workspace.data_ptr(), _stream())
    _lib.check("ditango_contrib", st)


def contrib_noalloc(lse_states: torch.Tensor, lse_out: torch.Tensor, w_part: torch.Tensor,
                    w_rows: Optional[torch.Tensor] = None) -> None:
    """ditango_contrib_noalloc: the weights with the library's fixed device
    scratch instead of a workspace (nothing is allocated)."""
    _dev(lse_states, lse_out, w_part, w_rows)
    P, B, H, q_len = lse_states.shape
    if lse_states.dtype != torch.float32 or lse_out.dtype != torch.float32:
        raise ValueError("lse_states and lse_out must be float32")
    if tuple(lse_out.shape) != (B, H, q_len):
        raise ValueError("lse_out must be [B, H, q_len]")
    if tuple(w_part.shape) != (P,) or w_part.dtype != torch.float32:
        raise ValueError("w_part must be float32 [P]")
    if w_rows is not None and (tuple(w_rows.shape) != (B, H, q_len, P) or w_rows.dtype != torch.float32):
        raise ValueError("w_rows must be float32 [B, H, q_len, P]")
    st = _lib.lib().ditango_contrib_noalloc(
        lse_states.data_ptr(), lse_out.data_ptr(), P, B, H, q_len,
        w_rows.data_ptr() if w_rows is not None else None, w_part.data_ptr(), _stream())
    _lib.check("ditango_contrib_noalloc", st)


def norms_workspace_bytes(B: int, H: int, D: int, q_len: int, n_slots: int) -> int:
    return int(_lib.lib().ditango_norms_workspace_bytes(B, H, D, q_len, n_slots))


def state_norms(out_states: torch.Tensor, norms: torch.Tensor, workspace: torch.Tensor,
                slots: Optional[Sequence[int]] = None, ref: Optional[torch.Tensor] = None) -> None:
    """norms[i] = ||out_states[slots[i]] - ref||_2 (ditango_state_norms); ref None = 0."""
    _dev(out_states, norms, workspace, ref)
    P, B, q_len, H, D = out_states.shape
    if ref is not None and (tuple(ref.shape) != (B, q_len, H, D) or ref.dtype != out_states.dtype):
        raise ValueError("ref must be [B, q_len, H, D] in the state dtype")
    if slots is None:
        sl, n = None, P
    else:
        n = len(slots)
        sl = (ctypes.c_int32 * n)(*[int(s) for s in slots])
    if tuple(norms.shape) != (n,) or norms.dtype != torch.float32:
        raise ValueError("norms must be float32 [n_slots]")
    need = norms_workspace_bytes(B, H, D, q_len, n)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace too small: need {need} bytes")
    st = _lib.lib().ditango_state_norms(
        out_states.data_ptr(), _dtype(out_states), P, sl, n, B, H, D, q_len,
        ref.data_ptr() if ref is not None else None, norms.data_ptr(), workspace.data_ptr(), _stream())
    _lib.check("ditango_state_norms", st)


def probe_mfma_bf16(n_workgroups: int, iters: int, sink: torch.Tensor) -> float:
    """Enqueue the MFMA-rate probe (ditango_probe_mfma_bf16) on the current
    stream; returns the flops the launch performs.  ``sink`` is a float32
    device tensor of at least n_workgroups * 256 elements."""
    _dev(sink)
    if sink.dtype != torch.float32 or sink.numel() < n_workgroups * 256:
        raise ValueError("sink must be float32 with n_workgroups * 256 elements")
    st = _lib.lib().ditango_probe_mfma_bf16(n_workgroups, iters, sink.data_ptr(), _stream())
    _lib.check("ditango_probe_mfma_bf16", st)
    return float(n_workgroups) * 4 * iters * 4 * 32768
