"""ctypes loader of libditango.so: the C ABI declared in include/ditango.h.

The library is built in-tree (``paper_2607_15650_amd/libditango.so``).  When
it is missing, loading fails loudly: there is no CPU or PyTorch fallback for
any entry point.
"""
from __future__ import annotations

import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libditango.so")

OK, ERR_INVALID, ERR_UNSUPPORTED, ERR_HIP = 0, 1, 2, 3
F32, BF16 = 0, 1
MAX_PARTITIONS = 64
CONTRIB_SCRATCH_BYTES = 1 << 20

# Every symbol include/ditango.h declares, with (restype, argtypes).
_c = ctypes
SIGNATURES = {
    "ditango_attn_partition_states": (_c.c_int, [
        _c.c_void_p, _c.c_void_p, _c.c_void_p, _c.c_int,
        _c.c_int, _c.c_int, _c.c_int, _c.c_int64,
        _c.POINTER(_c.c_int64), _c.c_int, _c.POINTER(_c.c_uint8), _c.c_float,
        _c.c_void_p, _c.c_void_p, _c.c_void_p]),
    "ditango_attn_partition_states_ex": (_c.c_int, [
        _c.c_void_p, _c.c_void_p, _c.c_void_p, _c.c_int,
        _c.c_int, _c.c_int, _c.c_int, _c.c_int64,
        _c.POINTER(_c.c_int64), _c.c_int, _c.POINTER(_c.c_uint8), _c.c_float,
        _c.c_void_p, _c.c_int, _c.c_void_p, _c.c_void_p]),
    "ditango_attn_partition_states_ws": (_c.c_int, [
        _c.c_void_p, _c.c_void_p, _c.c_void_p, _c.c_int,
        _c.c_int, _c.c_int, _c.c_int, _c.c_int64,
        _c.POINTER(_c.c_int64), _c.c_int, _c.POINTER(_c.c_uint8), _c.c_float,
        _c.c_void_p, _c.c_int, _c.c_void_p, _c.c_void_p, _c.c_size_t, _c.c_void_p]),
    "ditango_attn_workspace_bytes": (_c.c_size_t, [
        _c.c_int, _c.c_int, _c.c_int, _c.c_int, _c.c_int64,
        _c.POINTER(_c.c_int64), _c.c_int, _c.POINTER(_c.c_uint8)]),
    "ditango_merge_states": (_c.c_int, [
        _c.c_void_p, _c.c_void_p, _c.c_int,
        _c.c_int, _c.POINTER(_c.c_int32), _c.c_int,
        _c.c_int, _c.c_int, _c.c_int, _c.c_int64,
        _c.c_void_p, _c.c_int, _c.c_void_p, _c.c_void_p]),
    "ditango_contrib_workspace_bytes": (_c.c_size_t, [_c.c_int, _c.c_int, _c.c_int64, _c.c_int]),
    "ditango_contrib": (_c.c_int, [
        _c.c_void_p, _c.c_void_p, _c.c_int,
        _c.c_int, _c.c_int, _c.c_int64,
        _c.c_void_p, _c.c_void_p, _c.c_void_p, _c.c_void_p]),
    "ditango_contrib_noalloc": (_c.c_int, [
        _c.c_void_p, _c.c_void_p, _c.c_int,
        _c.c_int, _c.c_int, _c.c_int64,
        _c.c_void_p, _c.c_void_p, _c.c_void_p]),
    "ditango_norms_workspace_bytes": (_c.c_size_t, [_c.c_int, _c.c_int, _c.c_int, _c.c_int64, _c.c_int]),
    "ditango_state_norms": (_c.c_int, [
        _c.c_void_p, _c.c_int, _c.c_int, _c.POINTER(_c.c_int32), _c.c_int,
        _c.c_int, _c.c_int, _c.c_int, _c.c_int64, _c.c_void_p,
        _c.c_void_p, _c.c_void_p, _c.c_void_p]),
    "ditango_probe_mfma_bf16": (_c.c_int, [_c.c_int, _c.c_int, _c.c_void_p, _c.c_void_p]),
    "ditango_status_string": (_c.c_char_p, [_c.c_int]),
    "ditango_version": (_c.c_char_p, []),
}

_lock = threading.Lock()
_handle = None


class DitangoError(RuntimeError):
    def __init__(self, fn: str, status: int):
        msg = "unknown"
        try:
            msg = lib().ditango_status_string(status).decode()
        except Exception:   # pragma: no cover - the library itself is broken
            pass
        super().__init__(f"{fn} failed: status {status} ({msg})")
        self.status = status


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _handle
    if _handle is not None:
        return _handle
    with _lock:
        if _handle is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    f"{LIB_PATH} is missing: build it with `python -m paper_2607_15650_amd.build` "
                    "(the hot path has no fallback)")
            h = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in SIGNATURES.items():
                fn = getattr(h, name)
                fn.restype = res
                fn.argtypes = args
            _handle = h
    return _handle


def check(fn: str, status: int) -> None:
    if status != OK:
        raise DitangoError(fn, status)
