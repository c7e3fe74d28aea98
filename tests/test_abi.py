"""The C-ABI library loads, exports every symbol the header declares, and
rejects bad arguments with a status code before launching anything.  Runs
without a GPU: only calls that fail argument validation are made."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ditango.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ditango_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    from paper_2607_15650_amd import _lib
    return _lib.lib()


def test_every_declared_symbol_is_exported(L):
    names = header_functions()
    assert "ditango_attn_partition_states" in names and "ditango_merge_states" in names
    assert "ditango_contrib" in names
    for n in names:
        assert hasattr(L, n), n
    from paper_2607_15650_amd import _lib
    assert set(names) == set(_lib.SIGNATURES)


def test_status_strings_and_version(L):
    assert L.ditango_status_string(0) == b"ok"
    assert L.ditango_status_string(1) == b"invalid argument"
    assert L.ditango_status_string(2) == b"unsupported configuration"
    assert L.ditango_status_string(3) == b"HIP runtime error"
    assert re.match(rb"\d+\.\d+\.\d+", L.ditango_version())


FAKE = 0x1000  # never dereferenced: every call below fails validation first


def attn(L, q=FAKE, k=FAKE, v=FAKE, dt=1, B=1, H=2, D=128, q_len=10, offs=(0, 5, 10),
         sel=(1, 1), scale=0.1, out=FAKE, lse=FAKE):
    P = len(offs) - 1 if offs is not None else 1
    o = (ctypes.c_int64 * len(offs))(*offs) if offs is not None else None
    s = (ctypes.c_uint8 * len(sel))(*sel) if sel is not None else None
    return L.ditango_attn_partition_states(q, k, v, dt, B, H, D, q_len, o, P, s,
                                           scale, out, lse, None)


def test_attn_argument_validation(L):
    assert attn(L, q=None) == 1
    assert attn(L, out=None) == 1
    assert attn(L, lse=None) == 1
    assert attn(L, offs=None) == 1
    assert attn(L, sel=None) == 1
    assert attn(L, dt=7) == 1
    assert attn(L, B=0) == 1
    assert attn(L, H=0) == 1
    assert attn(L, q_len=0) == 1
    assert attn(L, q_len=-3) == 1
    assert attn(L, D=96) == 2
    assert attn(L, D=256) == 2
    assert attn(L, H=513, D=128) == 2                     # H*D beyond 65536
    assert attn(L, H=1025, D=64) == 2
    assert attn(L, offs=(0, 6, 5), sel=(1, 1)) == 1       # decreasing offsets
    assert attn(L, offs=(1, 6, 10), sel=(1, 1)) == 1      # offsets[0] != 0
    assert attn(L, scale=float("nan")) == 1
    assert attn(L, scale=float("inf")) == 1
    # the kernels need scale > 0: masked tail keys are -inf before scaling
    # and the running maximum is taken over unscaled scores
    assert attn(L, scale=0.0) == 1
    assert attn(L, scale=-0.0) == 1
    assert attn(L, scale=-0.125) == 1
    assert attn(L, scale=float("-inf")) == 1
    big = tuple(range(66))
    assert attn(L, offs=big, sel=(1,) * 65) == 2          # more than 64 partitions


def test_attn_empty_selection_launches_nothing(L):
    # valid arguments, nothing selected: returns OK without touching the GPU
    assert attn(L, sel=(0, 0)) == 0


def merge(L, st=FAKE, lse=FAKE, sdt=1, P=4, slots=None, n=0, B=1, H=2, D=64, q_len=8,
          out=FAKE, odt=1, lse_out=FAKE):
    sl = (ctypes.c_int32 * len(slots))(*slots) if slots is not None else None
    return L.ditango_merge_states(st, lse, sdt, P, sl, n, B, H, D, q_len, out, odt, lse_out, None)


def test_merge_argument_validation(L):
    assert merge(L, st=None) == 1
    assert merge(L, lse=None) == 1
    assert merge(L, out=None) == 1
    assert merge(L, sdt=3) == 1
    assert merge(L, odt=-1) == 1
    assert merge(L, P=0) == 1
    assert merge(L, P=65) == 2
    assert merge(L, D=32) == 2
    assert merge(L, q_len=0) == 1
    assert merge(L, slots=[0, 4], n=2) == 1               # slot out of range
    assert merge(L, slots=[-1], n=1) == 1
    assert merge(L, slots=[0], n=0) == 1                  # empty list


def test_contrib_argument_validation(L):
    c = L.ditango_contrib
    assert c(None, FAKE, 4, 1, 2, 8, None, FAKE, FAKE, None) == 1
    assert c(FAKE, None, 4, 1, 2, 8, None, FAKE, FAKE, None) == 1
    assert c(FAKE, FAKE, 4, 1, 2, 8, None, None, FAKE, None) == 1
    assert c(FAKE, FAKE, 4, 1, 2, 8, None, FAKE, None, None) == 1
    assert c(FAKE, FAKE, 0, 1, 2, 8, None, FAKE, FAKE, None) == 1
    assert c(FAKE, FAKE, 65, 1, 2, 8, None, FAKE, FAKE, None) == 2
    assert c(FAKE, FAKE, 4, 1, 2, 8, None, FAKE, FAKE + 4, None) == 1   # misaligned workspace


def test_contrib_workspace_size(L):
    f = L.ditango_contrib_workspace_bytes
    assert f(1, 40, 9450, 8) == ((40 * 9450 + 511) // 512) * 8 * 4
    assert f(0, 1, 1, 1) == 0
    assert f(1, 1, 1, 1) == 4


def test_state_norms_argument_validation(L):
    f = L.ditango_state_norms
    assert f(None, 1, 4, None, 0, 1, 2, 64, 8, None, FAKE, FAKE, None) == 1
    assert f(FAKE, 1, 4, None, 0, 1, 2, 64, 8, None, None, FAKE, None) == 1
    assert f(FAKE, 1, 4, None, 0, 1, 2, 64, 8, None, FAKE, None, None) == 1
    assert f(FAKE, 9, 4, None, 0, 1, 2, 64, 8, None, FAKE, FAKE, None) == 1
    assert f(FAKE, 1, 0, None, 0, 1, 2, 64, 8, None, FAKE, FAKE, None) == 1
    assert f(FAKE, 1, 65, None, 0, 1, 2, 64, 8, None, FAKE, FAKE, None) == 2
    assert f(FAKE, 1, 4, None, 0, 1, 2, 96, 8, None, FAKE, FAKE, None) == 2
    assert f(FAKE, 1, 4, None, 0, 1, 2, 64, 8, None, FAKE, FAKE + 8, None) == 1
    bad = (ctypes.c_int32 * 2)(0, 4)
    assert f(FAKE, 1, 4, bad, 2, 1, 2, 64, 8, None, FAKE, FAKE, None) == 1
    assert L.ditango_norms_workspace_bytes(1, 40, 128, 9450, 8) == ((40 * 9450 * 128 // 8 + 4095) // 4096) * 8 * 4


def test_probe_argument_validation(L):
    f = L.ditango_probe_mfma_bf16
    assert f(0, 10, FAKE, None) == 1
    assert f(4, 0, FAKE, None) == 1
    assert f(4, 10, None, None) == 1
    assert f((1 << 20) + 1, 10, FAKE, None) == 1
    assert f(4, (1 << 20) + 1, FAKE, None) == 1


def test_attn_ex_state_dtype_validation(L):
    f = L.ditango_attn_partition_states_ex
    o = (ctypes.c_int64 * 3)(0, 5, 10)
    s = (ctypes.c_uint8 * 2)(1, 1)
    call = lambda dt, sdt: f(FAKE, FAKE, FAKE, dt, 1, 2, 128, 10, o, 2, s, 0.1, FAKE, sdt, FAKE, None)
    assert call(1, 7) == 1            # unknown state dtype
    assert call(0, 1) == 2            # float32 inputs with bf16 states: not built
    o_bad = (ctypes.c_int64 * 3)(0, 6, 5)
    assert f(FAKE, FAKE, FAKE, 1, 1, 2, 128, 10, o_bad, 2, s, 0.1, FAKE, 0, FAKE, None) == 1


def attn_ws(L, ws=0x1000, ws_bytes=4096, D=128, dt=1, state_dt=1, offs=(0, 5, 10), sel=(1, 1), q=FAKE):
    P = len(offs) - 1
    o = (ctypes.c_int64 * len(offs))(*offs)
    s = (ctypes.c_uint8 * len(sel))(*sel)
    return L.ditango_attn_partition_states_ws(q, FAKE, FAKE, dt, 1, 2, D, 10, o, P, s, 0.1,
                                              FAKE, state_dt, FAKE, ws, ws_bytes, None)


def test_attn_ws_argument_validation(L):
    # the same checks as the other attention entry points, then the workspace
    assert attn_ws(L, q=None) == 1
    assert attn_ws(L, D=96) == 2
    assert attn_ws(L, offs=(0, 6, 5)) == 1
    assert attn_ws(L, dt=0, state_dt=1) == 2
    assert attn_ws(L, ws=0x1000 + 64) == 1          # not 256-byte aligned
    assert attn_ws(L, sel=(0, 0)) == 0              # nothing selected: nothing launched


def test_attn_workspace_bytes_without_a_split(L):
    o = (ctypes.c_int64 * 3)(0, 5, 10)
    s = (ctypes.c_uint8 * 2)(1, 1)
    none = (ctypes.c_uint8 * 2)(0, 0)
    # float32 inputs never split; invalid shapes and empty selections need nothing
    assert L.ditango_attn_workspace_bytes(0, 1, 2, 128, 10, o, 2, s) == 0
    assert L.ditango_attn_workspace_bytes(1, 1, 2, 96, 10, o, 2, s) == 0
    assert L.ditango_attn_workspace_bytes(1, 0, 2, 128, 10, o, 2, s) == 0
    assert L.ditango_attn_workspace_bytes(1, 1, 2, 128, 10, o, 2, none) == 0


def test_contrib_noalloc_validation_before_any_launch(L):
    """The allocation-free weights call rejects bad arguments and sizes whose
    partial sums would not fit its fixed device scratch, before touching the
    GPU."""
    from paper_2607_15650_amd import _lib
    f = L.ditango_contrib_noalloc
    assert _lib.CONTRIB_SCRATCH_BYTES == 1 << 20
    assert f(None, FAKE, 8, 1, 40, 9450, None, FAKE, None) == 1
    assert f(FAKE, None, 8, 1, 40, 9450, None, FAKE, None) == 1
    assert f(FAKE, FAKE, 8, 1, 40, 9450, None, None, None) == 1
    assert f(FAKE, FAKE, 0, 1, 40, 9450, None, FAKE, None) == 1
    assert f(FAKE, FAKE, 8, 1, 0, 9450, None, FAKE, None) == 1
    assert f(FAKE, FAKE, 8, 1, 40, 0, None, FAKE, None) == 1
    assert f(FAKE, FAKE, 65, 1, 40, 9450, None, FAKE, None) == 2
    # the largest row count whose partial sums fit, and one workgroup more
    per_block, P = 512, 8
    max_blocks = (1 << 20) // (4 * P)
    assert L.ditango_contrib_workspace_bytes(1, 1, max_blocks * per_block, P) == 1 << 20
    assert f(FAKE, FAKE, P, 1, 1, max_blocks * per_block + 1, None, FAKE, None) == 2
    assert f(FAKE, FAKE, 64, 4, 64, 9450, None, FAKE, None) == 2
