"""Build libditango.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

The library is built in-tree, next to this file, so that it travels with the
source tree.  ``python -m paper_2607_15650_amd.build`` rebuilds it.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libditango.so")
SOURCES = ["ditango_api.cpp", "attn_bf16.hip", "attn_f32.hip", "merge.hip", "norms.hip", "probe.hip"]
ARCH = "gfx950"
# Per-source compiler options.  The attention kernel is scheduled with the
# backend's iterative ILP strategy, which interleaves its MFMAs, LDS reads and
# softmax VALU work better than the default (2-4 % faster on both head dims).
SOURCE_FLAGS = {"attn_bf16.hip": ["-mllvm", "--amdgpu-sched-strategy=iterative-ilp"]}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; set HIPCC or install ROCm")


# options that decide the generated code (the rest only locate headers or
# select warnings)
CODEGEN_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 VALU forms are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def flags():
    return CODEGEN_FLAGS + ["-I", INCLUDE, "-I", CSRC, "-Wall", "-Wno-unused-function"]


# generated code a source includes besides internal.h
INCLUDES = {"attn_bf16.hip": ["attn_d128_loop.inc", "attn_d64_loop.inc"]}


def source_id(name: str) -> str:
    """SHA-256 prefix over a source file, the files it includes from csrc/
    and the options it is compiled with: changes whenever the code built
    from it can change."""
    import hashlib
    h = hashlib.sha256(open(os.path.join(CSRC, name), "rb").read())
    h.update(open(os.path.join(CSRC, "internal.h"), "rb").read())
    for inc in INCLUDES.get(name, []):
        h.update(open(os.path.join(CSRC, inc), "rb").read())
    h.update(" ".join(CODEGEN_FLAGS + SOURCE_FLAGS.get(name, [])).encode())
    return h.hexdigest()[:16]


def _compile(src: str, obj: str, extra) -> None:
    cmd = [hipcc()] + flags() + SOURCE_FLAGS.get(os.path.basename(src), []) + list(extra)
    if src.endswith(".cpp"):
        cmd += ["-x", "hip"]
    cmd += ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {os.path.basename(src)}:\n{r.stderr}")


def build(verbose: bool = False, extra=(), out: str = LIB, objdir: str = "") -> str:
    """Compile every source and link ``out``; ``extra`` flags go to each compile."""
    objdir = objdir or os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    jobs = []
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), 8)) as ex:
        for s in SOURCES:
            obj = os.path.join(objdir, os.path.splitext(s)[0] + ".o")
            jobs.append((obj, ex.submit(_compile, os.path.join(CSRC, s), obj, extra)))
        for _, f in jobs:
            f.result()
    tmp = out + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + [o for o, _ in jobs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    build(verbose=True, extra=sys.argv[1:])
