"""Workload definitions: the five synthetic cases the hot path is tested and measured on.

Each workload is one context-parallel rank's share of one DiT attention call:
the rank's query block (partition ``q`` of the token sequence) attends to ``P``
key/value partitions of the whole sequence.  Tokens are a T x Hg x W latent grid
flattened t-major, n = (t*Hg + h)*W + w, and the sequence is split into ``P``
contiguous chunks of ceil(S/P) tokens, the last taking the remainder, as
context parallelism splits a sequence across ranks (Sec. 2.1 and Sec. 2.2.3 of
the paper; partition adjacency follows Fig. 2).

Shapes follow the paper's video-DiT workloads (Table 1 of Sec. 6.1): the
75,600-token, 40-head, head-dim-128 case is Wan2.1-14B's 81-frame 720p latent;
the 131,072-token case stands for the long-context HunyuanVideo-scale sequence.
Batch is 1 in the five main workloads; the paper's classifier-free-guidance
batch of 2 (the conditional and unconditional branch of one denoising step)
is the separate ``videodit_cfg_bf16_b2_h40_d128_s75600_p8`` variant below,
beside the HunyuanVideo-like head-dim-64 shape.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                 # "f32" or "bf16": input dtype = state dtype = output dtype
    B: int
    H: int
    D: int
    grid: Tuple[int, int, int]  # (T, Hg, W) latent grid; S = T*Hg*W
    P: int                     # number of KV partitions
    q: int                     # query partition (the rank's local block)
    seed: int
    select: Tuple[int, ...]    # KV partitions computed fresh this step
    prev_noise: float = 0.0    # sigma of previous-step perturbation (0: no reuse case)
    sweep: Tuple[Tuple[int, ...], ...] = ()   # optional list of selections (long-context sweep)
    steps: int = 1             # multi-step workloads
    step_noise: float = 0.0    # per-step evolution sigma (multi-step workloads)
    anchors: Tuple[int, ...] = ()
    threshold: float = 0.0     # planner threshold on anchor contribution weight

    @property
    def S(self) -> int:
        T, Hg, W = self.grid
        return T * Hg * W

    @property
    def offsets(self) -> List[int]:
        return partition_offsets(self.S, self.P)

    @property
    def q_len(self) -> int:
        o = self.offsets
        return o[self.q + 1] - o[self.q]

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.D)

    def select_mask(self, select: Optional[Tuple[int, ...]] = None) -> List[int]:
        sel = self.select if select is None else select
        return [1 if j in sel else 0 for j in range(self.P)]

    def with_query(self, q: int) -> "Workload":
        d = dict(self.__dict__)
        d["q"] = q
        return Workload(**d)


def partition_offsets(S: int, P: int) -> List[int]:
    """Token offsets o_0=0 < ... < o_P=S of P contiguous chunks of ceil(S/P) tokens.

    The last chunk takes the remainder, so it can be shorter, or empty when
    P*ceil(S/P) - S >= ceil(S/P).
    """
    if P < 1 or S < 0:
        raise ValueError("need P >= 1 and S >= 0")
    chunk = -(-S // P) if S > 0 else 0
    return [min(j * chunk, S) for j in range(P)] + [S]


def nearest_first(P: int, q: int, k: int) -> Tuple[int, ...]:
    """The k partitions nearest to q, ordered by (|j - q|, j)."""
    order = sorted(range(P), key=lambda j: (abs(j - q), j))
    return tuple(order[:k])


WORKLOADS: Dict[str, Workload] = {}


def _add(w: Workload) -> None:
    WORKLOADS[w.name] = w


# Tiny single-rank plumbing case in fp32; all partitions fresh.
_add(Workload(name="plumbing_f32_h2_d64_s4096_p4", dtype="f32", B=1, H=2, D=64,
              grid=(4, 32, 32), P=4, q=0, seed=0, select=(0, 1, 2, 3)))
# Reuse path in bf16: fresh {2,3,4}, the rest reused from the previous step.
_add(Workload(name="reuse_bf16_h12_d64_s16384_p8", dtype="bf16", B=1, H=12, D=64,
              grid=(16, 32, 32), P=8, q=3, seed=1, select=(2, 3, 4), prev_noise=0.05))
# Video-DiT shape (Wan2.1-14B latent, 81 frames 720p): fresh |j-q| <= 1.
_add(Workload(name="videodit_bf16_h40_d128_s75600_p8", dtype="bf16", B=1, H=40, D=128,
              grid=(21, 45, 80), P=8, q=3, seed=2, select=(2, 3, 4), prev_noise=0.05))
# Long context: selection sizes 1,2,4,8,16 nearest-first; 16 = full attention.
_add(Workload(name="longctx_bf16_h24_d128_s131072_p16", dtype="bf16", B=1, H=24, D=128,
              grid=(32, 64, 64), P=16, q=7, seed=3, select=nearest_first(16, 7, 4),
              prev_noise=0.05,
              sweep=tuple(nearest_first(16, 7, k) for k in (1, 2, 4, 8, 16))))
# Planner-driven multi-step run: anchors at steps 0 and 5 compute everything.
_add(Workload(name="planner_bf16_h40_d128_s75600_p8_10steps", dtype="bf16", B=1, H=40, D=128,
              grid=(21, 45, 80), P=8, q=3, seed=4, select=tuple(range(8)),
              steps=10, step_noise=0.03, anchors=(0, 5), threshold=0.05))


# HunyuanVideo-like shape ([1, 119K, 48, 64]: 129 frames at 720p give a
# 33 x 45 x 80 latent grid), fresh |j-q| <= 1.
_add(Workload(name="hunyuan_bf16_h48_d64_s118800_p8", dtype="bf16", B=1, H=48, D=64,
              grid=(33, 45, 80), P=8, q=3, seed=5, select=(2, 3, 4), prev_noise=0.05))
# Wan2.1-14B shape with the classifier-free-guidance batch of 2
# ([2, 76K, 40, 128]), fresh |j-q| <= 1.
_add(Workload(name="videodit_cfg_bf16_b2_h40_d128_s75600_p8", dtype="bf16", B=2, H=40, D=128,
              grid=(21, 45, 80), P=8, q=3, seed=6, select=(2, 3, 4), prev_noise=0.05))

# Reduced planner-driven run (same partition structure, 2 heads, 16,384
# tokens) that the float64 oracle can follow over all steps and blocks.  On
# these inputs the anchor weights are close to uniform (about 0.12-0.14 for
# 8 partitions), so the threshold sits at the uniform level 1/8: some
# partitions of every block are reused.
_add(Workload(name="planner_bf16_h2_d128_s16384_p8_10steps", dtype="bf16", B=1, H=2, D=128,
              grid=(16, 32, 32), P=8, q=3, seed=4, select=tuple(range(8)),
              steps=10, step_noise=0.03, anchors=(0, 5), threshold=0.125))


def get_workload(name: str) -> Workload:
    try:
        return WORKLOADS[name]
    except KeyError:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}") from None
