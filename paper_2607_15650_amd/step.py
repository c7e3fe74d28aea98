"""Selective attention over denoising steps for one context-parallel rank.

Each query block owns a state cache (one OUT slot and one LSE slot per key /
value partition) that persists across steps: the paper's attention-state
cache (Sec. 5.2).  A step computes the selected partitions fresh into their
slots (the others keep the state of the step at which they were last
computed), composes all slots, and measures the contribution weights.  All
work runs in the HIP kernels behind the C ABI; this module only owns buffers
and calls them in order on the current stream.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import torch

from . import api
from .workspace import AttnWorkspace


class StateCache:
    """OUT slots [P, B, q_len, H, D] and LSE slots [P, B, H, q_len] of one query block."""

    def __init__(self, P: int, B: int, q_len: int, H: int, D: int, dtype: torch.dtype, device):
        self.out = torch.zeros((P, B, q_len, H, D), dtype=dtype, device=device)
        self.lse = torch.full((P, B, H, q_len), float("-inf"), dtype=torch.float32, device=device)
        self.computed_at = [-1] * P     # step at which each slot was last computed


class SelectiveAttention:
    """Runs fresh-state / compose / weights steps for a set of query blocks.

    ``offsets`` are the P+1 token offsets of the partitions; query block i is
    partition i of the same sequence.  ``state_dtype`` is the dtype of the
    cached states: the input dtype (default) or float32 for bf16 inputs; the
    composed output is in the input dtype either way.
    """

    def __init__(self, B: int, H: int, D: int, offsets: Sequence[int], scale: float,
                 dtype: torch.dtype = torch.bfloat16, device="cuda",
                 state_dtype: torch.dtype = None):
        self.B, self.H, self.D = B, H, D
        self.offsets = [int(o) for o in offsets]
        self.P = len(self.offsets) - 1
        self.scale = float(scale)
        self.dtype = dtype
        self.state_dtype = state_dtype if state_dtype is not None else dtype
        self.device = device
        self.caches = {}
        self._ws = {}
        self._attn_ws = AttnWorkspace(device)

    def cache(self, qb: int) -> StateCache:
        if qb not in self.caches:
            L = self.offsets[qb + 1] - self.offsets[qb]
            self.caches[qb] = StateCache(self.P, self.B, L, self.H, self.D, self.state_dtype, self.device)
        return self.caches[qb]

    def step(self, step: int, qb: int, q_all: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
             select: Sequence[int]) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
        """One step for query block ``qb``: returns (OUT, LSE, per-partition weights).

        q_all, k, v are [B, S, H, D] for the whole sequence; the query block is
        rows [offsets[qb], offsets[qb+1]) of q_all.
        """
        c = self.cache(qb)
        a, e = self.offsets[qb], self.offsets[qb + 1]
        q = q_all[:, a:e]
        if not q.is_contiguous():
            q = q.contiguous()
        ws = self._attn_ws.get(q.dtype, self.B, self.H, self.D, e - a, self.offsets, select)
        api.attn_partition_states(q, k, v, self.offsets, select, self.scale, c.out, c.lse, ws)
        for j, s in enumerate(select):
            if s:
                c.computed_at[j] = step
        L = e - a
        out = torch.empty((self.B, L, self.H, self.D), dtype=self.dtype, device=self.device)
        lse = torch.empty((self.B, self.H, L), dtype=torch.float32, device=self.device)
        api.merge_states(c.out, c.lse, out, lse)
        w_part = torch.empty(self.P, dtype=torch.float32, device=self.device)
        key = (self.B, self.H, L, self.P)
        if key not in self._ws:
            self._ws[key] = torch.empty(max(16, api.contrib_workspace_bytes(*key)), dtype=torch.uint8,
                                        device=self.device)
        api.contrib(c.lse, lse, w_part, self._ws[key])
        return out, lse, w_part
