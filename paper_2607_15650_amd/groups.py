"""Group states and Dynamic Group State Compose for one query block.

The paper organises the P partition states of a rank into groups of g
contiguous partitions (Sec. 4.2.1), decides COMPUTE or REUSE per group
(Sec. 4.2.2), caches one composed state per group (Sec. 5.2: evict, compute,
store), and, when the cached states approach a memory budget, composes k
adjacent groups into one (Sec. 5.1, Eq. GroupCompose), recursively, until the
budget is met or an anchor step resets the grouping.  The local (diagonal)
partition is handled separately and always computed.

Layout: the state of group [a, b) lives in slot a of the block's cache (OUT
slots [P, B, q_len, H, D], LSE slots [P, B, H, q_len]).  Computing a group
writes its members' fresh states into slots a..b-1 (one attention launch for
all computing groups) and composes them in place into slot a; composing
groups [a, b) and [b, c) writes slot a in place.  The cache memory the
budget is checked against is the number of live group states times the
bytes of one state.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import torch

from . import api
from .workspace import AttnWorkspace


def base_groups(P: int, q: int, g: int) -> List[Tuple[int, int]]:
    """Contiguous runs [a, b) of the partitions j // g == i, without the local partition q."""
    out = []
    for i in range(0, P, g):
        members = [j for j in range(i, min(i + g, P)) if j != q]
        # the local partition splits its run; each side stays contiguous
        run: List[int] = []
        for j in members:
            if run and j != run[-1] + 1:
                out.append((run[0], run[-1] + 1))
                run = []
            run.append(j)
        if run:
            out.append((run[0], run[-1] + 1))
    return out


def compose_pairs(groups: Sequence[Tuple[int, int]], q: int, k: int = 2) -> List[List[Tuple[int, int]]]:
    """Partition of the group list into runs of up to k adjacent groups that
    are contiguous in partition index (never across the local partition)."""
    runs: List[List[Tuple[int, int]]] = []
    cur: List[Tuple[int, int]] = []
    for grp in groups:
        if cur and (len(cur) == k or cur[-1][1] != grp[0]):
            runs.append(cur)
            cur = []
        cur.append(grp)
    if cur:
        runs.append(cur)
    return runs


class GroupedSelectiveAttention:
    """Selective attention with group-granular state reuse for one query block."""

    def __init__(self, B: int, H: int, D: int, offsets: Sequence[int], q: int, g: int, scale: float,
                 dtype: torch.dtype = torch.bfloat16, device="cuda",
                 mem_budget_bytes: Optional[int] = None, k: int = 2):
        self.B, self.H, self.D = B, H, D
        self.offsets = [int(o) for o in offsets]
        self.P = len(self.offsets) - 1
        self.q, self.g, self.k = q, g, k
        self.scale = float(scale)
        self.dtype, self.device = dtype, device
        self.L = self.offsets[q + 1] - self.offsets[q]
        self.out = torch.zeros((self.P, B, self.L, H, D), dtype=dtype, device=device)
        self.lse = torch.full((self.P, B, H, self.L), float("-inf"), dtype=torch.float32, device=device)
        self._attn_ws = AttnWorkspace(device)
        self.budget = mem_budget_bytes
        self.groups = base_groups(self.P, q, g)
        self.computed_at = {grp: -1 for grp in self.groups}
        self._ws = None

    @property
    def state_bytes(self) -> int:
        return self.B * self.L * self.H * (self.D * self.out.element_size() + 4)

    def memory_bytes(self) -> int:
        """Bytes of the cached group states (the local partition's state is transient)."""
        return len(self.groups) * self.state_bytes

    def reset(self) -> None:
        """Anchor step: back to the base grouping (every group is recomputed)."""
        self.groups = base_groups(self.P, self.q, self.g)
        self.computed_at = {grp: -1 for grp in self.groups}

    def _merge_into(self, slots: Sequence[int]) -> None:
        a = slots[0]
        api.merge_states(self.out, self.lse, self.out[a], self.lse[a], slots=list(slots))

    def compose_once(self) -> bool:
        """One Dynamic Group State Compose pass (k adjacent groups -> 1).  Returns
        False when nothing can be composed any more."""
        runs = compose_pairs(self.groups, self.q, self.k)
        if all(len(r) == 1 for r in runs):
            return False
        new_groups, new_t = [], {}
        for r in runs:
            if len(r) > 1:
                self._merge_into([grp[0] for grp in r])
            grp = (r[0][0], r[-1][1])
            new_groups.append(grp)
            new_t[grp] = min(self.computed_at[x] for x in r)
        self.groups, self.computed_at = new_groups, new_t
        return True

    def fit_budget(self) -> int:
        """Compose until the cached states fit the budget; returns the number of passes."""
        n = 0
        while self.budget is not None and self.memory_bytes() > self.budget and self.compose_once():
            n += 1
        return n

    def step(self, step: int, q_all: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
             compute: Sequence[Tuple[int, int]]):
        """One step: the groups in ``compute`` (and the local partition) get fresh
        states, the others are reused; returns (OUT, LSE, weights per live group
        in the order of ``self.groups`` followed by the local partition)."""
        compute = set(compute)
        sel = [0] * self.P
        sel[self.q] = 1
        for grp in self.groups:
            if grp in compute:
                for j in range(*grp):
                    sel[j] = 1
        a, e = self.offsets[self.q], self.offsets[self.q + 1]
        qb = q_all[:, a:e]
        if not qb.is_contiguous():
            qb = qb.contiguous()
        ws = self._attn_ws.get(qb.dtype, self.B, self.H, self.D, self.L, self.offsets, sel)
        api.attn_partition_states(qb, k, v, self.offsets, sel, self.scale, self.out, self.lse, ws)
        for grp in self.groups:
            if grp in compute:
                if grp[1] - grp[0] > 1:
                    self._merge_into(list(range(*grp)))
                self.computed_at[grp] = step
        slots = [grp[0] for grp in self.groups] + [self.q]
        out = torch.empty((self.B, self.L, self.H, self.D), dtype=self.dtype, device=self.device)
        lse = torch.empty((self.B, self.H, self.L), dtype=torch.float32, device=self.device)
        api.merge_states(self.out, self.lse, out, lse, slots=slots)
        # weights of the live groups: contrib over a compact copy of their LSE slots
        lse_live = self.lse[slots].contiguous()
        n = len(slots)
        if self._ws is None or self._ws.numel() < api.contrib_workspace_bytes(self.B, self.H, self.L, n):
            self._ws = torch.empty(max(16, api.contrib_workspace_bytes(self.B, self.H, self.L, self.P)),
                                   dtype=torch.uint8, device=self.device)
        w = torch.empty(n, dtype=torch.float32, device=self.device)
        api.contrib(lse_live, lse, w, self._ws)
        return out, lse, w
