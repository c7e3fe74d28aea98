"""Anchor-guided, error-model selection of groups to compute (the paper's
Alg. 1, Sec. 4.1-4.2) on top of group states, for one query block.

Per step t:
  1. The local (diagonal) partition is computed first (it always is).
  2. Error model (Sec. 4.1.2): the drift of the local state since step t_c,
     d(t_c) = ||OUT_t(loc) - OUT_tc(loc)||, is extrapolated to partition j by
     its scale ratio alpha(j) = ||OUT_ta(j)|| / ||OUT_ta(loc)|| measured at the
     anchor t_a (Eq. scale_ratio, Eq. error_extrapolation); a group cached at
     t_c gets ASE(G) = sum_{j in G} w(j) * alpha(j) * d(t_c), with w(j) the
     anchor weights (Eq. lse_weight, Eq. ase_decomposition).
  3. Anchor when every group's ASE exceeds eps or the relative local drift
     d(t_a) / ||OUT_ta(loc)|| exceeds eps_local (Sec. 4.2.4); otherwise
     compute the groups with ASE > eps (Eq. error_based_selection).
  4. At an anchor every partition is recomputed; the anchor correction error
     of each group, w(G) * ||fresh(G) - cached(G)||, is recorded and eps
     becomes the R-quantile of all correction errors seen so far, R being the
     target fraction of reused groups; w, alpha and the local snapshot are
     refreshed and every group's t_c is reset.  Before the first correction
     errors exist, eps is the R-quantile of the current step's ASE values.

Norms: ||.|| is the Frobenius norm of a state's output over all
(batch, row, head, dim), computed by ditango_state_norms.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import api
from .workspace import AttnWorkspace
from .groups import base_groups


def quantile_r(values: Sequence[float], r: float) -> float:
    """The smallest value with at least a fraction r of ``values`` at or below
    it (the ceil(r*m)-th smallest of m values; the smallest for r <= 0)."""
    v = np.sort(np.asarray(values, dtype=np.float64))
    k = min(max(int(math.ceil(r * v.size)), 1), v.size)
    return float(v[k - 1])


def accuracy_stats(predicted: Sequence[float], measured: Sequence[float]) -> Dict[str, float]:
    """How well predicted errors match measured ones: R^2 of the prediction as
    it stands (1 - sum (m - p)^2 / sum (m - mean m)^2, no fitted line),
    Pearson's r, RMSE and MAE, over paired samples."""
    p = np.asarray(predicted, dtype=np.float64)
    m = np.asarray(measured, dtype=np.float64)
    if p.size < 2:
        return {"n": int(p.size), "r2": float("nan"), "pearson": float("nan"),
                "rmse": float("nan"), "mae": float("nan")}
    res = m - p
    ss_tot = float(np.sum((m - m.mean()) ** 2))
    r2 = 1.0 - float(np.sum(res ** 2)) / ss_tot if ss_tot > 0 else float("nan")
    sp, sm = p.std(), m.std()
    pearson = float(np.mean((p - p.mean()) * (m - m.mean())) / (sp * sm)) if sp > 0 and sm > 0 else float("nan")
    return {"n": int(p.size), "r2": r2, "pearson": pearson, "rmse": float(np.sqrt(np.mean(res ** 2))),
            "mae": float(np.mean(np.abs(res)))}


class ErrorModelSelectiveAttention:
    def __init__(self, B: int, H: int, D: int, offsets: Sequence[int], q: int, g: int, scale: float,
                 reuse_ratio: float, eps_local: float, dtype=torch.bfloat16, device="cuda",
                 evaluate: bool = False):
        self.B, self.H, self.D = B, H, D
        self.offsets = [int(o) for o in offsets]
        self.P = len(self.offsets) - 1
        self.q, self.g = q, g
        self.scale = float(scale)
        self.R, self.eps_local = float(reuse_ratio), float(eps_local)
        self.dtype, self.device = dtype, device
        # evaluation of the error model (costs a full attention pass per
        # step): record the error every cached group state actually carries
        self.evaluate = bool(evaluate)
        self.L = self.offsets[q + 1] - self.offsets[q]
        shp = (self.P, B, self.L, H, D)
        self.cache = torch.zeros(shp, dtype=dtype, device=device)
        self.cache_lse = torch.full((self.P, B, H, self.L), float("-inf"), dtype=torch.float32, device=device)
        self.fresh = torch.zeros(shp, dtype=dtype, device=device)
        self.fresh_lse = torch.full((self.P, B, H, self.L), float("-inf"), dtype=torch.float32, device=device)
        self.groups = base_groups(self.P, q, g)
        self.t_c: Dict[Tuple[int, int], int] = {grp: -1 for grp in self.groups}
        self.t_a: Optional[int] = None
        self.w: List[float] = []
        self.alpha: List[float] = []
        # snapshots of OUT(loc) at the steps still referenced (t_a and every
        # group's t_c), kept in slots of one preallocated buffer so that the
        # drift norms read them in place
        self.snapbuf = torch.zeros((len(self.groups) + 2, B, self.L, H, D), dtype=dtype, device=device)
        self.snap: Dict[int, int] = {}               # step -> snapbuf slot
        self.corrections: List[float] = []
        self.eps: Optional[float] = None
        nws = max(api.norms_workspace_bytes(B, H, D, self.L, self.P), api.contrib_workspace_bytes(B, H, self.L, self.P))
        self._ws = torch.empty(max(16, nws), dtype=torch.uint8, device=device)
        self._attn_ws = AttnWorkspace(device)

    # ---------------------------------------------------------------- helpers
    def _norms(self, states: torch.Tensor, slots: Sequence[int], ref: Optional[torch.Tensor] = None) -> List[float]:
        out = torch.empty(len(slots), dtype=torch.float32, device=self.device)
        api.state_norms(states, out, self._ws, slots=list(slots), ref=ref)
        return out.cpu().tolist()

    def _snapshot(self, t: int) -> None:
        """OUT(loc) of step t into a free snapshot slot."""
        used = set(self.snap.values())
        slot = next(i for i in range(self.snapbuf.shape[0]) if i not in used)
        self.snapbuf[slot].copy_(self.cache[self.q])
        self.snap[t] = slot

    def _attn(self, q, k, v, sel, states, lses):
        ws = self._attn_ws.get(q.dtype, q.shape[0], q.shape[2], q.shape[3], q.shape[1], self.offsets, sel)
        api.attn_partition_states(q, k, v, self.offsets, sel, self.scale, states, lses, ws)

    def _compose_group(self, states, lses, grp):
        if grp[1] - grp[0] > 1:
            a = grp[0]
            api.merge_states(states, lses, states[a], lses[a], slots=list(range(*grp)))

    # ---------------------------------------------------------------- one step
    def step(self, t: int, q_all: torch.Tensor, k: torch.Tensor, v: torch.Tensor):
        """Returns (OUT, LSE, info) with info = dict(anchor, compute, ase, eps, drift), and,
        when the model is evaluated, ``measured`` (group -> the error its cached
        state actually carries) at every step after the first."""
        a, e = self.offsets[self.q], self.offsets[self.q + 1]
        qb = q_all[:, a:e].contiguous()
        loc = [0] * self.P
        loc[self.q] = 1
        self._attn(qb, k, v, loc, self.cache, self.cache_lse)          # local partition first
        info = {"ase": {}, "eps": self.eps, "drift": None}
        if self.t_a is None:
            anchor = True
        else:
            tcs = sorted(set(self.t_c.values()) | {self.t_a})
            cur = self.cache[self.q]
            d = dict(zip(tcs, self._norms(self.snapbuf, [self.snap[tc] for tc in tcs], ref=cur)))
            n_loc = self.alpha_ref
            drift = d[self.t_a] / n_loc if n_loc > 0 else 0.0
            ase = {grp: sum(self.w[j] * self.alpha[j] for j in range(*grp)) * d[self.t_c[grp]] for grp in self.groups}
            if self.eps is None:
                self.eps = quantile_r(list(ase.values()), self.R)
            info.update(ase=ase, eps=self.eps, drift=drift)
            anchor = all(x > self.eps for x in ase.values()) or drift > self.eps_local
            if self.evaluate:
                info["measured"] = self._measure(qb, k, v)
        if anchor:
            compute = list(self.groups)
            self._anchor(t, qb, k, v)
        else:
            compute = [grp for grp in self.groups if info["ase"][grp] > self.eps]
            sel = [0] * self.P
            for grp in compute:
                for j in range(*grp):
                    sel[j] = 1
            if any(sel):
                self._attn(qb, k, v, sel, self.cache, self.cache_lse)
                for grp in compute:
                    self._compose_group(self.cache, self.cache_lse, grp)
                    self.t_c[grp] = t
                self._snapshot(t)
        live = set(self.t_c.values()) | {self.t_a}
        self.snap = {tc: i for tc, i in self.snap.items() if tc in live}
        slots = [grp[0] for grp in self.groups] + [self.q]
        out = torch.empty((self.B, self.L, self.H, self.D), dtype=self.dtype, device=self.device)
        lse = torch.empty((self.B, self.H, self.L), dtype=torch.float32, device=self.device)
        api.merge_states(self.cache, self.cache_lse, out, lse, slots=slots)
        info.update(anchor=anchor, compute=compute)
        return out, lse, info

    def _measure(self, qb, k, v) -> Dict[Tuple[int, int], float]:
        """The error each cached group state carries at this step, the
        quantity the ASE of Eq. ase_decomposition models: w(G, t) ||AS_t(G) -
        AS_tc(G)||, with every partition computed fresh (evaluation only, in
        the anchor buffers, which are free between anchors), each group's
        fresh state composed, and w(G, t) its partitions' weights in the full
        composition of this step (Eq. lse_weight at t)."""
        self._attn(qb, k, v, [1] * self.P, self.fresh, self.fresh_lse)
        out = torch.empty((self.B, self.L, self.H, self.D), dtype=self.dtype, device=self.device)
        lse = torch.empty((self.B, self.H, self.L), dtype=torch.float32, device=self.device)
        api.merge_states(self.fresh, self.fresh_lse, out, lse)
        w = torch.empty(self.P, dtype=torch.float32, device=self.device)
        api.contrib(self.fresh_lse, lse, w, self._ws)
        w_t = w.cpu().tolist()
        measured = {}
        for grp in self.groups:
            self._compose_group(self.fresh, self.fresh_lse, grp)
            n = self._norms(self.fresh, [grp[0]], ref=self.cache[grp[0]])[0]
            measured[grp] = sum(w_t[j] for j in range(*grp)) * n
        return measured

    def _anchor(self, t: int, qb, k, v) -> None:
        sel = [1] * self.P
        self._attn(qb, k, v, sel, self.fresh, self.fresh_lse)
        # anchor weights per partition and scale ratios, before any composition
        out = torch.empty((self.B, self.L, self.H, self.D), dtype=self.dtype, device=self.device)
        lse = torch.empty((self.B, self.H, self.L), dtype=torch.float32, device=self.device)
        api.merge_states(self.fresh, self.fresh_lse, out, lse)
        w = torch.empty(self.P, dtype=torch.float32, device=self.device)
        api.contrib(self.fresh_lse, lse, w, self._ws)
        w_new = w.cpu().tolist()
        norms = self._norms(self.fresh, range(self.P))
        for grp in self.groups:
            self._compose_group(self.fresh, self.fresh_lse, grp)
        if self.t_a is not None:
            # anchor correction errors: fresh group state against the cached one
            for grp in self.groups:
                n = self._norms(self.fresh, [grp[0]], ref=self.cache[grp[0]])[0]
                self.corrections.append(sum(self.w[j] for j in range(*grp)) * n)
            self.eps = quantile_r(self.corrections, self.R)
        self.cache.copy_(self.fresh)
        self.cache_lse.copy_(self.fresh_lse)
        self.w = w_new
        self.alpha_ref = norms[self.q]
        self.alpha = [nj / norms[self.q] if norms[self.q] > 0 else 0.0 for nj in norms]
        self.t_a = t
        self.t_c = {grp: t for grp in self.groups}
        self.snap = {}
        self._snapshot(t)
