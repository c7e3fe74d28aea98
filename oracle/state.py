"""Float64 NumPy oracle of the selective attention-state hot path.

Test infrastructure only (see the package docstring): never imported by the
product.

Readings of the paper taken here (where it is silent or loose):

* Eq. attention_state writes exp(q.k) with no softmax scale; DiT attention
  uses scale = 1/sqrt(D), so every exponent here is ``scale*q.k`` and LSE
  includes the scale.  The scale is passed in explicitly.
* Logarithms are natural.  The stored state is the normalised output OUT and
  LSE as in Eq. attention_state.
* A partition with no keys (or a row whose keys are all absent) has
  LSE = -inf and OUT = 0; it then carries weight 0 in every composition.
* The per-partition contribution scalar is the mean of the per-row weights
  exp(LSE_j - LSE) over all (batch, head, row); the paper defines w per row in
  Eq. lse_weight but uses it as one number per partition in Eq. ase_decomposition.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np

F64 = np.float64


def partition_state(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Attention state of one key/value partition (Sec. 2.2.4, Eq. attention_state).

    q: [B, Lq, H, D], k and v: [B, L, H, D] (any float dtype; computed in float64).
    Returns OUT [B, Lq, H, D] and LSE [B, H, Lq] where, per (b, h, query row r),
    LSE = log sum_c exp(scale * q_r . k_c) and
    OUT = sum_c exp(scale * q_r . k_c - LSE) v_c.
    The max-subtraction below is the usual exact rewrite of these sums.
    """
    q = np.asarray(q, dtype=F64)
    k = np.asarray(k, dtype=F64)
    v = np.asarray(v, dtype=F64)
    B, Lq, H, D = q.shape
    L = k.shape[1]
    out = np.zeros((B, Lq, H, D), dtype=F64)
    lse = np.full((B, H, Lq), -np.inf, dtype=F64)
    if L == 0 or Lq == 0:
        return out, lse
    s = F64(scale)
    for b in range(B):
        for h in range(H):
            sc = s * (q[b, :, h, :] @ k[b, :, h, :].T)          # [Lq, L]
            m = sc.max(axis=1)                                   # [Lq]
            e = np.exp(sc - m[:, None])
            l = e.sum(axis=1)
            out[b, :, h, :] = (e @ v[b, :, h, :]) / l[:, None]
            lse[b, h, :] = m + np.log(l)
    return out, lse


def partition_states(q, k, v, offsets: Sequence[int], scale: float,
                     which: Optional[Sequence[int]] = None):
    """States of partitions ``which`` (default all) of k/v split at ``offsets``.

    Returns lists OUT_j, LSE_j indexed by partition (None for partitions not
    in ``which``).
    """
    P = len(offsets) - 1
    which = range(P) if which is None else which
    outs: List[Optional[np.ndarray]] = [None] * P
    lses: List[Optional[np.ndarray]] = [None] * P
    for j in which:
        a, e = offsets[j], offsets[j + 1]
        outs[j], lses[j] = partition_state(q, k[:, a:e], v[:, a:e], scale)
    return outs, lses


def compose2(out_i, lse_i, out_j, lse_j):
    """Binary state composition (Sec. 2.2.4, Eq. composition).

    OUT = (e^{L_i} OUT_i + e^{L_j} OUT_j) / (e^{L_i} + e^{L_j}),
    LSE = log(e^{L_i} + e^{L_j}), with both exponentials shifted by
    max(L_i, L_j) so they cannot overflow.  OUT is [B, Lq, H, D], LSE [B, H, Lq].
    """
    li = np.asarray(lse_i, F64)
    lj = np.asarray(lse_j, F64)
    m = np.maximum(li, lj)
    dead = np.isneginf(m)
    ms = np.where(dead, 0.0, m)
    ei = np.exp(li - ms)
    ej = np.exp(lj - ms)
    den = ei + ej
    lse = np.where(dead, -np.inf, ms + np.log(np.where(dead, 1.0, den)))
    wi = np.where(dead, 0.0, ei / np.where(dead, 1.0, den))
    wj = np.where(dead, 0.0, ej / np.where(dead, 1.0, den))
    # weights are [B, H, Lq]; outputs are [B, Lq, H, D]
    wi_ = np.transpose(wi, (0, 2, 1))[..., None]
    wj_ = np.transpose(wj, (0, 2, 1))[..., None]
    out = wi_ * np.asarray(out_i, F64) + wj_ * np.asarray(out_j, F64)
    return out, lse


def merge(outs: Sequence[np.ndarray], lses: Sequence[np.ndarray]):
    """n-ary composition of states (Eq. composition applied over all states at once).

    With M = max_j LSE_j: LSE = M + log sum_j e^{LSE_j - M},
    OUT = sum_j e^{LSE_j - LSE} OUT_j.  All-(-inf) rows give OUT = 0, LSE = -inf.
    """
    if len(outs) == 0:
        raise ValueError("merge of zero states")
    L = np.stack([np.asarray(x, F64) for x in lses])           # [n, B, H, Lq]
    O = np.stack([np.asarray(x, F64) for x in outs])           # [n, B, Lq, H, D]
    M = L.max(axis=0)
    dead = np.isneginf(M)
    Ms = np.where(dead, 0.0, M)
    E = np.exp(L - Ms[None])
    tot = E.sum(axis=0)
    lse = np.where(dead, -np.inf, Ms + np.log(np.where(dead, 1.0, tot)))
    W = np.where(dead[None], 0.0, E / np.where(dead, 1.0, tot)[None])   # [n, B, H, Lq]
    Wt = np.transpose(W, (0, 1, 3, 2))[..., None]                        # [n, B, Lq, H, 1]
    out = (Wt * O).sum(axis=0)
    return out, lse


def full_attention(q, k, v, scale: float):
    """One-shot softmax attention over all keys: the state of the whole sequence."""
    return partition_state(q, k, v, scale)


def selective_step(q, k, v, q_prev, k_prev, v_prev, offsets, select, scale):
    """One selective step (Sec. 2.2.4, Fig. 4; Sec. 5.2 'partition status').

    Partitions j with select[j] get a fresh state from the current tensors;
    the others reuse the state computed from the previous step's tensors.
    All P states are then composed.  Returns (OUT, LSE, outs, lses).
    """
    P = len(offsets) - 1
    outs, lses = [None] * P, [None] * P
    for j in range(P):
        a, e = offsets[j], offsets[j + 1]
        if select[j]:
            outs[j], lses[j] = partition_state(q, k[:, a:e], v[:, a:e], scale)
        else:
            outs[j], lses[j] = partition_state(q_prev, k_prev[:, a:e], v_prev[:, a:e], scale)
    out, lse = merge(outs, lses)
    return out, lse, outs, lses


def contrib(lses: Sequence[np.ndarray], lse: np.ndarray):
    """Contribution weights of each partition state to the composed state.

    Per row: W_j = e^{LSE_j} / sum_k e^{LSE_k} = e^{LSE_j - LSE}
    (w_i of Sec. 4.1.1; Eq. lse_weight).  Returns W [B, H, Lq, P] and the
    per-partition means wbar [P] over all (b, h, r).  Rows whose composed LSE
    is -inf get W = 0.
    """
    L = np.stack([np.asarray(x, F64) for x in lses], axis=-1)     # [B, H, Lq, P]
    lse = np.asarray(lse, F64)[..., None]
    dead = np.isneginf(lse)
    W = np.where(dead, 0.0, np.exp(L - np.where(dead, 0.0, lse)))
    W = np.where(np.isneginf(L), 0.0, W)
    wbar = W.reshape(-1, W.shape[-1]).mean(axis=0) if W.size else np.zeros(W.shape[-1])
    return W, wbar


def rank_partitions(wbar: Sequence[float], q: int) -> List[int]:
    """Partitions ordered by decreasing contribution, ties by (|j - q|, j)."""
    return sorted(range(len(wbar)), key=lambda j: (-float(wbar[j]), abs(j - q), j))


def plan_threshold(wbar: Sequence[float], q: int, thr: float) -> List[int]:
    """Next-step selection from anchor weights: the query partition plus every
    partition whose mean contribution weight strictly exceeds ``thr``.

    The local (diagonal) partition is always computed (Sec. 4.1.2); anchor
    weights stand in for the current ones over the following steps
    (Eq. lse_weight).
    """
    return [1 if (j == q or float(wbar[j]) > thr) else 0 for j in range(len(wbar))]
