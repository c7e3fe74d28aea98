"""Host-side selection of the partitions to compute fresh at the next step.

The planner-driven workload follows the paper's anchor scheme in its simplest
form: at anchor steps every partition is computed and the per-partition
contribution weights are recorded (Sec. 4.1.2, Eq. lse_weight, which keeps the
anchor weights for the following steps); at the other steps the query
(local, diagonal) partition is always computed (Sec. 4.1.2) together with
every partition whose anchor weight exceeds the threshold.  The paper's full
error-model planner (Alg. 1: age penalty, group errors, adaptive threshold)
is not part of this module.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np


def rank_partitions(wbar: Sequence[float], q: int) -> List[int]:
    """Partitions by decreasing contribution weight; equal weights by distance
    to the query partition q, then by index (numpy's stable lexicographic
    sort, whose last key is the primary one)."""
    w = np.asarray(wbar, dtype=np.float64)
    idx = np.arange(w.size)
    return [int(j) for j in np.lexsort((idx, np.abs(idx - q), -w))]


def plan_threshold(wbar: Sequence[float], q: int, thr: float) -> List[int]:
    """Mask of partitions to compute: q, and every j with weight strictly above thr."""
    m = (np.asarray(wbar, dtype=np.float64) > float(thr)).astype(np.int64)
    m[q] = 1
    return [int(x) for x in m]


class AnchorPlanner:
    """Per-query-block selection over denoising steps.

    ``select(step)`` returns the mask for ``step``; ``observe(step, wbar)``
    records the weights measured at that step (kept only at anchors).
    """

    def __init__(self, P: int, q: int, anchors: Sequence[int], threshold: float):
        self.P, self.q = P, q
        self.anchors = set(int(a) for a in anchors)
        self.threshold = float(threshold)
        self.anchor_wbar: Optional[List[float]] = None

    def is_anchor(self, step: int) -> bool:
        return step in self.anchors or self.anchor_wbar is None

    def select(self, step: int) -> List[int]:
        if self.is_anchor(step):
            return [1] * self.P
        return plan_threshold(self.anchor_wbar, self.q, self.threshold)

    def observe(self, step: int, wbar: Sequence[float]) -> None:
        if self.is_anchor(step):
            self.anchor_wbar = [float(x) for x in wbar]
