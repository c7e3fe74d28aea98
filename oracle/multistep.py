"""Oracle of the planner-driven multi-step workload (test infrastructure only).

Per step and query block: partitions selected for the step get a state from
that step's tensors; the others keep the state computed at the step they were
last selected (Sec. 2.2.4 reuse; Sec. 5.2 state cache).  Anchor steps select
every partition and record the per-partition weights; other steps select the
query partition plus every partition whose anchor weight exceeds the
threshold (Sec. 4.1.2, Eq. lse_weight; the local partition is always
computed).  Everything in float64.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from .state import contrib, merge, partition_state, plan_threshold


def run(steps: Sequence[Dict[str, np.ndarray]], offsets: Sequence[int], blocks: Sequence[int],
        anchors: Sequence[int], threshold: float, scale: float, force=None):
    """``steps[s]`` holds float64 q, k, v [B, S, H, D] of step s.

    Returns a list over steps of dicts {block: (mask, out, lse, wbar)}.
    ``force`` (optional) maps (step, block) to a mask used instead of the
    rule's: a test re-synchronises with a run whose mask differed on a
    near-tie.
    """
    P = len(offsets) - 1
    cache = {qb: [None] * P for qb in blocks}
    anchor_w = {qb: None for qb in blocks}
    results = []
    for s, x in enumerate(steps):
        res = {}
        for qb in blocks:
            if s in anchors or anchor_w[qb] is None:
                mask = [1] * P
            else:
                mask = plan_threshold(anchor_w[qb], qb, threshold)
            if force is not None and (s, qb) in force:
                mask = list(force[(s, qb)])
            q = x["q"][:, offsets[qb]:offsets[qb + 1]]
            for j in range(P):
                if mask[j]:
                    a, e = offsets[j], offsets[j + 1]
                    cache[qb][j] = partition_state(q, x["k"][:, a:e], x["v"][:, a:e], scale)
            outs = [cache[qb][j][0] for j in range(P)]
            lses = [cache[qb][j][1] for j in range(P)]
            out, lse = merge(outs, lses)
            _, wbar = contrib(lses, lse)
            if s in anchors or anchor_w[qb] is None:
                anchor_w[qb] = list(wbar)
            res[qb] = (mask, out, lse, wbar)
        results.append(res)
    return results
