"""Oracle of group states and Dynamic Group State Compose (test infrastructure only).

Groups of g contiguous partitions, the local partition kept apart (Sec. 4.2.1);
a computed group's state is the composition of its members' fresh states, a
reused group keeps the state of the step it was last computed (Sec. 4.2.2,
Sec. 5.2); when more than ``max_states`` group states are cached at the start
of a non-anchor step, runs of k adjacent groups are composed into one
(Sec. 5.1, Eq. GroupCompose), repeatedly; an anchor step recomputes every
partition and restores the base grouping.  Non-anchor steps compute the
groups whose anchor weight (the sum of the anchor weights of the base groups
they contain) exceeds the threshold.  float64 throughout.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

from .state import contrib, merge, partition_state


def groups_of(P: int, q: int, g: int) -> List[Tuple[int, int]]:
    """Base groups: maximal contiguous runs of {j : j // g == i, j != q}."""
    result = []
    for i in range(0, P, g):
        js = [j for j in range(i, min(i + g, P)) if j != q]
        while js:
            a = js[0]
            b = a + 1
            while b in js:
                b += 1
            result.append((a, b))
            js = [j for j in js if j >= b]
    return result


def compose_runs(groups: List[Tuple[int, int]], k: int) -> List[List[Tuple[int, int]]]:
    runs: List[List[Tuple[int, int]]] = []
    for grp in groups:
        if runs and len(runs[-1]) < k and runs[-1][-1][1] == grp[0]:
            runs[-1].append(grp)
        else:
            runs.append([grp])
    return runs


def run(steps: Sequence[Dict[str, np.ndarray]], offsets: Sequence[int], q: int, g: int, k: int,
        max_states: int, anchors: Sequence[int], threshold: float, scale: float):
    """Returns per step: (groups, computed groups, OUT, LSE, weights of groups + local)."""
    P = len(offsets) - 1
    base = groups_of(P, q, g)
    groups = list(base)
    state: Dict[Tuple[int, int], tuple] = {}
    anchor_w: Dict[Tuple[int, int], float] = {}
    out_steps = []
    for s, x in enumerate(steps):
        qx = x["q"][:, offsets[q]:offsets[q + 1]]
        anchor = s in anchors or not anchor_w
        if anchor:
            groups = list(base)
            compute = list(groups)
        else:
            while len(groups) > max_states:
                runs = compose_runs(groups, k)
                if all(len(r) == 1 for r in runs):
                    break
                new = []
                for r in runs:
                    grp = (r[0][0], r[-1][1])
                    if len(r) > 1:
                        state[grp] = merge([state[x_][0] for x_ in r], [state[x_][1] for x_ in r])
                    new.append(grp)
                groups = new
            compute = [grp for grp in groups
                       if sum(anchor_w[b] for b in base if grp[0] <= b[0] and b[1] <= grp[1]) > threshold]
        for grp in compute:
            sts = [partition_state(qx, x["k"][:, offsets[j]:offsets[j + 1]], x["v"][:, offsets[j]:offsets[j + 1]],
                                   scale) for j in range(*grp)]
            state[grp] = merge([t[0] for t in sts], [t[1] for t in sts])
        local = partition_state(qx, x["k"][:, offsets[q]:offsets[q + 1]], x["v"][:, offsets[q]:offsets[q + 1]], scale)
        outs = [state[grp][0] for grp in groups] + [local[0]]
        lses = [state[grp][1] for grp in groups] + [local[1]]
        out, lse = merge(outs, lses)
        _, w = contrib(lses, lse)
        if anchor:
            anchor_w = {grp: float(w[i]) for i, grp in enumerate(groups)}
        out_steps.append((list(groups), list(compute), out, lse, w))
    return out_steps
