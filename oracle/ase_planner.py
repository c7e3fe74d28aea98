"""Oracle of the error-model selection (the paper's Alg. 1 with group states),
float64, test infrastructure only.  Same readings as the product: norms are
Frobenius norms of a state's output; a group cached at t_c has
ASE = sum_j w(j) alpha(j) ||OUT_t(loc) - OUT_tc(loc)|| (Eq. ase_decomposition,
Eq. scale_ratio, Eq. error_extrapolation); anchors when every group exceeds
eps or the relative local drift exceeds eps_local (Sec. 4.2.4); eps is the
R-quantile of the anchor correction errors w(G) ||fresh(G) - cached(G)||,
and before any exist the R-quantile of the current step's ASE values.

Each step's result also records the step every group was last computed at
(``t_c``) and every anchor correction error recorded so far
(``corrections``, in the order they were recorded: anchor by anchor, groups
in order).
"""
from __future__ import annotations

import math
from typing import Dict, Sequence

import numpy as np

from .groups import groups_of
from .state import contrib, merge, partition_state


def r_quantile(values, r):
    v = sorted(values)
    return v[max(0, min(len(v) - 1, int(math.ceil(r * len(v))) - 1))]


def run(steps: Sequence[Dict[str, np.ndarray]], offsets, q, g, R, eps_local, scale, force=None,
        evaluate=False):
    """``force`` (optional) maps a step t to a decision (anchor, groups to
    compute) taken instead of the rule's, after the rule's inputs (ASE,
    drift, eps) have been formed: a test re-synchronises with a run whose
    decision differed on a near-tie.

    ``evaluate``: at every non-anchor step also record, for every group, the
    error its cached state actually carries, the quantity ASE predicts
    (Eq. ase_decomposition with the true state change instead of
    Eq. error_extrapolation): w(G, t) ||AS_t(G) - AS_tc(G)||, with AS_t(G)
    the group's state composed from fresh states of step t, AS_tc(G) its
    cached state before the step's recomputation, and w(G, t) the sum of its
    partitions' weights in the full composition at step t (Eq. lse_weight at
    t).  Evaluation only: it costs a full attention pass per step."""
    P = len(offsets) - 1
    groups = groups_of(P, q, g)
    part = lambda qx, x, j: partition_state(qx, x["k"][:, offsets[j]:offsets[j + 1]],
                                            x["v"][:, offsets[j]:offsets[j + 1]], scale)
    cache, t_c, snap = {}, {}, {}
    t_a, w, alpha, n_loc, eps = None, None, None, None, None
    corrections = []
    results = []
    for t, x in enumerate(steps):
        qx = x["q"][:, offsets[q]:offsets[q + 1]]
        local = part(qx, x, q)
        ase, drift, measured = {}, None, None
        if t_a is None:
            anchor = True
        else:
            d = {tc: float(np.linalg.norm(local[0] - snap[tc])) for tc in set(t_c.values()) | {t_a}}
            drift = d[t_a] / n_loc if n_loc > 0 else 0.0
            for grp in groups:
                ase[grp] = sum(w[j] * alpha[j] for j in range(*grp)) * d[t_c[grp]]
            if eps is None:
                eps = r_quantile(list(ase.values()), R)
            anchor = all(ase[grp] > eps for grp in groups) or drift > eps_local
            if evaluate:
                sts = [part(qx, x, j) for j in range(P)]
                _, full_lse = merge([s_[0] for s_ in sts], [s_[1] for s_ in sts])
                _, w_t = contrib([s_[1] for s_ in sts], full_lse)
                measured = {}
                for grp in groups:
                    fresh_g = merge([sts[j][0] for j in range(*grp)], [sts[j][1] for j in range(*grp)])
                    measured[grp] = (sum(w_t[j] for j in range(*grp)) *
                                     float(np.linalg.norm(fresh_g[0] - cache[grp][0])))
        forced = force is not None and t in force
        if forced:
            anchor = bool(force[t][0])
        if anchor:
            compute = list(groups)
            sts = [part(qx, x, j) for j in range(P)]
            full_out, full_lse = merge([s_[0] for s_ in sts], [s_[1] for s_ in sts])
            _, w_new = contrib([s_[1] for s_ in sts], full_lse)
            norms = [float(np.linalg.norm(s_[0])) for s_ in sts]
            fresh = {grp: merge([sts[j][0] for j in range(*grp)], [sts[j][1] for j in range(*grp)]) for grp in groups}
            if t_a is not None:
                for grp in groups:
                    corrections.append(sum(w[j] for j in range(*grp)) *
                                       float(np.linalg.norm(fresh[grp][0] - cache[grp][0])))
                eps = r_quantile(corrections, R)
            cache = dict(fresh)
            w = list(w_new)
            n_loc = norms[q]
            alpha = [nj / n_loc if n_loc > 0 else 0.0 for nj in norms]
            t_a = t
            t_c = {grp: t for grp in groups}
            snap = {t: local[0]}
        else:
            compute = [grp for grp in groups if ase[grp] > eps]
            if forced:
                compute = [tuple(grp) for grp in force[t][1]]
            for grp in compute:
                sts = [part(qx, x, j) for j in range(*grp)]
                cache[grp] = merge([s_[0] for s_ in sts], [s_[1] for s_ in sts])
                t_c[grp] = t
            if compute:
                snap[t] = local[0]
        out, lse = merge([cache[grp][0] for grp in groups] + [local[0]],
                         [cache[grp][1] for grp in groups] + [local[1]])
        results.append(dict(anchor=anchor, compute=compute, ase=ase, eps=eps, drift=drift, out=out, lse=lse,
                            t_c=dict(t_c), corrections=list(corrections), measured=measured))
    return results
