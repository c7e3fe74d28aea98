"""Pins of the multi-step oracles (group states with Dynamic Group State
Compose, and the error-model planner of Alg. 1) against things other than
themselves, on the CPU.

What fixes the expected values:
* composition is exact (Sec. 2.2.4, Eq. composition): with the same tensors
  at every step, any mix of fresh, reused and composed group states must
  give full softmax attention, whatever the grouping, budget or selection;
* the grouping and compose rules of Sec. 4.2.1 and Sec. 5.1 worked by hand
  on a small case;
* a construction where the error model's inputs have closed forms: scaling
  V by (1 + c) scales every partition's OUT by (1 + c) and leaves every LSE
  (hence every weight) unchanged, so the local drift is exactly c and the
  extrapolated error of a group (Eq. ase_decomposition with the scale ratios
  of Eq. scale_ratio and the local drift of Eq. error_extrapolation) is
  exactly c * sum_{j in G} w_j ||OUT_j||.
"""
import math

import numpy as np
import pytest

import oracle
from oracle import ase_planner, groups as og
from fixtures.workloads import partition_offsets


def seq(seed, S=40, H=2, D=8, B=1):
    rng = np.random.default_rng(seed)
    return {n: rng.standard_normal((B, S, H, D)) for n in ("q", "k", "v")}


def full(x, offs, q, scale):
    return oracle.full_attention(x["q"][:, offs[q]:offs[q + 1]], x["k"], x["v"], scale)


# ------------------------------------------------ group states and compose

@pytest.mark.parametrize("g,k,max_states,thr", [(1, 2, 99, 0.1), (2, 2, 2, 0.0), (2, 3, 1, 0.2), (3, 2, 1, 1.0)])
def test_group_run_with_unchanged_tensors_is_full_attention(g, k, max_states, thr):
    x = seq(3)
    S, P, q, scale = 40, 8, 3, 0.35
    offs = partition_offsets(S, P)
    res = og.run([x] * 5, offs, q, g, k, max_states, anchors=(0,), threshold=thr, scale=scale)
    fo, fl = full(x, offs, q, scale)
    for groups, compute, out, lse, w in res:
        np.testing.assert_allclose(out, fo, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(lse, fl, rtol=1e-13)
        np.testing.assert_allclose(np.sum(w, axis=0), 1.0, rtol=1e-12)


def test_group_run_worked_example_of_the_compose_rule():
    # P=8, local partition 3, g=2: base groups {0,1} {2} {4,5} {6,7}
    # (Sec. 4.2.1, the local partition kept apart); at a non-anchor step with
    # room for 2 cached group states, runs of k=2 adjacent groups are composed:
    # {0,1}+{2} -> {0,1,2}, {4,5}+{6,7} -> {4..7} (Sec. 5.1, Eq. GroupCompose)
    x = seq(4)
    offs = partition_offsets(40, 8)
    res = og.run([x] * 3, offs, 3, 2, 2, 2, anchors=(0,), threshold=1.0, scale=0.35)
    assert res[0][0] == [(0, 2), (2, 3), (4, 6), (6, 8)]        # anchor: base grouping, all computed
    assert res[0][1] == [(0, 2), (2, 3), (4, 6), (6, 8)]
    assert res[1][0] == [(0, 3), (4, 8)]                        # composed under the budget
    assert res[1][1] == []                                      # threshold 1.0: nothing recomputed
    assert res[2][0] == [(0, 3), (4, 8)]


def test_group_run_reused_states_come_from_their_own_step():
    # changed tensors: a group that is not recomputed keeps the state of the
    # step where it was last computed, composed from that step's tensors
    S, P, q, scale = 40, 8, 3, 0.35
    offs = partition_offsets(S, P)
    xs = [seq(10 + s) for s in range(3)]
    res = og.run(xs, offs, q, 2, 2, 99, anchors=(0,), threshold=1.0, scale=scale)
    qx = [x["q"][:, offs[q]:offs[q + 1]] for x in xs]
    # threshold 1.0: after the anchor at step 0 no group is recomputed, so at
    # step 2 every group state is the one computed at step 0 (from step 0's
    # queries, keys and values), composed with step 2's local state
    sts0 = [oracle.partition_state(qx[0], xs[0]["k"][:, offs[j]:offs[j + 1]], xs[0]["v"][:, offs[j]:offs[j + 1]],
                                   scale) for j in range(P) if j != q]
    local2 = oracle.partition_state(qx[2], xs[2]["k"][:, offs[q]:offs[q + 1]], xs[2]["v"][:, offs[q]:offs[q + 1]],
                                    scale)
    eo, el = oracle.merge([s_[0] for s_ in sts0] + [local2[0]], [s_[1] for s_ in sts0] + [local2[1]])
    groups, compute, out, lse, _ = res[2]
    assert compute == []
    np.testing.assert_allclose(out, eo, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, el, rtol=1e-13)


def test_group_run_budget_and_coverage_invariants():
    S, P, q = 48, 12, 5
    offs = partition_offsets(S, P)
    xs = [seq(20 + s, S=S) for s in range(6)]
    for g in (1, 2, 3):
        for k in (2, 3):
            for max_states in (1, 2, 3, 5):
                res = og.run(xs, offs, q, g, k, max_states, anchors=(0, 3), threshold=0.15, scale=0.3)
                base = og.groups_of(P, q, g)
                for s, (groups, compute, _, _, w) in enumerate(res):
                    covered = sorted(j for a, b in groups for j in range(a, b))
                    assert covered == [j for j in range(P) if j != q]          # every partition once
                    assert all(not (a <= q < b) for a, b in groups)            # never across the local one
                    assert set(compute) <= set(groups)
                    assert len(w) == len(groups) + 1
                    if s in (0, 3):
                        assert groups == base and compute == base
                    else:
                        runs = og.compose_runs(groups, k)
                        # either within the budget, or no two groups left to compose
                        assert len(groups) <= max_states or all(len(r) == 1 for r in runs)


def test_base_groups_hand_examples():
    assert og.groups_of(8, 3, 2) == [(0, 2), (2, 3), (4, 6), (6, 8)]
    assert og.groups_of(8, 5, 4) == [(0, 4), (4, 5), (6, 8)]
    assert og.groups_of(8, 0, 3) == [(1, 3), (3, 6), (6, 8)]
    assert og.groups_of(4, 2, 1) == [(0, 1), (1, 2), (3, 4)]
    assert og.compose_runs([(0, 2), (2, 3), (4, 6), (6, 8)], 2) == [[(0, 2), (2, 3)], [(4, 6), (6, 8)]]
    assert og.compose_runs([(0, 1), (1, 2), (3, 4)], 3) == [[(0, 1), (1, 2)], [(3, 4)]]


# ------------------------------------------------------- error-model planner

def test_quantile_hand_examples():
    assert ase_planner.r_quantile([4.0, 1.0, 3.0, 2.0], 0.5) == 2.0
    assert ase_planner.r_quantile([4.0, 1.0, 3.0, 2.0], 0.75) == 3.0
    assert ase_planner.r_quantile([5.0, 1.0, 3.0], 1.0) == 5.0
    assert ase_planner.r_quantile([5.0, 1.0, 3.0], 0.0) == 1.0
    assert ase_planner.r_quantile([7.0], 0.4) == 7.0


def test_error_planner_with_unchanged_tensors_reuses_everything_exactly():
    S, P, q, scale = 40, 8, 3, 0.35
    offs = partition_offsets(S, P)
    x = seq(5)
    res = ase_planner.run([x] * 4, offs, q, 2, 0.5, 0.1, scale)
    fo, fl = full(x, offs, q, scale)
    assert res[0]["anchor"]
    for r in res[1:]:
        assert not r["anchor"] and r["compute"] == [] and r["drift"] == 0.0
        assert all(v == 0.0 for v in r["ase"].values())
    for r in res:
        np.testing.assert_allclose(r["out"], fo, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(r["lse"], fl, rtol=1e-13)


@pytest.mark.parametrize("c", [0.02, 0.3])
def test_error_planner_closed_forms_under_a_value_scaling(c):
    S, P, q, scale, g = 40, 8, 3, 0.35, 2
    offs = partition_offsets(S, P)
    x0 = seq(6)
    x1 = dict(x0, v=x0["v"] * (1.0 + c))
    eps_local = 0.1
    res = ase_planner.run([x0, x1], offs, q, g, 0.5, eps_local, scale)
    qx = x0["q"][:, offs[q]:offs[q + 1]]
    sts = [oracle.partition_state(qx, x0["k"][:, offs[j]:offs[j + 1]], x0["v"][:, offs[j]:offs[j + 1]], scale)
           for j in range(P)]
    _, lse = oracle.merge([s_[0] for s_ in sts], [s_[1] for s_ in sts])
    _, wbar = oracle.contrib([s_[1] for s_ in sts], lse)
    r = res[1]
    assert r["drift"] == pytest.approx(c, rel=1e-12)                 # ||dOUT_loc|| / ||OUT_loc||
    for (a, b), ase in r["ase"].items():
        expect = c * sum(wbar[j] * np.linalg.norm(sts[j][0]) for j in range(a, b))
        assert ase == pytest.approx(expect, rel=1e-10)
    # a relative local drift above eps_local makes the step an anchor (Sec. 4.2.4)
    assert r["anchor"] == (c > eps_local)


# ---- several anchors: the eps adaptation, group snapshots and corrections
#
# Q and K fixed, V_t = (1 + c_t) V_0.  No LSE moves, so every anchor weight
# stays w_j (step 0's), every partition and group output is (1 + c_t) times
# its step-0 value, and with A_G = sum_{j in G} w_j ||OUT_0(j)|| and
# B_G = w(G) ||OUT_0(G)||, w(G) = sum_{j in G} w_j:
#   ASE_t(G)        = |c_t - c_{t_c(G)}| A_G           (local snapshot at t_c)
#   relative drift  = |c_t - c_{t_a}| / (1 + c_{t_a})
#   correction(G)   = |c_t - c_{t_c(G)}| B_G           (at an anchor t)
#   measured error  = |c_t - c_{t_c(G)}| B_G           (any step t > t_a)
#   composed LSE    = the full-attention LSE at every step.
# The step-0 quantities come from torch's float64 attention and scipy's
# logsumexp over each partition's and group's key range, not from the oracle.

def _truth_by_key_range(x, offs, q, scale):
    torch = pytest.importorskip("torch")
    from scipy.special import logsumexp
    Q = x["q"][:, offs[q]:offs[q + 1]]

    def out(a, e):
        t = lambda y: torch.from_numpy(np.ascontiguousarray(y)).permute(0, 2, 1, 3)
        o = torch.nn.functional.scaled_dot_product_attention(t(Q), t(x["k"][:, a:e]), t(x["v"][:, a:e]), scale=scale)
        return o.permute(0, 2, 1, 3).numpy()

    def lse(a, e):
        return logsumexp(scale * np.einsum("brhd,bchd->bhrc", Q, x["k"][:, a:e]), axis=-1)

    return out, lse


def test_error_planner_eps_adaptation_over_several_anchors():
    S, P, q, scale, g, R, eps_local = 40, 8, 3, 0.35, 2, 0.5, 0.1
    offs = partition_offsets(S, P)
    x0 = seq(7)
    c = [0.0, 0.05, 0.08, 0.3, 0.32, 0.6, 0.62]
    xs = [dict(x0, v=x0["v"] * (1.0 + ct)) for ct in c]
    res = ase_planner.run(xs, offs, q, g, R, eps_local, scale, evaluate=True)

    out_of, lse_of = _truth_by_key_range(x0, offs, q, scale)
    lse_full = lse_of(0, S)
    w = [float(np.mean(np.exp(lse_of(offs[j], offs[j + 1]) - lse_full))) for j in range(P)]
    n_part = [float(np.linalg.norm(out_of(offs[j], offs[j + 1]))) for j in range(P)]
    groups = og.groups_of(P, q, g)
    assert groups == [(0, 2), (2, 3), (4, 6), (6, 8)]
    A = {G: sum(w[j] * n_part[j] for j in range(*G)) for G in groups}
    Bc = {G: sum(w[j] for j in range(*G)) * float(np.linalg.norm(out_of(offs[G[0]], offs[G[1]]))) for G in groups}

    # the rule, followed on the closed forms: eps from step 1's ASE until
    # the first correction errors exist, then their R-quantile
    # (sorted[ceil(R m) - 1]) over every anchor so far
    quant = lambda v: sorted(v)[int(math.ceil(R * len(v))) - 1]
    t_c, t_a, eps, corr = {G: 0 for G in groups}, 0, None, []
    anchors = []
    for t in range(1, len(c)):
        r = res[t]
        ase = {G: abs(c[t] - c[t_c[G]]) * A[G] for G in groups}
        # the error each cached group state actually carries (evaluation)
        for G in groups:
            assert r["measured"][G] == pytest.approx(abs(c[t] - c[t_c[G]]) * Bc[G], rel=1e-9, abs=1e-15), (t, G)
        drift = abs(c[t] - c[t_a]) / (1.0 + c[t_a])
        assert r["drift"] == pytest.approx(drift, rel=1e-9, abs=1e-15)
        for G in groups:
            assert r["ase"][G] == pytest.approx(ase[G], rel=1e-9, abs=1e-15), (t, G)
        if eps is None:
            eps = quant(list(ase.values()))
        anchor = all(v > eps for v in ase.values()) or drift > eps_local
        assert r["anchor"] == anchor, t
        if anchor:
            corr += [abs(c[t] - c[t_c[G]]) * Bc[G] for G in groups]
            eps = quant(corr)
            t_c, t_a = {G: t for G in groups}, t
            anchors.append(t)
        else:
            comp = [G for G in groups if ase[G] > eps]
            assert r["compute"] == comp, t
            for G in comp:
                t_c[G] = t
        assert r["eps"] == pytest.approx(eps, rel=1e-9), t
        assert r["t_c"] == t_c, t
        np.testing.assert_allclose(r["corrections"], corr, rtol=1e-9)
        # no LSE moved: the composed LSE is full attention's at every step
        np.testing.assert_allclose(r["lse"], lse_full, rtol=1e-12)

    # the schedule reaches every branch: groups recomputed between anchors
    # (three different snapshot steps at the second anchor), two anchors
    # after the first, and a quantile over the corrections of both
    assert anchors == [3, 5]
    assert sorted(set(res[2]["t_c"].values())) == [0, 1, 2]
    assert len(res[5]["corrections"]) == 8 and len(res[4]["corrections"]) == 4
    assert res[5]["eps"] == pytest.approx(sorted(res[5]["corrections"])[3], rel=0)


def test_error_planner_measured_errors_by_key_range_on_changing_tensors():
    """Tensors that change at every step (LSEs and weights move): the
    measured error of a group, w(G, t) ||AS_t(G) - AS_tc(G)||, recomputed
    from torch's float64 attention over the group's key range at steps t and
    t_c (a group's composed state is attention over the union of its keys)
    and scipy's logsumexp for the current weight."""
    from scipy.special import logsumexp
    torch = pytest.importorskip("torch")
    S, P, q, scale, g = 48, 8, 3, 0.35, 2
    offs = partition_offsets(S, P)
    xs = [seq(30 + s, S=S) for s in range(5)]
    res = ase_planner.run(xs, offs, q, g, 0.5, 10.0, scale, evaluate=True)
    groups = og.groups_of(P, q, g)

    def attn(x, a, e):
        t = lambda y: torch.from_numpy(np.ascontiguousarray(y)).permute(0, 2, 1, 3)
        Q = x["q"][:, offs[q]:offs[q + 1]]
        o = torch.nn.functional.scaled_dot_product_attention(t(Q), t(x["k"][:, a:e]), t(x["v"][:, a:e]), scale=scale)
        return o.permute(0, 2, 1, 3).numpy()

    def lse(x, a, e):
        Q = x["q"][:, offs[q]:offs[q + 1]]
        return logsumexp(scale * np.einsum("brhd,bchd->bhrc", Q, x["k"][:, a:e]), axis=-1)

    checked = 0
    for t in range(1, len(xs)):
        r = res[t]
        t_c = res[t - 1]["t_c"]                 # before this step's recomputation
        assert r["measured"] is not None
        for G in groups:
            a, e = offs[G[0]], offs[G[1]]
            w = float(np.mean(np.exp(lse(xs[t], a, e) - lse(xs[t], 0, S))))
            expect = w * float(np.linalg.norm(attn(xs[t], a, e) - attn(xs[t_c[G]], a, e)))
            assert r["measured"][G] == pytest.approx(expect, rel=1e-9), (t, G)
            checked += 1
    assert res[0]["measured"] is None and checked == 4 * len(groups)
    # groups were recomputed between steps, so several cache ages were seen
    assert len({tc for t in range(len(xs)) for tc in res[t]["t_c"].values()}) > 2
