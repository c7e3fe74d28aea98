"""Host planner (product) against the oracle's selection rule, and the
anchor sequencing of the planner-driven workload.  CPU only."""
import numpy as np

import oracle
from paper_2607_15650_amd import planner


def test_plan_and_rank_match_oracle_on_random_weights():
    rng = np.random.default_rng(0)
    for trial in range(500):
        P = int(rng.integers(1, 17))
        q = int(rng.integers(0, P))
        w = rng.dirichlet(np.ones(P))
        if trial % 3 == 0:                       # plant exact ties and threshold hits
            w[rng.integers(0, P)] = 0.05
            w = np.round(w, 2)
        thr = float(rng.choice([0.0, 0.05, 0.1, 0.3]))
        assert planner.plan_threshold(w, q, thr) == oracle.plan_threshold(w, q, thr)
        assert planner.rank_partitions(w, q) == oracle.rank_partitions(w, q)


def test_anchor_planner_sequence():
    p = planner.AnchorPlanner(P=8, q=3, anchors=(0, 5), threshold=0.05)
    assert p.select(0) == [1] * 8
    w = [0.01, 0.02, 0.3, 0.4, 0.2, 0.04, 0.051, 0.0]
    p.observe(0, w)
    assert p.select(1) == [0, 0, 1, 1, 1, 0, 1, 0]
    p.observe(1, [1.0] * 8)                      # non-anchor observations are ignored
    assert p.select(2) == [0, 0, 1, 1, 1, 0, 1, 0]
    assert p.select(5) == [1] * 8
    p.observe(5, [0.0] * 8)
    assert p.select(6) == [0, 0, 0, 1, 0, 0, 0, 0]   # the query partition is always computed


def test_oracle_multistep_reuse_semantics_tiny():
    """Unchanged tensors across steps: every step equals full attention, and
    the anchor-then-threshold masks are what the rule says."""
    from fixtures.workloads import partition_offsets
    rng = np.random.default_rng(1)
    S, P, H, D = 48, 4, 2, 8
    x = {k: rng.standard_normal((1, S, H, D)) for k in ("q", "k", "v")}
    offs = partition_offsets(S, P)
    from oracle import multistep
    res = multistep.run([x, x, x], offs, [0, 2], anchors=(0,), threshold=0.3, scale=0.4)
    for s in range(3):
        for qb in (0, 2):
            mask, out, lse, wbar = res[s][qb]
            fo, fl = oracle.full_attention(x["q"][:, offs[qb]:offs[qb + 1]], x["k"], x["v"], 0.4)
            np.testing.assert_allclose(out, fo, rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(lse, fl, rtol=1e-13)
            if s == 0:
                assert mask == [1] * P
            else:
                assert mask == oracle.plan_threshold(res[0][qb][3], qb, 0.3)


def test_quantile_rule_matches_oracle():
    from paper_2607_15650_amd.ase import quantile_r
    from oracle.ase_planner import r_quantile
    rng = np.random.default_rng(3)
    for _ in range(300):
        v = list(rng.random(int(rng.integers(1, 20))))
        r = float(rng.random())
        assert quantile_r(v, r) == r_quantile(v, r)
    assert quantile_r([3.0, 1.0, 2.0, 4.0], 0.5) == 2.0
    assert quantile_r([3.0, 1.0, 2.0, 4.0], 0.75) == 3.0
    assert quantile_r([3.0], 0.1) == 3.0


def test_product_rank_hand_examples():
    # decreasing weight; equal weights by distance to q, then by index
    assert planner.rank_partitions([0.1, 0.3, 0.3, 0.2, 0.1], 2) == [2, 1, 3, 0, 4]
    assert planner.rank_partitions([0.25] * 4, 1) == [1, 0, 2, 3]
    assert planner.rank_partitions([0.5, 0.0, 0.5], 2) == [2, 0, 1]
    assert planner.rank_partitions([0.0, 0.1, 0.2, 0.3, 0.4], 0) == [4, 3, 2, 1, 0]
    assert planner.rank_partitions([0.7], 0) == [0]


def test_product_threshold_hand_examples():
    # strictly above the threshold, and the query partition always
    assert planner.plan_threshold([0.05, 0.050001, 0.2, 0.0], 3, 0.05) == [0, 1, 1, 1]
    assert planner.plan_threshold([0.05, 0.050001, 0.2, 0.0], 3, 0.3) == [0, 0, 0, 1]
    assert planner.plan_threshold([0.4, 0.3, 0.3], 0, 0.0) == [1, 1, 1]
    assert planner.plan_threshold([0.0, 0.0, 0.0], 1, 0.0) == [0, 1, 0]


def test_product_quantile_hand_examples():
    from paper_2607_15650_amd.ase import quantile_r
    v = [4.0, 1.0, 3.0, 2.0]
    assert quantile_r(v, 0.0) == 1.0          # the smallest
    assert quantile_r(v, 0.25) == 1.0         # ceil(1) = 1st
    assert quantile_r(v, 0.26) == 2.0         # ceil(1.04) = 2nd
    assert quantile_r(v, 0.5) == 2.0
    assert quantile_r(v, 0.51) == 3.0
    assert quantile_r(v, 1.0) == 4.0
    assert quantile_r([0.3, 0.1, 0.2, 0.9, 0.5, 0.7, 0.8, 0.6], 0.5) == 0.5   # 4th of 8


def test_accuracy_stats_hand_examples():
    from paper_2607_15650_amd.ase import accuracy_stats
    st = accuracy_stats([1.0, 2.0, 3.0], [1.0, 2.0, 3.0])
    assert st["r2"] == 1.0 and abs(st["pearson"] - 1.0) < 1e-15 and st["rmse"] == 0.0 and st["mae"] == 0.0
    # prediction off by a constant 1: r = 1, R^2 = 1 - 3/2, RMSE = MAE = 1
    st = accuracy_stats([2.0, 3.0, 4.0], [1.0, 2.0, 3.0])
    assert abs(st["pearson"] - 1.0) < 1e-15 and st["r2"] == -0.5 and st["rmse"] == 1.0 and st["mae"] == 1.0
    # anti-correlated: r = -1
    st = accuracy_stats([3.0, 2.0, 1.0], [1.0, 2.0, 3.0])
    assert abs(st["pearson"] + 1.0) < 1e-15 and st["r2"] == 1.0 - 8.0 / 2.0
    st = accuracy_stats([0.0, 1.0], [1.0, 0.0])
    assert st["n"] == 2 and st["mae"] == 1.0
