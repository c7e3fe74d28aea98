"""Group bookkeeping of the product (CPU): base groups and compose runs
against the oracle's independent statement of the same rules."""
from oracle import groups as og
from paper_2607_15650_amd import groups as pg


def test_base_groups_match_oracle():
    for P in range(1, 17):
        for q in range(P):
            for g in (1, 2, 3, 4, 8):
                assert pg.base_groups(P, q, g) == og.groups_of(P, q, g), (P, q, g)


def test_compose_runs_match_oracle_and_never_cross_the_local_partition():
    for P in (4, 8, 16):
        for q in range(P):
            for g in (1, 2, 4):
                groups = pg.base_groups(P, q, g)
                for k in (2, 3):
                    runs = pg.compose_pairs(groups, q, k)
                    assert runs == og.compose_runs(groups, k)
                    for r in runs:
                        assert len(r) <= k
                        assert not (r[0][0] <= q < r[-1][1])
                        for a, b in zip(r, r[1:]):
                            assert a[1] == b[0]


def test_local_group_has_one_member_fewer():
    # Sec. 4.2.1: the group holding the local partition has g-1 members
    assert pg.base_groups(8, 3, 2) == [(0, 2), (2, 3), (4, 6), (6, 8)]
    assert pg.base_groups(8, 5, 4) == [(0, 4), (4, 5), (6, 8)]
