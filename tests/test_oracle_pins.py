"""Pins of the float64 oracle against things other than itself.

Each test states what fixes the expected value: the pure-Python brute force
of the definitions, a library routine (torch's scaled-dot-product attention,
scipy's logsumexp), a closed form, an invariant of the composition (Sec. 2.2.4,
Eq. composition: associative and commutative), or the paper's first-order
error analysis (Sec. 4.1.1, Eq. error_composition and Eq. error_bound).
"""
import itertools
import math

import numpy as np
import pytest

import oracle
from oracle import brute
from fixtures import workloads as wl

RTOL = 1e-12


def rnd(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def tiny(seed=0, B=1, Lq=3, S=8, H=2, D=4):
    q = rnd((B, Lq, H, D), seed)
    k = rnd((B, S, H, D), seed + 1)
    v = rnd((B, S, H, D), seed + 2)
    return q, k, v


# ---------------------------------------------------------------- brute force

@pytest.mark.parametrize("P", [1, 2, 4])
def test_partition_states_match_brute_force(P):
    q, k, v = tiny(seed=P)
    S = k.shape[1]
    offs = wl.partition_offsets(S, P)
    scale = 1 / math.sqrt(q.shape[-1])
    outs, lses = oracle.partition_states(q, k, v, offs, scale)
    for j in range(P):
        a, e = offs[j], offs[j + 1]
        bo, bl = brute.state(q.tolist(), k[:, a:e].tolist(), v[:, a:e].tolist(), scale)
        np.testing.assert_allclose(outs[j], np.array(bo), rtol=RTOL, atol=1e-13)
        np.testing.assert_allclose(lses[j], np.array(bl), rtol=RTOL, atol=1e-13)
    # composed state vs brute composition
    out, lse = oracle.merge(outs, lses)
    bo, bl = brute.compose([(np.array(o).tolist(), np.array(l).tolist()) for o, l in zip(outs, lses)])
    np.testing.assert_allclose(out, np.array(bo), rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(lse, np.array(bl), rtol=1e-12, atol=1e-13)
    # weights vs brute weights
    W, wbar = oracle.contrib(lses, lse)
    for b, h, r in itertools.product(range(q.shape[0]), range(q.shape[2]), range(q.shape[1])):
        np.testing.assert_allclose(W[b, h, r], brute.weights([l.tolist() for l in lses], b, h, r), rtol=1e-11)


# ---------------------------------------------------------------- library routines

def test_full_attention_matches_torch_sdpa_float64():
    torch = pytest.importorskip("torch")
    q, k, v = tiny(seed=11, B=2, Lq=5, S=37, H=3, D=8)
    scale = 0.3
    out, lse = oracle.full_attention(q, k, v, scale)
    tq = torch.from_numpy(q).permute(0, 2, 1, 3)     # [B,H,L,D]
    tk = torch.from_numpy(k).permute(0, 2, 1, 3)
    tv = torch.from_numpy(v).permute(0, 2, 1, 3)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale)
    np.testing.assert_allclose(out, ref.permute(0, 2, 1, 3).numpy(), rtol=1e-12, atol=1e-13)


def test_lse_matches_scipy_logsumexp():
    from scipy.special import logsumexp
    q, k, v = tiny(seed=12, B=1, Lq=4, S=50, H=2, D=6)
    scale = 0.7
    _, lse = oracle.full_attention(q, k, v, scale)
    for h in range(2):
        sc = scale * np.einsum("rd,cd->rc", q[0, :, h], k[0, :, h])
        np.testing.assert_allclose(lse[0, h], logsumexp(sc, axis=1), rtol=1e-13)


# ---------------------------------------------------------------- composition invariants

@pytest.mark.parametrize("P", [2, 3, 5, 8])
def test_merge_of_all_fresh_partitions_equals_full_attention(P):
    q, k, v = tiny(seed=20 + P, B=2, Lq=6, S=41, H=2, D=8)
    offs = wl.partition_offsets(41, P)
    outs, lses = oracle.partition_states(q, k, v, offs, 0.35)
    out, lse = oracle.merge(outs, lses)
    fo, fl = oracle.full_attention(q, k, v, 0.35)
    np.testing.assert_allclose(out, fo, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, fl, rtol=1e-13)


def test_merge_is_order_and_tree_independent():
    q, k, v = tiny(seed=31, B=1, Lq=7, S=64, H=2, D=8)
    offs = wl.partition_offsets(64, 8)
    outs, lses = oracle.partition_states(q, k, v, offs, 0.4)
    ref_o, ref_l = oracle.merge(outs, lses)
    rng = np.random.default_rng(5)
    for _ in range(6):
        perm = rng.permutation(8)
        o, l = oracle.merge([outs[i] for i in perm], [lses[i] for i in perm])
        np.testing.assert_allclose(o, ref_o, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(l, ref_l, rtol=1e-13)
        # random binary tree of compose2
        items = [(outs[i], lses[i]) for i in perm]
        while len(items) > 1:
            i = int(rng.integers(0, len(items) - 1))
            a, b = items[i], items[i + 1]
            items[i:i + 2] = [oracle.compose2(a[0], a[1], b[0], b[1])]
        np.testing.assert_allclose(items[0][0], ref_o, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(items[0][1], ref_l, rtol=1e-13)


def test_composed_cached_group_is_a_valid_reuse_unit():
    """Sec. 2.2.4 / Fig. 4: rank 0 of CP=4 computes partitions 0 and 1 fresh and
    reuses the cached composition of 2 and 3; with an unchanged cache the
    result equals all-fresh attention."""
    q, k, v = tiny(seed=41, B=1, Lq=5, S=32, H=2, D=8)
    offs = wl.partition_offsets(32, 4)
    outs, lses = oracle.partition_states(q, k, v, offs, 0.5)
    g23 = oracle.compose2(outs[2], lses[2], outs[3], lses[3])
    o, l = oracle.merge([outs[0], outs[1], g23[0]], [lses[0], lses[1], g23[1]])
    fo, fl = oracle.full_attention(q, k, v, 0.5)
    np.testing.assert_allclose(o, fo, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l, fl, rtol=1e-13)


def test_reuse_with_unchanged_cache_equals_fresh():
    """Non-contiguous selection {0,2,3,4,5} fresh, {1,6,7} reused (Sec. 5.2 example)."""
    q, k, v = tiny(seed=51, B=1, Lq=4, S=80, H=2, D=8)
    offs = wl.partition_offsets(80, 8)
    sel = [1, 0, 1, 1, 1, 1, 0, 0]
    o, l, _, _ = oracle.selective_step(q, k, v, q, k, v, offs, sel, 0.45)
    fo, fl, _, _ = oracle.selective_step(q, k, v, q, k, v, offs, [1] * 8, 0.45)
    assert np.array_equal(o, fo) and np.array_equal(l, fl)
    # and a changed cache really changes the reused partitions
    o2, _, _, _ = oracle.selective_step(q, k, v, q, k + 0.1, v + 0.1, offs, sel, 0.45)
    assert np.abs(o2 - o).max() > 1e-4


# ---------------------------------------------------------------- closed forms / special cases

def test_zero_query_gives_mean_of_values_and_log_length():
    _, k, v = tiny(seed=61, B=1, Lq=1, S=13, H=2, D=4)
    q = np.zeros((1, 3, 2, 4))
    out, lse = oracle.partition_state(q, k, v, 0.9)
    np.testing.assert_allclose(out, np.broadcast_to(v.mean(axis=1, keepdims=True), out.shape), rtol=1e-13)
    np.testing.assert_allclose(lse, np.log(13.0), rtol=1e-15)


def test_single_key_state():
    q, k, v = tiny(seed=62, B=1, Lq=3, S=1, H=2, D=4)
    out, lse = oracle.partition_state(q, k, v, 0.25)
    np.testing.assert_allclose(out, np.broadcast_to(v, out.shape), rtol=1e-15)
    np.testing.assert_allclose(lse, 0.25 * np.einsum("brhd,bchd->bhr", q, k), rtol=1e-15)


def test_two_key_worked_example():
    """q=(1,0), keys (1,0),(0,1), values e1,e2, scale 1: LSE = log(e+1),
    OUT = (e/(e+1), 1/(e+1)); composing the two single-key states gives the same."""
    q = np.array([[[[1.0, 0.0]]]])
    k = np.array([[[[1.0, 0.0]], [[0.0, 1.0]]]])
    v = np.array([[[[1.0, 0.0]], [[0.0, 1.0]]]])
    out, lse = oracle.partition_state(q, k, v, 1.0)
    e = math.e
    assert abs(lse[0, 0, 0] - math.log(e + 1)) < 1e-15
    np.testing.assert_allclose(out[0, 0, 0], [e / (e + 1), 1 / (e + 1)], rtol=1e-15)
    s1 = oracle.partition_state(q, k[:, :1], v[:, :1], 1.0)
    s2 = oracle.partition_state(q, k[:, 1:], v[:, 1:], 1.0)
    assert abs(s1[1][0, 0, 0] - 1.0) < 1e-15 and abs(s2[1][0, 0, 0]) < 1e-15
    o, l = oracle.compose2(s1[0], s1[1], s2[0], s2[1])
    np.testing.assert_allclose(o, out, rtol=1e-15)
    np.testing.assert_allclose(l, lse, rtol=1e-15)


def test_empty_partition_is_neutral():
    q, k, v = tiny(seed=63, B=1, Lq=4, S=9, H=2, D=4)
    out_e, lse_e = oracle.partition_state(q, k[:, :0], v[:, :0], 0.5)
    assert np.all(np.isneginf(lse_e)) and np.all(out_e == 0)
    o, l = oracle.partition_state(q, k, v, 0.5)
    mo, ml = oracle.merge([o, out_e], [l, lse_e])
    np.testing.assert_allclose(mo, o, rtol=1e-15)
    np.testing.assert_allclose(ml, l, rtol=1e-15)
    W, wbar = oracle.contrib([l, lse_e], ml)
    assert np.all(W[..., 1] == 0) and wbar[1] == 0 and not np.isnan(W).any()
    # all partitions empty: OUT 0, LSE -inf, no NaN
    zo, zl = oracle.merge([out_e, out_e], [lse_e, lse_e])
    assert np.all(zo == 0) and np.all(np.isneginf(zl))
    W, wbar = oracle.contrib([lse_e, lse_e], zl)
    assert not np.isnan(W).any() and np.all(wbar == 0)


def test_uneven_offsets_last_partition_shorter_and_empty():
    assert wl.partition_offsets(75600, 8) == [j * 9450 for j in range(9)]
    assert wl.partition_offsets(10, 4) == [0, 3, 6, 9, 10]
    assert wl.partition_offsets(9, 4) == [0, 3, 6, 9, 9]   # last partition empty
    q, k, v = tiny(seed=64, B=1, Lq=3, S=9, H=2, D=4)
    offs = wl.partition_offsets(9, 4)
    outs, lses = oracle.partition_states(q, k, v, offs, 0.5)
    o, l = oracle.merge(outs, lses)
    fo, fl = oracle.full_attention(q, k, v, 0.5)
    np.testing.assert_allclose(o, fo, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(l, fl, rtol=1e-13)


# ---------------------------------------------------------------- weights

def test_weights_sum_to_one_and_special_values():
    q, k, v = tiny(seed=71, B=2, Lq=6, S=40, H=3, D=8)
    offs = wl.partition_offsets(40, 5)
    outs, lses = oracle.partition_states(q, k, v, offs, 0.5)
    _, lse = oracle.merge(outs, lses)
    W, wbar = oracle.contrib(lses, lse)
    np.testing.assert_allclose(W.sum(-1), 1.0, rtol=1e-13)
    assert abs(wbar.sum() - 1.0) < 1e-13
    # P = 1 -> weight 1
    W1, wb1 = oracle.contrib([lse], lse)
    assert np.all(W1 == 1.0) and wb1[0] == 1.0
    # equal LSE -> 1/n
    eq = [lses[0]] * 4
    _, l4 = oracle.merge([outs[0]] * 4, eq)
    W4, wb4 = oracle.contrib(eq, l4)
    np.testing.assert_allclose(W4, 0.25, rtol=1e-14)


def test_rank_and_threshold_plan():
    wbar = [0.01, 0.2, 0.3, 0.2, 0.05, 0.24]
    # ties (0.2 at 1 and 3) broken by distance to q=2, then index
    assert oracle.rank_partitions(wbar, 2) == [2, 5, 1, 3, 4, 0]
    assert oracle.rank_partitions(wbar, 4) == [2, 5, 3, 1, 4, 0]
    # strict '>' and the query partition always computed
    assert oracle.plan_threshold(wbar, 0, 0.05) == [1, 1, 1, 1, 0, 1]
    assert oracle.plan_threshold(wbar, 4, 0.2) == [0, 0, 1, 0, 1, 1]


# ---------------------------------------------------------------- error propagation (Sec. 4.1.1)

def _random_states(n, seed, R=5, D=6):
    rng = np.random.default_rng(seed)
    outs = [rng.standard_normal((1, R, 1, D)) for _ in range(n)]
    lses = [rng.standard_normal((1, 1, R)) * 2.0 for _ in range(n)]
    return outs, lses


def test_error_composition_first_order():
    """Eq. error_composition: perturbing (OUT_i, LSE_i) by eps moves the composed
    state by w1 dO1 + w2 dO2 + w1 w2 (O1 - O2)(dL1 - dL2) and w1 dL1 + w2 dL2,
    up to O(eps^2)."""
    outs, lses = _random_states(2, 81)
    rng = np.random.default_rng(82)
    dO = [rng.standard_normal(o.shape) for o in outs]
    dL = [rng.standard_normal(l.shape) for l in lses]
    o0, l0 = oracle.compose2(outs[0], lses[0], outs[1], lses[1])
    w1 = np.exp(lses[0] - l0)
    w2 = np.exp(lses[1] - l0)
    tw = lambda w: np.transpose(w, (0, 2, 1))[..., None]   # [B,H,R] -> [B,R,H,1]
    pred_dO = (tw(w1) * dO[0] + tw(w2) * dO[1]
               + tw(w1 * w2) * (outs[0] - outs[1]) * tw(dL[0] - dL[1]))
    pred_dL = w1 * dL[0] + w2 * dL[1]
    for eps in (1e-4, 1e-5):
        o, l = oracle.compose2(outs[0] + eps * dO[0], lses[0] + eps * dL[0],
                               outs[1] + eps * dO[1], lses[1] + eps * dL[1])
        res_o = np.abs((o - o0) - eps * pred_dO).max()
        res_l = np.abs((l - l0) - eps * pred_dL).max()
        assert res_o < 50 * eps ** 2 and res_l < 50 * eps ** 2, (eps, res_o, res_l)
    # the first-order term itself is not negligible (the test has teeth)
    assert np.abs(pred_dO).max() > 0.1


def test_error_bound_holds_for_n_partitions():
    """Eq. error_bound: ||dOUT|| <= sum w_i ||dO_i|| + sum_{i<j} w_i w_j ||O_i - O_j|| |dL_i - dL_j|
    for small perturbations of n = 6 states (first order, so a tiny O(eps^2) slack)."""
    n = 6
    outs, lses = _random_states(n, 91)
    rng = np.random.default_rng(92)
    o0, l0 = oracle.merge(outs, lses)
    W, _ = oracle.contrib(lses, l0)               # [1,1,R,n]
    eps = 1e-6
    for _ in range(20):
        dO = [rng.standard_normal(o.shape) for o in outs]
        dL = [rng.standard_normal(l.shape) for l in lses]
        o, _ = oracle.merge([x + eps * d for x, d in zip(outs, dO)],
                            [x + eps * d for x, d in zip(lses, dL)])
        lhs = np.linalg.norm((o - o0)[0, :, 0, :], axis=-1)            # per row
        rhs = np.zeros_like(lhs)
        for i in range(n):
            rhs += W[0, 0, :, i] * np.linalg.norm(eps * dO[i][0, :, 0, :], axis=-1)
            for j in range(i + 1, n):
                rhs += (W[0, 0, :, i] * W[0, 0, :, j]
                        * np.linalg.norm((outs[i] - outs[j])[0, :, 0, :], axis=-1)
                        * np.abs(eps * (dL[i] - dL[j])[0, 0]))
        assert np.all(lhs <= rhs * (1 + 1e-5) + 1e-15)
