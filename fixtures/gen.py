"""Seeded tensor generation for the synthetic workloads.

Recipe (all draws with numpy's PCG64 ``default_rng``):

* ``Zq, Zk, Zv = rng.standard_normal((B, S, H, D), float32)`` in that order from
  ``default_rng(seed)``, then the previous-step noise ``Nq, Nk, Nv`` likewise.
* A smooth positional component shared by Q, K and V and by all heads,
  ``pos[t,h,w,d] = 0.5*sin(wt[d]*t + wh[d]*h + ww[d]*w + phi[d])`` with
  ``w_a[d] = 2*pi*g_a[d]/N_a``, ``g_a ~ U(0,2)`` cycles across axis ``a`` of
  extent N_a, ``phi ~ U(0, 2*pi)``, drawn in float64 from
  ``default_rng(seed + 1000)``.  Because Q and K share it, q.k is largest for
  nearby tokens, so nearer partitions carry more attention weight, the
  distance-decaying contribution the paper observes in Fig. 2 and Fig. 5.
* ``X = Z + pos`` in float32; the previous step is ``X + sigma*N``.
* Multi-step workloads evolve a float32 master copy:
  ``X_{s+1} = X_s + sigma*N(0,1)`` with the noise from ``default_rng([seed, s])``.
* bf16 inputs are the round-to-nearest-even bf16 values of the float32 arrays;
  both the kernels and the oracle see exactly those values.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

from .workloads import Workload


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of float32 ``x`` rounded to bf16, round-to-nearest-even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    nan = np.isnan(x)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    r = r.astype(np.uint16)
    if nan.any():
        r[nan] = np.uint16(0x7FC0)
    return r


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 array holding the bf16-rounded values of ``x`` (exactly representable)."""
    return (bf16_bits(x).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _positional(w: Workload) -> np.ndarray:
    T, Hg, W = w.grid
    rng = np.random.default_rng(w.seed + 1000)
    D = w.D
    g = rng.uniform(0.0, 2.0, size=(3, D))
    phi = rng.uniform(0.0, 2.0 * np.pi, size=D)
    om_t = 2.0 * np.pi * g[0] / T
    om_h = 2.0 * np.pi * g[1] / Hg
    om_w = 2.0 * np.pi * g[2] / W
    t = np.arange(T, dtype=np.float64)[:, None, None, None]
    h = np.arange(Hg, dtype=np.float64)[None, :, None, None]
    x = np.arange(W, dtype=np.float64)[None, None, :, None]
    ang = om_t * t + om_h * h + om_w * x + phi
    pos = 0.5 * np.sin(ang)                      # [T, Hg, W, D]
    return pos.reshape(T * Hg * W, 1, D).astype(np.float32)   # [S, 1(head), D]


def gen_qkv(w: Workload, with_prev: Optional[bool] = None) -> Dict[str, np.ndarray]:
    """Current-step (and optionally previous-step) float32 Q, K, V of shape [B, S, H, D].

    Returns keys ``q, k, v`` and, when a previous step is requested (default:
    when the workload reuses states, ``prev_noise > 0``), ``q_prev, k_prev,
    v_prev``.  Values are float32; callers round to bf16 with ``bf16_round``
    for bf16 workloads.
    """
    if with_prev is None:
        with_prev = w.prev_noise > 0.0
    shape = (w.B, w.S, w.H, w.D)
    rng = np.random.default_rng(w.seed)
    pos = _positional(w)
    out: Dict[str, np.ndarray] = {}
    for name in ("q", "k", "v"):
        z = rng.standard_normal(shape, dtype=np.float32)
        z += pos[None]
        out[name] = z
    if with_prev:
        sig = np.float32(w.prev_noise)
        for name in ("q", "k", "v"):
            n = rng.standard_normal(shape, dtype=np.float32)
            n *= sig
            n += out[name]
            out[name + "_prev"] = n
    return out


def gen_evolved(w: Workload, x: Dict[str, np.ndarray], s: int) -> Dict[str, np.ndarray]:
    """Step s+1 of a multi-step workload from step s: ``X + step_noise*N(0,1)``."""
    rng = np.random.default_rng([w.seed, s])
    sig = np.float32(w.step_noise)
    out = {}
    for name in ("q", "k", "v"):
        n = rng.standard_normal(x[name].shape, dtype=np.float32)
        n *= sig
        n += x[name]
        out[name] = n
    return out


def sample_rows(q_len: int, n: int, seed: int, tile: int = 128) -> np.ndarray:
    """Sorted seeded sample of query rows for row-sampled parity checks.

    Always includes the tile-boundary rows 0, 1, 63, 64, 127, 128, q_len-1 and
    every row of the last partial ``tile``-row tile.
    """
    must = {0, 1, 63, 64, 127, 128, q_len - 1}
    last_full = (q_len // tile) * tile
    must.update(range(last_full, q_len))
    must = {r for r in must if 0 <= r < q_len}
    rng = np.random.default_rng(seed + 7)
    k = max(0, min(n, q_len) - len(must))
    pool = np.setdiff1d(np.arange(q_len), np.fromiter(must, dtype=np.int64))
    extra = rng.choice(pool, size=min(k, pool.size), replace=False) if k else np.array([], np.int64)
    return np.unique(np.concatenate([np.fromiter(must, dtype=np.int64), extra.astype(np.int64)]))


def query_block(x: np.ndarray, offsets: Sequence[int], q: int) -> np.ndarray:
    """Rows [o_q, o_{q+1}) of a [B, S, H, D] tensor: the rank's query block."""
    return x[:, offsets[q]:offsets[q + 1]]
