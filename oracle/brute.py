"""Pure-Python brute force of the attention state, composition and weights.

Test infrastructure only.  Triple loops with ``math.exp`` and ``math.log``,
straight from the definitions of Sec. 2.2.4 (Eq. attention_state and
Eq. composition) without any max-shift, so only tiny, well-scaled inputs are
meaningful.  Inputs are nested lists or arrays indexed [b][row][h][d].
"""
from __future__ import annotations

import math


def state(q, k, v, scale):
    """Returns (out[b][r][h][d], lse[b][h][r]) for keys k, values v."""
    B, Lq, H, D = len(q), len(q[0]), len(q[0][0]), len(q[0][0][0])
    L = len(k[0])
    out = [[[[0.0] * D for _ in range(H)] for _ in range(Lq)] for _ in range(B)]
    lse = [[[float("-inf")] * Lq for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for h in range(H):
            for r in range(Lq):
                ex = []
                for c in range(L):
                    dot = 0.0
                    for d in range(D):
                        dot += float(q[b][r][h][d]) * float(k[b][c][h][d])
                    ex.append(math.exp(scale * dot))
                z = sum(ex)
                if L == 0:
                    continue
                lse[b][h][r] = math.log(z)
                for d in range(D):
                    acc = 0.0
                    for c in range(L):
                        acc += ex[c] / z * float(v[b][c][h][d])
                    out[b][r][h][d] = acc
    return out, lse


def compose(states):
    """Composition of a list of (out, lse) states by Eq. composition, unshifted."""
    B = len(states[0][0])
    Lq = len(states[0][0][0])
    H = len(states[0][0][0][0])
    D = len(states[0][0][0][0][0])
    out = [[[[0.0] * D for _ in range(H)] for _ in range(Lq)] for _ in range(B)]
    lse = [[[0.0] * Lq for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for h in range(H):
            for r in range(Lq):
                es = [math.exp(s[1][b][h][r]) for s in states]
                z = sum(es)
                lse[b][h][r] = math.log(z)
                for d in range(D):
                    out[b][r][h][d] = sum(e * s[0][b][r][h][d] for e, s in zip(es, states)) / z
    return out, lse


def weights(lses, b, h, r):
    """w_i = e^{LSE_i} / sum_k e^{LSE_k} for one row (Sec. 4.1.1)."""
    es = [math.exp(l[b][h][r]) for l in lses]
    z = sum(es)
    return [e / z for e in es]
