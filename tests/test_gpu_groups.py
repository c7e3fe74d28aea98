"""GPU parity of group states and Dynamic Group State Compose on the reduced
planner workload (2 heads, 16,384 tokens, 8 partitions, groups of 2, at most
3 cached group states, anchors at steps 0 and 5): groups, compute decisions,
composed outputs, LSE and group weights against the float64 oracle."""
import numpy as np
import pytest

from oracle import groups as og
from fixtures import gen_qkv, gen_evolved, get_workload

from helpers import TOL, exact_inputs, max_abs, to_gpu

pytestmark = pytest.mark.gpu

G, K, MAX_STATES, THR = 2, 2, 3, 0.25


def test_group_states_and_compose():
    import torch
    from paper_2607_15650_amd.groups import GroupedSelectiveAttention

    w = get_workload("planner_bf16_h2_d128_s16384_p8_10steps")
    x = gen_qkv(w, with_prev=False)
    steps = [x]
    for s in range(7):
        steps.append(gen_evolved(w, steps[-1], s))
    offs = w.offsets
    for qb in (3, 0):
        gs = GroupedSelectiveAttention(w.B, w.H, w.D, offs, qb, G, w.scale, torch.bfloat16, "cuda",
                                       mem_budget_bytes=None, k=K)
        gs.budget = MAX_STATES * gs.state_bytes
        anchor_w = {}
        base = list(gs.groups)
        gpu = []
        for s, xs in enumerate(steps):
            q, k, v = (to_gpu(xs[n], "bf16") for n in ("q", "k", "v"))
            anchor = s in w.anchors or not anchor_w
            if anchor:
                gs.reset()
                compute = list(gs.groups)
            else:
                gs.fit_budget()
                compute = [grp for grp in gs.groups
                           if sum(anchor_w[b] for b in base if grp[0] <= b[0] and b[1] <= grp[1]) > THR]
            out, lse, wg = gs.step(s, q, k, v, compute)
            wg = wg.cpu().numpy()
            if anchor:
                anchor_w = {grp: float(wg[i]) for i, grp in enumerate(gs.groups)}
            gpu.append((list(gs.groups), list(compute), out.float().cpu().numpy(), lse.cpu().numpy(), wg))
        orc = og.run([{n: exact_inputs(v_, "bf16") for n, v_ in xs.items()} for xs in steps],
                     offs, qb, G, K, MAX_STATES, w.anchors, THR, w.scale)
        tol = TOL["bf16"]
        composed = 0
        for s in range(len(steps)):
            gg, gc, go, gl, gw = gpu[s]
            og_, oc, oo, ol, ow = orc[s]
            assert gg == og_, (qb, s, gg, og_)
            composed += len(gg) < len(base)
            if gc != oc:
                a = max(a_ for a_ in w.anchors if a_ <= s)
                margin = min(abs(sum(v_ for b, v_ in zip(orc[a][0], orc[a][4]) if grp[0] <= b[0] and b[1] <= grp[1])
                                 - THR) for grp in gg)
                assert margin <= tol["w"], (qb, s, gc, oc, margin)
                break       # the caches differ from here on
            assert max_abs(go, oo) <= tol["out"], (qb, s)
            assert max_abs(gl, ol) <= tol["lse"], (qb, s)
            assert max_abs(gw, ow) <= tol["w"], (qb, s)
        assert composed > 0      # the budget really forced Dynamic Group State Compose
