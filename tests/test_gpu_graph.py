"""A step (queue-counter reset, fresh states with a split last round and
its fix-up, composition, contribution weights) captured once as a HIP graph
and replayed: every replay must equal the eager step bit for bit, with eager
launches that share the attention workspace (and leave its counters stale)
and synchronisations between the replays.
"""
import numpy as np
import pytest

from helpers import to_gpu

pytestmark = pytest.mark.gpu


def api():
    from paper_2607_15650_amd import api as _api
    return _api


def test_step_graph_replays_match_eager():
    import torch
    a = api()
    D, H, B = 128, 8, 1
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    lens = [900, 1300, 700, 1100]
    offs = [0]
    for n in lens:
        offs.append(offs[-1] + n)
    P, S = len(lens), offs[-1]
    mask = [1, 1, 0, 0]
    per_tile = H * B * sum(mask)
    q_tiles = (cus + 16 + per_tile - 1) // per_tile    # one full round and a few tasks more: split
    q_len = (q_tiles - 1) * 256 + 100
    rng = np.random.default_rng(11)
    q = to_gpu(rng.standard_normal((B, q_len, H, D), dtype=np.float32), "bf16")
    k = to_gpu(rng.standard_normal((B, S, H, D), dtype=np.float32), "bf16")
    v = to_gpu(rng.standard_normal((B, S, H, D), dtype=np.float32), "bf16")
    k2 = to_gpu(rng.standard_normal((B, S, H, D), dtype=np.float32), "bf16")
    scale = D ** -0.5
    need = a.attn_workspace_bytes(torch.bfloat16, B, H, D, q_len, offs, mask)
    print(f"graph case q_len={q_len} tasks={q_tiles * per_tile} cus={cus} ws={need}", flush=True)
    assert need > 256, "the captured step should include the split and its fix-up"
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    states = torch.zeros((P, B, q_len, H, D), dtype=torch.bfloat16, device="cuda")
    lses = torch.zeros((P, B, H, q_len), dtype=torch.float32, device="cuda")
    a.attn_partition_states(q, k, v, offs, [1] * P, scale, states, lses)   # the cache of an earlier step
    out = torch.empty((B, q_len, H, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((B, H, q_len), dtype=torch.float32, device="cuda")
    w_part = torch.empty(P, dtype=torch.float32, device="cuda")
    cws = torch.empty(max(16, a.contrib_workspace_bytes(B, H, q_len, P)), dtype=torch.uint8, device="cuda")

    def step():
        a.attn_partition_states(q, k2, v, offs, mask, scale, states, lses, workspace=ws)
        a.merge_states(states, lses, out, lse)
        a.contrib(lses, lse, w_part, cws)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (states, lses, out, lse, w_part)]

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()

    other_states = torch.zeros_like(states)
    other_lses = torch.zeros_like(lses)
    for rep in range(4):
        # eager work between the replays, on the same attention workspace
        a.attn_partition_states(q, k, v, offs, [0, 1, 1, 0], scale, other_states, other_lses, workspace=ws)
        other_states.mul_(1.0)
        torch.cuda.synchronize()
        for t in (out, lse, w_part):
            t.fill_(7.0)
        graph.replay()
        torch.cuda.synchronize()
        for name, t, r in zip(("states", "lses", "out", "lse", "w_part"), (states, lses, out, lse, w_part), ref):
            assert torch.equal(t.view(torch.uint8), r.view(torch.uint8)), (rep, name)


def test_allocation_free_step_graph_replays_match_eager():
    """The step with nothing allocated by the library: the static attention
    launch (no workspace), the composition and ditango_contrib_noalloc (the
    weights' partial sums in the library's fixed device array), captured as
    a graph.  Between replays an eager call of the same entry point on other
    sizes overwrites that array; every replay must still equal the eager step
    bit for bit (each call writes every partial sum it reads)."""
    import torch
    a = api()
    D, H, B = 128, 4, 1
    lens = [500, 700, 300]
    offs = [0]
    for n in lens:
        offs.append(offs[-1] + n)
    P, S = len(lens), offs[-1]
    q_len = 613
    rng = np.random.default_rng(12)
    q = to_gpu(rng.standard_normal((B, q_len, H, D), dtype=np.float32), "bf16")
    k = to_gpu(rng.standard_normal((B, S, H, D), dtype=np.float32), "bf16")
    v = to_gpu(rng.standard_normal((B, S, H, D), dtype=np.float32), "bf16")
    scale = D ** -0.5
    states = torch.zeros((P, B, q_len, H, D), dtype=torch.bfloat16, device="cuda")
    lses = torch.zeros((P, B, H, q_len), dtype=torch.float32, device="cuda")
    a.attn_partition_states(q, k, v, offs, [1] * P, scale, states, lses)
    out = torch.empty((B, q_len, H, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((B, H, q_len), dtype=torch.float32, device="cuda")
    w_part = torch.empty(P, dtype=torch.float32, device="cuda")
    w_rows = torch.empty((B, H, q_len, P), dtype=torch.float32, device="cuda")
    # other sizes, for eager calls between the replays
    o_l = torch.randn((5, 2, 3, 2000), device="cuda")
    o_lse = torch.logsumexp(o_l, dim=0)
    o_wp = torch.empty(5, dtype=torch.float32, device="cuda")

    def step():
        a.attn_partition_states(q, k, v, offs, [1, 0, 1], scale, states, lses)
        a.merge_states(states, lses, out, lse)
        a.contrib_noalloc(lses, lse, w_part, w_rows)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (states, lses, out, lse, w_part, w_rows)]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for rep in range(4):
        a.contrib_noalloc(o_l, o_lse, o_wp)
        torch.cuda.synchronize()
        for t in (out, lse, w_part, w_rows):
            t.fill_(7.0)
        graph.replay()
        torch.cuda.synchronize()
        for name, t, r in zip(("states", "lses", "out", "lse", "w_part", "w_rows"),
                              (states, lses, out, lse, w_part, w_rows), ref):
            assert torch.equal(t.view(torch.uint8), r.view(torch.uint8)), (rep, name)
