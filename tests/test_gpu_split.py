"""Tail-split launches (ditango_attn_partition_states_ws): the tasks of a
last, partly filled round are split over key ranges, their partial states
composed by a fix-up kernel.  Checked against the float64 oracle, against
the unsplit launch, for determinism, and for leaving unselected slots alone.

Shapes are chosen from the device's compute-unit count so that one full
round plus 16 tasks is launched: the 16 tail tasks are split 7 or 8 ways,
and the last key range of each ends in a partial tile.
"""
import numpy as np
import pytest

import oracle
from helpers import TOL, exact_inputs, max_abs, new_state_cache, to_gpu

pytestmark = pytest.mark.gpu

# query rows per workgroup of the kernel each head dim's launches here run
# (D=64 launches of fewer than four rounds run the compiled kernel)
ROWS = {128: 256, 64: 384}


def api():
    from paper_2607_15650_amd import api as _api
    return _api


# (D, partition lengths, selected partitions, state dtype): the last
# selected partition owns the split tail tasks
CASES = [
    (128, [500, 2081, 90], (0, 1), "bf16"),     # long tail partition: 33 tiles, 7 ranges of 5 (the last 3)
    (128, [2081, 500, 90], (0, 1), "bf16"),     # short tail partition: 8 tiles, one per range
    (64, [700, 1234, 33], (0, 1), "bf16"),
    (128, [300, 1000, 0], (0, 1), "f32"),       # float32 states for bf16 inputs
]


@pytest.mark.parametrize("D,lens,select,state_dt", CASES)
def test_tail_split_matches_oracle_and_unsplit(D, lens, select, state_dt):
    import torch
    a = api()
    H, B = 8, 1
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    per_tile = H * B * len(select)
    q_tiles = (cus + 16 + per_tile - 1) // per_tile
    q_len = (q_tiles - 1) * ROWS[D] + 100
    offs = [0]
    for n in lens:
        offs.append(offs[-1] + n)
    P, S = len(lens), offs[-1]
    mask = [1 if j in select else 0 for j in range(P)]
    rng = np.random.default_rng(D + lens[0])
    q = rng.standard_normal((B, q_len, H, D), dtype=np.float32)
    k = rng.standard_normal((B, S, H, D), dtype=np.float32) + 0.2
    v = rng.standard_normal((B, S, H, D), dtype=np.float32)
    scale = D ** -0.5
    gq, gk, gv = to_gpu(q, "bf16"), to_gpu(k, "bf16"), to_gpu(v, "bf16")

    need = a.attn_workspace_bytes(torch.bfloat16, B, H, D, q_len, offs, mask)
    print(f"split case D={D} lens={lens} q_len={q_len} tasks={q_tiles * per_tile} cus={cus} ws={need}", flush=True)
    # more than the 256 bytes of queue counters: the plan asks for the
    # partial states of a split tail
    assert need > 256, "one full round plus 16 tasks must split the tail"
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")

    sdt = torch.float32 if state_dt == "f32" else torch.bfloat16

    def launch(workspace):
        st = torch.empty((P, B, q_len, H, D), dtype=sdt, device="cuda")
        ls = torch.empty((P, B, H, q_len), dtype=torch.float32, device="cuda")
        st.view(torch.int16 if sdt == torch.bfloat16 else torch.int32).fill_(0x3F3F)
        ls.view(torch.int32).fill_(0x3F3F3F3F)
        a.attn_partition_states(gq, gk, gv, offs, mask, scale, st, ls, workspace=workspace)
        torch.cuda.synchronize()
        return st, ls

    s_split, l_split = launch(ws)
    s_again, l_again = launch(ws)
    s_plain, l_plain = launch(None)
    s_small, l_small = launch(ws[: need // 2])        # too small to split: balanced, unsplit
    s_queue, l_queue = launch(ws[:256])                # the queue counters only

    # bitwise: the split launch repeats; a short workspace balances without
    # splitting, which is the static launch's arithmetic
    assert torch.equal(s_split.view(torch.uint8), s_again.view(torch.uint8))
    assert torch.equal(l_split.view(torch.int32), l_again.view(torch.int32))
    for s_b, l_b in ((s_small, l_small), (s_queue, l_queue)):
        assert torch.equal(s_b.view(torch.uint8), s_plain.view(torch.uint8))
        assert torch.equal(l_b.view(torch.int32), l_plain.view(torch.int32))
    # the split path really ran: the composed key ranges round differently
    # from the single pass somewhere in the split tasks' rows
    assert not torch.equal(l_split.view(torch.int32), l_plain.view(torch.int32))
    # unselected slots untouched
    ity = torch.int16 if sdt == torch.bfloat16 else torch.int32
    for j in range(P):
        if not mask[j]:
            assert bool((s_split[j].view(ity) == 0x3F3F).all())
            assert bool((l_split[j].view(torch.int32) == 0x3F3F3F3F).all())

    Q, K, V = (exact_inputs(t, "bf16") for t in (q, k, v))
    tol = TOL["bf16"]
    for j in select:
        o_out, o_lse = oracle.partition_state(Q, K[:, offs[j]:offs[j + 1]], V[:, offs[j]:offs[j + 1]], scale)
        g_out = s_split[j].float().cpu().numpy()
        g_lse = l_split[j].cpu().numpy()
        assert max_abs(g_out, o_out) <= tol["out"], (j, max_abs(g_out, o_out))
        assert max_abs(g_lse, o_lse) <= tol["lse"], (j, max_abs(g_lse, o_lse))
        # split and unsplit differ by rounding only: each key range keeps its
        # own running maximum, so the bf16 probabilities of the P.V products
        # round differently (OUT), and the composition adds its own (LSE)
        assert max_abs(g_lse, l_plain[j].cpu().numpy()) <= 1e-4
        assert max_abs(g_out, s_plain[j].float().cpu().numpy()) <= tol["out"]


def test_no_split_of_short_tasks_in_a_single_round():
    """192 tasks of 32 key tiles (8 heads, 8 query tiles, 3 partitions of
    2,048 keys) on 256 compute units: one partial round, and splitting it
    would make units whose fixed costs (queries loaded again, float32
    partial states written and composed) outweigh the shorter round."""
    import torch
    a = api()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    if cus <= 192:
        pytest.skip("needs more than 192 compute units")
    offs = [2048 * j for j in range(9)]
    sel = [0, 0, 1, 1, 1, 0, 0, 0]
    assert a.attn_workspace_bytes(torch.bfloat16, 1, 8, 64, 2048, offs, sel) == 256


def test_no_split_when_the_last_round_is_full():
    import torch
    a = api()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    H = 8
    q_tiles = (2 * cus) // H                        # exactly two rounds with one partition
    if q_tiles * H != 2 * cus:
        pytest.skip("compute-unit count not a multiple of 8")
    q_len = q_tiles * ROWS[128]
    # the queue counters only; fp32 inputs use no workspace
    assert a.attn_workspace_bytes(torch.bfloat16, 1, H, 128, q_len, [0, 640], [1]) == 256
    assert a.attn_workspace_bytes(torch.float32, 1, H, 128, q_len + 1, [0, 640], [1]) == 0
