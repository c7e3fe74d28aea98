"""Balanced launches of ditango_attn_partition_states_ws: the last rounds of
tasks are claimed from queue counters in the workspace, so that faster XCDs
take more of them.  Balancing moves tasks between workgroups and changes no
arithmetic: a balanced unsplit launch must equal the static launch bit for
bit, every time, whatever the workspace held before (the counters are reset
by the launch itself).  The static launch is checked against the oracle by
the parity tests.
"""
import numpy as np
import pytest

from helpers import to_gpu

pytestmark = pytest.mark.gpu

# query rows per workgroup of the kernel each head dim's launches here run
# (D=64 launches of fewer than four rounds run the compiled kernel)
ROWS = {128: 256, 64: 384}


def api():
    from paper_2607_15650_amd import api as _api
    return _api


# (D, H, partition lengths, selected, query tiles): unequal partition
# lengths make tasks of unequal cost; enough tasks that most run static and
# the last rounds from the queues
CASES = [
    (128, 8, [3000, 200, 1500, 64, 0], (0, 1, 2, 3), 40),
    (64, 8, [2500, 900, 33], (0, 2), 60),
    (128, 4, [700], (0,), 17),            # few tasks: every one is claimed
]


@pytest.mark.parametrize("D,H,lens,select,q_tiles", CASES)
def test_balanced_launch_equals_static(D, H, lens, select, q_tiles):
    import torch
    a = api()
    B = 1
    q_len = (q_tiles - 1) * ROWS[D] + 77
    offs = [0]
    for n in lens:
        offs.append(offs[-1] + n)
    P, S = len(lens), offs[-1]
    mask = [1 if j in select else 0 for j in range(P)]
    rng = np.random.default_rng(1000 + D + lens[0])
    gq = to_gpu(rng.standard_normal((B, q_len, H, D), dtype=np.float32), "bf16")
    gk = to_gpu(rng.standard_normal((B, S, H, D), dtype=np.float32), "bf16")
    gv = to_gpu(rng.standard_normal((B, S, H, D), dtype=np.float32), "bf16")
    print(f"balance case D={D} H={H} lens={lens} q_len={q_len} tasks={q_tiles * H * len(select)}", flush=True)

    def launch(workspace):
        st = torch.empty((P, B, q_len, H, D), dtype=torch.bfloat16, device="cuda")
        ls = torch.empty((P, B, H, q_len), dtype=torch.float32, device="cuda")
        st.view(torch.int16).fill_(0x3F3F)
        ls.view(torch.int32).fill_(0x3F3F3F3F)
        a.attn_partition_states(gq, gk, gv, offs, mask, D ** -0.5, st, ls, workspace=workspace)
        torch.cuda.synchronize()
        return st, ls

    s_static, l_static = launch(None)
    queue = torch.empty(256, dtype=torch.uint8, device="cuda")
    for rep, fill in enumerate((0x00, 0x7F, 0xFF, 0x01, 0x7F)):
        queue.fill_(fill)                   # stale counters: the launch resets them
        s_bal, l_bal = launch(queue)
        assert torch.equal(s_bal.view(torch.uint8), s_static.view(torch.uint8)), (rep, fill)
        assert torch.equal(l_bal.view(torch.int32), l_static.view(torch.int32)), (rep, fill)
    for j in range(P):
        if not mask[j]:
            assert bool((s_bal[j].view(torch.int16) == 0x3F3F).all())
            assert bool((l_bal[j].view(torch.int32) == 0x3F3F3F3F).all())


def test_balanced_and_split_launch_repeats_with_a_reused_workspace():
    """The full workspace (counters and split partials) reused by back-to-back
    launches of two shapes: each launch equals its own first result."""
    import torch
    a = api()
    D, H, B = 128, 8, 1
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    lens = [1800, 950]
    offs = [0, lens[0], lens[0] + lens[1]]
    rng = np.random.default_rng(7)
    gk = to_gpu(rng.standard_normal((B, offs[-1], H, D), dtype=np.float32), "bf16")
    gv = to_gpu(rng.standard_normal((B, offs[-1], H, D), dtype=np.float32), "bf16")
    shapes = []
    for extra in (16, 40):
        q_tiles = (2 * cus + extra + 2 * H - 1) // (2 * H)
        q_len = q_tiles * ROWS[D] - 5
        gq = to_gpu(rng.standard_normal((B, q_len, H, D), dtype=np.float32), "bf16")
        need = a.attn_workspace_bytes(torch.bfloat16, B, H, D, q_len, offs, [1, 1])
        shapes.append((q_len, gq, need))
    ws = torch.empty(max(n for _, _, n in shapes), dtype=torch.uint8, device="cuda")

    def launch(q_len, gq):
        st = torch.empty((2, B, q_len, H, D), dtype=torch.bfloat16, device="cuda")
        ls = torch.empty((2, B, H, q_len), dtype=torch.float32, device="cuda")
        a.attn_partition_states(gq, gk, gv, offs, [1, 1], D ** -0.5, st, ls, workspace=ws)
        return st, ls

    first = [launch(q_len, gq) for q_len, gq, _ in shapes]
    for _ in range(3):
        for (q_len, gq, _), (s0, l0) in zip(shapes, first):
            s1, l1 = launch(q_len, gq)
            torch.cuda.synchronize()
            assert torch.equal(s1.view(torch.uint8), s0.view(torch.uint8))
            assert torch.equal(l1.view(torch.int32), l0.view(torch.int32))
