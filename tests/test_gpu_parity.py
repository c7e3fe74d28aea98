"""GPU parity: the HIP path through the C ABI against the float64 oracle on the
same seeded inputs.

Tolerances (max-abs, against the oracle evaluated on the exact input values
the kernels see):
  bf16 inputs, float32 accumulation: OUT <= 1e-2, LSE <= 2e-3 (V unit variance)
  float32 inputs:                    OUT <= 1e-5, LSE <= 1e-5
Selections are given; rankings of the contribution weights must agree exactly
wherever the oracle's adjacent gap exceeds the weight tolerance.
"""
import math

import numpy as np
import pytest

import fixtures
import oracle
from fixtures import gen_qkv, get_workload, sample_rows
from fixtures.workloads import Workload, partition_offsets

from helpers import TOL, exact_inputs, max_abs, new_state_cache, per_head, to_gpu, torch_dtype

pytestmark = pytest.mark.gpu


def api():
    from paper_2607_15650_amd import api as _api
    return _api


def run_step(w, x, select, rows_prev=True):
    """Populate the cache from the previous step (all partitions), then compute
    the selected partitions fresh from the current step, merge and contrib.
    Returns GPU results as numpy."""
    import torch
    a = api()
    offs = w.offsets
    P = w.P
    qa, qb = offs[w.q], offs[w.q + 1]
    q_len = qb - qa
    dev = {k: to_gpu(v, w.dtype) for k, v in x.items()}
    out_states, lse_states = new_state_cache(P, w.B, q_len, w.H, w.D, w.dtype)
    if "q_prev" in dev:
        a.attn_partition_states(dev["q_prev"][:, qa:qb].contiguous(), dev["k_prev"], dev["v_prev"],
                                offs, [1] * P, w.scale, out_states, lse_states)
    # the current step as bench.py launches it: with the workspace whose
    # queue counters balance the launch over the XCDs (and that splits the
    # last round of a launch of few rounds)
    mask = [1 if j in select else 0 for j in range(P)]
    n_ws = a.attn_workspace_bytes(torch_dtype(w.dtype), w.B, w.H, w.D, q_len, offs, mask)
    ws_attn = torch.empty(n_ws, dtype=torch.uint8, device="cuda") if n_ws > 0 else None
    a.attn_partition_states(dev["q"][:, qa:qb].contiguous(), dev["k"], dev["v"], offs, mask, w.scale,
                            out_states, lse_states, ws_attn)
    out = torch.empty((w.B, q_len, w.H, w.D), dtype=torch_dtype(w.dtype), device="cuda")
    lse = torch.empty((w.B, w.H, q_len), dtype=torch.float32, device="cuda")
    a.merge_states(out_states, lse_states, out, lse)
    w_part = torch.empty(P, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(16, a.contrib_workspace_bytes(w.B, w.H, q_len, P)), dtype=torch.uint8, device="cuda")
    w_rows = torch.empty((w.B, w.H, q_len, P), dtype=torch.float32, device="cuda")
    a.contrib(lse_states, lse, w_part, ws, w_rows)
    torch.cuda.synchronize()
    f = lambda t: t.float().cpu().numpy()
    return dict(out_states=f(out_states), lse_states=f(lse_states), out=f(out), lse=f(lse),
                w_part=f(w_part), w_rows=f(w_rows))


def oracle_step(w, x, select, rows):
    """Oracle on query rows ``rows`` of the query block (rows and heads are
    independent: the heads run in parallel and are stacked back)."""
    offs = w.offsets
    qa, qb = offs[w.q], offs[w.q + 1]
    sel = [1 if j in select else 0 for j in range(w.P)]

    def one(h):
        # the exact input values of head h only (float64 copies per head)
        qrow = lambda name: exact_inputs(x[name][:, qa:qb][:, rows][:, :, h:h + 1], w.dtype)
        kv = lambda name: exact_inputs(x[name][:, :, h:h + 1], w.dtype)
        if "q_prev" in x:
            _, _, outs, lses = oracle.selective_step(
                qrow("q"), kv("k"), kv("v"), qrow("q_prev"), kv("k_prev"), kv("v_prev"), offs, sel, w.scale)
        else:
            outs, lses = oracle.partition_states(qrow("q"), kv("k"), kv("v"), offs, w.scale)
        return outs, lses

    parts = per_head(one, w.H)
    outs = [np.concatenate([p[0][j] for p in parts], axis=2) for j in range(w.P)]
    lses = [np.concatenate([p[1][j] for p in parts], axis=1) for j in range(w.P)]
    out, lse = oracle.merge(outs, lses)
    W, wbar = oracle.contrib(lses, lse)
    return dict(outs=outs, lses=lses, out=out, lse=lse, W=W, wbar=wbar)


def compare(w, g, o, rows, tol, check_wbar=True):
    """Slot states, composed state and per-row weights at ``rows``, and the
    per-partition mean weights with their ranking (R3: exact wherever the
    oracle's adjacent gap exceeds the weight tolerance).  With all rows the
    GPU's w_part is compared with the oracle's mean; with sampled rows the
    GPU's per-row weights are averaged over the same rows as the oracle's,
    and w_part is checked to be the mean of the GPU's per-row weights over
    all rows."""
    sampled = len(rows) < w.q_len
    worst = {}
    for j in range(w.P):
        e_out = max_abs(g["out_states"][j][:, rows], o["outs"][j])
        e_lse = max_abs(g["lse_states"][j][:, :, rows], o["lses"][j])
        worst[f"slot{j}"] = (e_out, e_lse)
        assert e_out <= tol["out"], (j, e_out)
        assert e_lse <= tol["lse"], (j, e_lse)
    e_out = max_abs(g["out"][:, rows], o["out"])
    e_lse = max_abs(g["lse"][:, :, rows], o["lse"])
    assert e_out <= tol["out"], ("merged", e_out)
    assert e_lse <= tol["lse"], ("merged", e_lse)
    e_w = max_abs(g["w_rows"][:, :, rows], o["W"])
    assert e_w <= 2 * tol["lse"] + 1e-6, ("w_rows", e_w)
    if not check_wbar:
        return worst
    if not sampled:
        assert max_abs(g["w_part"], o["wbar"]) <= tol["w"]
        check_ranking(g["w_part"], o["wbar"], w.q, tol["w"])
    else:
        g_mean = g["w_rows"][:, :, rows].astype(np.float64).reshape(-1, w.P).mean(axis=0)
        assert max_abs(g_mean, o["wbar"]) <= tol["w"], ("sampled wbar", g_mean, o["wbar"])
        check_ranking(g_mean, o["wbar"], w.q, tol["w"])
        full_mean = g["w_rows"].astype(np.float64).reshape(-1, w.P).mean(axis=0)
        assert max_abs(g["w_part"], full_mean) <= 1e-5
    return worst


def check_ranking(w_gpu, w_orc, q, tau):
    """Ranks agree wherever the oracle's adjacent gap exceeds tau."""
    r_o = oracle.rank_partitions(w_orc, q)
    r_g = sorted(range(len(w_gpu)), key=lambda j: (-float(w_gpu[j]), abs(j - q), j))
    vals = [w_orc[j] for j in r_o]
    # split the oracle ranking into blocks separated by gaps > tau; each block
    # must hold the same set of partitions in both rankings
    start = 0
    for i in range(1, len(r_o) + 1):
        if i == len(r_o) or vals[i - 1] - vals[i] > tau:
            assert set(r_o[start:i]) == set(r_g[start:i]), (r_o, r_g)
            start = i


# --------------------------------------------------------------------- workloads

def test_plumbing_f32_all_fresh():
    w = get_workload("plumbing_f32_h2_d64_s4096_p4")
    x = gen_qkv(w)
    g = run_step(w, x, w.select)
    rows = np.arange(w.q_len)
    o = oracle_step(w, x, w.select, rows)
    compare(w, g, o, rows, TOL["f32"])
    # composing all fresh partitions is full attention
    X = {k: exact_inputs(v, "f32") for k, v in x.items()}
    offs = w.offsets
    fo, fl = oracle.full_attention(X["q"][:, offs[0]:offs[1]], X["k"], X["v"], w.scale)
    assert max_abs(g["out"], fo) <= 1e-5 and max_abs(g["lse"], fl) <= 1e-5


def test_reuse_bf16_all_rows():
    w = get_workload("reuse_bf16_h12_d64_s16384_p8")
    x = gen_qkv(w)
    g = run_step(w, x, w.select)
    rows = np.arange(w.q_len)
    o = oracle_step(w, x, w.select, rows)
    compare(w, g, o, rows, TOL["bf16"])


@pytest.mark.slow
def test_videodit_bf16_sampled_rows():
    w = get_workload("videodit_bf16_h40_d128_s75600_p8")
    x = gen_qkv(w)
    g = run_step(w, x, w.select)
    rows = sample_rows(w.q_len, 1024, w.seed)
    o = oracle_step(w, x, w.select, rows)
    compare(w, g, o, rows, TOL["bf16"])


@pytest.mark.slow
@pytest.mark.parametrize("k", [4, 16])
def test_longctx_bf16_sampled_rows(k):
    """Nearest-first selections of 4 and of all 16 partitions (16 = full
    attention over 131,072 keys), 1024 sampled rows."""
    from fixtures.workloads import nearest_first
    w = get_workload("longctx_bf16_h24_d128_s131072_p16")
    select = tuple(nearest_first(w.P, w.q, k))
    x = gen_qkv(w, with_prev=k < w.P)
    g = run_step(w, x, select)
    rows = sample_rows(w.q_len, 1024, w.seed)
    o = oracle_step(w, x, select, rows)
    compare(w, g, o, rows, TOL["bf16"])


@pytest.mark.slow
def test_hunyuan_d64_bf16_sampled_rows():
    w = get_workload("hunyuan_bf16_h48_d64_s118800_p8")
    x = gen_qkv(w)
    g = run_step(w, x, w.select)
    rows = sample_rows(w.q_len, 1024, w.seed)
    o = oracle_step(w, x, w.select, rows)
    compare(w, g, o, rows, TOL["bf16"])


@pytest.mark.slow
def test_videodit_cfg_batch2_sampled_rows():
    w = get_workload("videodit_cfg_bf16_b2_h40_d128_s75600_p8")
    x = gen_qkv(w)
    g = run_step(w, x, w.select)
    rows = sample_rows(w.q_len, 1024, w.seed)
    o = oracle_step(w, x, w.select, rows)
    compare(w, g, o, rows, TOL["bf16"])


# --------------------------------------------------------------------- ragged / edge shapes

EDGE = [
    # (dtype, D, H, q_len, partition lengths)
    ("bf16", 128, 3, 300, [0, 1, 63, 65, 200]),
    ("bf16", 64, 2, 1, [7, 64, 129]),
    ("bf16", 128, 1, 257, [256, 255, 1]),
    ("bf16", 64, 5, 513, [100, 0, 333]),
    # exact multiples of the key tiles (64 keys) and of the
    # query tiles (256 rows), and one key either side
    ("bf16", 128, 2, 256, [64, 128, 63, 65]),
    # 3, 3, 5, 6, 7 and 9 key tiles: the loop ends in each of its four
    # unrolled positions and masks a partial last tile from each of them
    ("bf16", 128, 2, 300, [130, 192, 300, 321, 440, 513]),
    # the same at D=64, with enough heads for four rounds of tasks (the
    # hand-scheduled D=64 kernel runs launches of at least four rounds)
    ("bf16", 64, 128, 300, [130, 192, 300, 321, 440, 513]),
    # full last tiles of 5, 8, 9 and 12 key tiles: the steady iterations run
    # in blocks of four while none of them is the last, so the loop leaves a
    # block straight for the last iteration (5, 9), after one or two blocks
    # and a tail of three (8, 12)
    ("bf16", 128, 2, 300, [320, 512, 576, 768]),
    ("bf16", 64, 128, 300, [320, 512, 576, 768]),
    ("bf16", 64, 128, 257, [64, 128, 63, 65]),
    ("bf16", 64, 4, 384, [96, 192, 95, 97]),    # 1.5 and 3 tiles of 64 keys, 1.5 query tiles
    ("bf16", 64, 1, 385, [288, 1, 383]),
    ("f32", 128, 2, 129, [31, 33, 96]),
    ("f32", 64, 3, 40, [0, 5, 70]),
]


@pytest.mark.parametrize("dtype,D,H,q_len,lens", EDGE)
def test_ragged_shapes(dtype, D, H, q_len, lens):
    import torch
    a = api()
    rng = np.random.default_rng(q_len * 7 + D)
    B = 2 if q_len < 100 else 1
    S = sum(lens)
    offs = [0]
    for n in lens:
        offs.append(offs[-1] + n)
    P = len(lens)
    q = rng.standard_normal((B, q_len, H, D), dtype=np.float32)
    k = rng.standard_normal((B, S, H, D), dtype=np.float32) + 0.3
    v = rng.standard_normal((B, S, H, D), dtype=np.float32)
    scale = 1 / math.sqrt(D)
    out_states, lse_states = new_state_cache(P, B, q_len, H, D, dtype)
    a.attn_partition_states(to_gpu(q, dtype), to_gpu(k, dtype), to_gpu(v, dtype), offs, [1] * P, scale,
                            out_states, lse_states)
    out = torch.empty((B, q_len, H, D), dtype=torch_dtype(dtype), device="cuda")
    lse = torch.empty((B, H, q_len), dtype=torch.float32, device="cuda")
    a.merge_states(out_states, lse_states, out, lse)
    torch.cuda.synchronize()
    Q, K, V = (exact_inputs(t, dtype) for t in (q, k, v))
    outs, lses = oracle.partition_states(Q, K, V, offs, scale)
    tol = TOL[dtype]
    for j in range(P):
        gl = lse_states[j].cpu().numpy()
        go = out_states[j].float().cpu().numpy()
        if lens[j] == 0:
            assert np.all(np.isneginf(gl)) and np.all(go == 0)
        assert max_abs(go, outs[j]) <= tol["out"], j
        assert max_abs(gl, lses[j]) <= tol["lse"], j
    mo, ml = oracle.merge(outs, lses)
    assert max_abs(out.float().cpu().numpy(), mo) <= tol["out"]
    assert max_abs(lse.cpu().numpy(), ml) <= tol["lse"]
    # the same launch with the attention workspace (queue counters, and a
    # split last round when the plan asks for one): bit for bit the static
    # launch when unsplit, within the tolerance of the oracle when split
    need = a.attn_workspace_bytes(torch_dtype(dtype), B, H, D, q_len, offs, [1] * P)
    if need > 0:
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        ws.fill_(0x5A)                                  # stale counters
        s2, l2 = new_state_cache(P, B, q_len, H, D, dtype)
        a.attn_partition_states(to_gpu(q, dtype), to_gpu(k, dtype), to_gpu(v, dtype), offs, [1] * P, scale,
                                s2, l2, ws)
        torch.cuda.synchronize()
        if need == 256:
            assert torch.equal(s2.view(torch.uint8), out_states.view(torch.uint8))
            assert torch.equal(l2.view(torch.int32), lse_states.view(torch.int32))
        else:
            for j in range(P):
                assert max_abs(s2[j].float().cpu().numpy(), outs[j]) <= tol["out"], j
                assert max_abs(l2[j].cpu().numpy(), lses[j]) <= tol["lse"], j


@pytest.mark.parametrize("dtype,D", [("bf16", 128), ("bf16", 64), ("f32", 64)])
def test_twenty_partitions_attn_merge_contrib(dtype, D):
    """P = 20 (three of them empty): the attention launch over 17 selected
    partitions, the merge of all 20 slots and the weights of 20 partitions
    run the instantiations for more than 16 slots; every result against the
    oracle, the ranking by R3, and a 17-slot subset list."""
    import torch
    a = api()
    rng = np.random.default_rng(20 + D)
    lens = [33, 0, 64, 65, 1, 190, 0, 96, 97, 5, 128, 200, 7, 0, 63, 129, 40, 2, 250, 31]
    P = len(lens)
    offs = [0]
    for n in lens:
        offs.append(offs[-1] + n)
    S = offs[-1]
    B, H, q_len = 1, 2, 301
    q = rng.standard_normal((B, q_len, H, D), dtype=np.float32)
    k = rng.standard_normal((B, S, H, D), dtype=np.float32) + 0.25
    v = rng.standard_normal((B, S, H, D), dtype=np.float32)
    # key norms differ per partition so that the weights are well separated
    k *= np.repeat(np.linspace(0.3, 1.6, P), lens).astype(np.float32)[None, :, None, None]
    scale = 1 / math.sqrt(D)
    qg, kg, vg = (to_gpu(t, dtype) for t in (q, k, v))
    mask = [1] * P
    st, ls = new_state_cache(P, B, q_len, H, D, dtype)
    n_ws = a.attn_workspace_bytes(torch_dtype(dtype), B, H, D, q_len, offs, mask)
    ws_attn = torch.empty(n_ws, dtype=torch.uint8, device="cuda") if n_ws > 0 else None
    a.attn_partition_states(qg, kg, vg, offs, mask, scale, st, ls, ws_attn)
    out = torch.empty((B, q_len, H, D), dtype=torch_dtype(dtype), device="cuda")
    lse = torch.empty((B, H, q_len), dtype=torch.float32, device="cuda")
    a.merge_states(st, ls, out, lse)
    sub = [19, 0, 2, 3, 4, 5, 7, 8, 9, 10, 11, 12, 14, 15, 16, 17, 18]      # 17 slots, empty ones left out
    out_s = torch.empty_like(out)
    lse_s = torch.empty_like(lse)
    a.merge_states(st, ls, out_s, lse_s, slots=sub)
    w_part = torch.empty(P, dtype=torch.float32, device="cuda")
    w_rows = torch.empty((B, H, q_len, P), dtype=torch.float32, device="cuda")
    cws = torch.empty(a.contrib_workspace_bytes(B, H, q_len, P), dtype=torch.uint8, device="cuda")
    a.contrib(ls, lse, w_part, cws, w_rows)
    torch.cuda.synchronize()
    Q, K, V = (exact_inputs(t, dtype) for t in (q, k, v))
    outs, lses = oracle.partition_states(Q, K, V, offs, scale)
    tol = TOL[dtype]
    for j in range(P):
        go, gl = st[j].float().cpu().numpy(), ls[j].cpu().numpy()
        if lens[j] == 0:
            assert np.all(np.isneginf(gl)) and np.all(go == 0), j
        # a partition of a few keys has OUT of the size of one V row: its bf16
        # state carries the store rounding 2^-8 |OUT| and the rounding of the
        # probabilities in the P.V product, up to 2^-8 max|v|, which at unit
        # variance can exceed 1e-2 (the bar assumes OUT averaged over many keys)
        t_out = tol["out"]
        if dtype == "bf16" and lens[j] > 0:
            vmax = float(np.abs(V[:, offs[j]:offs[j + 1]]).max())
            t_out = max(t_out, 2.0 ** -8 * (float(np.abs(outs[j]).max()) + vmax) + 2.0 ** -12)
        assert max_abs(go, outs[j]) <= t_out, (j, max_abs(go, outs[j]), t_out)
        assert max_abs(gl, lses[j]) <= tol["lse"], j
    mo, ml = oracle.merge(outs, lses)
    assert max_abs(out.float().cpu().numpy(), mo) <= tol["out"]
    assert max_abs(lse.cpu().numpy(), ml) <= tol["lse"]
    # the empty partitions carry weight 0: the subset composes to the same state
    so, sl = oracle.merge([outs[j] for j in sub], [lses[j] for j in sub])
    assert max_abs(out_s.float().cpu().numpy(), so) <= tol["out"]
    assert max_abs(lse_s.cpu().numpy(), sl) <= tol["lse"]
    W, wbar = oracle.contrib(lses, ml)
    assert max_abs(w_rows.cpu().numpy(), W) <= 2 * tol["lse"] + 1e-6
    wp = w_part.cpu().numpy()
    assert max_abs(wp, wbar) <= tol["w"]
    assert all(wp[j] == 0.0 for j in range(P) if lens[j] == 0)
    check_ranking(wp, wbar, 9, tol["w"])


@pytest.mark.parametrize("D", [128, 64])
def test_running_max_far_below_and_above(D):
    """Score ranges that force the kernel to raise its running maximum in the
    middle of a partition: per head, the key norms ramp up along the sequence
    (later tiles score far above the first one, up to overflow of exp2
    against a stale maximum), ramp down (later tiles underflow against the
    first), or jump once.  Queries scaled by 32 make scores span hundreds, so
    against the first tile's maximum exp2 would overflow float32.  Such rows
    are nearly one-hot, where the bf16 rounding of the probabilities bounds
    the OUT error by 2^-8 max|v| (+ 2^-9 |OUT| for the bf16 store); V is
    scaled by 1/4 to keep that bound (0.0065 here) under the 1e-2 tolerance,
    which is stated for unit-variance V."""
    import torch
    a = api()
    rng = np.random.default_rng(99 + D)
    B, H, q_len, dtype = 1, 3, 300, "bf16"
    lens = [1000, 130]
    S = sum(lens)
    offs = [0, lens[0], S]
    q = rng.standard_normal((B, q_len, H, D), dtype=np.float32) * 32.0
    k = rng.standard_normal((B, S, H, D), dtype=np.float32)
    ramp = np.linspace(0.05, 1.0, S, dtype=np.float32)
    k[:, :, 0, :] *= ramp[None, :, None]                        # rising
    k[:, :, 1, :] *= ramp[::-1][None, :, None]                  # falling
    k[:, :, 2, :] *= np.where(np.arange(S) < 400, 0.05, 1.0).astype(np.float32)[None, :, None]   # jump
    v = rng.standard_normal((B, S, H, D), dtype=np.float32) * 0.25
    scale = 1 / math.sqrt(D)
    P = len(lens)
    out_states, lse_states = new_state_cache(P, B, q_len, H, D, dtype)
    a.attn_partition_states(to_gpu(q, dtype), to_gpu(k, dtype), to_gpu(v, dtype), offs, [1] * P, scale,
                            out_states, lse_states)
    torch.cuda.synchronize()
    Q, K, V = (exact_inputs(t, dtype) for t in (q, k, v))
    outs, lses = oracle.partition_states(Q, K, V, offs, scale)
    for j in range(P):
        go = out_states[j].float().cpu().numpy()
        gl = lse_states[j].cpu().numpy()
        assert np.all(np.isfinite(go)) and np.all(np.isfinite(gl)), j
        assert max_abs(go, outs[j]) <= TOL[dtype]["out"], j
        assert max_abs(gl, lses[j]) <= TOL[dtype]["lse"], j
    # premise: in some row, the partition's top score exceeds the first 64-key
    # tile's top score by more than 128 (base 2): exp2 against the first
    # tile's maximum overflows float32 there
    sc = np.einsum("bqhd,bkhd->bhqk", Q, K[:, :lens[0]]) * scale
    gap = (sc.max(axis=3) - sc[..., :64].max(axis=3)) / math.log(2.0)
    assert gap.max() > 128.0, gap.max()


@pytest.mark.parametrize("D", [128, 64])
def test_running_max_redo_in_a_long_launch(D):
    """The hand-scheduled kernel runs a fast key loop that keeps tile 0's
    maximum and, in a workgroup where a row sum left [0, 2^40], runs the task
    again in the checked loop that raises the maximum.  A launch long enough
    for the hand-scheduled kernel at both head dims (at least four rounds of
    256-row tasks) with three heads whose later keys score far above tile 0
    (queries scaled by 32; key norms rising, falling, jumping) and 61 plain
    heads: tasks of both kinds in one launch, against the oracle on sampled
    rows of every head, and bitwise equal on a second launch."""
    import torch
    a = api()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    rng = np.random.default_rng(7 + D)
    B, H, dtype = 1, 64, "bf16"
    lens = [700, 150]
    S = sum(lens)
    offs = [0, lens[0], S]
    q_tiles = -(-4 * cus // (H * len(lens)))
    q_len = q_tiles * 256 - 37
    q = rng.standard_normal((B, q_len, H, D), dtype=np.float32)
    q[:, :, :3, :] *= 32.0
    k = rng.standard_normal((B, S, H, D), dtype=np.float32)
    ramp = np.linspace(0.05, 1.0, S, dtype=np.float32)
    k[:, :, 0, :] *= ramp[None, :, None]
    k[:, :, 1, :] *= ramp[::-1][None, :, None]
    k[:, :, 2, :] *= np.where(np.arange(S) < 400, 0.05, 1.0).astype(np.float32)[None, :, None]
    v = rng.standard_normal((B, S, H, D), dtype=np.float32) * 0.25
    scale = 1 / math.sqrt(D)
    P = len(lens)
    dq, dk, dv = to_gpu(q, dtype), to_gpu(k, dtype), to_gpu(v, dtype)
    print(f"redo case D={D} H={H} q_len={q_len} tasks={q_tiles * H * P} cus={cus}", flush=True)
    res = []
    for _ in range(2):
        out_states, lse_states = new_state_cache(P, B, q_len, H, D, dtype)
        n_ws = a.attn_workspace_bytes(torch_dtype(dtype), B, H, D, q_len, offs, [1] * P)
        ws = torch.empty(n_ws, dtype=torch.uint8, device="cuda") if n_ws > 0 else None
        a.attn_partition_states(dq, dk, dv, offs, [1] * P, scale, out_states, lse_states, ws)
        torch.cuda.synchronize()
        res.append((out_states.float().cpu().numpy(), lse_states.cpu().numpy()))
    assert np.array_equal(res[0][0], res[1][0]) and np.array_equal(res[0][1], res[1][1])
    go, gl = res[0]
    rows = np.unique(np.concatenate([[0, 1, 63, 64, 255, 256, q_len - 1],
                                     rng.choice(q_len, 96, replace=False)]))
    Q, K, V = (exact_inputs(t, dtype) for t in (q, k, v))
    outs, lses = oracle.partition_states(Q[:, rows], K, V, offs, scale)
    for j in range(P):
        assert np.all(np.isfinite(go[j])) and np.all(np.isfinite(gl[j])), j
        assert max_abs(go[j][:, rows], outs[j]) <= TOL[dtype]["out"], j
        assert max_abs(gl[j][:, :, rows], lses[j]) <= TOL[dtype]["lse"], j
    # premise: partition 0's top score lies far (> 128, base 2) above its first
    # tile's in some row of the scaled heads, and within 30 in every row of
    # the plain ones (their tasks keep the fast loop's result)
    sc = np.einsum("bqhd,bkhd->bhqk", Q[:, rows], K[:, :lens[0]]) * scale
    gap = (sc.max(axis=3) - sc[..., :64].max(axis=3)) / math.log(2.0)
    assert gap[:, :3].max() > 128.0, gap[:, :3].max()
    assert gap[:, 3:].max() < 30.0, gap[:, 3:].max()


@pytest.mark.parametrize("D", [128, 64])
def test_fp32_states_for_bf16_inputs(D):
    """bf16 inputs with the states kept in float32 (the _ex entry point): the
    states match the oracle, differ from the bf16 states by the bf16 store
    rounding only, and compose into a bf16 or a float32 output."""
    import torch
    a = api()
    rng = np.random.default_rng(5 + D)
    B, H, q_len, lens = 1, 4, 333, [150, 0, 449, 64]
    S = sum(lens)
    offs = [0]
    for n in lens:
        offs.append(offs[-1] + n)
    P = len(lens)
    q = rng.standard_normal((B, q_len, H, D), dtype=np.float32)
    k = rng.standard_normal((B, S, H, D), dtype=np.float32) + 0.2
    v = rng.standard_normal((B, S, H, D), dtype=np.float32)
    scale = 1 / math.sqrt(D)
    qg, kg, vg = (to_gpu(t, "bf16") for t in (q, k, v))
    st32, ls32 = new_state_cache(P, B, q_len, H, D, "f32")
    st16, ls16 = new_state_cache(P, B, q_len, H, D, "bf16")
    a.attn_partition_states(qg, kg, vg, offs, [1] * P, scale, st32, ls32)
    a.attn_partition_states(qg, kg, vg, offs, [1] * P, scale, st16, ls16)
    out16 = torch.empty((B, q_len, H, D), dtype=torch.bfloat16, device="cuda")
    out32 = torch.empty((B, q_len, H, D), dtype=torch.float32, device="cuda")
    lse = torch.empty((B, H, q_len), dtype=torch.float32, device="cuda")
    a.merge_states(st32, ls32, out16, lse)
    a.merge_states(st32, ls32, out32, None)
    torch.cuda.synchronize()
    assert st32.dtype == torch.float32
    Q, K, V = (exact_inputs(t, "bf16") for t in (q, k, v))
    outs, lses = oracle.partition_states(Q, K, V, offs, scale)
    g32 = st32.cpu().numpy()
    g16 = st16.float().cpu().numpy()
    for j in range(P):
        assert max_abs(g32[j], outs[j]) <= TOL["bf16"]["out"], j
        assert max_abs(ls32[j].cpu().numpy(), lses[j]) <= TOL["bf16"]["lse"], j
        # same kernel arithmetic: the bf16 states are the float32 ones rounded
        assert np.all(np.abs(g16[j] - g32[j]) <= np.abs(g32[j]) * 2.0 ** -8 + 1e-30), j
        assert np.array_equal(ls32[j].cpu().numpy(), ls16[j].cpu().numpy()), j
    mo, ml = oracle.merge(outs, lses)
    assert max_abs(out16.float().cpu().numpy(), mo) <= TOL["bf16"]["out"]
    assert max_abs(out32.cpu().numpy(), mo) <= TOL["bf16"]["out"]
    assert max_abs(lse.cpu().numpy(), ml) <= TOL["bf16"]["lse"]


def test_repeated_launches_bitwise_identical():
    """Every launch of the same inputs gives the same bits: a race between
    the waves of a workgroup on the LDS tile ring (a tile overwritten while
    another wave still reads it) shows up as launch-to-launch differences.
    Keys differ strongly from tile to tile so that a stale or early tile
    changes the result."""
    import torch
    a = api()
    rng = np.random.default_rng(2024)
    B, H, q_len, D = 1, 16, 1000, 128
    lens = [700, 333, 64, 901]
    S = sum(lens)
    offs = [0]
    for n in lens:
        offs.append(offs[-1] + n)
    P = len(lens)
    q = rng.standard_normal((B, q_len, H, D), dtype=np.float32) * 4.0
    k = rng.standard_normal((B, S, H, D), dtype=np.float32)
    k *= np.repeat(rng.uniform(0.1, 1.5, size=(S + 63) // 64), 64)[:S].astype(np.float32)[None, :, None, None]
    v = rng.standard_normal((B, S, H, D), dtype=np.float32)
    qg, kg, vg = (to_gpu(t, "bf16") for t in (q, k, v))
    first = None
    for rep in range(8):
        st, ls = new_state_cache(P, B, q_len, H, D, "bf16")
        a.attn_partition_states(qg, kg, vg, offs, [1] * P, 1 / math.sqrt(D), st, ls)
        torch.cuda.synchronize()
        cur = (st.view(torch.int16).cpu().numpy(), ls.cpu().numpy().view(np.int32))
        if first is None:
            first = cur
        else:
            assert np.array_equal(cur[0], first[0]) and np.array_equal(cur[1], first[1]), rep


def test_unselected_slots_untouched_bitwise():
    import torch
    a = api()
    w = Workload(name="t", dtype="bf16", B=1, H=3, D=128, grid=(4, 16, 16), P=8, q=3, seed=9, select=(2, 3, 4))
    x = gen_qkv(w, with_prev=False)
    offs = w.offsets
    qa, qb = offs[w.q], offs[w.q + 1]
    out_states, lse_states = new_state_cache(w.P, w.B, w.q_len, w.H, w.D, "bf16", fill=0x5A5A)
    before_o = out_states.clone()
    before_l = lse_states.clone()
    a.attn_partition_states(to_gpu(x["q"][:, qa:qb], "bf16"), to_gpu(x["k"], "bf16"), to_gpu(x["v"], "bf16"),
                            offs, w.select_mask(), w.scale, out_states, lse_states)
    torch.cuda.synchronize()
    for j in range(w.P):
        same_o = torch.equal(out_states[j].view(torch.int16), before_o[j].view(torch.int16))
        same_l = torch.equal(lse_states[j].view(torch.int32), before_l[j].view(torch.int32))
        assert same_o == same_l == (j not in w.select), j


def test_determinism_and_reuse_with_unchanged_cache_bitwise():
    import torch
    a = api()
    w = Workload(name="t", dtype="bf16", B=1, H=4, D=128, grid=(8, 16, 16), P=8, q=3, seed=10, select=(2, 3, 4))
    x = gen_qkv(w, with_prev=False)
    offs = w.offsets
    qa, qb = offs[w.q], offs[w.q + 1]
    q, k, v = (to_gpu(t, "bf16") for t in (x["q"][:, qa:qb], x["k"], x["v"]))

    def full():
        os_, ls_ = new_state_cache(w.P, w.B, w.q_len, w.H, w.D, "bf16")
        a.attn_partition_states(q, k, v, offs, [1] * w.P, w.scale, os_, ls_)
        return os_, ls_

    o1, l1 = full()
    o2, l2 = full()
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)
    # reuse with an unchanged cache: recompute only the selection over a cache
    # computed from the same tensors -> bitwise equal to all fresh
    o3, l3 = o1.clone(), l1.clone()
    a.attn_partition_states(q, k, v, offs, w.select_mask(), w.scale, o3, l3)
    outs = []
    for os_, ls_ in ((o1, l1), (o3, l3)):
        out = torch.empty((w.B, w.q_len, w.H, w.D), dtype=torch.float32, device="cuda")
        lse = torch.empty((w.B, w.H, w.q_len), dtype=torch.float32, device="cuda")
        a.merge_states(os_, ls_, out, lse)
        outs.append((out, lse))
    torch.cuda.synchronize()
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    # slot order only changes rounding of the float32 composition
    perm = [5, 2, 7, 0, 3, 6, 1, 4]
    out_p = torch.empty_like(outs[0][0])
    lse_p = torch.empty_like(outs[0][1])
    a.merge_states(o1, l1, out_p, lse_p, slots=perm)
    torch.cuda.synchronize()
    assert (out_p - outs[0][0]).abs().max().item() <= 1e-6
    assert (lse_p - outs[0][1]).abs().max().item() <= 1e-6
    # contrib is bitwise reproducible
    wp = []
    for _ in range(2):
        w_part = torch.empty(w.P, dtype=torch.float32, device="cuda")
        ws = torch.empty(a.contrib_workspace_bytes(w.B, w.H, w.q_len, w.P), dtype=torch.uint8, device="cuda")
        a.contrib(l1, outs[0][1], w_part, ws)
        wp.append(w_part)
    torch.cuda.synchronize()
    assert torch.equal(wp[0], wp[1])


# --------------------------------------------------------------------- merge / contrib in isolation

@pytest.mark.parametrize("state_dt,out_dt,D", [("bf16", "bf16", 128), ("bf16", "f32", 64), ("f32", "f32", 128)])
def test_merge_kernel_on_oracle_states(state_dt, out_dt, D):
    """Merge of given states (including -inf rows and a subset slot list)
    against the oracle's composition of the same stored values."""
    import torch
    a = api()
    rng = np.random.default_rng(D)
    P, B, q_len, H = 6, 2, 77, 3
    outs = rng.standard_normal((P, B, q_len, H, D)).astype(np.float32)
    lses = (rng.standard_normal((P, B, H, q_len)) * 3).astype(np.float32)
    lses[1, 0, 1, :10] = -np.inf                   # one partition empty for some rows
    lses[:, 1, 2, 5] = -np.inf                     # one row with every partition empty
    slots = [4, 0, 1, 5, 2]
    st = to_gpu(outs, state_dt)
    ls = torch.from_numpy(lses).cuda()
    out = torch.empty((B, q_len, H, D), dtype=torch_dtype(out_dt), device="cuda")
    lse = torch.empty((B, H, q_len), dtype=torch.float32, device="cuda")
    a.merge_states(st.contiguous(), ls, out, lse, slots=slots)
    torch.cuda.synchronize()
    O = exact_inputs(outs, state_dt)
    mo, ml = oracle.merge([O[j] for j in slots], [lses[j].astype(np.float64) for j in slots])
    go = out.float().cpu().numpy()
    gl = lse.cpu().numpy()
    assert not np.isnan(go).any() and not np.isnan(gl).any()
    assert np.all(go[1, 5, 2] == 0) and np.isneginf(gl[1, 2, 5])
    # float32 output: float32 arithmetic; bf16 output: plus one bf16 rounding
    tol_out = 1e-5 if out_dt == "f32" else float(np.abs(mo).max()) * 2.0 ** -8 + 1e-6
    assert max_abs(go, mo) <= tol_out
    assert max_abs(gl, ml) <= 5e-6


def test_contrib_kernel_against_oracle():
    import torch
    a = api()
    rng = np.random.default_rng(3)
    P, B, H, q_len = 8, 1, 7, 3001
    lses = (rng.standard_normal((P, B, H, q_len)) * 2).astype(np.float32)
    lses[3] -= 4.0
    lses[0, 0, 0, :100] = -np.inf
    mo, ml = oracle.merge([np.zeros((B, q_len, H, 1))] * P, [l.astype(np.float64) for l in lses])
    ml32 = ml.astype(np.float32)
    W, wbar = oracle.contrib([l.astype(np.float64) for l in lses], ml32.astype(np.float64))
    ls = torch.from_numpy(lses).cuda()
    lo = torch.from_numpy(ml32).cuda()
    w_part = torch.empty(P, dtype=torch.float32, device="cuda")
    w_rows = torch.empty((B, H, q_len, P), dtype=torch.float32, device="cuda")
    ws = torch.empty(a.contrib_workspace_bytes(B, H, q_len, P), dtype=torch.uint8, device="cuda")
    a.contrib(ls, lo, w_part, ws, w_rows)
    torch.cuda.synchronize()
    assert max_abs(w_rows.cpu().numpy(), W) <= 1e-6
    assert max_abs(w_part.cpu().numpy(), wbar) <= 1e-6
    check_ranking(w_part.cpu().numpy(), wbar, 3, 1e-6)
