#!/usr/bin/env python3
"""Bench of the selective attention-state hot path on one MI355X.

One step = one pass of the whole hot path for one context-parallel rank's
query block: fresh states of the selected key/value partitions
(ditango_attn_partition_states), composition with the cached states of the
others (ditango_merge_states), and contribution weights
(ditango_contrib).  The state cache is filled from the previous step's
tensors before timing; all inputs are resident in HBM when timing starts.

Default workload: the video-DiT shape (Wan2.1-14B latent, 75,600 tokens,
40 heads, head dim 128, 8 partitions of 9,450 tokens, query partition 3,
fresh partitions {2,3,4}).

Prints one JSON line.  ``value`` is the effective attention throughput of the
whole step: algorithmic flops of the fresh partitions, 4*B*H*q_len*D*sum(L_j),
divided by the step time.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "selective-attn step time (ms) + effective TFLOP/s and % bf16 MFMA peak, 1 GPU"
DEFAULT_WORKLOAD = "videodit_bf16_h40_d128_s75600_p8"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3        # MI355X fp32 MFMA / vector
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E

# HBM bytes per launch of the attention kernel at the default workload, from
# rocprofv3 --pmc FETCH_SIZE and WRITE_SIZE (each scaled so that a plain 1 GiB
# elementwise copy reads / writes 1 GiB), keyed by the build id (source and
# compile options) of the kernel they were taken on; reported only while the
# build id matches.
ATTN_TRAFFIC = {"build_id": "f6b4934c947b132e", "workload": "videodit_bf16_h40_d128_s75600_p8", "mode": "queue",
                # the balanced attention kernel (mean of 5 launches: the order
                # in which tasks are claimed moves the reads by up to 1 %); the
                # counter reset moves about 1 KiB
                "fetch_bytes": 766106.5 * 1024 * 2.0, "write_bytes": 287960.6 * 1024 * 1.0}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--select", default=None, help="comma-separated fresh partitions (default: the workload's)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle baseline sample (0 disables it)")
    ap.add_argument("--threshold", type=float, default=None,
                    help="planner-driven workload: anchor-weight threshold (default: the workload's)")
    ap.add_argument("--planner", choices=("threshold", "error-model"), default="threshold",
                    help="planner-driven workload: anchor-weight threshold, or the error-model planner "
                         "(groups of 2, target reuse ratio --reuse, local drift limit --eps-local)")
    ap.add_argument("--reuse", type=float, default=0.5)
    ap.add_argument("--eps-local", type=float, default=0.1)
    ap.add_argument("--error-accuracy", action="store_true",
                    help="error-model planner: also measure, at every step after the first, the error each "
                         "cached group state actually carries (a full-cost fresh pass, evaluation only) and "
                         "report how well the predicted errors match it (R^2, Pearson, RMSE, MAE)")
    ap.add_argument("--sweep", action="store_true",
                    help="time the step for each selection of the workload's sweep (long-context workload)")
    ap.add_argument("--attn-workspace", choices=("full", "queue", "none"), default="full",
                    help="workspace of the attention launch: queue counters and tail-split partials (full), "
                         "the queue counters only (balanced, unsplit), or none (static launch)")
    ap.add_argument("--graph", action="store_true",
                    help="time the step as one captured HIP graph (counter reset, attention, merge, weights) "
                         "replayed --steps times; the per-kernel times stay eager")
    ap.add_argument("--no-selection-sweep", dest="selection_sweep", action="store_false",
                    help="skip the step-time-against-selected-fraction points")
    ap.add_argument("--power-seconds", type=float, default=3.0,
                    help="sample socket power and clocks for this long per kernel after timing (0 disables)")
    ap.add_argument("--no-other-workloads", dest="other_workloads", action="store_false",
                    help="default workload: skip the long-context sweep and the planner-driven run that "
                         "the line also carries")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="before timing, run one plain elementwise copy of this many MiB "
                         "(the reference kernel that scales profiler byte counters)")
    return ap.parse_args()


def algorithmic(w, select):
    offs = w.offsets
    q_len = w.q_len
    keys = sum(offs[j + 1] - offs[j] for j in select)
    flops = 4.0 * w.B * w.H * q_len * w.D * keys
    s_state = 2 if w.dtype == "bf16" else 4
    rows = w.B * w.H * q_len
    merge_bytes = w.P * rows * (w.D * s_state + 4) + rows * (w.D * s_state + 4)
    contrib_bytes = (w.P + 1) * rows * 4 + w.P * 4
    return flops, merge_bytes, contrib_bytes


# MFMA utilisation of the same attention build at the same workload, from
# rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE SQ_LDS_BANK_CONFLICT
# (busy fraction = busy cycles / (1024 SIMDs x GRBM cycles / 8 XCDs); clock =
# GRBM cycles / 8 / the traced kernel duration); reported under the same rule.
ATTN_COUNTERS = {"mfma_busy": 0.851, "lds_bank_conflicts": 2269440, "clock_ghz": 1.56}


# HBM bytes per launch of the merge kernel at the default workload (all P
# slots), from the same two counter runs and scaled the same way; reported
# only while merge.hip's build id matches.
MERGE_TRAFFIC = {"build_id": "b8d356210acd6f42", "workload": "videodit_bf16_h40_d128_s75600_p8",
                 "fetch_bytes": 401726.0 * 1024 * 2.0, "write_bytes": 100415.0 * 1024 * 1.0}


def merge_traffic(w):
    from paper_2607_15650_amd import build
    if build.source_id("merge.hip") != MERGE_TRAFFIC["build_id"] or w.name != MERGE_TRAFFIC["workload"]:
        return None
    return MERGE_TRAFFIC["fetch_bytes"] + MERGE_TRAFFIC["write_bytes"]


def attn_mode(ws):
    """How the attention launch runs with this workspace: "static" (none),
    "queue" (balanced over the XCDs) or "split" (balanced, last round split)."""
    if ws is None:
        return "static"
    return "split" if ws.numel() > 256 else "queue"


def attn_kernels(ws, w, select):
    """The kernels of one attention launch: the hand-scheduled kernel at
    D=128, and at D=64 for launches of at least four rounds of 256-row tasks
    (shorter D=64 launches run the compiled kernel)."""
    import torch
    mode = attn_mode(ws)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    tasks = -(-w.q_len // 256) * w.H * w.B * len(select)
    asm = w.D == 128 or tasks >= 4 * cus
    k = f"attn_bf16_asm_kernel<{w.D}>" if asm else f"attn_bf16_kernel<{w.D}>"
    return {"static": k, "queue": f"attn_queue_reset_kernel + {k}",
            "split": f"attn_queue_reset_kernel + {k} + attn_split_fixup_kernel"}[mode]


def attn_counters(w, select, mode):
    return dict(ATTN_COUNTERS) if attn_traffic(w, select, mode) is not None else None


def attn_traffic(w, select, mode):
    """Profiled HBM bytes per attention launch, or None when the kernel build,
    the workload, the selection or the launch mode differs from the one the
    counters were taken on."""
    from paper_2607_15650_amd import build
    if build.source_id("attn_bf16.hip") != ATTN_TRAFFIC["build_id"] or mode != ATTN_TRAFFIC["mode"]:
        return None
    if w.name != ATTN_TRAFFIC["workload"] or tuple(select) != w.select:
        return None
    return ATTN_TRAFFIC["fetch_bytes"] + ATTN_TRAFFIC["write_bytes"]


def cpu_baseline(w, x, select, target_s):
    """The float64 oracle, as it stands, on a bounded sample of query rows of
    the same step; scaled to the whole step by the row fraction.  The heads
    are independent in every oracle function, so the fresh states run one
    head per task in a pool of len(os.sched_getaffinity(0)) threads (NumPy's
    matrix products and exponentials release the interpreter lock), each
    with single-threaded BLAS; the composition and the weights then run over
    all heads at once.  Returns (rows, seconds, seconds per whole step,
    workers)."""
    import concurrent.futures as cf
    import numpy as np
    import oracle
    from fixtures import bf16_round
    from threadpoolctl import threadpool_limits
    offs = w.offsets
    qa, qb = offs[w.q], offs[w.q + 1]
    cvt = (lambda a: bf16_round(a).astype(np.float64)) if w.dtype == "bf16" else (lambda a: a.astype(np.float64))
    K, V = cvt(x["k"]), cvt(x["v"])
    Kp = cvt(x["k_prev"]) if "k_prev" in x else K
    Vp = cvt(x["v_prev"]) if "v_prev" in x else V
    Qall = cvt(x["q"][:, qa:qb])
    Qp_all = cvt(x["q_prev"][:, qa:qb]) if "q_prev" in x else Qall
    rng = np.random.default_rng(w.seed + 99)
    workers = max(1, min(len(os.sched_getaffinity(0)), w.H * w.B))
    sel = [j for j in range(w.P) if j in select]

    def states(Q, Kx, Vx, parts, pool):
        """oracle.partition_state of every partition in `parts`, one head per task."""
        def head(h):
            return [oracle.partition_state(Q[:, :, h:h + 1], Kx[:, offs[j]:offs[j + 1], h:h + 1],
                                           Vx[:, offs[j]:offs[j + 1], h:h + 1], w.scale) for j in parts]
        res = list(pool.map(head, range(w.H)))
        return {j: (np.concatenate([r[i][0] for r in res], axis=2), np.concatenate([r[i][1] for r in res], axis=1))
                for i, j in enumerate(parts)}

    def one(n, pool):
        rows = np.sort(rng.choice(w.q_len, size=n, replace=False))
        Q = Qall[:, rows]
        Qp = Qp_all[:, rows]
        # cached states of the unselected partitions: filled before timing
        cached = states(Qp, Kp, Vp, [j for j in range(w.P) if j not in select], pool)
        t0 = time.perf_counter()
        fresh = states(Q, K, V, sel, pool)
        outs = [fresh[j][0] if j in fresh else cached[j][0] for j in range(w.P)]
        lses = [fresh[j][1] if j in fresh else cached[j][1] for j in range(w.P)]
        out, lse = oracle.merge(outs, lses)
        oracle.contrib(lses, lse)
        return time.perf_counter() - t0

    with threadpool_limits(1), cf.ThreadPoolExecutor(workers) as pool:
        n0 = min(w.q_len, 32)
        t0 = one(n0, pool)
        n = int(min(w.q_len, max(n0, n0 * target_s / max(t0, 1e-3))))
        t = one(n, pool) if n > n0 else t0
    per_step_s = t * w.q_len / n
    return n, t, per_step_s, workers


def cpu_description():
    """The host the oracle baseline ran on: CPU model, logical CPUs this
    process may use, NumPy version and the BLAS libraries NumPy calls (as
    threadpoolctl reports them: library, version, threading layer, threads)."""
    import numpy as np
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:   # pragma: no cover
        pass
    blas = []
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                blas.append({k: i.get(k) for k in ("internal_api", "version", "threading_layer", "num_threads",
                                                   "architecture")})
    except Exception:   # pragma: no cover
        pass
    return {"cpu_model": model, "affinity_cpus": len(os.sched_getaffinity(0)), "numpy": np.__version__,
            "blas": blas}


def device_reference(torch):
    """What this GPU sustains, measured in the same process, as context for
    the roofline fractions (clocks and power limits vary from card to card):
    a stream of independent bf16 MFMAs filling the chip (the library's probe
    kernel), a large bf16 GEMM through torch.matmul and a 1 GiB device copy."""
    from paper_2607_15650_amd import api
    def timed(fn, it):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(it):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / it
    n_wg = 2 * torch.cuda.get_device_properties(0).multi_processor_count
    sink = torch.empty(n_wg * 256, dtype=torch.float32, device="cuda")
    probe_flops = [0.0]

    def probe():
        probe_flops[0] = api.probe_mfma_bf16(n_wg, 20000, sink)
    probe_ms = timed(probe, 5)
    del sink
    n = 8192
    a = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    c = torch.empty(n, n, device="cuda", dtype=torch.bfloat16)
    gemm_ms = timed(lambda: torch.matmul(a, b, out=c), 10)
    del a, b, c
    src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    copy_ms = timed(lambda: dst.copy_(src), 10)
    del src, dst
    return {"bf16_mfma_probe_tflops": probe_flops[0] / (probe_ms * 1e-3) / 1e12,
            "bf16_gemm_8192_tflops": 2 * n ** 3 / (gemm_ms * 1e-3) / 1e12,
            "copy_1gib_gbs": 2 * (1 << 30) / (copy_ms * 1e-3) / 1e9}


def power_during(torch, fn, seconds=3.0):
    """Socket power and XCD (GFX) clocks sampled with amd-smi while fn runs
    back to back for about `seconds`: shows whether a kernel runs at the
    power limit (and at what clock).  None when amd-smi is unavailable."""
    import re
    import shutil
    import subprocess
    import threading
    tool = shutil.which("amd-smi")
    if tool is None:
        return None
    samples, done = [], threading.Event()

    def sampler():
        while not done.is_set():
            try:
                r = subprocess.run([tool, "metric", "-p", "-c"], capture_output=True, text=True, timeout=10)
            except Exception:
                return
            pw = re.findall(r"SOCKET_POWER:\s*([0-9.]+)\s*W", r.stdout)
            clk = re.findall(r"GFX_\d+:\s*\n\s*CLK:\s*([0-9.]+)\s*MHz", r.stdout)
            if pw and clk:
                samples.append((float(pw[0]), [float(c) for c in clk]))
            done.wait(0.2)

    fn()
    torch.cuda.synchronize()
    th = threading.Thread(target=sampler, daemon=True)
    th.start()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(4):
            fn()
        torch.cuda.synchronize()
    done.set()
    th.join(timeout=15)
    use = samples[1:] or samples      # the first sample can predate the load
    if not use:
        return None
    clocks = [c for _, cs in use for c in cs]
    return {"socket_w": sum(p for p, _ in use) / len(use), "gfx_mhz_mean": sum(clocks) / len(clocks),
            "gfx_mhz_min": min(clocks), "gfx_mhz_max": max(clocks), "samples": len(use)}


def planner_result(w, thresholds):
    """Planner-driven run: every query block, w.steps denoising steps; for
    each threshold, anchors compute every partition and other steps the query
    partition plus every partition whose anchor weight exceeds it.  One set of
    evolving inputs serves every threshold and the all-fresh reference.
    Returns, per threshold, the selective attention time, the all-fresh time
    and the drift of the selective output from fresh full attention."""
    import numpy as np
    import torch
    from fixtures import bf16_bits, gen_qkv, gen_evolved
    from paper_2607_15650_amd.planner import AnchorPlanner
    from paper_2607_15650_amd.step import SelectiveAttention

    offs = w.offsets
    blocks = list(range(w.P))
    g = lambda a: torch.from_numpy(bf16_bits(a).view(np.int16)).view(torch.bfloat16).cuda()
    runs = {thr: {"sa": SelectiveAttention(w.B, w.H, w.D, offs, w.scale, torch.bfloat16),
                  "pl": {qb: AnchorPlanner(w.P, qb, w.anchors, thr) for qb in blocks},
                  "t": 0.0, "flops": 0.0, "per_step": []} for thr in thresholds}
    ref = SelectiveAttention(w.B, w.H, w.D, offs, w.scale, torch.bfloat16)
    x = gen_qkv(w, with_prev=False)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    t_full = flops_full = 0.0
    for s in range(w.steps):
        q, k, v = g(x["q"]), g(x["k"]), g(x["v"])
        torch.cuda.synchronize()
        fresh = {}
        for qb in blocks:
            e0, e1 = ev(), ev()
            e0.record()
            fo, _, _ = ref.step(s, qb, q, k, v, [1] * w.P)
            e1.record()
            torch.cuda.synchronize()
            t_full += e0.elapsed_time(e1)
            L = offs[qb + 1] - offs[qb]
            flops_full += 4.0 * w.B * w.H * L * w.D * offs[-1]
            fresh[qb] = fo.float()
        for thr, r in runs.items():
            masks, drift, maxabs = [], [], []
            for qb in blocks:
                mask = r["pl"][qb].select(s)
                L = offs[qb + 1] - offs[qb]
                e0, e1 = ev(), ev()
                e0.record()
                out, _, wp = r["sa"].step(s, qb, q, k, v, mask)
                e1.record()
                torch.cuda.synchronize()
                r["t"] += e0.elapsed_time(e1)
                keys = sum(offs[j + 1] - offs[j] for j in range(w.P) if mask[j])
                r["flops"] += 4.0 * w.B * w.H * L * w.D * keys
                wp_h = wp.cpu().numpy()
                r["pl"][qb].observe(s, wp_h)
                if r["pl"][qb].is_anchor(s):
                    # how far the anchor weights sit from the threshold (the
                    # query partition is selected whatever its weight)
                    m = min(abs(float(wp_h[j]) - thr) for j in range(w.P) if j != qb)
                    r["margin"] = min(r.get("margin", float("inf")), m)
                d = out.float() - fresh[qb]
                drift.append(float(d.norm() / fresh[qb].norm()))
                maxabs.append(float(d.abs().max()))
                masks.append("".join(str(m) for m in mask))
            r["per_step"].append({"step": s, "anchor": s in w.anchors, "masks": masks,
                                  "drift_rel_l2_max": max(drift), "drift_maxabs_max": max(maxabs)})
            print(f"[bench] {w.name} thr {thr} step {s} masks {masks} drift {max(drift):.3e}",
                  file=sys.stderr, flush=True)
        del fresh
        if s + 1 < w.steps:
            x = gen_evolved(w, x, s)
    out = {}
    for thr, r in runs.items():
        out[str(thr)] = {"threshold": thr, "selective_ms_per_step": r["t"] / w.steps,
                         "all_fresh_ms_per_step": t_full / w.steps, "speedup_vs_all_fresh": t_full / r["t"],
                         "computed_fraction": r["flops"] / flops_full,
                         "anchor_weight_margin_min": r.get("margin"),
                         "tflops_selective": r["flops"] / (r["t"] * 1e-3) / 1e12, "per_step": r["per_step"]}
    return {"workload": w.name, "steps": w.steps, "query_blocks": len(blocks), "anchors": list(w.anchors),
            "by_threshold": out,
            "note": "times are the calls of each block's step on the stream (attention, composition, "
                    "weights); each block's step is synchronised to read its weights back for the planner"}


def multistep(args, w):
    """Planner-driven run at one threshold (the workload's or --threshold)."""
    thr = w.threshold
    r = planner_result(w, [thr])
    t = r["by_threshold"][str(thr)]
    res = {
        "metric": METRIC, "value": t["tflops_selective"], "unit": "TFLOP/s", "n_gpus": 1,
        "steps": w.steps, "warmup": 0, "ms_per_step": t["selective_ms_per_step"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic (seeded; each step adds 0.03*N(0,1) to Q, K, V)",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "D": w.D, "S": w.S, "P": w.P,
                   "query_blocks": r["query_blocks"], "anchors": r["anchors"], "threshold": thr},
        "selective_ms_total": t["selective_ms_per_step"] * w.steps,
        "all_fresh_ms_total": t["all_fresh_ms_per_step"] * w.steps,
        "speedup_vs_all_fresh": t["speedup_vs_all_fresh"], "computed_fraction": t["computed_fraction"],
        "per_step": t["per_step"], "note": r["note"],
    }
    print(json.dumps(res), flush=True)


def multistep_error_model(args, w):
    """Error-model planner (groups of 2) on every query block over w.steps
    steps: selective time (planning included), all-fresh time, drift."""
    import numpy as np
    import torch
    from fixtures import bf16_bits, gen_qkv, gen_evolved
    from paper_2607_15650_amd.ase import ErrorModelSelectiveAttention, accuracy_stats
    from paper_2607_15650_amd.step import SelectiveAttention

    offs = w.offsets
    blocks = list(range(w.P))
    g = lambda a: torch.from_numpy(bf16_bits(a).view(np.int16)).view(torch.bfloat16).cuda()
    ems = {qb: ErrorModelSelectiveAttention(w.B, w.H, w.D, offs, qb, 2, w.scale, args.reuse, args.eps_local,
                                            evaluate=args.error_accuracy)
           for qb in blocks}
    pairs = []
    ref = SelectiveAttention(w.B, w.H, w.D, offs, w.scale, torch.bfloat16)
    x = gen_qkv(w, with_prev=False)
    t_sel = t_full = 0.0
    per_step = []
    n_groups = n_computed = 0
    for s in range(w.steps):
        q, k, v = g(x["q"]), g(x["k"]), g(x["v"])
        torch.cuda.synchronize()
        anchors, drift = [], []
        for qb in blocks:
            t0 = time.perf_counter()
            out, _, info = ems[qb].step(s, q, k, v)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            fo, _, _ = ref.step(s, qb, q, k, v, [1] * w.P)
            torch.cuda.synchronize()
            t2 = time.perf_counter()
            t_sel += (t1 - t0) * 1e3
            t_full += (t2 - t1) * 1e3
            anchors.append(int(info["anchor"]))
            if "measured" in info:
                pairs += [(info["ase"][grp], info["measured"][grp]) for grp in info["ase"]]
            n_groups += len(ems[qb].groups)
            n_computed += len(info["compute"])
            d = out.float() - fo.float()
            drift.append(float(d.norm() / fo.float().norm()))
        per_step.append({"step": s, "anchor_blocks": anchors, "drift_rel_l2_max": max(drift)})
        print(f"[bench] step {s} anchors {anchors} drift {max(drift):.3e}", file=sys.stderr, flush=True)
        if s + 1 < w.steps:
            x = gen_evolved(w, x, s)
    res = {
        "metric": METRIC, "value": None, "unit": "TFLOP/s", "n_gpus": 1, "steps": w.steps, "warmup": 0,
        "ms_per_step": t_sel / w.steps, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.dtype, "data": "synthetic (seeded; each step adds 0.03*N(0,1) to Q, K, V)",
        "config": {"workload": w.name, "planner": "error-model", "groups_of": 2, "reuse_target": args.reuse,
                   "eps_local": args.eps_local, "query_blocks": len(blocks)},
        "selective_ms_total": t_sel, "all_fresh_ms_total": t_full, "speedup_vs_all_fresh": t_full / t_sel,
        "computed_group_fraction": n_computed / n_groups, "per_step": per_step,
        "note": "wall-clock per block step including the planner's host work and norm read-backs",
    }
    if args.error_accuracy:
        st = accuracy_stats([p_ for p_, _ in pairs], [m_ for _, m_ in pairs])
        res["error_model_accuracy"] = dict(
            st, data="synthetic", points="every group of every query block at every step after the first",
            predicted="ASE(G,t) = sum_j w(j,t_a) alpha(j) ||OUT_t(loc) - OUT_tc(loc)||",
            measured="w(G,t) ||OUT_t(G) - OUT_tc(G)|| with every partition computed fresh (evaluation only)",
            paper_context="R^2 0.9792, Pearson 0.9899, RMSE 32.46, MAE 21.88 on Wan2.1 activations (other "
                          "models, layers and error units; not a target)")
        res["note"] += "; the selective time includes the evaluation passes"
    print(json.dumps(res), flush=True)


def sweep_result(w, steps, warmup):
    """Step time for each selection of the workload's sweep (nearest-first
    sizes), the other partitions' states read from the cache, and the line
    through step time against the selected fraction."""
    import numpy as np
    import torch
    from fixtures import bf16_bits, gen_qkv
    from paper_2607_15650_amd import api

    offs = w.offsets
    qa, qb = offs[w.q], offs[w.q + 1]
    x = gen_qkv(w, with_prev=True)
    g = lambda a: torch.from_numpy(bf16_bits(np.ascontiguousarray(a)).view(np.int16)).view(torch.bfloat16).cuda()
    q, k, v = g(x["q"][:, qa:qb]), g(x["k"]), g(x["v"])
    qp, kp, vp = g(x["q_prev"][:, qa:qb]), g(x["k_prev"]), g(x["v_prev"])
    del x
    L = w.q_len
    st = torch.empty((w.P, w.B, L, w.H, w.D), dtype=torch.bfloat16, device="cuda")
    ls = torch.empty((w.P, w.B, w.H, L), dtype=torch.float32, device="cuda")
    out = torch.empty((w.B, L, w.H, w.D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((w.B, w.H, L), dtype=torch.float32, device="cuda")
    wp = torch.empty(w.P, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(16, api.contrib_workspace_bytes(w.B, w.H, L, w.P)), dtype=torch.uint8, device="cuda")
    api.attn_partition_states(qp, kp, vp, offs, [1] * w.P, w.scale, st, ls)
    del qp, kp, vp
    rows = []
    for sel in w.sweep:
        mask = [1 if j in sel else 0 for j in range(w.P)]
        n_ws = api.attn_workspace_bytes(torch.bfloat16, w.B, w.H, w.D, L, offs, mask)
        ws_k = torch.empty(n_ws, dtype=torch.uint8, device="cuda") if n_ws > 0 else None

        def step():
            api.attn_partition_states(q, k, v, offs, mask, w.scale, st, ls, ws_k)
            api.merge_states(st, ls, out, lse)
            api.contrib(ls, lse, wp, ws)
        for _ in range(warmup):
            step()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        # the attention call alone: events around it in a second pass
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        for ea, eb in evs:
            ea.record()
            api.attn_partition_states(q, k, v, offs, mask, w.scale, st, ls, ws_k)
            eb.record()
            api.merge_states(st, ls, out, lse)
            api.contrib(ls, lse, wp, ws)
        torch.cuda.synchronize()
        attn_ms = sum(ea.elapsed_time(eb) for ea, eb in evs) / steps
        flops = algorithmic(w, sel)[0]
        rows.append({"k": len(sel), "fraction": len(sel) / w.P, "ms_per_step": ms,
                     "tflops": flops / (ms * 1e-3) / 1e12, "attn_ms": attn_ms,
                     "attn_frac_of_peak": flops / (attn_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS})
        print(f"[bench] {w.name} k={len(sel)} {ms:.3f} ms (attention {attn_ms:.3f} ms)", file=sys.stderr, flush=True)
    res = {"workload": w.name, "steps": steps, "warmup": warmup, "points": rows}
    if len(rows) > 1:
        ks = np.array([r["fraction"] for r in rows])
        ts = np.array([r["ms_per_step"] for r in rows])
        slope, icpt = np.polyfit(ks, ts, 1)
        res["linear_fit_ms"] = {"slope_per_fraction": float(slope), "intercept": float(icpt)}
    return res


def sweep(args, w):
    r = sweep_result(w, args.steps, args.warmup)
    full = r["points"][-1]
    res = {
        "metric": METRIC, "value": full["tflops"], "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": full["ms_per_step"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "D": w.D, "S": w.S, "P": w.P,
                   "query_partition": w.q, "q_len": w.q_len},
        "sweep": r["points"], "linear_fit_ms": r.get("linear_fit_ms"),
    }
    print(json.dumps(res), flush=True)


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from fixtures import bf16_bits, gen_qkv, get_workload
    from paper_2607_15650_amd import api

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)

    w = get_workload(args.workload)
    if args.threshold is not None:
        import dataclasses
        w = dataclasses.replace(w, threshold=args.threshold)
    if w.steps > 1 and args.planner == "error-model":
        return multistep_error_model(args, w)
    if w.steps > 1:
        return multistep(args, w)
    if args.sweep:
        return sweep(args, w)
    select = tuple(int(s) for s in args.select.split(",")) if args.select else w.select
    mask = [1 if j in select else 0 for j in range(w.P)]
    offs = w.offsets
    qa, qb = offs[w.q], offs[w.q + 1]
    q_len = w.q_len

    t_gen = time.perf_counter()
    x = gen_qkv(w, with_prev=True)

    def gpu(a):
        if w.dtype == "bf16":
            return torch.from_numpy(bf16_bits(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()

    q = gpu(np.ascontiguousarray(x["q"][:, qa:qb]))
    k = gpu(x["k"])
    v = gpu(x["v"])
    qp = gpu(np.ascontiguousarray(x["q_prev"][:, qa:qb]))
    kp = gpu(x["k_prev"])
    vp = gpu(x["v_prev"])
    t_gen = time.perf_counter() - t_gen
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32

    out_states = torch.empty((w.P, w.B, q_len, w.H, w.D), dtype=dt, device="cuda")
    lse_states = torch.empty((w.P, w.B, w.H, q_len), dtype=torch.float32, device="cuda")
    out = torch.empty((w.B, q_len, w.H, w.D), dtype=dt, device="cuda")
    lse = torch.empty((w.B, w.H, q_len), dtype=torch.float32, device="cuda")
    w_part = torch.empty(w.P, dtype=torch.float32, device="cuda")
    ws = torch.empty(max(16, api.contrib_workspace_bytes(w.B, w.H, q_len, w.P)), dtype=torch.uint8, device="cuda")
    # workspace of the attention launch: queue counters that balance its
    # last tasks over the XCDs, and room to split the tasks of a partly
    # filled last round over key ranges (None: the static launch)
    def attn_ws(sel_mask):
        if args.attn_workspace == "none":
            return None
        n = api.attn_workspace_bytes(dt, w.B, w.H, w.D, q_len, offs, sel_mask)
        if args.attn_workspace == "queue":
            n = min(n, 256)
        return torch.empty(n, dtype=torch.uint8, device="cuda") if n > 0 else None
    ws_attn = attn_ws(mask)

    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # previous step: every partition's state into the cache (not timed)
    api.attn_partition_states(qp, kp, vp, offs, [1] * w.P, w.scale, out_states, lse_states)
    torch.cuda.synchronize()

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        api.attn_partition_states(q, k, v, offs, mask, w.scale, out_states, lse_states, ws_attn)
        if ev is not None:
            ev[1].record()
        api.merge_states(out_states, lse_states, out, lse)
        if ev is not None:
            ev[2].record()
        api.contrib(lse_states, lse, w_part, ws)
        if ev is not None:
            ev[3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] workload {w.name} select {list(select)} warmup {args.warmup} done", file=sys.stderr, flush=True)

    # pass 1: whole-step wall clock (events only at the ends); with --graph
    # the step is captured once and replayed
    run_step = step
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        run_step = graph.replay
        for _ in range(max(1, args.warmup)):
            run_step()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for _ in range(args.steps):
        run_step()
    stop.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(stop) / args.steps

    # pass 2: per-kernel durations with events between the calls
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    t_attn = sorted(e[0].elapsed_time(e[1]) for e in evs)
    t_merge = sorted(e[1].elapsed_time(e[2]) for e in evs)
    t_contrib = sorted(e[2].elapsed_time(e[3]) for e in evs)
    mean = lambda a: sum(a) / len(a)
    med = lambda a: a[len(a) // 2]

    flops, merge_bytes, contrib_bytes = algorithmic(w, select)
    attn_ms = mean(t_attn)
    merge_ms = mean(t_merge)
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    achieved = flops / (attn_ms * 1e-3) / 1e12
    merge_gbs = merge_bytes / (merge_ms * 1e-3) / 1e9

    # pass 3: the merge alone with a cold cache (a 1 GiB write before each
    # launch evicts the states from L2 and the 256 MB Infinity Cache)
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    t_cold = []
    for i in range(max(3, min(args.steps, 10))):
        flush.fill_(float(i))
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        api.merge_states(out_states, lse_states, out, lse)
        e1.record()
        torch.cuda.synchronize()
        t_cold.append(e0.elapsed_time(e1))
    del flush
    merge_cold_ms = mean(t_cold)

    # step time against the fraction of partitions computed fresh: the same
    # step with nearest-first selections of k partitions (the others reused),
    # and a least-squares line through the points
    from fixtures.workloads import nearest_first
    scaling = None
    if args.selection_sweep and w.P > 1:
        ks = sorted(set([1, 2, len(select), (w.P + 1) // 2, w.P]))
        pts = []
        for kk in ks:
            sel_k = nearest_first(w.P, w.q, kk)
            mask_k = [1 if j in sel_k else 0 for j in range(w.P)]
            ws_k = attn_ws(mask_k)

            def step_k():
                api.attn_partition_states(q, k, v, offs, mask_k, w.scale, out_states, lse_states, ws_k)
                api.merge_states(out_states, lse_states, out, lse)
                api.contrib(lse_states, lse, w_part, ws)
            step_k()
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            n_it = max(3, min(args.steps, 10))
            e0.record()
            for _ in range(n_it):
                step_k()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / n_it
            pts.append({"k": kk, "fraction": kk / w.P, "fresh": list(sel_k), "ms_per_step": ms,
                        "tflops": algorithmic(w, sel_k)[0] / (ms * 1e-3) / 1e12})
        xs = [p_["fraction"] for p_ in pts]
        ys = [p_["ms_per_step"] for p_ in pts]
        mx, my = mean(xs), mean(ys)
        slope = sum((x_ - mx) * (y_ - my) for x_, y_ in zip(xs, ys)) / sum((x_ - mx) ** 2 for x_ in xs)
        scaling = {"points": pts, "linear_fit_ms": {"per_unit_fraction": slope, "intercept": my - slope * mx},
                   "note": "nearest-first selections around the query partition, the other partitions' "
                           "states read from the cache; 10 steps per point"}

    ref = device_reference(torch)
    if w.dtype == "bf16":
        ref["attn_frac_of_probe"] = achieved / ref["bf16_mfma_probe_tflops"]
    # power and clocks while the attention kernel, then the MFMA-only probe,
    # run back to back (after the timed passes, so timing is unaffected)
    n_wg = 2 * torch.cuda.get_device_properties(0).multi_processor_count
    sink = torch.empty(n_wg * 256, dtype=torch.float32, device="cuda")
    if args.power_seconds > 0:
        ref["power"] = {
            "attn_partition_states": power_during(
                torch, lambda: api.attn_partition_states(q, k, v, offs, mask, w.scale, out_states, lse_states,
                                                         ws_attn),
                args.power_seconds),
            "mfma_probe": power_during(torch, lambda: api.probe_mfma_bf16(n_wg, 20000, sink), args.power_seconds),
        }
        # the attention rate against the peak at the clock the card ran the
        # attention launches at (the published peak assumes 2.4 GHz)
        mhz = ref["power"]["attn_partition_states"].get("gfx_mhz_mean") if ref["power"]["attn_partition_states"] else None
        if w.dtype == "bf16" and mhz:
            ref["attn_frac_of_peak_at_sampled_clock"] = achieved / (PEAK_BF16_TFLOPS * mhz / 2400.0)
    del sink

    cpu = None
    if args.cpu_seconds > 0:
        print("[bench] timing the CPU oracle baseline", file=sys.stderr, flush=True)
        n, t, per_step, cores = cpu_baseline(w, x, select, args.cpu_seconds)
        cpu = {"value": flops / per_step / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
               "sample": f"{n} of {q_len} query rows (all {w.H} heads, all keys of the fresh partitions), "
                         f"{t:.2f} s; scaled by {q_len}/{n} to {per_step:.1f} s per step",
               "parallelism": f"fresh states one head per task on {cores} threads, single-threaded BLAS each; "
                              "composition and weights over all heads in one thread"}
        cpu.update(cpu_description())

    res = {
        "metric": METRIC,
        "value": flops / (ms_per_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded N(0,1) plus shared sinusoidal positional component)",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "D": w.D, "S": w.S, "P": w.P,
                   "query_partition": w.q, "q_len": q_len, "fresh_partitions": list(select),
                   "fresh_fraction": len(select) / w.P,
                   "attn_launch": attn_mode(ws_attn), "step_graph": bool(args.graph),
                   "attn_workspace_bytes": int(ws_attn.numel()) if ws_attn is not None else 0},
        "roofline": {"bound": "mfma",
                     "kernel": attn_kernels(ws_attn, w, select) if w.dtype == "bf16" else "attn_f32_kernel",
                     "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
                     "traffic": attn_traffic(w, select, attn_mode(ws_attn)),
                     "counters": attn_counters(w, select, attn_mode(ws_attn))},
        "kernels_ms": {"attn_partition_states": {"mean": attn_ms, "median": med(t_attn)},
                       "merge_states": {"mean": merge_ms, "median": med(t_merge)},
                       "contrib": {"mean": mean(t_contrib), "median": med(t_contrib)}},
        "merge_roofline": {"bound": "hbm", "achieved": merge_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                           "frac": merge_gbs / PEAK_HBM_GBS, "bytes_per_launch": merge_bytes,
                           "traffic": merge_traffic(w),
                           "cold_cache": {"ms": merge_cold_ms,
                                          "achieved": merge_bytes / (merge_cold_ms * 1e-3) / 1e9,
                                          "frac": merge_bytes / (merge_cold_ms * 1e-3) / 1e9 / PEAK_HBM_GBS}},
        "attn_tflops_per_step_flops": flops / 1e12,
        "selection_scaling": scaling,
        "device_reference": ref,
        "cpu_baseline": cpu,
        "input_gen_s": t_gen,
    }
    if args.other_workloads and args.workload == DEFAULT_WORKLOAD:
        res["other_workloads"] = other_workloads()
    print(json.dumps(res), flush=True)


def other_workloads():
    """The other workloads of the hot path, measured in the same run: the
    long-context selection sweep (131,072 tokens, 24 heads, 16 partitions,
    nearest-first fresh sets of 1, 2, 4, 8 and 16 partitions), the
    HunyuanVideo-like head-dim-64 step (118,800 tokens, 48 heads, fresh
    {2,3,4} of 8) and the planner-driven run (75,600 tokens, 40 heads, all 8
    query blocks over 10 steps, anchors at steps 0 and 5) at the specified
    weight threshold 0.05 and at the uniform level 1/8.  Reported beside the
    headline figure, not in it."""
    import dataclasses
    import gc
    import torch
    from fixtures import get_workload
    out = {}
    t0 = time.perf_counter()
    gc.collect()
    torch.cuda.empty_cache()
    print("[bench] other workloads: long-context sweep", file=sys.stderr, flush=True)
    out["longctx_sweep"] = sweep_result(get_workload("longctx_bf16_h24_d128_s131072_p16"), steps=5, warmup=2)
    gc.collect()
    torch.cuda.empty_cache()
    print("[bench] other workloads: head dim 64", file=sys.stderr, flush=True)
    wh = get_workload("hunyuan_bf16_h48_d64_s118800_p8")
    out["hunyuan_d64"] = sweep_result(dataclasses.replace(wh, sweep=(wh.select,)), steps=10, warmup=2)
    gc.collect()
    torch.cuda.empty_cache()
    print("[bench] other workloads: planner-driven run", file=sys.stderr, flush=True)
    r = planner_result(get_workload("planner_bf16_h40_d128_s75600_p8_10steps"), [0.05, 0.125])
    for t in r["by_threshold"].values():
        # the per-step masks of 8 blocks x 10 steps stay in the planner mode's own line
        t["drift_rel_l2_max_by_step"] = [p["drift_rel_l2_max"] for p in t.pop("per_step")]
    out["planner"] = r
    gc.collect()
    torch.cuda.empty_cache()
    out["wall_s"] = time.perf_counter() - t0
    return out


if __name__ == "__main__":
    main()
