"""The bench line's denominators, pinned by hand: the algorithmic flops of
the fresh partitions (4*B*H*q_len*D*sum of their key counts: 2D for the
scores and 2D for P V per query row, key and head) and the merge's
algorithmic bytes (every listed state slot read once, OUT and LSE written
once), at the workload shapes the bench reports; and the rule that profiled
traffic is reported only for the kernel build it was taken on (CPU only)."""
import importlib
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    sys.path.insert(0, ROOT)
    return importlib.import_module("bench")


def test_videodit_flops_and_merge_bytes(bench):
    from fixtures import get_workload
    w = get_workload("videodit_bf16_h40_d128_s75600_p8")
    flops, merge_bytes, contrib_bytes = bench.algorithmic(w, (2, 3, 4))
    # 75,600 tokens in 8 partitions of 9,450; query block 9,450 rows
    assert flops == 4 * 40 * 9450 * 128 * (3 * 9450)
    assert abs(flops - 5.487e12) < 1e9
    # 8 slots of bf16 OUT (256 B per row and head) + float32 LSE, one output
    rows = 40 * 9450
    assert merge_bytes == 8 * rows * (256 + 4) + rows * (256 + 4)
    assert abs(merge_bytes - 884.52e6) < 1e4
    assert contrib_bytes == 9 * rows * 4 + 8 * 4


def test_long_context_and_head_dim_64_flops(bench):
    from fixtures import get_workload
    w = get_workload("longctx_bf16_h24_d128_s131072_p16")
    one = bench.algorithmic(w, (7,))[0]
    assert one == 4 * 24 * 8192 * 128 * 8192              # 0.8246 TFLOP per partition
    assert bench.algorithmic(w, tuple(range(16)))[0] == 16 * one
    h = get_workload("hunyuan_bf16_h48_d64_s118800_p8")
    assert bench.algorithmic(h, (2, 3, 4))[0] == 4 * 48 * 14850 * 64 * (3 * 14850)   # 8.129 TFLOP


def test_profiled_traffic_only_for_its_build(bench, monkeypatch):
    from fixtures import get_workload
    from paper_2607_15650_amd import build
    w = get_workload("videodit_bf16_h40_d128_s75600_p8")
    t = bench.ATTN_TRAFFIC
    monkeypatch.setattr(build, "source_id", lambda name: t["build_id"])
    got = bench.attn_traffic(w, w.select, "queue")
    assert got == t["fetch_bytes"] + t["write_bytes"]
    assert bench.attn_counters(w, w.select, "queue") == bench.ATTN_COUNTERS
    # another launch mode, selection or build: no figures
    assert bench.attn_traffic(w, w.select, "split") is None
    assert bench.attn_traffic(w, (3,), "queue") is None
    monkeypatch.setattr(build, "source_id", lambda name: "0" * 16)
    assert bench.attn_traffic(w, w.select, "queue") is None
    assert bench.attn_counters(w, w.select, "queue") is None

