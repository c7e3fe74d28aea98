"""Seeded input generation: bf16 rounding, reproducibility, workload shapes."""
import numpy as np
import pytest

from fixtures import bf16_bits, bf16_round, gen_qkv, get_workload, sample_rows, WORKLOADS
from fixtures.workloads import Workload, nearest_first, partition_offsets


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 3,
                        np.array([0.0, -0.0, 1e-40, 3.0e38, -1.0000001, 65504.0], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf16_bits(x), ref)
    assert np.array_equal(bf16_round(x), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_workload_shapes():
    w = get_workload("videodit_bf16_h40_d128_s75600_p8")
    assert w.S == 75600 and w.q_len == 9450 and w.offsets[-1] == 75600
    w4 = get_workload("longctx_bf16_h24_d128_s131072_p16")
    assert w4.S == 131072 and w4.q_len == 8192
    assert w4.sweep[0] == (7,) and set(w4.sweep[2]) == {5, 6, 7, 8}
    assert set(w4.sweep[3]) == set(range(3, 11)) and len(w4.sweep[4]) == 16
    assert nearest_first(8, 3, 3) == (3, 2, 4)
    assert get_workload("reuse_bf16_h12_d64_s16384_p8").select_mask() == [0, 0, 1, 1, 1, 0, 0, 0]
    assert partition_offsets(4096, 4) == [0, 1024, 2048, 3072, 4096]


def test_generator_reproducible_and_prev_noise():
    w = Workload(name="t", dtype="bf16", B=1, H=2, D=8, grid=(2, 4, 4), P=2, q=0, seed=5,
                 select=(0,), prev_noise=0.05)
    a = gen_qkv(w)
    b = gen_qkv(w)
    for key in a:
        assert np.array_equal(a[key], b[key])
    d = a["k_prev"] - a["k"]
    assert 0.03 < d.std() < 0.07
    assert a["q"].shape == (1, 32, 2, 8) and a["q"].dtype == np.float32


def test_nearer_tokens_have_larger_positional_similarity():
    """The positional component makes q.k larger at small token distance."""
    w = Workload(name="t", dtype="f32", B=1, H=1, D=64, grid=(8, 8, 8), P=8, q=3, seed=0,
                 select=(3,))
    x = gen_qkv(w)
    q = x["q"][0, :, 0]
    k = x["k"][0, :, 0]
    offs = w.offsets
    qb = q[offs[3]:offs[4]]
    means = [float((qb @ k[offs[j]:offs[j + 1]].T).mean()) for j in range(8)]
    assert means[3] == max(means)
    assert means[3] > means[0] and means[3] > means[7]


def test_sample_rows_includes_boundaries():
    r = sample_rows(9450, 1024, seed=2)
    for must in (0, 1, 63, 64, 127, 128, 9449):
        assert must in r
    assert all(x in r for x in range(9344, 9450))
    assert len(r) >= 1024 and np.all(np.diff(r) > 0)


def test_all_workloads_have_local_partition_selected():
    for w in WORKLOADS.values():
        assert w.q in w.select
