"""The seeded input generator: shapes, determinism, storage rounding, recipe."""
import numpy as np

from paper_2609_15030_amd import workloads as wl


def test_bf16_rounding_is_nearest_even():
    # 1 + 2^-8 is halfway between bf16 neighbours 1 and 1 + 2^-7: ties to even (1.0)
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1e-3], np.float32)
    r = wl.round_to_bf16(x)
    assert r[0] == 1.0 and r[1] == 1.0 + 2 ** -6 and r[2] == -2.5
    assert np.array_equal(wl.round_to_bf16(r), r)          # idempotent
    assert np.all(wl.bf16_bits(r).astype(np.uint32) << 16 == r.view(np.uint32))


def test_tiny_fp32_recipe():
    w = wl.tiny_fp32()
    x = w.inputs
    assert x.q.shape == (256, 1, 64) and x.v.shape == (256, 1, 64) and x.g.shape == (256, 1)
    assert w.interval == 16 and x.io_dtype == wl.F32
    assert np.allclose(np.linalg.norm(x.q.astype(np.float64), axis=-1), 1, atol=1e-6)
    assert np.all(x.g < 0) and np.all((x.beta > 0) & (x.beta < 1))
    assert np.array_equal(wl.tiny_fp32().inputs.k, x.k)      # deterministic


def test_bf16_workload_values_are_representable():
    x = wl.tp_rank_3584().inputs
    assert x.q.shape == (3584, 8, 128) and x.io_dtype == wl.BF16
    for a in (x.q, x.k, x.v):
        assert np.array_equal(wl.round_to_bf16(a), a)
    assert np.allclose(np.linalg.norm(x.k.astype(np.float64), axis=-1), 1, atol=1e-2)
    # -softplus(N(0,1)) has mean about -0.81
    assert -0.9 < float(x.g.mean()) < -0.7


def test_varlen_recipe():
    w = wl.batched_varlen(with_data=False)
    lens = np.diff(w.inputs.cu_seqlens)
    assert len(lens) == 16 and np.all(lens % 16 == 0)
    assert np.all((lens >= 1024) & (lens <= 8192))
    assert sorted(w.page_perm.tolist()) == list(range(4096))
    assert set(w.modes) <= {"cold", "complete", "partial"}
    for n, m, k, a in zip(lens, w.modes, w.kept, w.available):
        usable = (n - 1) // 256
        if m == "partial":
            assert 0 <= k < usable and a == k * 256
        elif m == "cold":
            assert a == 0
        else:
            assert a == n


def test_sweep_lengths():
    ws = wl.nine_length_sweep()
    assert [w.inputs.total_tokens for w in ws] == [512 * i for i in range(1, 10)]
