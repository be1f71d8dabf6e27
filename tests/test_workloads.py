"""The seeded input generators: determinism, exact lengths, bf16 rounding."""

import numpy as np
import pytest

from paper_2408_00539_amd import workloads as W


def test_rescale_exact_and_positive():
    rng = np.random.default_rng(0)
    for _ in range(200):
        n = int(rng.integers(1, 40))
        x = rng.lognormal(0, 2, size=n)
        total = int(rng.integers(n, 5000))
        f = W.rescale_lengths(x, total)
        assert f.sum() == total and f.min() >= 1


@pytest.mark.parametrize("index,batch,n,segs_per", [(1, 8, 4096, 16),
                                                    (2, 2, 16384, 48),
                                                    (4, 4, 8192, 32)])
def test_layouts(index, batch, n, segs_per):
    s = W.make_segments(index, index)
    assert s.batch == batch and s.num_segs == batch * segs_per
    assert np.all(np.diff(s.cu_seqlens) == n)
    assert np.all(np.diff(s.cu_segs) >= 1)
    assert set(s.cu_seqlens.tolist()) <= set(s.cu_segs.tolist())
    # alternate query / answer, starting with a query
    for b in range(batch):
        flags = s.seg_is_query[b * segs_per:(b + 1) * segs_per]
        assert flags.tolist() == [1, 0] * (segs_per // 2)


def test_workload0_bounds_and_determinism():
    for seed in range(20):
        s = W.make_segments(0, seed)
        lens = np.diff(s.cu_segs)
        assert s.total <= 320 and s.num_segs == 8
        assert lens[0::2].min() >= 8 and lens[0::2].max() <= 32
        assert lens[1::2].min() >= 16 and lens[1::2].max() <= 48
    a = W.make_workload(0)
    b = W.make_workload(0)
    np.testing.assert_array_equal(a.q, b.q)
    np.testing.assert_array_equal(a.segs.cu_segs, b.segs.cu_segs)
    c = W.make_workload(0, seed=1)
    n = min(len(a.q), len(c.q))
    assert not np.array_equal(a.q[:n], c.q[:n])


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10,
                        np.array([0.0, -0.0, 1.0, 65504.0, 1e-30, -3.3e38],
                                 dtype=np.float32)])
    ours = W.to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy()
    np.testing.assert_array_equal(ours, ref.view(np.uint16))
    back = W.bf16_bits_to_f32(ours)
    np.testing.assert_array_equal(
        back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_dialogue_slices_regenerate():
    s = W.make_segments(0, 0)
    full = W.packed_tensor(0, W.Q, s.cu_seqlens, 1, 64)
    again = W.normal_bf16(0, W.Q, 0, (s.total, 1, 64))
    np.testing.assert_array_equal(full, again)


def test_cache_workload_small_batch_is_prefix():
    w = W.make_workload(3, tensors=False)
    assert w.new_lens.min() >= 64 and w.new_lens.max() <= 512
    assert len(w.new_lens) == 32
    assert np.all(np.diff(w.hist.cu_seqlens) == 8192)
    w2 = W.make_workload(3, tensors=True, batch=1, steps=3)
    assert w2.k_cache.shape == (1, 32, W.CACHE_CAP, 128)
    assert w2.q_dec.shape == (3, 1, 32, 128)
    np.testing.assert_array_equal(w2.new_lens, w.new_lens[:1])
    np.testing.assert_array_equal(
        w2.k_cache[0, :, :8192], W.history_slice(3, W.K_HIST, 0, 32, 8192, 128))
    assert not w2.k_cache[0, :, 8192:].any()


def test_bench_flop_accounting_matches_oracle():
    """bench.py counts useful pairs on its own; it must agree with the
    oracle's count from the dense mask rule."""
    import bench
    import oracle
    for i in (0, 1, 2, 4):
        s = W.make_segments(i, i)
        assert bench.visible_pairs(s) == oracle.visible_pairs(
            s.cu_seqlens, s.cu_segs, s.seg_is_query)
