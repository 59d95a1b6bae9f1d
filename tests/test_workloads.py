"""CPU checks of the seeded input generators against the recipe they follow: the
layouts, sizes and keep counts of the five configurations, the structure of the
NMT-shaped set (whole embedding rows zero or drawn, dense tensors drawn), the
per-tensor scales of the Student-t MLP, the server shard's pushes, and that the
same seed gives the same bytes.  No GPU needed."""
import numpy as np
import pytest

import oracle
from paper_1704_05021_amd import workloads as wl


def test_layout_sizes_and_keep_counts():
    mnist = wl.workload("mnist_mlp_784_512_512_10").layout
    assert mnist.offsets.tolist() == [0, 401408, 401920, 664064, 664576, 669696, 669706]
    assert oracle.keep_count(mnist.numel, 0.99) == 6697  # the MNIST-shaped config's k
    mlp = wl.workload("mlp_784_4096_4096_10_t3").layout
    assert mlp.offsets.tolist() == [0, 3211264, 3215360, 19992576, 19996672, 20037632, 20037642]
    assert oracle.keep_count(mlp.numel, 0.99) == 200376
    nmt = wl.workload("nmt_85k_per_tensor").layout
    assert nmt.numel == 136_875_744 and nmt.num_tensors == 27
    assert nmt.shapes[:3] == ((85000, 500),) * 3
    assert sum(oracle.keep_count(n, 0.99) for n in nmt.sizes) == 1_368_750  # per tensor
    assert oracle.keep_count(nmt.numel, 0.99) == 1_368_757                  # global
    assert oracle.keep_count(wl.SHARD_FULL["n"], 0.99) == 370_000


def test_nmt_rows_are_whole_and_scaled():
    w = wl.workload("nmt_small_per_tensor")
    g = w.grad(0)
    off = w.layout.offsets.astype(np.int64)
    for t, shape in enumerate(w.layout.shapes):
        x = g[off[t]:off[t + 1]]
        if t < 3:  # an embedding: each row all zero or all drawn
            rows = x.reshape(shape)
            nz = np.count_nonzero(rows, axis=1)
            assert set(np.unique(nz).tolist()) <= {0, shape[1]}
            hit = int(np.count_nonzero(nz))
            assert 0 < hit <= 140  # at most one row per token drawn
            # Zipf: the most frequent words (lowest ranks) are always hit
            assert nz[0] == shape[1]
        else:
            assert np.count_nonzero(x) == x.size
        v = x[x != 0].astype(np.float64)
        # N(0, 1e-3): sample mean and spread within five standard errors
        assert abs(v.mean()) < 5 * 1e-3 / np.sqrt(v.size)
        assert abs(v.std() - 1e-3) < 5 * 1e-3 / np.sqrt(2 * v.size)


def test_nmt_full_size_row_count():
    # 3,000 Zipf(1.1) tokens over 85,000 ranks hit on the order of a thousand distinct rows
    w = wl.workload("nmt_85k_per_tensor")
    rng = wl.rng_for(w.seed, 0, 0)
    cdf = wl.zipf_cdf(85000, 1.1)
    rows = np.unique(np.minimum(np.searchsorted(cdf, rng.random(3000), side="right"), 84999))
    assert 900 <= rows.size <= 1500


def test_student_t_scales_fixed_per_tensor():
    w = wl.workload("mlp_784_256_256_10_t3_small")
    scales = wl.tensor_scales_loguniform(w.layout, w.seed)
    assert np.all((scales >= 1e-4) & (scales <= 1e-2))
    g0, g1 = w.grad(0), w.grad(1)
    assert not np.array_equal(g0, g1)  # a new draw each step, the same scales
    off = w.layout.offsets.astype(np.int64)
    big = int(np.argmax(w.layout.sizes))
    for g in (g0, g1):
        x = g[off[big]:off[big + 1]].astype(np.float64) / scales[big]
        # StudentT(3): median |x| is about 0.765
        assert 0.7 < np.median(np.abs(x)) < 0.83


def test_server_shard_pushes():
    s = wl.server_shard(**wl.SHARD_SMALL)
    n, nnz = wl.SHARD_SMALL["n"], wl.SHARD_SMALL["nnz"]
    assert s.params.dtype == np.float32 and s.params.size == n
    seen = np.zeros(0, np.int64)
    for c, (ix, v) in enumerate(zip(s.idx, s.val)):
        assert ix.dtype == np.uint32 and v.dtype == np.float32 and ix.size == v.size == nnz
        assert np.all(np.diff(ix.astype(np.int64)) > 0) and int(ix[-1]) < n  # ascending, unique, in the shard
        shared = np.intersect1d(ix.astype(np.int64), seen).size
        assert shared == (0 if c == 0 else round(0.05 * nnz))
        seen = np.union1d(seen, ix.astype(np.int64))
    with pytest.raises(ValueError):
        wl.server_shard(n=2, clients=3, nnz=1, dup_frac=0.0, seed=1)


def test_same_seed_same_bytes():
    w = wl.workload("nmt_small_per_tensor")
    assert np.array_equal(w.grad(2).view(np.uint32), w.grad(2).view(np.uint32))
    a, b = wl.server_shard(**wl.SHARD_SMALL), wl.server_shard(**wl.SHARD_SMALL)
    assert all(np.array_equal(x, y) for x, y in zip(a.idx, b.idx))
    assert np.array_equal(a.params.view(np.uint32), b.params.view(np.uint32))
