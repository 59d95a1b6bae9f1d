"""GPU parity of the sampled-threshold mode (Section 4: select on a sample).

The HIP path (``gd_compress_sampled`` through the C ABI) against the oracle's
``gdo_compress_sampled`` on the same bytes, with the same sample positions:
bit-exact on sent indices, values, per-tensor counts and residuals.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1704_05021_amd import gd, workloads as wl
from parity import Result, assert_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gd.load()
    torch.cuda.set_device(0)


def gpu_sampled(comp, grad, residual, drop, per_tensor, sample_ppm, seed, base=None, capacity=None,
                quant=0) -> Result:
    dev = comp.device
    g = torch.from_numpy(np.ascontiguousarray(grad, np.float32)).to(dev)
    r = torch.from_numpy(np.ascontiguousarray(residual, np.float32)).to(dev)
    b = None if base is None else torch.from_numpy(np.ascontiguousarray(base, np.float32)).to(dev)
    o = comp.compress_sampled(g, r, drop, per_tensor=per_tensor, sample_ppm=sample_ppm, seed=seed, base=b,
                              capacity=capacity, quant=quant)
    torch.cuda.synchronize()
    counts = o.tensor_counts[:comp.T].cpu().numpy().view(np.uint32).copy()
    k = int(counts.astype(np.int64).sum())
    res = Result(idx=o.idx[:k].cpu().numpy().view(np.uint32).copy(), val=o.val[:k].cpu().numpy().copy(),
                 residual=r.cpu().numpy(), tensor_counts=counts)
    if quant:
        res.sign_bits = o.sign_bits[:(k + 31) // 32].cpu().numpy().view(np.uint32).copy()
        res.means = o.means[:comp.quant_centres(quant)].cpu().numpy().copy()
    return res


def oracle_sampled(grad, residual, offsets, drop, per_tensor, sample_ppm, seed, base=None, capacity=None, quant=0,
                   columns=None):
    o = oracle.compress_sampled(grad, residual, offsets, drop, per_tensor=per_tensor, sample_ppm=sample_ppm,
                                seed=seed, base=base, capacity=capacity, quant=quant, columns=columns)
    return Result(o.idx, o.val, o.residual, o.tensor_counts, o.sign_bits, o.means)


def check(grad, residual, offsets, drop, per, ppm, seed, base=None, capacity=None, comp=None, what="", quant=0,
          columns=None):
    """comp must already have ``columns`` set when it is passed in with quant 4."""
    if comp is None:
        comp = gd.Compressor(offsets)
        if columns is not None:
            comp.set_columns(columns)
    g = gpu_sampled(comp, grad, residual, drop, per, ppm, seed, base, capacity, quant)
    o = oracle_sampled(grad, residual, offsets, drop, per, ppm, seed, base, capacity, quant, columns)
    assert_parity(g, o, quant, what, offsets=offsets, columns=columns)
    return o


def _values(rng, n, kind):
    if kind == "gauss":
        return rng.normal(0, 1e-2, n).astype(np.float32)
    if kind == "ties":
        levels = np.array([0.0, 0.25, 0.5, 1.0, 1.5, 3.0, 1e-3, 2.0 ** -130], np.float32)
        return (levels[rng.integers(0, levels.size, n)] * np.where(rng.random(n) < 0.5, -1, 1)).astype(np.float32)
    return (rng.standard_t(3, n) * 1e-3).astype(np.float32)


@pytest.mark.parametrize("seed", range(8))
def test_random_layouts(seed):
    rng = np.random.default_rng(1000 + seed)
    T = int(rng.integers(1, 9))
    sizes = rng.integers(0, 300_000, T)
    sizes[rng.random(T) < 0.2] = 0
    offsets = [0] + np.cumsum(sizes).tolist()
    N = offsets[-1]
    if N == 0:
        offsets[-1] = N = 1
    kind = ["gauss", "ties", "heavy"][seed % 3]
    g, r = _values(rng, N, kind), _values(rng, N, kind)
    comp = gd.Compressor(offsets)
    for per in (False, True):
        for ppm, drop in ((1000, 0.99), (20_000, 0.99), (50_000, 0.9), (1_000_000, 0.99)):
            check(g, r, offsets, drop, per, ppm, seed * 7919 + ppm, comp=comp, what=f"{kind} per={per} ppm={ppm}")


@pytest.mark.parametrize("N", [1, 3, 17, 1023, 1024, 1025, 4096 + 5, 70_001])
def test_edge_sizes(N):
    rng = np.random.default_rng(N)
    g, r = _values(rng, N, "gauss"), _values(rng, N, "ties")
    offsets = [0, N // 3, N]
    comp = gd.Compressor(offsets)
    for per in (False, True):
        for drop in (0.99, 0.5, 0.0, 1.0):
            for ppm in (1000, 300_000, 1_000_000):
                check(g, r, offsets, drop, per, ppm, 5, comp=comp, what=f"N={N} per={per} drop={drop} ppm={ppm}")


def test_capacity_overflow():
    rng = np.random.default_rng(5)
    offsets = [0, 200_000, 200_500, 600_000]
    N = offsets[-1]
    g, r = _values(rng, N, "heavy"), _values(rng, N, "gauss")
    comp = gd.Compressor(offsets)
    full = oracle_sampled(g, r, offsets, 0.99, False, 20_000, 9)
    K = full.idx.size
    assert K > 1000
    for per in (False, True):
        for cap in (0, 1, K // 3, K - 1, K, K + 10):
            check(g, r, offsets, 0.99, per, 20_000, 9, capacity=cap, comp=comp, what=f"per={per} cap={cap}")


def test_pull_delta():
    rng = np.random.default_rng(6)
    offsets = [0, 150_000, 400_000]
    N = offsets[-1]
    p0 = rng.normal(0, 0.1, N).astype(np.float32)
    p1 = (p0 + rng.normal(0, 1e-3, N)).astype(np.float32)
    r = _values(rng, N, "gauss") * np.float32(1e-2)
    for per in (False, True):
        check(p1, r, offsets, 0.99, per, 10_000, 3, base=p0, what=f"pull per={per}")


@pytest.mark.parametrize("name", ["nmt_small_per_tensor", "mlp_784_256_256_10_t3_small"])
def test_workload_streams(name):
    """Several steps of a workload stream, teacher-forced from the oracle's residual."""
    w = wl.workload(name)
    offsets = w.layout.offsets.astype(np.int64).tolist()
    comp = gd.Compressor(offsets)
    res = np.zeros(w.layout.numel, np.float32)
    for step in range(3):
        g = w.grad(step)
        o = check(g, res, offsets, w.drop, w.per_tensor, 1000, step, comp=comp, what=f"{name} step {step}")
        res = o.residual


def test_full_size_nmt():
    """The 136,875,744-element NMT-shaped set at the paper's 0.1% sample, both threshold modes."""
    w = wl.workload("nmt_85k_per_tensor")
    offsets = w.layout.offsets.astype(np.int64).tolist()
    comp = gd.Compressor(offsets)
    g = w.grad(0)
    r = (w.grad(1) * np.float32(0.5)).astype(np.float32)
    for per in (True, False):
        check(g, r, offsets, 0.99, per, 1000, 11, capacity=4 * w.layout.numel // 100, comp=comp,
              what=f"nmt full per={per}")


def test_matches_exact_mode_with_full_sample():
    """Every entry sampled and distinct magnitudes: the same result as gd_compress."""
    rng = np.random.default_rng(8)
    offsets = [0, 50_000, 50_001, 130_000]
    N = offsets[-1]
    g = (rng.permutation(np.arange(1, N + 1)) * np.where(rng.random(N) < 0.5, -1, 1)).astype(np.float32)
    r = np.zeros(N, np.float32)
    comp = gd.Compressor(offsets)
    for per in (False, True):
        s = gpu_sampled(comp, g, r, 0.99, per, 1_000_000, 1)
        dev = comp.device
        gg, rr = torch.from_numpy(g).to(dev), torch.from_numpy(r).to(dev)
        o = comp.compress(gg, rr, 0.99, per_tensor=per)
        torch.cuda.synchronize()
        assert np.array_equal(s.idx, o.idx[:o.k].cpu().numpy().view(np.uint32))
        assert np.array_equal(bits32(s.residual), bits32(rr.cpu().numpy()))


def bits32(a):
    return np.ascontiguousarray(a, np.float32).view(np.uint32)


def test_errors():
    comp = gd.Compressor([0, 1000])
    g = torch.zeros(1000, device="cuda")
    r = torch.zeros(1000, device="cuda")
    for ppm in (0, 1_000_001):
        with pytest.raises(gd.GDError):
            comp.compress_sampled(g, r, 0.99, sample_ppm=ppm)
    with pytest.raises(gd.GDError):
        comp.compress_sampled(g, r, 1.5)
    with pytest.raises(gd.GDError):
        comp.compress_sampled(torch.zeros(1001, device="cuda")[1:], r)  # not 16-byte aligned


def test_many_tensors():
    """70,000 small tensors under a per-tensor sampled threshold (one sampler block row per tensor)."""
    rng = np.random.default_rng(70)
    T = 70_000
    sizes = rng.integers(0, 40, T)
    sizes[rng.integers(0, T, 2)] = [30_000, 5_000]
    offsets = [0] + np.cumsum(sizes).tolist()
    N = offsets[-1]
    g, r = _values(rng, N, "heavy"), _values(rng, N, "gauss")
    comp = gd.Compressor(offsets)
    for per in (True, False):
        check(g, r, offsets, 0.9, per, 50_000, 4, comp=comp, what=f"T={T} per={per}")


QUANT = {"sign_mean": gd.GD_QUANT_SIGN_MEAN, "threshold": gd.GD_QUANT_THRESHOLD,
         "global_mean": gd.GD_QUANT_GLOBAL_MEAN, "column_mean": gd.GD_QUANT_COLUMN_MEAN}


def _divisor_columns(rng, sizes):
    cols = []
    for n in sizes:
        divs = [d for d in range(1, min(int(n), 2048) + 1) if n % d == 0] if n else [1, 5]
        cols.append(int(rng.choice(divs)))
    return cols


@pytest.mark.parametrize("kind", list(QUANT))
@pytest.mark.parametrize("seed", range(3))
def test_quantised(kind, seed):
    """Each 1-bit form of Section 5.4 over what the sampled threshold sends, short output buffers included."""
    rng = np.random.default_rng(2000 + seed)
    T = int(rng.integers(1, 7))
    sizes = rng.integers(0, 120_000, T)
    sizes[rng.random(T) < 0.2] = 0
    offsets = [0] + np.cumsum(sizes).tolist()
    if offsets[-1] == 0:
        offsets[-1] = 1
        sizes[-1] = 1
    N = offsets[-1]
    g, r = _values(rng, N, ["gauss", "ties", "heavy"][seed % 3]), _values(rng, N, "gauss")
    q = QUANT[kind]
    cols = _divisor_columns(rng, sizes) if q == gd.GD_QUANT_COLUMN_MEAN else None
    comp = gd.Compressor(offsets)
    if cols is not None:
        comp.set_columns(cols)
    for per in (False, True):
        full = oracle_sampled(g, r, offsets, 0.99, per, 20_000, seed)
        K = full.idx.size
        for ppm, cap in ((1000, None), (20_000, None), (20_000, K // 2), (20_000, 0)):
            check(g, r, offsets, 0.99, per, ppm, seed, capacity=cap, comp=comp, quant=q, columns=cols,
                  what=f"{kind} per={per} ppm={ppm} cap={cap}")


@pytest.mark.parametrize("kind", list(QUANT))
def test_quantised_full_size_nmt(kind):
    """The 136,875,744-element NMT-shaped set, global threshold on a 0.1% sample, each 1-bit form."""
    w = wl.workload("nmt_85k_global_signmean")
    offsets = w.layout.offsets.astype(np.int64).tolist()
    q = QUANT[kind]
    cols = [int(c) for c in w.layout.columns] if q == gd.GD_QUANT_COLUMN_MEAN else None
    comp = gd.Compressor(offsets)
    if cols is not None:
        comp.set_columns(cols)
    g = w.grad(0)
    r = (w.grad(1) * np.float32(0.5)).astype(np.float32)
    check(g, r, offsets, 0.99, False, 1000, 3, capacity=4 * w.layout.numel // 100, comp=comp, quant=q, columns=cols,
          what=f"nmt {kind}")


def test_quantised_errors():
    comp = gd.Compressor([0, 1000])
    g = torch.zeros(1000, device="cuda")
    r = torch.zeros(1000, device="cuda")
    with pytest.raises(gd.GDError):
        comp.compress_sampled(g, r, 0.99, quant=7)
    out = comp.alloc_out(1.0, capacity=100)  # no sign_bits or means
    with pytest.raises(gd.GDError):
        comp.compress_sampled(g, r, 0.99, quant=gd.GD_QUANT_SIGN_MEAN, out=out, capacity=100)


@pytest.mark.parametrize("block", range(2))
def test_random_cases(block):
    """Seeded random cases: 1 to 60 tensors, every value family, sample rates
    from 0.01% to all, short output buffers, pull deltas and 1-bit forms."""
    for case in range(block * 40, (block + 1) * 40):
        rng = np.random.default_rng(20_000 + case)
        T = int(rng.choice([1, 2, 5, 60]))
        sizes = rng.integers(0, int(rng.choice([200, 20_000, 400_000])), T)
        offsets = [0] + np.cumsum(sizes).tolist()
        if offsets[-1] == 0:
            offsets[-1] = 1
            sizes[-1] = 1
        N = offsets[-1]
        kind = ["gauss", "ties", "heavy"][case % 3]
        g, r = _values(rng, N, kind), _values(rng, N, "gauss")
        base = _values(rng, N, "gauss") if rng.random() < 0.2 else None
        drop = float(rng.choice([0.0, 0.5, 0.9, 0.99, 0.999, 1.0]))
        per = bool(rng.random() < 0.5)
        ppm = int(rng.choice([100, 1000, 20_000, 300_000, 1_000_000]))
        q = int(rng.choice([0, 0, 1, 2, 3, 4]))
        cols = _divisor_columns(rng, sizes) if q == gd.GD_QUANT_COLUMN_MEAN else None
        cap = None
        if rng.random() < 0.25:
            full = oracle_sampled(g, r, offsets, drop, per, ppm, case, base)
            cap = int(full.idx.size * rng.uniform(0.0, 0.9))
        comp = gd.Compressor(offsets)
        if cols is not None:
            comp.set_columns(cols)
        check(g, r, offsets, drop, per, ppm, case, base=base, capacity=cap, comp=comp, quant=q, columns=cols,
              what=f"case {case}: N={N} T={T} {kind} drop={drop} per={per} ppm={ppm} q={q} cap={cap} "
                   f"base={base is not None}")
        comp.close()
