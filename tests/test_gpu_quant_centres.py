"""GPU parity of the other 1-bit centres of Section 5.4.

Threshold (every survivor sent as +-T, T the smallest kept magnitude of its
segment), one global average of each sign, and column-wise averages over each
tensor's row-major matrix view: the HIP path through the C ABI against the
oracle on the same bytes.  Indices, sign bits, counts and dropped residuals are
bit-exact; centres and the residuals built from them are within 1e-6 relative
(column sums are fp64 atomics, so their order varies); threshold centres are
bit-exact.
"""
import numpy as np
import pytest
import torch

from paper_1704_05021_amd import gd, workloads as wl
from parity import bits, check_case

pytestmark = pytest.mark.gpu

KINDS = {"threshold": gd.GD_QUANT_THRESHOLD, "global_mean": gd.GD_QUANT_GLOBAL_MEAN,
         "column_mean": gd.GD_QUANT_COLUMN_MEAN}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gd.load()
    torch.cuda.set_device(0)


def divisor_columns(rng, sizes):
    """A column count dividing each size (a random divisor up to 4096)."""
    cols = []
    for n in sizes:
        divs = [d for d in range(1, min(int(n), 4096) + 1) if n % d == 0] if n else [1, 3, 7]
        cols.append(int(rng.choice(divs)))
    return cols


@pytest.mark.parametrize("kind", list(KINDS))
@pytest.mark.parametrize("seed", range(4))
def test_random_layouts(kind, seed):
    rng = np.random.default_rng(300 + seed)
    T = int(rng.integers(1, 7))
    sizes = rng.integers(0, 60_000, T)
    sizes[rng.random(T) < 0.2] = 0
    offsets = [0] + np.cumsum(sizes).tolist()
    if offsets[-1] == 0:
        offsets[-1] = 1
        sizes[-1] = 1
    N = offsets[-1]
    g = (rng.standard_t(3, N) * 10.0 ** rng.uniform(-4, -1)).astype(np.float32)
    r = rng.normal(0, 1e-3, N).astype(np.float32)
    cols = divisor_columns(rng, sizes)
    comp = gd.Compressor(offsets)
    comp.set_columns(cols)
    for per in (False, True):
        for drop in (0.99, 0.9):
            check_case(g, r, offsets, drop, per, KINDS[kind], comp=comp, columns=cols,
                       what=f"{kind} seed={seed} per={per} drop={drop}")


@pytest.mark.parametrize("kind", list(KINDS))
def test_nmt_small_stream(kind):
    """Three carried steps of the scaled NMT stream, teacher-forced, both thresholds."""
    w = wl.workload("nmt_small_per_tensor")
    offsets = w.layout.offsets.astype(np.int64).tolist()
    sizes = np.diff(offsets)
    cols = [int(c) for c in w.layout.columns] if hasattr(w.layout, "columns") else divisor_columns(
        np.random.default_rng(1), sizes)
    comp = gd.Compressor(offsets)
    comp.set_columns(cols)
    for per in (True, False):
        res = np.zeros(w.layout.numel, np.float32)
        for step in range(3):
            o = check_case(w.grad(step), res, offsets, w.drop, per, KINDS[kind], comp=comp, columns=cols,
                           what=f"{kind} per={per} step={step}")
            res = o.residual


def test_threshold_centres_are_the_threshold():
    """The sent centre is +-(the smallest kept magnitude) of the segment, bit for bit."""
    rng = np.random.default_rng(9)
    offsets = [0, 40_000, 40_100, 90_000]
    g = rng.normal(0, 1, 90_000).astype(np.float32)
    r = np.zeros_like(g)
    for per in (False, True):
        o = check_case(g, r, offsets, 0.99, per, gd.GD_QUANT_THRESHOLD, what=f"per={per}")
        for t in range(3):
            a, b = offsets[t], offsets[t + 1]
            kept = o.idx[(o.idx >= a) & (o.idx < b)] if per else o.idx
            if kept.size:
                tmag = np.min(np.abs((g + r)[kept]))
                assert bits(o.means[2 * t:2 * t + 1])[0] == bits(np.array([tmag], np.float32))[0]


def test_full_size_nmt_column_mean():
    """The full NMT-shaped set under a global threshold with column-wise centres (matrices by row)."""
    w = wl.workload("nmt_85k_global_signmean")
    offsets = w.layout.offsets.astype(np.int64).tolist()
    sizes = np.diff(offsets)
    # embeddings 85000 x 500, recurrent 1024 x 500 and 1024 x 1024, biases as one row
    cols = [500 if n % 500 == 0 else 1024 if n % 1024 == 0 else int(n) for n in sizes]
    comp = gd.Compressor(offsets)
    comp.set_columns(cols)
    g = w.grad(0)
    r = (w.grad(1) * np.float32(0.5)).astype(np.float32)
    check_case(g, r, offsets, 0.99, False, gd.GD_QUANT_COLUMN_MEAN, comp=comp, columns=cols, what="nmt column")


def test_set_columns_errors():
    comp = gd.Compressor([0, 10, 10, 25])
    with pytest.raises(gd.GDError):
        comp.set_columns([3, 1, 5])  # 3 does not divide 10
    with pytest.raises(gd.GDError):
        comp.set_columns([0, 1, 5])
    with pytest.raises(gd.GDError):
        comp.set_columns([5, 1, 25])  # 25 does not divide 15
    comp.set_columns([5, 7, 15])  # an empty tensor takes any count
    assert comp.quant_centres(gd.GD_QUANT_COLUMN_MEAN) == 2 * (5 + 7 + 15)
    assert comp.quant_centres(gd.GD_QUANT_THRESHOLD) == 6
    assert comp.quant_centres(gd.GD_QUANT_NONE) == 0
