"""GPU parity over seeded random cases: layouts of 1 to 300 tensors and up to
tens of millions of elements, Gaussian, Student-t, row-sparse and tie-heavy
values, every drop ratio from 0 to 1, both threshold scopes, every 1-bit form
and every forced bracket mode, each compared with the oracle at the bar of
the other parity tests (bit-exact, centres within 1e-6)."""
import numpy as np
import pytest
import torch

from paper_1704_05021_amd import gd
from parity import check_case

pytestmark = pytest.mark.gpu

CASES = 600
BLOCKS = 12


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gd.load()
    torch.cuda.set_device(0)


def _case(case):
    rng = np.random.default_rng(10_000 + case)
    T = int(rng.choice([1, 2, 3, 5, 8, 30, 300]))
    scale = int(rng.choice([100, 3000, 30000, 300000]))
    sizes = rng.integers(0, scale, size=T)
    if rng.random() < 0.3:
        sizes[rng.integers(0, T)] = int(rng.choice([0, 1, 1023, 1024, 1025, 4096, 65537, 1 << 20]))
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64).tolist()
    N = offsets[-1]
    if N == 0:
        offsets[-1] = N = 1
        sizes[-1] = 1
    kind = rng.integers(0, 4)
    if kind == 0:
        g = rng.normal(0, 1, N).astype(np.float32)
    elif kind == 1:
        g = (rng.standard_t(3, N) * 10.0 ** rng.uniform(-4, -1)).astype(np.float32)
    elif kind == 2:  # runs of 100 entries, 5% of them nonzero
        g = rng.normal(0, 1e-3, N).astype(np.float32) * (rng.random(N // 100 + 1) < 0.05).repeat(100)[:N]
    else:  # few distinct magnitudes: ties everywhere
        g = rng.choice(np.array([0.0, 0.5, 1.0, -1.0, 2.0 ** -140], np.float32), N)
    r = (rng.normal(0, 1e-3, N) * (rng.random(N) < rng.random())).astype(np.float32)
    drop = float(rng.choice([0.0, 0.5, 0.9, 0.99, 0.999, 0.9999, 1.0]))
    per = bool(rng.random() < 0.5)
    quant = int(rng.choice([0, 0, 1, 2, 3, 4])) if rng.random() < 0.5 else 0
    debug = int(rng.choice([0, 0, 0, 1, 2, 3, 4]))
    columns = None
    if quant == gd.GD_QUANT_COLUMN_MEAN:  # a divisor of each size
        columns = []
        for sz in sizes:
            divs = [d for d in range(1, min(int(sz), 512) + 1) if sz % d == 0] if sz else [1]
            columns.append(int(rng.choice(divs)))
    return offsets, g, r, drop, per, quant, debug, columns


@pytest.mark.parametrize("block", range(BLOCKS))
def test_random_cases(block):
    for case in range(block * CASES // BLOCKS, (block + 1) * CASES // BLOCKS):
        offsets, g, r, drop, per, quant, debug, columns = _case(case)
        comp = gd.Compressor(offsets)
        if columns is not None:
            comp.set_columns(columns)
        check_case(g, r, offsets, drop, per, quant, comp=comp, debug_bracket=debug, columns=columns,
                   what=f"case {case}: N={offsets[-1]} T={len(offsets) - 1} drop={drop} per={per} "
                        f"quant={quant} debug={debug}")
        comp.close()
