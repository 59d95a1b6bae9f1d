"""GPU parity of the server-side apply of quantised pushes (Sections 3 and 5.4).

Clients' quantised outputs (indices, sign bits, centre pairs) of every kind,
from the oracle, are decoded and applied by gd_apply_quantised through the C
ABI and by the oracle's gdo_apply_quantised: bit-exact (sums in push order
from +0 on both sides).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1704_05021_amd import gd, workloads as wl
from parity import bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gd.load()
    torch.cuda.set_device(0)


def _push(o):
    return (torch.from_numpy(o.idx.view(np.int32)).cuda(),
            torch.from_numpy((o.sign_bits if o.sign_bits.size else np.zeros(1, np.uint32)).view(np.int32)).cuda(),
            torch.from_numpy(o.means).cuda())


def run_case(offsets, grads, quant, lr, columns=None, per_flags=None, what=""):
    N = offsets[-1]
    outs = []
    for c, g in enumerate(grads):
        per = bool(per_flags[c]) if per_flags is not None else bool(c % 2)
        outs.append(oracle.compress(g, np.zeros(N, np.float32), offsets, 0.99, per_tensor=per, quant=quant,
                                    columns=columns))
    p0 = np.random.default_rng(len(grads)).normal(0, 0.1, N).astype(np.float32)
    want = oracle.apply_quantised(p0, offsets, [o.idx for o in outs], [o.sign_bits for o in outs],
                                  [o.means for o in outs], quant, lr, columns=columns)
    comp = gd.Compressor(offsets)
    if columns is not None:
        comp.set_columns(columns)
    pushes = [_push(o) for o in outs]
    p = torch.from_numpy(p0).cuda()
    comp.apply_quantised(p, [x[0] for x in pushes], [x[1] for x in pushes], [x[2] for x in pushes], quant, lr)
    torch.cuda.synchronize()
    got = p.cpu().numpy()
    if not np.array_equal(bits(got), bits(want)):
        bad = np.nonzero(bits(got) != bits(want))[0]
        raise AssertionError(f"{what}: {bad.size} parameters differ, first at {bad[0]}")


@pytest.mark.parametrize("quant", [1, 2, 3, 4])
def test_small_nmt_layout(quant, apply_form):
    w = wl.workload("nmt_small_per_tensor")
    offsets = w.layout.offsets.astype(np.int64).tolist()
    grads = [w.grad(s) for s in range(3)]
    run_case(offsets, grads, quant, 1.0, columns=w.layout.columns if quant == 4 else None, what=f"quant={quant}")


@pytest.mark.parametrize("quant", [1, 4])
def test_random_layout_many_pushes(quant, apply_form):
    rng = np.random.default_rng(40 + quant)
    sizes = [7000, 1, 0, 33_000, 640]
    offsets = [0] + np.cumsum(sizes).tolist()
    columns = [70, 1, 5, 330, 64]
    grads = [(rng.standard_t(3, offsets[-1]) * 1e-2).astype(np.float32) for _ in range(9)]
    run_case(offsets, grads, quant, 0.5, columns=columns if quant == 4 else None, what=f"quant={quant}")


def test_full_nmt_layout_sign_mean(apply_form):
    """Two pushes of the full NMT-shaped layout (1.37M entries each) under a global threshold."""
    w = wl.workload("nmt_85k_global_signmean")
    offsets = w.layout.offsets.astype(np.int64).tolist()
    run_case(offsets, [w.grad(0), w.grad(1)], 1, 1.0, per_flags=[0, 0], what="nmt full")


def test_errors():
    comp = gd.Compressor([0, 100])
    p = torch.zeros(100, device="cuda")
    i = torch.zeros(1, dtype=torch.int32, device="cuda")
    b = torch.zeros(1, dtype=torch.int32, device="cuda")
    m = torch.zeros(2, device="cuda")
    with pytest.raises(gd.GDError):
        comp.apply_quantised(p, [i], [b], [m], 0)  # not a quantised form
