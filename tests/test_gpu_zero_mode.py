"""Segments with fewer nonzero |acc| than k, HIP path against the oracle.

Such a segment keeps every nonzero entry and then its lowest-index zeros
(Algorithm 1, Section 4: the k largest |acc|, ties to the lower index; here
the threshold is 0).  Under an exact threshold such segments take the zero
mode (no fallback to every element), with or without 1-bit forms.  Results must match the oracle bit for bit: indices, values
(-0 kept as -0), residuals (+0 where sent) and per-tensor counts.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_1704_05021_amd import gd, workloads as wl
from parity import check_case

pytestmark = pytest.mark.gpu

# big sparse tensor, empty tensor, big sparse tensor, tiny dense tensor,
# big sparse tensor; boundaries off the 1024-element units
OFF = [0, 300_001, 300_001, 700_000, 700_100, 1_500_003]
DENSITY = [0.002, 0.0, 0.004, 0.5, 0.001]


def _sparse_inputs(seed: int, density=DENSITY):
    rng = np.random.default_rng(seed)
    n = OFF[-1]
    g = np.zeros(n, np.float32)
    for t, d in enumerate(density):
        a, b = OFF[t], OFF[t + 1]
        nz = rng.random(b - a) < d
        g[a:b][nz] = rng.normal(0.0, 1e-3, int(nz.sum())).astype(np.float32)
    g[(g == 0) & (rng.random(n) < 0.5)] = np.float32(-0.0)  # zeros of both signs
    r = np.zeros(n, np.float32)
    nz = np.nonzero(g)[0]
    cancel = nz[rng.random(nz.size) < 0.2]
    r[cancel] = -g[cancel]  # acc = +0 exactly
    extra = rng.choice(n, 300, replace=False)
    r[extra] = rng.normal(0.0, 1e-3, extra.size).astype(np.float32)
    return g, r


def _segments(comp, per_tensor):
    segs, _ = comp.debug_state()
    return segs if per_tensor else segs[:1]


@pytest.mark.parametrize("drop", [0.99, 0.9])
@pytest.mark.parametrize("per_tensor", [True, False], ids=["per_tensor", "global"])
def test_zero_mode(per_tensor, drop):
    g, r = _sparse_inputs(21)
    comp = gd.Compressor(OFF)
    check_case(g, r, OFF, drop, per_tensor, False, comp=comp, what=f"zero mode per_tensor={per_tensor} drop={drop}")
    segs = _segments(comp, per_tensor)
    if per_tensor:
        assert [s["zero"] for s in segs] == [1, 0, 1, 0, 1]
    else:
        assert segs[0]["zero"] == 1 and segs[0]["thr"] == 0
    assert not any(s["miss"] for s in segs)


def test_zero_mode_with_base():
    g, r = _sparse_inputs(22)
    base = np.zeros_like(g)
    base[::5] = g[::5]  # g - base = 0 there
    comp = gd.Compressor(OFF)
    check_case(g, r, OFF, 0.99, True, False, base=base, comp=comp, what="zero mode with a base")
    assert _segments(comp, True)[0]["zero"] == 1


def test_zero_mode_over_steps():
    # the residual fills in over the steps: from the zero mode to a regular threshold
    rng = np.random.default_rng(23)
    comp = gd.Compressor(OFF)
    r = np.zeros(OFF[-1], np.float32)
    modes = []
    for step in range(4):
        g, _ = _sparse_inputs(30 + step)
        g = g * np.float32(1.0 + 0.1 * rng.random())
        o = check_case(g, r, OFF, 0.99, True, False, comp=comp, what=f"zero mode step {step}")
        modes.append([s["zero"] for s in _segments(comp, True)])
        r = o.residual
    assert modes[0] == [1, 0, 1, 0, 1]


@pytest.mark.parametrize("per_tensor", [True, False], ids=["per_tensor", "global"])
@pytest.mark.parametrize("quant", [gd.GD_QUANT_SIGN_MEAN, gd.GD_QUANT_THRESHOLD, gd.GD_QUANT_GLOBAL_MEAN],
                         ids=["sign_mean", "threshold", "global_mean"])
def test_zero_mode_quantised(quant, per_tensor):
    # kept zeros are positive values (not below zero): they count in the
    # positive centre's average, and under threshold centres T = 0
    g, r = _sparse_inputs(24)
    comp = gd.Compressor(OFF)
    check_case(g, r, OFF, 0.99, per_tensor, quant, comp=comp,
               what=f"zero mode, quant={quant}, per_tensor={per_tensor}")
    segs = _segments(comp, per_tensor)
    assert segs[0]["zero"] == 1 and not any(s["miss"] for s in segs)


@pytest.mark.parametrize("per_tensor", [True, False], ids=["per_tensor", "global"])
def test_zero_mode_column_centres(per_tensor):
    # the column sums are taken over the sent list, kept zeros included
    g, r = _sparse_inputs(26)
    cols = [13, 1, 3, 4, 1]  # 300001 = 23077 x 13, 399999 = 133333 x 3, 100 = 25 x 4
    comp = gd.Compressor(OFF)
    comp.set_columns(cols)
    check_case(g, r, OFF, 0.99, per_tensor, gd.GD_QUANT_COLUMN_MEAN, comp=comp, columns=cols,
               what=f"zero mode, column centres, per_tensor={per_tensor}")
    seg = _segments(comp, per_tensor)[0]
    assert seg["zero"] == 1 and seg["miss"] == 0


@pytest.mark.parametrize("per_tensor", [True, False], ids=["per_tensor", "global"])
def test_zero_mode_pull_from_copy(per_tensor):
    # no residual: acc = p - copy, and a kept zero updates the copy to
    # copy + acc, which turns a -0 copy under a +0 difference into +0
    g, _ = _sparse_inputs(25)
    rng = np.random.default_rng(27)
    copy = np.zeros_like(g)
    copy[rng.random(g.size) < 0.3] = np.float32(-0.0)
    same = rng.random(g.size) < 0.1
    copy[same] = g[same]  # p - copy = +0 there
    comp = gd.Compressor(OFF)
    p_t = torch.from_numpy(g).to(comp.device)
    c_t = torch.from_numpy(copy).to(comp.device)
    out = comp.compress_pull(p_t, c_t, 0.99, per_tensor=per_tensor)
    torch.cuda.synchronize()
    o, o_copy = oracle.compress_pull(g, copy, OFF, 0.99, per_tensor=per_tensor)
    k = out.k
    assert np.array_equal(out.idx[:k].cpu().numpy().view(np.uint32), o.idx)
    assert np.array_equal(out.val[:k].cpu().numpy().view(np.uint32), o.val.view(np.uint32))
    assert np.array_equal(c_t.cpu().numpy().view(np.uint32), o_copy.view(np.uint32))
    assert np.array_equal(out.tensor_counts[:comp.T].cpu().numpy().view(np.uint32), o.tensor_counts)
    assert _segments(comp, per_tensor)[0]["zero"] == 1


@pytest.mark.parametrize("per_tensor", [True, False], ids=["per_tensor", "global"])
def test_zero_mode_full_size_sparse_step(per_tensor):
    w = wl.workload("nmt_85k_per_tensor")
    g = wl.grad_nmt(w.layout, w.seed, 1, tokens=800)
    comp = gd.Compressor(w.layout.offsets)
    check_case(g, np.zeros_like(g), w.layout.offsets, 0.99, per_tensor, False, comp=comp,
               what=f"NMT set, 800 tokens, per_tensor={per_tensor}")
    segs = _segments(comp, per_tensor)
    # per tensor the three embeddings are short of nonzeros; globally the
    # dense tensors supply more than k nonzeros
    assert [s["zero"] for s in segs[:4]] == ([1, 1, 1, 0] if per_tensor else [0])


@pytest.mark.parametrize("quant", [False, gd.GD_QUANT_SIGN_MEAN], ids=["plain", "sign_mean"])
@pytest.mark.parametrize("per_tensor", [True, False], ids=["per_tensor", "global"])
def test_zero_mode_all_zero(per_tensor, quant):
    # tensors with no nonzero entry at all: no candidates and no tiles, so
    # their kept zeros and counts come from the fill alone
    off = [0, 100_000, 100_000, 100_003, 400_000]
    rng = np.random.default_rng(28)
    g = np.where(rng.random(off[-1]) < 0.5, np.float32(-0.0), np.float32(0.0)).astype(np.float32)
    comp = gd.Compressor(off)
    check_case(g, np.zeros_like(g), off, 0.99, per_tensor, quant, comp=comp,
               what=f"all zero, per_tensor={per_tensor}, quant={quant}")
    segs = _segments(comp, per_tensor)
    if per_tensor:
        assert [s["zero"] for s in segs] == [1, 0, 0, 1]  # the 3-element tensor keeps nothing
    else:
        assert segs[0]["zero"] == 1
