"""Helpers for GPU-vs-oracle parity tests (imported by the ``-m gpu`` tests).

The GPU side always goes through the C ABI (``paper_1704_05021_amd.gd``); the
reference side is the CPU oracle.  Both receive the same bytes.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np
import torch

import oracle
from paper_1704_05021_amd import gd

# Tolerance for results whose float reductions may be reordered on the GPU
# (quantisation centres summed in fp64 in a different order).
REL_TOL = 1e-6
QUANT_COLUMN_MEAN = 4


def bits(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


@dataclass
class Result:
    idx: np.ndarray
    val: np.ndarray
    residual: np.ndarray
    tensor_counts: np.ndarray
    sign_bits: Optional[np.ndarray] = None
    means: Optional[np.ndarray] = None


def gpu_compress(comp: gd.Compressor, grad: np.ndarray, residual: np.ndarray, drop: float, per_tensor: bool,
                 quant: bool, base: Optional[np.ndarray] = None, out: Optional[gd.SparseOut] = None) -> Result:
    dev = comp.device
    g = torch.from_numpy(np.ascontiguousarray(grad, np.float32)).to(dev)
    r = torch.from_numpy(np.ascontiguousarray(residual, np.float32)).to(dev)
    b = None if base is None else torch.from_numpy(np.ascontiguousarray(base, np.float32)).to(dev)
    o = comp.compress(g, r, drop, per_tensor=per_tensor, quant=quant, base=b, out=out)
    torch.cuda.synchronize()
    k = o.k
    res = Result(
        idx=o.idx[:k].cpu().numpy().view(np.uint32).copy(),
        val=o.val[:k].cpu().numpy().copy(),
        residual=r.cpu().numpy(),
        tensor_counts=o.tensor_counts[:comp.T].cpu().numpy().view(np.uint32).copy(),
    )
    if quant:
        res.sign_bits = o.sign_bits[:(k + 31) // 32].cpu().numpy().view(np.uint32).copy()
        res.means = o.means[:comp.quant_centres(int(quant))].cpu().numpy().copy()
    return res


def oracle_compress(grad, residual, offsets, drop, per_tensor, quant, base=None, columns=None) -> Result:
    o = oracle.compress(grad, residual, offsets, drop, per_tensor=per_tensor, quant=quant, base=base,
                        columns=columns)
    return Result(o.idx, o.val, o.residual, o.tensor_counts, o.sign_bits, o.means)


def centre_slots(idx: np.ndarray, bits_words: np.ndarray, offsets: Sequence[int], quant: int,
                 columns: Optional[Sequence[int]] = None) -> np.ndarray:
    """Position in the centre array of the centre each kept entry is sent as:
    2 * group + sign bit, where the group is the entry's tensor, or under
    column-wise centres its column (tensor t's columns follow those of the
    tensors before it)."""
    off = np.asarray(offsets, np.int64)
    i = idx.astype(np.int64)
    t = np.searchsorted(off, i, side="right") - 1  # last tensor starting at or before i (skips empty ones)
    if int(quant) == QUANT_COLUMN_MEAN:
        cols = np.asarray(columns if columns is not None else np.ones(off.size - 1), np.int64)
        colbase = np.concatenate([[0], np.cumsum(cols)])
        grp = colbase[t] + (i - off[t]) % cols[t]
    else:
        grp = t
    j = np.arange(idx.size, dtype=np.int64)
    bit = (bits_words[j >> 5].astype(np.int64) >> (j & 31)) & 1
    return 2 * grp + bit


def assert_parity(g: Result, o: Result, quant, what: str = "", offsets: Optional[Sequence[int]] = None,
                  columns: Optional[Sequence[int]] = None) -> None:
    """Bit-exact on indices, values, counts, sign bits and unquantised residuals;
    quantisation centres within REL_TOL of the oracle's.  A quantised kept
    entry's residual is one binary32 subtraction, acc - centre: it must equal
    that subtraction bit for bit, taken with the GPU's own centre of the
    entry's group and sign (so each entry is judged against its own centre).
    ``offsets`` (and ``columns`` for the column-wise centres) are required
    for quantised results."""
    assert g.idx.shape == o.idx.shape, f"{what}: kept {g.idx.size} vs oracle {o.idx.size}"
    if not np.array_equal(g.idx, o.idx):
        bad = np.nonzero(g.idx != o.idx)[0]
        raise AssertionError(f"{what}: {bad.size} index mismatches, first at {bad[0]}: gpu {g.idx[bad[0]]} "
                             f"oracle {o.idx[bad[0]]}")
    assert np.array_equal(bits(g.val), bits(o.val)), f"{what}: kept values differ"
    assert np.array_equal(g.tensor_counts, o.tensor_counts), f"{what}: tensor counts {g.tensor_counts} vs {o.tensor_counts}"
    if not quant:
        if not np.array_equal(bits(g.residual), bits(o.residual)):
            bad = np.nonzero(bits(g.residual) != bits(o.residual))[0]
            raise AssertionError(f"{what}: {bad.size} residual mismatches, first at {bad[0]}: "
                                 f"gpu {g.residual[bad[0]]!r} oracle {o.residual[bad[0]]!r}")
        return
    assert np.array_equal(g.sign_bits, o.sign_bits), f"{what}: sign bits differ"
    m_g, m_o = g.means.astype(np.float64), o.means.astype(np.float64)
    assert np.all(np.abs(m_g - m_o) <= REL_TOL * np.abs(m_o)), f"{what}: centres {m_g} vs {m_o}"
    kept = np.zeros(o.residual.size, bool)
    kept[o.idx] = True
    assert np.array_equal(bits(g.residual[~kept]), bits(o.residual[~kept])), f"{what}: dropped residuals differ"
    assert offsets is not None, "quantised parity needs the layout's offsets"
    slot = centre_slots(g.idx, g.sign_bits, offsets, int(quant), columns)
    want = np.ascontiguousarray(g.val, np.float32) - g.means.astype(np.float32)[slot]  # one binary32 rounding
    got = g.residual[g.idx]
    if not np.array_equal(bits(got), bits(want)):
        bad = np.nonzero(bits(got) != bits(want))[0]
        raise AssertionError(f"{what}: {bad.size} quantised residuals are not fl32(acc - own centre), first at "
                             f"index {g.idx[bad[0]]}: gpu {got[bad[0]]!r}, want {want[bad[0]]!r}")
    if np.array_equal(bits(g.means), bits(o.means)):
        assert np.array_equal(bits(g.residual), bits(o.residual)), f"{what}: equal centres but residuals differ"


def check_case(grad, residual, offsets: Sequence[int], drop: float, per_tensor: bool, quant,
               base=None, comp: Optional[gd.Compressor] = None, debug_bracket: int = 0,
               what: str = "", columns: Optional[Sequence[int]] = None) -> Result:
    """quant: False/True or a GD_QUANT_* form; columns: the matrix view for the column-wise centres
    (``comp`` must already have them set when it is passed in)."""
    if comp is None:
        comp = gd.Compressor(offsets)
        if columns is not None:
            comp.set_columns(columns)
    comp.debug_force_bracket(debug_bracket)
    try:
        g = gpu_compress(comp, grad, residual, drop, per_tensor, quant, base)
    finally:
        comp.debug_force_bracket(0)
    o = oracle_compress(grad, residual, offsets, drop, per_tensor, quant, base, columns)
    assert_parity(g, o, quant, what, offsets=offsets, columns=columns)
    return o
