"""The quantised-residual check of the GPU parity tests, pinned on the CPU.

``parity.centre_slots`` says which centre each kept entry was sent as; the
GPU parity tests then require residual = fl32(acc - that centre) bit for bit.
Here the same rule is checked on the oracle's own results for every 1-bit
form (Section 5.4 and readings R5, R10): if the helper picked a wrong group,
sign or column, the oracle, whose residuals follow that rule by construction,
would fail it.
"""
import numpy as np
import pytest

import oracle
from parity import bits, centre_slots


@pytest.mark.parametrize("quant", [1, 2, 3, 4])
@pytest.mark.parametrize("per_tensor", [False, True])
def test_oracle_residuals_follow_their_own_centres(quant, per_tensor):
    rng = np.random.default_rng(quant * 10 + per_tensor)
    sizes = [600, 0, 1, 96 * 7, 4 * 33, 0, 250]
    cols = [20, 1, 1, 96, 33, 1, 5]
    off = [0] + np.cumsum(sizes).tolist()
    n = off[-1]
    g = (rng.standard_t(3, n) * 1e-2).astype(np.float32)
    g[rng.random(n) < 0.2] = 0.0
    r = rng.normal(0, 1e-2, n).astype(np.float32)
    o = oracle.compress(g, r, off, 0.9, per_tensor=per_tensor, quant=quant, columns=cols if quant == 4 else None)
    slot = centre_slots(o.idx, o.sign_bits, off, quant, cols if quant == 4 else None)
    want = o.val - o.means.astype(np.float32)[slot]
    assert np.array_equal(bits(o.residual[o.idx]), bits(want))
    # a plausible slip, the wrong sign's centre, is caught
    wrong = o.val - o.means.astype(np.float32)[slot ^ 1]
    assert not np.array_equal(bits(o.residual[o.idx]), bits(wrong))
    if quant == 4:  # and so is taking the column from the row
        t = np.searchsorted(np.asarray(off), o.idx.astype(np.int64), side="right") - 1
        row = (o.idx.astype(np.int64) - np.asarray(off)[t]) // np.asarray(cols)[t]
        colbase = np.concatenate([[0], np.cumsum(cols)])
        bad_slot = 2 * (colbase[t] + row % np.asarray(cols)[t]) + (slot & 1)
        assert not np.array_equal(bits(o.residual[o.idx]), bits(o.val - o.means.astype(np.float32)[bad_slot]))
