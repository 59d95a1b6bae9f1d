"""Pins for the CPU oracle: checks that do not re-use the oracle's own code.

Each ``pin_*`` function takes a loaded oracle library and raises
``AssertionError`` when the oracle disagrees with something the paper or the
mathematics fixes:

* hand-worked examples of Algorithm 1 (``golden/hand_examples.json``),
* brute force by full sort on tiny inputs (exhaustive) and on random inputs
  with heavy ties,
* the closed form of k and the kept-count stated for the 784-512-512-10 MLP,
* invariants that hold for any input,
* exact rational arithmetic (``fractions.Fraction``) for the quantisation
  centres and the server apply.

The same functions run against deliberately broken builds of the oracle in
``test_oracle_mutants.py``: every planted mistake must trip at least one pin.
"""
from __future__ import annotations

import itertools
import json
import math
import os
from fractions import Fraction
from typing import Dict, List, Sequence, Tuple

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hand_examples.json")


def f32(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float32)


def bits(a) -> np.ndarray:
    return f32(a).view(np.uint32)


def keys(a) -> np.ndarray:
    return bits(a) & np.uint32(0x7FFFFFFF)


# ---------------------------------------------------------------------------
# brute force: full sort by (|acc| descending, index ascending)
# ---------------------------------------------------------------------------

def brute_keep(acc: np.ndarray, offsets: Sequence[int], keep_ppm: int, per_tensor: bool) -> np.ndarray:
    """Keep mask from a full sort; magnitudes compared as Python floats (finite inputs)."""
    keep = np.zeros(acc.size, dtype=bool)
    segs = [(offsets[t], offsets[t + 1]) for t in range(len(offsets) - 1)] if per_tensor else [(0, acc.size)]
    for a, b in segs:
        n = b - a
        k = n * keep_ppm // 1_000_000
        order = sorted(range(a, b), key=lambda i: (-abs(float(acc[i])), i))
        keep[order[:k]] = True
    return keep


def check_against_brute(lib, grad, residual, offsets, keep_ppm, per_tensor):
    drop = 1.0 - keep_ppm / 1e6
    acc = f32(grad) + f32(residual)
    out = oracle.compress(grad, residual, offsets, drop, per_tensor=per_tensor, lib=lib)
    keep = brute_keep(acc, offsets, keep_ppm, per_tensor)
    want_idx = np.nonzero(keep)[0].astype(np.uint32)
    assert np.array_equal(out.idx, want_idx), (out.idx, want_idx)
    assert np.array_equal(bits(out.val), bits(acc[want_idx]))
    want_res = np.where(keep, np.float32(0.0), acc).astype(np.float32)
    assert np.array_equal(bits(out.residual), bits(want_res))
    T = len(offsets) - 1
    want_counts = [int(keep[offsets[t]:offsets[t + 1]].sum()) for t in range(T)]
    assert list(out.tensor_counts) == want_counts


# ---------------------------------------------------------------------------
# invariants (hold for every input)
# ---------------------------------------------------------------------------

def check_invariants(acc: np.ndarray, offsets, keep_ppm: int, per_tensor: bool, idx, val, residual, counts):
    """Properties any correct exact-k gradient drop must satisfy (finite or not)."""
    N = acc.size
    segs = [(offsets[t], offsets[t + 1]) for t in range(len(offsets) - 1)] if per_tensor else [(0, N)]
    idx = np.asarray(idx, dtype=np.int64)
    assert np.all(np.diff(idx) > 0), "indices must be strictly ascending"
    kept = np.zeros(N, dtype=bool)
    kept[idx] = True
    kk = keys(acc)
    k_total = 0
    for a, b in segs:
        n = b - a
        k = n * keep_ppm // 1_000_000
        k_total += k
        seg_kept = kept[a:b]
        assert int(seg_kept.sum()) == k, "kept count must equal k"
        if 0 < k < n:
            kmin = kk[a:b][seg_kept].min()
            kmax = kk[a:b][~seg_kept].max()
            assert kmin >= kmax, "a dropped |value| exceeds a kept one"
            if kmin == kmax:  # ties at the threshold: kept ones come first
                tie = np.nonzero(kk[a:b] == kmin)[0]
                tk = seg_kept[tie]
                assert np.all(tk[:int(tk.sum())]) and not np.any(tk[int(tk.sum()):]), "ties not by lower index"
    assert idx.size == k_total
    assert int(np.asarray(counts, dtype=np.int64).sum()) == k_total
    # sent + residual == acc, bit for bit
    assert np.array_equal(bits(val), bits(acc[idx]))
    assert np.all(bits(residual)[kept] == 0), "kept residual must be +0.0"
    assert np.array_equal(bits(residual)[~kept], bits(acc)[~kept])


# ---------------------------------------------------------------------------
# exact rational helpers
# ---------------------------------------------------------------------------

def ulp32(x: np.float32) -> Fraction:
    x = np.float32(abs(x))
    up = np.nextafter(x, np.float32(np.inf))
    return Fraction(float(up)) - Fraction(float(x))


def within_half_ulp(got: np.float32, exact: Fraction) -> bool:
    g = Fraction(float(np.float32(got)))
    return abs(g - exact) <= ulp32(np.float32(got)) / 2 * Fraction(1000001, 1000000)


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------

def pin_keep_count(lib):
    # the 784-512-512-10 MLP gradient (669,706 entries) keeps 6,697 at a 99% drop
    assert oracle.keep_count(669_706, 0.99, lib) == 6_697
    # closed form floor(n * (1 - R)) in exact arithmetic for decimal drop ratios
    for n in (0, 1, 7, 8, 99, 100, 101, 12345, 37_000_000, 42_500_000):
        for r in ("0", "0.5", "0.9", "0.99", "0.999", "0.625", "1"):
            want = math.floor(n * (1 - Fraction(r)))
            assert oracle.keep_count(n, float(r), lib) == want, (n, r)
    # R = 1/3 is quantised to 666,667 parts per million of kept entries
    assert oracle.keep_count(6, 1 / 3, lib) == 4
    assert oracle.keep_count(3_000_000, 1 / 3, lib) == 2_000_001


def pin_golden_compress(lib):
    with open(GOLDEN) as f:
        gold = json.load(f)
    for case in gold["compress"]:
        res = None
        for st in case["steps"]:
            r_in = res if st["residual_in"] == "previous" else f32(st["residual_in"])
            out = oracle.compress(f32(st["grad"]), r_in, case["offsets"], case["drop"],
                                  per_tensor=case.get("per_tensor", False), quant=case.get("quant", False), lib=lib)
            assert out.idx.tolist() == st["idx"], (case["name"], out.idx)
            assert np.array_equal(bits(out.val), bits(st["val"])), case["name"]
            assert np.array_equal(bits(out.residual), bits(st["residual_out"])), (case["name"], out.residual)
            assert out.tensor_counts.tolist() == st["tensor_counts"], case["name"]
            if "sign_bits" in st:
                assert out.sign_bits.tolist() == st["sign_bits"], case["name"]
                assert np.array_equal(bits(out.means), bits(st["means"])), case["name"]
            res = out.residual


def pin_golden_apply(lib):
    with open(GOLDEN) as f:
        gold = json.load(f)
    for case in gold["apply"]:
        p0 = f32(case["params"])
        idx = [np.array(pi, np.uint32) for pi, _ in case["pushes"]]
        val = [f32(pv) for _, pv in case["pushes"]]
        p1 = oracle.apply_sparse(p0, idx, val, case["lr"], lib=lib)
        assert np.array_equal(bits(p1), bits(case["params_out"])), (case["name"], p1)
        if "pull" in case:
            pl = case["pull"]
            out = oracle.compress(p1, np.zeros_like(p1), [0, p1.size], pl["drop"], base=p0, lib=lib)
            assert out.idx.tolist() == pl["idx"]
            assert np.array_equal(bits(out.val), bits(pl["val"]))
            assert np.array_equal(bits(out.residual), bits(pl["residual_out"]))


def pin_brute_exhaustive(lib):
    """Every vector of length <= 4 over {0, -0, +-1, +-2}, and every vector of
    length 5 to 7 over {0, -0, +1, -1} (ties and signed zeros everywhere), with
    every k."""
    for alphabet, sizes in (([0.0, -0.0, 1.0, -1.0, 2.0, -2.0], range(1, 5)), ([0.0, -0.0, 1.0, -1.0], range(5, 8))):
        for n in sizes:
            z = np.zeros(n, np.float32)
            for vec in itertools.product(alphabet, repeat=n):
                g = f32(vec)
                for k in range(n + 1):
                    # smallest ppm giving exactly k of n
                    ppm = -(-k * 1_000_000 // n)
                    check_against_brute(lib, g, z, [0, n], ppm, False)


def pin_brute_random_ties(lib):
    rng = np.random.default_rng(12345)
    for trial in range(60):
        T = int(rng.integers(1, 6))
        sizes = rng.integers(0, 400, size=T)
        if trial % 7 == 0:
            sizes[rng.integers(0, T)] = 0
        offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64).tolist()
        N = offsets[-1]
        if N == 0:
            continue
        levels = f32([0.0, 0.25, 0.5, 1.0, 1.5, 3.0, 1e-3, 2.0 ** -130])
        g = levels[rng.integers(0, levels.size, N)] * np.where(rng.random(N) < 0.5, -1, 1).astype(np.float32)
        r = (levels[rng.integers(0, levels.size, N)] * np.where(rng.random(N) < 0.5, -1, 1)).astype(np.float32)
        r[rng.random(N) < 0.5] = 0.0
        ppm = int(rng.choice([0, 1_000, 10_000, 100_000, 333_334, 500_000, 900_000, 1_000_000]))
        per = bool(trial % 2)
        check_against_brute(lib, g, r, offsets, ppm, per)
        out = oracle.compress(g, r, offsets, 1 - ppm / 1e6, per_tensor=per, lib=lib)
        check_invariants(g + r, offsets, ppm, per, out.idx, out.val, out.residual, out.tensor_counts)


def pin_invariants_large(lib):
    """Gaussian and heavy-tailed draws at a 99% drop, several tensors, both modes."""
    rng = np.random.default_rng(7)
    offsets = [0, 50_000, 50_017, 120_000, 120_000, 200_003]
    N = offsets[-1]
    g = (rng.standard_t(3, N) * 1e-3).astype(np.float32)
    r = (rng.normal(0, 1e-3, N)).astype(np.float32)
    for per in (False, True):
        out = oracle.compress(g, r, offsets, 0.99, per_tensor=per, lib=lib)
        check_invariants(g + r, offsets, 10_000, per, out.idx, out.val, out.residual, out.tensor_counts)


def pin_special_cases(lib):
    rng = np.random.default_rng(3)
    g = rng.normal(0, 1, 1000).astype(np.float32)
    r = rng.normal(0, 1, 1000).astype(np.float32)
    acc = g + r
    # R = 0 keeps everything, residual all +0
    out = oracle.compress(g, r, [0, 1000], 0.0, lib=lib)
    assert out.idx.tolist() == list(range(1000)) and np.all(bits(out.residual) == 0)
    # R = 1 keeps nothing, residual is acc
    out = oracle.compress(g, r, [0, 1000], 1.0, lib=lib)
    assert out.idx.size == 0 and np.array_equal(bits(out.residual), bits(acc))
    # one tensor: per-tensor equals global
    a = oracle.compress(g, r, [0, 1000], 0.9, per_tensor=False, lib=lib)
    b = oracle.compress(g, r, [0, 1000], 0.9, per_tensor=True, lib=lib)
    assert np.array_equal(a.idx, b.idx) and np.array_equal(bits(a.residual), bits(b.residual))
    # all zeros: the lowest indices are kept
    z = np.zeros(100, np.float32)
    out = oracle.compress(z, z, [0, 100], 0.9, lib=lib)
    assert out.idx.tolist() == list(range(10))
    # equal magnitudes with random signs: indices 0..k-1
    s = np.where(rng.random(100) < 0.5, -0.75, 0.75).astype(np.float32)
    out = oracle.compress(s, z, [0, 100], 0.95, lib=lib)
    assert out.idx.tolist() == list(range(5))
    # Inf above finite, NaN above Inf; +-Inf tie by index
    v = f32([1.0, np.inf, np.nan, -np.inf, 2.0])
    out = oracle.compress(v, np.zeros(5, np.float32), [0, 5], 0.6, lib=lib)
    assert out.idx.tolist() == [1, 2]
    out = oracle.compress(v, np.zeros(5, np.float32), [0, 5], 0.4, lib=lib)
    assert out.idx.tolist() == [1, 2, 3]
    # signed zeros: -0 + -0 = -0 keeps its sign bit; -0 + +0 = +0
    gz = f32([-0.0, 0.0, -0.0])
    rz = f32([-0.0, -0.0, 0.0])
    out = oracle.compress(gz, rz, [0, 3], 0.6666, lib=lib)  # keep_ppm 333400 -> k = 1
    assert out.idx.tolist() == [0] and bits(out.val).tolist() == [0x80000000]
    assert bits(out.residual).tolist() == [0, 0, 0]
    # denormals survive the add and the copy
    d = f32([2.0 ** -149, -(2.0 ** -148), 2.0 ** -140, 0.0])
    out = oracle.compress(d, d, [0, 4], 0.5, lib=lib)
    assert out.idx.tolist() == [1, 2]
    assert np.array_equal(bits(out.val), bits(f32([-(2.0 ** -147), 2.0 ** -139])))
    assert np.array_equal(bits(out.residual), bits(f32([2.0 ** -148, 0, 0, 0])))


def pin_quant_exact(lib):
    """Sign-mean centres and residuals against exact rational arithmetic."""
    rng = np.random.default_rng(11)
    offsets = [0, 700, 701, 1500, 1500, 2600]
    N = offsets[-1]
    for trial in range(6):
        g = (rng.standard_t(3, N) * 10.0 ** rng.uniform(-4, 0)).astype(np.float32)
        r = rng.normal(0, 1e-3, N).astype(np.float32)
        per = bool(trial % 2)
        out = oracle.compress(g, r, offsets, 0.9, per_tensor=per, quant=True, lib=lib)
        acc = g + r
        k = out.idx.size
        first = 0
        for t in range(len(offsets) - 1):
            last = first + int(out.tensor_counts[t])
            v = out.val[first:last]
            assert np.array_equal(bits(v), bits(acc[out.idx[first:last]]))
            pos = [Fraction(float(x)) for x in v if not (x < 0)]
            neg = [Fraction(float(x)) for x in v if x < 0]
            mp, mn = out.means[2 * t], out.means[2 * t + 1]
            assert mp >= 0 >= mn
            if pos:
                assert within_half_ulp(mp, sum(pos) / len(pos)), (t, mp)
            else:
                assert bits([mp])[0] == 0
            if neg:
                assert within_half_ulp(mn, sum(neg) / len(neg)), (t, mn)
            else:
                assert bits([mn])[0] == 0
            for q in range(first, last):
                neg_q = bool(out.val[q] < 0)
                bit = (int(out.sign_bits[q >> 5]) >> (q & 31)) & 1
                assert bit == int(neg_q)
                centre = mn if neg_q else mp
                res = out.residual[out.idx[q]]
                assert within_half_ulp(res, Fraction(float(out.val[q])) - Fraction(float(centre)))
            first = last
        assert first == k
        # bits beyond k are zero
        if k % 32:
            assert int(out.sign_bits[-1]) >> (k % 32) == 0
        # dropped residuals untouched by quantisation
        dropped = np.ones(N, bool)
        dropped[out.idx] = False
        assert np.array_equal(bits(out.residual[dropped]), bits(acc[dropped]))


def _check_sign_bits(out, k):
    for q in range(k):
        bit = (int(out.sign_bits[q >> 5]) >> (q & 31)) & 1
        assert bit == int(bool(out.val[q] < 0))
    if k % 32:
        assert int(out.sign_bits[-1]) >> (k % 32) == 0


def _exact_avg(vals):
    return sum(Fraction(float(x)) for x in vals) / len(vals)


def pin_quant_other_centres(lib):
    """Threshold, global-average and column-wise centres (Section 5.4) against exact arithmetic."""
    rng = np.random.default_rng(12)
    offsets = [0, 700, 701, 1500, 1500, 2600]
    columns = [7, 1, 17, 3, 11]  # each divides its tensor's size (799 = 17 * 47)
    T, N = len(offsets) - 1, offsets[-1]
    tensor_of = np.searchsorted(np.array(offsets[1:]), np.arange(N), side="right")
    for trial in range(6):
        g = (rng.standard_t(3, N) * 10.0 ** rng.uniform(-4, 0)).astype(np.float32)
        r = rng.normal(0, 1e-3, N).astype(np.float32)
        acc = g + r
        per = bool(trial % 2)
        # threshold: +-(smallest kept magnitude of the segment)
        out = oracle.compress(g, r, offsets, 0.9, per_tensor=per, quant=2, lib=lib)
        k = out.idx.size
        _check_sign_bits(out, k)
        kt = tensor_of[out.idx]
        for t in range(T):
            seg = (kt == t) if per else np.ones(k, bool)
            if seg.any():
                tmag = np.min(np.abs(out.val[seg]))
                assert bits([out.means[2 * t]])[0] == bits([tmag])[0]
                assert bits([out.means[2 * t + 1]])[0] == bits([-tmag])[0]
            else:
                assert bits(out.means[2 * t:2 * t + 2]).tolist() == [0, 0]
        for q in range(k):
            c = out.means[2 * kt[q] + int(out.val[q] < 0)]
            assert within_half_ulp(out.residual[out.idx[q]], Fraction(float(out.val[q])) - Fraction(float(c)))
        # global average: one pair over every kept entry
        out = oracle.compress(g, r, offsets, 0.9, per_tensor=per, quant=3, lib=lib)
        k = out.idx.size
        _check_sign_bits(out, k)
        pos = [x for x in out.val if not (x < 0)]
        neg = [x for x in out.val if x < 0]
        for t in range(T):
            mp, mn = out.means[2 * t], out.means[2 * t + 1]
            assert within_half_ulp(mp, _exact_avg(pos)) if pos else bits([mp])[0] == 0
            assert within_half_ulp(mn, _exact_avg(neg)) if neg else bits([mn])[0] == 0
        assert np.all(bits(out.means[0::2]) == bits(out.means[0])) and np.all(bits(out.means[1::2]) == bits(out.means[1]))
        # column-wise average
        out = oracle.compress(g, r, offsets, 0.9, per_tensor=per, quant=4, columns=columns, lib=lib)
        k = out.idx.size
        _check_sign_bits(out, k)
        colbase = np.concatenate([[0], np.cumsum(columns)])
        assert out.means.size == 2 * colbase[-1]
        col = np.array([colbase[t] + (int(i) - offsets[t]) % columns[t] for i, t in zip(out.idx, tensor_of[out.idx])],
                       dtype=np.int64)
        for c in range(colbase[-1]):
            v = out.val[col == c]
            pos = [x for x in v if not (x < 0)]
            neg = [x for x in v if x < 0]
            mp, mn = out.means[2 * c], out.means[2 * c + 1]
            assert within_half_ulp(mp, _exact_avg(pos)) if pos else bits([mp])[0] == 0
            assert within_half_ulp(mn, _exact_avg(neg)) if neg else bits([mn])[0] == 0
        for q in range(k):
            cq = out.means[2 * col[q] + int(out.val[q] < 0)]
            assert within_half_ulp(out.residual[out.idx[q]], Fraction(float(out.val[q])) - Fraction(float(cq)))
        dropped = np.ones(N, bool)
        dropped[out.idx] = False
        assert np.array_equal(bits(out.residual[dropped]), bits(acc[dropped]))


def pin_quant_column_limits(lib):
    """One column per tensor is the per-tensor sign mean; one column per entry sends every value exactly."""
    rng = np.random.default_rng(13)
    offsets = [0, 900, 960, 2000]
    N = offsets[-1]
    g = rng.normal(0, 1, N).astype(np.float32)
    r = rng.normal(0, 0.1, N).astype(np.float32)
    for per in (False, True):
        a = oracle.compress(g, r, offsets, 0.95, per_tensor=per, quant=1, lib=lib)
        b = oracle.compress(g, r, offsets, 0.95, per_tensor=per, quant=4, columns=[1, 1, 1], lib=lib)
        assert np.array_equal(bits(a.means), bits(b.means)) and np.array_equal(bits(a.residual), bits(b.residual))
        sizes = [offsets[t + 1] - offsets[t] for t in range(3)]
        c = oracle.compress(g, r, offsets, 0.95, per_tensor=per, quant=4, columns=sizes, lib=lib)
        assert np.all(bits(c.residual[c.idx]) == 0), "a column of one kept value sends it exactly"
        assert np.array_equal(bits(c.val), bits((g + r)[c.idx]))


def pin_pull_copy(lib):
    """Pulls from the last pulled copy (Section 4): the delta sent and what the copy becomes."""
    rng = np.random.default_rng(14)
    offsets = [0, 3000, 3005, 8000]
    N = offsets[-1]
    copy0 = rng.normal(0, 0.1, N).astype(np.float32)
    p = (copy0 * (1 + rng.normal(0, 1e-2, N))).astype(np.float32)  # within a factor 2: p - copy is exact
    for per in (False, True):
        out, copy1 = oracle.compress_pull(p, copy0, offsets, 0.99, per_tensor=per, lib=lib)
        # the sent part is Algorithm 1 on the delta (the exact mode, pinned by brute force)
        ref = oracle.compress(p, np.zeros(N, np.float32), offsets, 0.99, per_tensor=per, base=copy0, lib=lib)
        assert np.array_equal(out.idx, ref.idx) and np.array_equal(bits(out.val), bits(ref.val))
        # Sterbenz: the delta is exact, so the client (copy + sent) holds p exactly where sent
        assert np.array_equal(bits(copy1[out.idx]), bits(p[out.idx]))
        unsent = np.ones(N, bool)
        unsent[out.idx] = False
        assert np.array_equal(bits(copy1[unsent]), bits(copy0[unsent]))
    # scales far apart: the client holds copy + fl32(p - copy), which is not p
    c = f32([1.0, 1.0, -2.0, 3.0])
    q = f32([1e-8, 5.0, -2.0 - 2.0 ** -22, 3.0])
    out, c1 = oracle.compress_pull(q, c, [0, 4], 0.5, lib=lib)  # k = 2: |delta| 4.0 and 1.0 - 1e-8
    assert out.idx.tolist() == [0, 1]
    assert bits(out.val).tolist() == bits(f32([-1.0, 4.0])).tolist()  # 1e-8 - 1 rounds to -1
    assert bits(c1).tolist() == bits(f32([0.0, 5.0, -2.0, 3.0])).tolist()
    # a delta of -0 is sent as -0 (no residual is added to it)
    out, _ = oracle.compress_pull(f32([-0.0, 1.0]), f32([0.0, 0.0]), [0, 2], 0.0, lib=lib)
    assert bits(out.val).tolist() == [0x80000000, bits(f32([1.0]))[0]]
    # pulling a fixed p repeatedly at 50% drains the difference (Sterbenz holds)
    cc = copy0.copy()
    for _ in range(40):
        _, cc = oracle.compress_pull(p, cc, offsets, 0.5, lib=lib)
    assert np.array_equal(bits(cc), bits(p))


def pin_apply_quantised(lib):
    """Quantised pushes decode to the centres each client subtracted (its error feedback), then sum as R6."""
    rng = np.random.default_rng(15)
    offsets = [0, 1200, 1210, 3000]
    columns = [40, 10, 179]  # each divides its tensor (1790 = 10 * 179)
    N = offsets[-1]
    for quant in (1, 2, 3, 4):
        cols = columns if quant == 4 else None
        pushes = []
        for c in range(3):
            g = (rng.standard_t(3, N) * 1e-2).astype(np.float32)
            out = oracle.compress(g, np.zeros(N, np.float32), offsets, 0.9, per_tensor=bool(c % 2), quant=quant,
                                  columns=cols, lib=lib)
            pushes.append((g, out))
        decoded = []
        for g, out in pushes:
            # one push on p = 0 with lr = -1 leaves exactly the decoded values at the pushed indices
            d = oracle.apply_quantised(np.zeros(N, np.float32), offsets, [out.idx], [out.sign_bits], [out.means],
                                       quant, -1.0, columns=cols, lib=lib)[out.idx]
            # the client kept acc - centre as its residual: the decode must give that centre back
            assert np.array_equal(bits(out.val - d), bits(out.residual[out.idx])), quant
            decoded.append(d)
        p0 = rng.normal(0, 0.1, N).astype(np.float32)
        got = oracle.apply_quantised(p0, offsets, [o.idx for _, o in pushes], [o.sign_bits for _, o in pushes],
                                     [o.means for _, o in pushes], quant, 0.5, columns=cols, lib=lib)
        want = oracle.apply_sparse(p0, [o.idx for _, o in pushes], decoded, 0.5, lib=lib)
        assert np.array_equal(bits(got), bits(want)), quant


def pin_apply_exact(lib):
    rng = np.random.default_rng(5)
    n = 5000
    p = rng.normal(0, 0.1, n).astype(np.float32)
    # no duplicates, lr = 1: one rounding, p - v
    ix = np.sort(rng.choice(n, 300, replace=False)).astype(np.uint32)
    v = (rng.standard_t(3, 300) * 1e-3).astype(np.float32)
    got = oracle.apply_sparse(p, [ix], [v], 1.0, lib=lib)
    want = p.copy()
    want[ix] = p[ix] - v
    assert np.array_equal(bits(got), bits(want))
    # duplicates across 4 clients: within a few ulps of the exact rational result
    idx, val = [], []
    for c in range(4):
        ixc = np.sort(rng.choice(400, 120, replace=False)).astype(np.uint32)
        idx.append(ixc)
        val.append((rng.standard_t(3, 120) * 1e-3).astype(np.float32))
    lr = np.float32(0.5)
    got = oracle.apply_sparse(p, idx, val, float(lr), lib=lib)
    exact: Dict[int, Fraction] = {}
    for ixc, vc in zip(idx, val):
        for i, x in zip(ixc.tolist(), vc.tolist()):
            exact[i] = exact.get(i, Fraction(0)) + Fraction(x)
    touched = np.zeros(n, bool)
    for i, s in exact.items():
        touched[i] = True
        want = Fraction(float(p[i])) - Fraction(float(lr)) * s
        tol = 8 * ulp32(np.float32(abs(float(p[i])) + float(lr) * sum(abs(float(vc[j])) for ixc, vc in zip(idx, val)
                                                                 for j in np.nonzero(ixc == i)[0])))
        assert abs(Fraction(float(got[i])) - want) <= tol, i
    assert np.array_equal(bits(got[~touched]), bits(p[~touched]))


def pin_pull_delta(lib):
    rng = np.random.default_rng(9)
    p0 = rng.normal(0, 0.1, 3000).astype(np.float32)
    p1 = p0.copy()
    ix = rng.choice(3000, 200, replace=False)
    p1[ix] -= rng.normal(0, 1e-2, 200).astype(np.float32)
    res = rng.normal(0, 1e-4, 3000).astype(np.float32)
    delta = p1 - p0
    a = oracle.compress(p1, res, [0, 3000], 0.99, base=p0, lib=lib)
    b = oracle.compress(delta, res, [0, 3000], 0.99, lib=lib)
    assert np.array_equal(a.idx, b.idx) and np.array_equal(bits(a.residual), bits(b.residual))
    assert np.any(delta != 0)
    # a 99% drop of the delta keeps the 30 largest |delta + residual|
    acc = delta + res
    check_invariants(acc, [0, 3000], 10_000, False, a.idx, a.val, a.residual, a.tensor_counts)


# ---------------------------------------------------------------------------
# sampled threshold (Section 4: selection on a 0.1% sample, keep above it)
# ---------------------------------------------------------------------------

SPLITMIX = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "splitmix64.json")


def segments_of(offsets, per_tensor, N):
    return [(offsets[t], offsets[t + 1]) for t in range(len(offsets) - 1)] if per_tensor else [(0, N)]


def sampled_keep_brute(acc, offsets, keep_ppm, per_tensor, sample_ppm, seed, lib):
    """Keep mask of the sampled mode: the sample's threshold by a full numpy sort.

    Positions come from the oracle's generator (pinned separately against the
    published SplitMix64 outputs and the stratum property); the selection on
    the sample and the strict keep rule are recomputed here by brute force.
    """
    N = acc.size
    kk = keys(acc)
    keep = np.zeros(N, dtype=bool)
    for s, (a, b) in enumerate(segments_of(offsets, per_tensor, N)):
        n = b - a
        if n == 0 or keep_ppm == 0:
            continue
        m = -(-n * sample_ppm // 1_000_000)
        sk = np.sort(np.array([kk[oracle.sample_position(0 if seed is None else seed, s, a, n, m, j, lib=lib)]
                               for j in range(m)], dtype=np.int64))[::-1]
        km = m * keep_ppm // 1_000_000
        if km >= m:
            keep[a:b] = True
        else:
            keep[a:b] = kk[a:b] > sk[km]
    return keep


def pin_splitmix64_reference(lib):
    """The position generator reproduces SplitMix64's published outputs."""
    with open(SPLITMIX) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        got = [oracle.splitmix64(case["seed"], i, lib=lib) for i in range(len(case["outputs"]))]
        assert got == [int(x) for x in case["outputs"]], (case["seed"], got)


def pin_sample_positions(lib):
    """One position per stratum [floor(j n/m), floor((j+1) n/m)); a full sample is every entry once."""
    for (a, n, m, seed) in [(0, 1000, 10, 1), (17, 12345, 13, 2), (5, 7, 7, 3), (0, 100, 3, 4), (9, 2 ** 31, 4, 5)]:
        pos = [oracle.sample_position(seed, 3, a, n, m, j, lib=lib) for j in range(m)]
        for j, p in enumerate(pos):
            assert a + j * n // m <= p < a + (j + 1) * n // m, (a, n, m, j, p)
    pos = [oracle.sample_position(9, 0, 4, 50, 50, j, lib=lib) for j in range(50)]
    assert pos == list(range(4, 54))
    # the offsets within strata are spread, not a fixed column
    pos = [oracle.sample_position(11, 0, 0, 100_000, 100, j, lib=lib) - j * 1000 for j in range(100)]
    assert len(set(pos)) > 80


def pin_sampled_full_sample_is_exact(lib):
    """Every entry sampled and distinct magnitudes: the sampled mode keeps exactly the k largest."""
    rng = np.random.default_rng(21)
    offsets = [0, 3000, 3001, 7000, 7000, 10_000]
    g = rng.permutation(np.arange(1, 10_001, dtype=np.float32)) * np.where(rng.random(10_000) < 0.5, -1, 1)
    g = g.astype(np.float32)
    r = np.zeros(10_000, np.float32)
    for per in (False, True):
        for drop in (0.99, 0.9, 0.5, 0.0, 1.0):
            a = oracle.compress_sampled(g, r, offsets, drop, per_tensor=per, sample_ppm=1_000_000, seed=5, lib=lib)
            keep = brute_keep(g, offsets, oracle.keep_ppm(drop, lib=lib), per)
            assert np.array_equal(a.idx, np.nonzero(keep)[0].astype(np.uint32)), (per, drop)
            assert np.array_equal(bits(a.residual), bits(np.where(keep, np.float32(0), g)))


def pin_sampled_brute(lib):
    """Partial samples with heavy ties: selection on the sample and the strict rule by full sort."""
    rng = np.random.default_rng(22)
    for trial in range(12):
        T = int(rng.integers(1, 5))
        sizes = rng.integers(0, 4000, T)
        offsets = [0] + np.cumsum(sizes).tolist()
        N = offsets[-1]
        if N == 0:
            continue
        g = (rng.integers(-6, 7, N) * 0.25).astype(np.float32)
        r = (rng.integers(-2, 3, N) * 0.125).astype(np.float32)
        acc = g + r
        per = bool(trial % 2)
        ppm = int(rng.choice([2_000, 50_000, 300_000]))
        drop = float(rng.choice([0.99, 0.9, 0.7]))
        seed = int(rng.integers(0, 2 ** 63))
        out = oracle.compress_sampled(g, r, offsets, drop, per_tensor=per, sample_ppm=ppm, seed=seed, lib=lib)
        keep = sampled_keep_brute(acc, offsets, oracle.keep_ppm(drop, lib=lib), per, ppm, seed, lib)
        assert np.array_equal(out.idx, np.nonzero(keep)[0].astype(np.uint32)), trial
        assert np.array_equal(bits(out.val), bits(acc[keep]))
        assert np.array_equal(bits(out.residual), bits(np.where(keep, np.float32(0), acc)))
        assert list(out.tensor_counts) == [int(keep[offsets[t]:offsets[t + 1]].sum()) for t in range(T)]


def pin_sampled_capacity(lib):
    """A short output buffer sends the first entries; the rest stay in the residual."""
    rng = np.random.default_rng(23)
    offsets = [0, 40_000, 41_000, 100_000]
    g = rng.normal(0, 1, 100_000).astype(np.float32)
    r = rng.normal(0, 1, 100_000).astype(np.float32)
    acc = g + r
    full = oracle.compress_sampled(g, r, offsets, 0.99, per_tensor=False, sample_ppm=20_000, seed=3, lib=lib)
    K = full.idx.size
    assert K > 100
    for cap in (0, 1, K // 3, K - 1, K, K + 5):
        out = oracle.compress_sampled(g, r, offsets, 0.99, per_tensor=False, sample_ppm=20_000, seed=3,
                                      capacity=cap, lib=lib)
        c = min(cap, K)
        assert np.array_equal(out.idx, full.idx[:c])
        assert int(np.asarray(out.tensor_counts, np.int64).sum()) == c
        sent = np.zeros(acc.size, bool)
        sent[full.idx[:c]] = True
        assert np.array_equal(bits(out.residual), bits(np.where(sent, np.float32(0), acc)))


def pin_sampled_quant_full_sample_is_exact(lib):
    """Every entry sampled and distinct magnitudes: each 1-bit form under the sampled threshold is the exact one."""
    rng = np.random.default_rng(24)
    offsets = [0, 3000, 3001, 7000, 7000, 10_000]
    columns = [30, 1, 43, 9, 100]  # 3999 = 3 * 31 * 43
    g = rng.permutation(np.arange(1, 10_001, dtype=np.float32)) * np.where(rng.random(10_000) < 0.5, -1, 1)
    g = (g * np.float32(1e-3)).astype(np.float32)
    r = np.zeros(10_000, np.float32)
    for per in (False, True):
        for quant in (1, 2, 3, 4):
            cols = columns if quant == 4 else None
            a = oracle.compress_sampled(g, r, offsets, 0.9, per_tensor=per, sample_ppm=1_000_000, seed=2, lib=lib,
                                        quant=quant, columns=cols)
            b = oracle.compress(g, r, offsets, 0.9, per_tensor=per, quant=quant, columns=cols, lib=lib)
            assert np.array_equal(a.idx, b.idx) and np.array_equal(bits(a.val), bits(b.val)), (per, quant)
            assert np.array_equal(bits(a.means), bits(b.means)), (per, quant)
            assert np.array_equal(a.sign_bits, b.sign_bits), (per, quant)
            assert np.array_equal(bits(a.residual), bits(b.residual)), (per, quant)


def pin_sampled_quant_sent_entries(lib):
    """Under the sampled threshold and a short output buffer, centres, sign bits and error feedback cover exactly
    the entries sent (exact arithmetic); the threshold centre is the smallest sent magnitude."""
    rng = np.random.default_rng(25)
    offsets = [0, 2000, 2001, 5001]
    columns = [40, 1, 60]
    T, N = len(offsets) - 1, offsets[-1]
    tensor_of = np.searchsorted(np.array(offsets[1:]), np.arange(N), side="right")
    g = (rng.standard_t(3, N) * 1e-3).astype(np.float32)
    r = rng.normal(0, 1e-3, N).astype(np.float32)
    acc = g + r
    for per in (False, True):
        full = oracle.compress_sampled(g, r, offsets, 0.95, per_tensor=per, sample_ppm=100_000, seed=9, lib=lib)
        K = full.idx.size
        assert K > 40
        cap = K * 2 // 3
        for quant in (1, 2, 3, 4):
            out = oracle.compress_sampled(g, r, offsets, 0.95, per_tensor=per, sample_ppm=100_000, seed=9,
                                          capacity=cap, lib=lib, quant=quant, columns=columns if quant == 4 else None)
            k = out.idx.size
            assert k == cap and np.array_equal(out.idx, full.idx[:cap])
            _check_sign_bits(out, k)
            kt = tensor_of[out.idx]
            if quant == 4:
                colbase = np.concatenate([[0], np.cumsum(columns)])
                grp = np.array([colbase[t] + (int(i) - offsets[t]) % columns[t] for i, t in zip(out.idx, kt)])
                G = int(colbase[-1])
            elif quant == 3:
                grp, G = np.zeros(k, np.int64), 1
            else:
                grp, G = kt.astype(np.int64), T
            for q in range(k):
                c = out.means[2 * (kt[q] if quant == 3 else grp[q]) + int(out.val[q] < 0)]
                assert within_half_ulp(out.residual[out.idx[q]], Fraction(float(out.val[q])) - Fraction(float(c)))
            if quant == 2:
                for t in range(T):
                    seg = (kt == t) if per else np.ones(k, bool)
                    if seg.any():
                        assert bits([out.means[2 * t]])[0] == bits([np.min(np.abs(out.val[seg]))])[0]
            else:
                for gi in range(G):
                    v = out.val[grp == gi]
                    pos = [x for x in v if not (x < 0)]
                    neg = [x for x in v if x < 0]
                    mp, mn = out.means[2 * gi], out.means[2 * gi + 1]
                    assert within_half_ulp(mp, _exact_avg(pos)) if pos else bits([mp])[0] == 0
                    assert within_half_ulp(mn, _exact_avg(neg)) if neg else bits([mn])[0] == 0
            unsent = np.ones(N, bool)
            unsent[out.idx] = False
            assert np.array_equal(bits(out.residual[unsent]), bits(acc[unsent])), (per, quant)


def pin_sampled_statistics(lib):
    """On iid data the kept fraction tracks 1 - R; entries above the sample maximum when k_m = 0."""
    rng = np.random.default_rng(24)
    N = 2_000_000
    g = rng.standard_t(3, N).astype(np.float32)
    r = np.zeros(N, np.float32)
    out = oracle.compress_sampled(g, r, [0, N], 0.99, sample_ppm=1000, seed=77, lib=lib)
    # m = 2000 samples, k_m = 20: the kept fraction is Beta(m - 20, 21)-like, mean ~1.05%
    assert 0.004 * N < out.idx.size < 0.02 * N, out.idx.size
    kk = keys(g + r)
    assert kk[out.idx].min() > kk[np.setdiff1d(np.arange(N), out.idx)].max()
    # 50 samples at 1% keep: k_m = 0, the threshold is the largest sample key
    n = 50_000
    out = oracle.compress_sampled(g[:n], r[:n], [0, n], 0.99, sample_ppm=1000, seed=4, lib=lib)
    smax = max(int(kk[oracle.sample_position(4, 0, 0, n, 50, j, lib=lib)]) for j in range(50))
    assert np.array_equal(out.idx, np.nonzero(kk[:n] > smax)[0].astype(np.uint32))
    # R = 1 keeps nothing, R = 0 keeps everything
    assert oracle.compress_sampled(g[:n], r[:n], [0, n], 1.0, sample_ppm=1000, lib=lib).idx.size == 0
    assert oracle.compress_sampled(g[:n], r[:n], [0, n], 0.0, sample_ppm=1000, lib=lib).idx.size == n


ALL_PINS = [
    pin_keep_count,
    pin_golden_compress,
    pin_golden_apply,
    pin_brute_random_ties,
    pin_invariants_large,
    pin_special_cases,
    pin_quant_exact,
    pin_quant_other_centres,
    pin_quant_column_limits,
    pin_apply_exact,
    pin_pull_copy,
    pin_apply_quantised,
    pin_pull_delta,
    pin_splitmix64_reference,
    pin_sample_positions,
    pin_sampled_full_sample_is_exact,
    pin_sampled_brute,
    pin_sampled_capacity,
    pin_sampled_statistics,
    pin_sampled_quant_full_sample_is_exact,
    pin_sampled_quant_sent_entries,
    pin_brute_exhaustive,  # last: the slowest pin (about 10 s)
]
