"""CPU oracle for gradient dropping: TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  The product path (the HIP library and its
Python binding) never imports it.

The arithmetic lives in ``oracle.cpp`` (plain single-threaded C++ using
``std::nth_element``); this module builds it with g++ and marshals numpy
arrays through ctypes.  See ``oracle.cpp`` for the passages of the paper each
step follows and for the readings taken where the paper is silent.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import tempfile
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_LIB = os.path.join(_HERE, "libgdoracle.so")
CXXFLAGS = ["-O2", "-std=c++17", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared"]

_lib_cache = {}


def build(out: Optional[str] = None, defines: Sequence[str] = (), extra_flags: Sequence[str] = ()) -> str:
    """Compile the oracle with g++ into ``out`` (default: next to the source);
    ``extra_flags`` are added to the g++ line (e.g. sanitizers, for a test build)."""
    out = out or _LIB
    tmp = out + f".tmp{os.getpid()}"
    cmd = ["g++", *CXXFLAGS, *extra_flags, *[f"-D{d}" for d in defines], _SRC, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def _declare(lib: ctypes.CDLL) -> ctypes.CDLL:
    u64, u32, i32, dbl, f32 = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int, ctypes.c_double, ctypes.c_float
    vp = ctypes.c_void_p
    lib.gdo_keep_ppm.argtypes = [dbl]
    lib.gdo_keep_ppm.restype = u64
    lib.gdo_keep_count.argtypes = [u64, dbl]
    lib.gdo_keep_count.restype = u64
    lib.gdo_compress.argtypes = [vp, vp, vp, vp, u32, dbl, i32, i32, vp, vp, vp, vp, vp, u64, ctypes.POINTER(u64),
                                 vp]
    lib.gdo_compress.restype = i32
    lib.gdo_apply_sparse.argtypes = [vp, u64, u32, vp, vp, vp, f32]
    lib.gdo_apply_sparse.restype = i32
    lib.gdo_apply_quantised.argtypes = [vp, vp, u32, vp, u32, vp, vp, vp, vp, i32, f32]
    lib.gdo_apply_quantised.restype = i32
    lib.gdo_compress_pull.argtypes = [vp, vp, vp, u32, dbl, i32, vp, vp, vp, u64, ctypes.POINTER(u64)]
    lib.gdo_compress_pull.restype = i32
    lib.gdo_splitmix64.argtypes = [u64, u64]
    lib.gdo_splitmix64.restype = u64
    lib.gdo_sample_position.argtypes = [u64, u32, u64, u64, u64, u64]
    lib.gdo_sample_position.restype = u64
    lib.gdo_compress_sampled.argtypes = [vp, vp, vp, vp, u32, dbl, i32, u32, u64, i32, vp, vp, vp, vp, vp, u64,
                                         ctypes.POINTER(u64), vp]
    lib.gdo_compress_sampled.restype = i32
    return lib


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load the oracle library, building it first if it is missing or stale."""
    path = path or _LIB
    if path in _lib_cache:
        return _lib_cache[path]
    if path == _LIB and (not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC)):
        build(path)
    lib = _declare(ctypes.CDLL(path))
    _lib_cache[path] = lib
    return lib


def declare(lib: ctypes.CDLL) -> ctypes.CDLL:
    """Set the argument and result types of an oracle library loaded elsewhere."""
    return _declare(lib)


def build_variant(defines: Sequence[str]) -> ctypes.CDLL:
    """Build and load an oracle compiled with extra ``-D`` defines (mutation tests)."""
    d = tempfile.mkdtemp(prefix="gdo_")
    path = os.path.join(d, "libgdoracle_" + "_".join(defines) + ".so")
    build(path, defines)
    return _declare(ctypes.CDLL(path))


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def keep_ppm(drop_ratio: float, lib: Optional[ctypes.CDLL] = None) -> int:
    return int((lib or load()).gdo_keep_ppm(drop_ratio))


def keep_count(n: int, drop_ratio: float, lib: Optional[ctypes.CDLL] = None) -> int:
    return int((lib or load()).gdo_keep_count(n, drop_ratio))


@dataclass
class Compressed:
    idx: np.ndarray  # uint32 [k]
    val: np.ndarray  # float32 [k] (acc of kept entries)
    residual: np.ndarray  # float32 [N] new residual
    tensor_counts: np.ndarray  # uint32 [T]
    sign_bits: Optional[np.ndarray]  # uint32 [ceil(k/32)] when quantised
    means: Optional[np.ndarray]  # float32 [2T] (positive, negative) per tensor


def compress(
    grad: np.ndarray,
    residual: np.ndarray,
    offsets: Sequence[int],
    drop_ratio: float = 0.99,
    per_tensor: bool = False,
    quant=False,
    base: Optional[np.ndarray] = None,
    lib: Optional[ctypes.CDLL] = None,
    columns: Optional[Sequence[int]] = None,
) -> Compressed:
    """One call of Algorithm 1 over the layout ``offsets``; inputs are not modified.

    quant: False/0 none, True/1 per-tensor sign mean, 2 threshold, 3 global
    average, 4 column-wise average over the matrices ``columns`` describes.
    """
    lib = lib or load()
    g = np.ascontiguousarray(grad, dtype=np.float32)
    r = np.array(residual, dtype=np.float32, copy=True)
    b = None if base is None else np.ascontiguousarray(base, dtype=np.float32)
    off = np.ascontiguousarray(offsets, dtype=np.uint64)
    T = off.size - 1
    assert off[-1] == g.size == r.size
    cap = int(g.size)
    idx = np.zeros(max(cap, 1), np.uint32)
    val = np.zeros(max(cap, 1), np.float32)
    counts = np.zeros(T, np.uint32)
    quant = int(quant)
    cols = None if columns is None else np.ascontiguousarray(columns, dtype=np.uint32)
    groups = int(cols.astype(np.int64).sum()) if (quant == 4 and cols is not None) else T
    bits = np.zeros(max((cap + 31) // 32, 1), np.uint32) if quant else None
    means = np.zeros(2 * groups, np.float32) if quant else None
    k = ctypes.c_uint64(0)
    rc = lib.gdo_compress(_ptr(g), _ptr(b), _ptr(r), _ptr(off), T, float(drop_ratio), int(per_tensor), quant,
                          _ptr(idx), _ptr(val), _ptr(bits), _ptr(means), _ptr(counts), cap, ctypes.byref(k),
                          _ptr(cols))
    if rc != 0:
        raise ValueError(f"gdo_compress failed with status {rc}")
    k = int(k.value)
    return Compressed(idx[:k].copy(), val[:k].copy(), r, counts,
                      None if bits is None else bits[:(k + 31) // 32].copy(), means)


def compress_pull(params: np.ndarray, copy: np.ndarray, offsets: Sequence[int], drop_ratio: float = 0.99,
                  per_tensor: bool = False, lib: Optional[ctypes.CDLL] = None):
    """A pull as a delta from the last pulled copy (R11): returns (Compressed with
    idx/val/tensor_counts, the updated copy); inputs are not modified."""
    lib = lib or load()
    p = np.ascontiguousarray(params, dtype=np.float32)
    c = np.array(copy, dtype=np.float32, copy=True)
    off = np.ascontiguousarray(offsets, dtype=np.uint64)
    T = off.size - 1
    assert off[-1] == p.size == c.size
    cap = int(p.size)
    idx = np.zeros(max(cap, 1), np.uint32)
    val = np.zeros(max(cap, 1), np.float32)
    counts = np.zeros(T, np.uint32)
    k = ctypes.c_uint64(0)
    rc = lib.gdo_compress_pull(_ptr(p), _ptr(c), _ptr(off), T, float(drop_ratio), int(per_tensor), _ptr(idx),
                               _ptr(val), _ptr(counts), cap, ctypes.byref(k))
    if rc != 0:
        raise ValueError(f"gdo_compress_pull failed with status {rc}")
    k = int(k.value)
    return Compressed(idx[:k].copy(), val[:k].copy(), None, counts, None, None), c


def splitmix64(seed: int, i: int, lib: Optional[ctypes.CDLL] = None) -> int:
    """Output number i of SplitMix64 seeded with ``seed`` (the sample-position generator)."""
    return int((lib or load()).gdo_splitmix64(seed, i))


def sample_position(seed: int, s: int, a: int, n: int, m: int, j: int, lib: Optional[ctypes.CDLL] = None) -> int:
    """Flat position of sample j of m drawn from segment s = [a, a + n)."""
    return int((lib or load()).gdo_sample_position(seed, s, a, n, m, j))


def compress_sampled(
    grad: np.ndarray,
    residual: np.ndarray,
    offsets: Sequence[int],
    drop_ratio: float = 0.99,
    per_tensor: bool = False,
    sample_ppm: int = 1000,
    seed: int = 0,
    base: Optional[np.ndarray] = None,
    capacity: Optional[int] = None,
    lib: Optional[ctypes.CDLL] = None,
    quant=False,
    columns: Optional[Sequence[int]] = None,
) -> Compressed:
    """Algorithm 1 with the threshold selected on a sample (Section 4), optionally with the 1-bit
    quantisation of Section 5.4 over the entries sent (quant and columns as ``compress``); inputs are
    not modified."""
    lib = lib or load()
    g = np.ascontiguousarray(grad, dtype=np.float32)
    r = np.array(residual, dtype=np.float32, copy=True)
    b = None if base is None else np.ascontiguousarray(base, dtype=np.float32)
    off = np.ascontiguousarray(offsets, dtype=np.uint64)
    T = off.size - 1
    assert off[-1] == g.size == r.size
    cap = int(g.size) if capacity is None else int(capacity)
    idx = np.zeros(max(cap, 1), np.uint32)
    val = np.zeros(max(cap, 1), np.float32)
    counts = np.zeros(T, np.uint32)
    quant = int(quant)
    cols = None if columns is None else np.ascontiguousarray(columns, dtype=np.uint32)
    groups = int(cols.astype(np.int64).sum()) if (quant == 4 and cols is not None) else T
    bits = np.zeros(max((cap + 31) // 32, 1), np.uint32) if quant else None
    means = np.zeros(2 * groups, np.float32) if quant else None
    k = ctypes.c_uint64(0)
    rc = lib.gdo_compress_sampled(_ptr(g), _ptr(b), _ptr(r), _ptr(off), T, float(drop_ratio), int(per_tensor),
                                  int(sample_ppm), int(seed), quant, _ptr(idx), _ptr(val), _ptr(bits), _ptr(means),
                                  _ptr(counts), cap, ctypes.byref(k), _ptr(cols))
    if rc != 0:
        raise ValueError(f"gdo_compress_sampled failed with status {rc}")
    k = min(int(k.value), cap)
    return Compressed(idx[:k].copy(), val[:k].copy(), r, counts,
                      None if bits is None else bits[:(k + 31) // 32].copy(), means)


def apply_sparse(params: np.ndarray, idx: List[np.ndarray], val: List[np.ndarray], lr: float = 1.0,
                 lib: Optional[ctypes.CDLL] = None) -> np.ndarray:
    """Server-side apply of sparse pushes; returns the updated copy of ``params``."""
    lib = lib or load()
    p = np.array(params, dtype=np.float32, copy=True)
    C = len(idx)
    ix = [np.ascontiguousarray(a, dtype=np.uint32) for a in idx]
    vx = [np.ascontiguousarray(a, dtype=np.float32) for a in val]
    iptr = (ctypes.c_void_p * max(C, 1))(*[a.ctypes.data for a in ix])
    vptr = (ctypes.c_void_p * max(C, 1))(*[a.ctypes.data for a in vx])
    nnz = np.array([a.size for a in ix], dtype=np.uint64)
    rc = lib.gdo_apply_sparse(_ptr(p), p.size, C, ctypes.cast(iptr, ctypes.c_void_p),
                              ctypes.cast(vptr, ctypes.c_void_p), _ptr(nnz) if C else None, float(lr))
    if rc != 0:
        raise ValueError(f"gdo_apply_sparse failed with status {rc}")
    return p


def apply_quantised(params: np.ndarray, offsets: Sequence[int], idx: List[np.ndarray], sign_bits: List[np.ndarray],
                    means: List[np.ndarray], quant: int, lr: float = 1.0, columns: Optional[Sequence[int]] = None,
                    lib: Optional[ctypes.CDLL] = None) -> np.ndarray:
    """Server-side apply of quantised pushes (decoded per R12); returns the updated copy of ``params``."""
    lib = lib or load()
    p = np.array(params, dtype=np.float32, copy=True)
    off = np.ascontiguousarray(offsets, dtype=np.uint64)
    T = off.size - 1
    C = len(idx)
    ix = [np.ascontiguousarray(a, dtype=np.uint32) for a in idx]
    bx = [np.ascontiguousarray(b, dtype=np.uint32) if b.size else np.zeros(1, np.uint32) for b in sign_bits]
    mx = [np.ascontiguousarray(m, dtype=np.float32) for m in means]
    cols = None if columns is None else np.ascontiguousarray(columns, dtype=np.uint32)
    arr = lambda xs: (ctypes.c_void_p * max(C, 1))(*[a.ctypes.data for a in xs])
    ip, bp, mp = arr(ix), arr(bx), arr(mx)
    nnz = np.array([a.size for a in ix], dtype=np.uint64)
    rc = lib.gdo_apply_quantised(_ptr(p), _ptr(off), T, _ptr(cols), C, ctypes.cast(ip, ctypes.c_void_p),
                                 ctypes.cast(bp, ctypes.c_void_p), ctypes.cast(mp, ctypes.c_void_p),
                                 _ptr(nnz) if C else None, int(quant), float(lr))
    if rc != 0:
        raise ValueError(f"gdo_apply_quantised failed with status {rc}")
    return p
