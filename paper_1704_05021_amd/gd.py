"""Python binding of the HIP gradient-dropping library (``libgd.so``).

Argument marshalling only: torch supplies device memory and the current HIP
stream; every step of the compressor runs in the library's kernels.  There is
no CPU fallback: if ``libgd.so`` has not been built, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgd.so")

GD_GLOBAL, GD_PER_TENSOR = 0, 1
GD_QUANT_NONE, GD_QUANT_SIGN_MEAN, GD_QUANT_THRESHOLD, GD_QUANT_GLOBAL_MEAN, GD_QUANT_COLUMN_MEAN = 0, 1, 2, 3, 4

STATUS = {
    0: "GD_OK",
    1: "GD_ERR_ARG",
    2: "GD_ERR_LAYOUT",
    3: "GD_ERR_CAPACITY",
    4: "GD_ERR_ALIGN",
    5: "GD_ERR_OOM",
    6: "GD_ERR_HIP",
}

EXPORTS = [
    "gd_create",
    "gd_destroy",
    "gd_keep_count",
    "gd_keep_total",
    "gd_compress",
    "gd_compress_sampled",
    "gd_set_columns",
    "gd_compress_pull",
    "gd_apply_quantised",
    "gd_quant_centres",
    "gd_apply_sparse",
    "gd_status_string",
    "gd_profile_enable",
    "gd_profile_read",
    "gd_debug_force_bracket",
    "gd_debug_apply_form",
    "gd_debug_state",
    "gd_compress_static",
]


class GDError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {STATUS.get(status, status)} ({_lib().gd_status_string(status).decode()})")


class _Sparse(ctypes.Structure):
    _fields_ = [
        ("idx", ctypes.c_void_p),
        ("val", ctypes.c_void_p),
        ("sign_bits", ctypes.c_void_p),
        ("means", ctypes.c_void_p),
        ("tensor_counts", ctypes.c_void_p),
        ("capacity", ctypes.c_uint64),
    ]


_LIB = None


def _lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build the HIP library first (python -c "
                          "'import __graft_entry__ as g; g.build()')")
    lib = ctypes.CDLL(LIB_PATH)
    vp, u64, u32, dbl, i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_double, ctypes.c_int
    lib.gd_create.argtypes = [ctypes.POINTER(vp), vp, u32]
    lib.gd_create.restype = i32
    lib.gd_destroy.argtypes = [vp]
    lib.gd_destroy.restype = None
    lib.gd_keep_count.argtypes = [u64, dbl]
    lib.gd_keep_count.restype = u64
    lib.gd_keep_total.argtypes = [vp, dbl, i32]
    lib.gd_keep_total.restype = u64
    lib.gd_compress.argtypes = [vp, vp, vp, vp, dbl, i32, i32, ctypes.POINTER(_Sparse), vp]
    lib.gd_compress.restype = i32
    lib.gd_compress_sampled.argtypes = [vp, vp, vp, vp, dbl, i32, u32, u64, i32, ctypes.POINTER(_Sparse), vp]
    lib.gd_compress_sampled.restype = i32
    lib.gd_apply_quantised.argtypes = [vp, vp, u32, vp, vp, vp, vp, i32, ctypes.c_float, vp]
    lib.gd_apply_quantised.restype = i32
    lib.gd_compress_pull.argtypes = [vp, vp, vp, dbl, i32, ctypes.POINTER(_Sparse), vp]
    lib.gd_compress_pull.restype = i32
    lib.gd_set_columns.argtypes = [vp, vp]
    lib.gd_set_columns.restype = i32
    lib.gd_quant_centres.argtypes = [vp, i32]
    lib.gd_quant_centres.restype = u64
    lib.gd_apply_sparse.argtypes = [vp, u64, u32, vp, vp, vp, ctypes.c_float, vp]
    lib.gd_apply_sparse.restype = i32
    lib.gd_status_string.argtypes = [i32]
    lib.gd_status_string.restype = ctypes.c_char_p
    lib.gd_profile_enable.argtypes = [vp, i32]
    lib.gd_profile_enable.restype = i32
    lib.gd_profile_read.argtypes = [vp, ctypes.POINTER(dbl), ctypes.POINTER(u64)]
    lib.gd_profile_read.restype = i32
    lib.gd_debug_force_bracket.argtypes = [vp, i32]
    lib.gd_debug_force_bracket.restype = i32
    lib.gd_debug_apply_form.argtypes = [i32]
    lib.gd_debug_apply_form.restype = i32
    lib.gd_debug_state.argtypes = [vp, vp, u32, vp]
    lib.gd_debug_state.restype = i32
    lib.gd_compress_static.argtypes = [vp, u32, vp, vp, vp, dbl, i32, i32, ctypes.POINTER(_Sparse), vp]
    lib.gd_compress_static.restype = i32
    _LIB = lib
    return lib


def load() -> ctypes.CDLL:
    """Load ``libgd.so`` (raises ImportError when it has not been built)."""
    return _lib()


def keep_count(n: int, drop_ratio: float) -> int:
    return int(_lib().gd_keep_count(n, float(drop_ratio)))


def _stream_handle(stream: Optional[torch.cuda.Stream]) -> Optional[int]:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream or None


def _check_f32(t: torch.Tensor, name: str, n: int) -> None:
    if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous float32 tensor on the GPU")
    if t.numel() != n:
        raise ValueError(f"{name} has {t.numel()} elements, the layout has {n}")


@dataclass
class SparseOut:
    """Device buffers of one compressed gradient (views of length k)."""

    idx: torch.Tensor  # int32 storage holding uint32 indices
    val: torch.Tensor  # float32
    tensor_counts: torch.Tensor  # int32 storage holding uint32 counts
    sign_bits: Optional[torch.Tensor] = None  # int32 storage holding uint32 words
    means: Optional[torch.Tensor] = None  # float32 [2T]
    k: int = 0


class Compressor:
    """A gradient layout (tensor offsets) bound to the device scratch of ``gd_create``."""

    def __init__(self, offsets: Sequence[int], device: Optional[torch.device] = None):
        lib = _lib()
        off = (ctypes.c_uint64 * len(offsets))(*[int(o) for o in offsets])
        self.offsets = [int(o) for o in offsets]
        self.T = len(offsets) - 1
        self.N = self.offsets[-1]
        self.device = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        h = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            st = lib.gd_create(ctypes.byref(h), off, self.T)
        if st != 0:
            raise GDError(st, "gd_create")
        self._h = h

    def close(self) -> None:
        if getattr(self, "_h", None):
            _lib().gd_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def keep_total(self, drop_ratio: float, per_tensor: bool = False) -> int:
        return int(_lib().gd_keep_total(self._h, float(drop_ratio), GD_PER_TENSOR if per_tensor else GD_GLOBAL))

    def alloc_out(self, drop_ratio: float, per_tensor: bool = False, quant=False,
                  capacity: Optional[int] = None) -> SparseOut:
        k = self.keep_total(drop_ratio, per_tensor)
        cap = max(k if capacity is None else capacity, 1)
        dev = self.device
        out = SparseOut(
            idx=torch.empty(cap, dtype=torch.int32, device=dev),
            val=torch.empty(cap, dtype=torch.float32, device=dev),
            tensor_counts=torch.empty(max(self.T, 1), dtype=torch.int32, device=dev),
            k=k,
        )
        if quant:
            centres = int(_lib().gd_quant_centres(self._h, int(quant)))
            out.sign_bits = torch.empty(max((cap + 31) // 32, 1), dtype=torch.int32, device=dev)
            out.means = torch.empty(max(centres, 1), dtype=torch.float32, device=dev)
        return out

    def compress(self, grad: torch.Tensor, residual: torch.Tensor, drop_ratio: float = 0.99,
                 per_tensor: bool = False, quant=False, base: Optional[torch.Tensor] = None,
                 out: Optional[SparseOut] = None, stream: Optional[torch.cuda.Stream] = None) -> SparseOut:
        """One gd_compress call; ``residual`` is updated in place.

        quant: False/GD_QUANT_NONE, True/GD_QUANT_SIGN_MEAN, or another GD_QUANT_* form.
        """
        _check_f32(grad, "grad", self.N)
        _check_f32(residual, "residual", self.N)
        if base is not None:
            _check_f32(base, "base", self.N)
        if out is None:
            out = self.alloc_out(drop_ratio, per_tensor, quant)
        sp = _Sparse(
            out.idx.data_ptr(),
            out.val.data_ptr(),
            out.sign_bits.data_ptr() if (quant and out.sign_bits is not None) else None,
            out.means.data_ptr() if (quant and out.means is not None) else None,
            out.tensor_counts.data_ptr(),
            out.idx.numel(),
        )
        st = _lib().gd_compress(
            self._h, grad.data_ptr(), None if base is None else base.data_ptr(), residual.data_ptr(),
            float(drop_ratio), GD_PER_TENSOR if per_tensor else GD_GLOBAL,
            int(quant), ctypes.byref(sp), _stream_handle(stream))
        if st != 0:
            raise GDError(st, "gd_compress")
        out.k = self.keep_total(drop_ratio, per_tensor)
        return out

    def compress_pull(self, params: torch.Tensor, copy: torch.Tensor, drop_ratio: float = 0.99,
                      per_tensor: bool = False, out: Optional[SparseOut] = None,
                      stream: Optional[torch.cuda.Stream] = None) -> SparseOut:
        """gd_compress_pull: send params - copy; ``copy`` takes the sent values in place."""
        _check_f32(params, "params", self.N)
        _check_f32(copy, "copy", self.N)
        if out is None:
            out = self.alloc_out(drop_ratio, per_tensor)
        sp = _Sparse(out.idx.data_ptr(), out.val.data_ptr(), None, None, out.tensor_counts.data_ptr(),
                     out.idx.numel())
        st = _lib().gd_compress_pull(self._h, params.data_ptr(), copy.data_ptr(), float(drop_ratio),
                                     GD_PER_TENSOR if per_tensor else GD_GLOBAL, ctypes.byref(sp),
                                     _stream_handle(stream))
        if st != 0:
            raise GDError(st, "gd_compress_pull")
        out.k = self.keep_total(drop_ratio, per_tensor)
        return out

    def apply_quantised(self, params: torch.Tensor, idx, sign_bits, means, quant: int, lr: float = 1.0,
                        stream: Optional[torch.cuda.Stream] = None, validate: bool = False) -> None:
        """gd_apply_quantised: decode quantised pushes of this layout and apply them to params.

        validate: as for ``apply_sparse``, check first that each push's indices are strictly ascending.
        """
        _check_f32(params, "params", self.N)
        C = len(idx)
        if not (len(sign_bits) == len(means) == C):
            raise ValueError("idx, sign_bits and means must have one entry per push")
        for a, b, m in zip(idx, sign_bits, means):
            if a.dtype != torch.int32 or b.dtype != torch.int32 or m.dtype != torch.float32:
                raise TypeError("a push is int32 (uint32 bits) indices and sign words and float32 centres")
            if not (a.is_cuda and b.is_cuda and m.is_cuda and a.is_contiguous() and b.is_contiguous()
                    and m.is_contiguous()):
                raise TypeError("push tensors must be contiguous GPU tensors")
        if validate:
            _check_pushes_ascending(idx)
        arr = lambda xs: (ctypes.c_void_p * max(C, 1))(*[x.data_ptr() for x in xs])
        ip, bp, mp = arr(idx), arr(sign_bits), arr(means)
        nz = (ctypes.c_uint64 * max(C, 1))(*[a.numel() for a in idx])
        st = _lib().gd_apply_quantised(self._h, params.data_ptr(), C, ctypes.cast(ip, ctypes.c_void_p),
                                       ctypes.cast(bp, ctypes.c_void_p), ctypes.cast(mp, ctypes.c_void_p),
                                       ctypes.cast(nz, ctypes.c_void_p), int(quant), float(lr), _stream_handle(stream))
        if st != 0:
            raise GDError(st, "gd_apply_quantised")

    def set_columns(self, columns) -> None:
        """Matrix view of every tensor for the column-wise centres (gd_set_columns)."""
        import numpy as np

        c = np.ascontiguousarray(columns, dtype=np.uint32)
        if c.size != self.T:
            raise ValueError(f"need {self.T} column counts, got {c.size}")
        st = _lib().gd_set_columns(self._h, c.ctypes.data)
        if st != 0:
            raise GDError(st, "gd_set_columns")

    def quant_centres(self, quant: int) -> int:
        return int(_lib().gd_quant_centres(self._h, int(quant)))

    def compress_sampled(self, grad: torch.Tensor, residual: torch.Tensor, drop_ratio: float = 0.99,
                         per_tensor: bool = False, sample_ppm: int = 1000, seed: int = 0,
                         base: Optional[torch.Tensor] = None, out: Optional[SparseOut] = None,
                         capacity: Optional[int] = None, quant=False,
                         stream: Optional[torch.cuda.Stream] = None) -> SparseOut:
        """One gd_compress_sampled call; ``residual`` is updated in place.

        The number sent is data dependent: it is ``out.tensor_counts.sum()``
        (read it after the stream has run).  ``out.k`` is left as None.
        quant: as ``compress``, over the entries sent.
        """
        _check_f32(grad, "grad", self.N)
        _check_f32(residual, "residual", self.N)
        if base is not None:
            _check_f32(base, "base", self.N)
        if out is None:
            out = self.alloc_out(1.0, per_tensor, quant, capacity=self.N if capacity is None else capacity)
        sp = _Sparse(out.idx.data_ptr(), out.val.data_ptr(),
                     out.sign_bits.data_ptr() if (quant and out.sign_bits is not None) else None,
                     out.means.data_ptr() if (quant and out.means is not None) else None,
                     out.tensor_counts.data_ptr(),
                     out.idx.numel() if capacity is None else min(int(capacity), out.idx.numel()))
        st = _lib().gd_compress_sampled(
            self._h, grad.data_ptr(), None if base is None else base.data_ptr(), residual.data_ptr(),
            float(drop_ratio), GD_PER_TENSOR if per_tensor else GD_GLOBAL, int(sample_ppm), int(seed),
            int(quant), ctypes.byref(sp), _stream_handle(stream))
        if st != 0:
            raise GDError(st, "gd_compress_sampled")
        out.k = None
        return out

    def debug_force_bracket(self, mode: int) -> None:
        st = _lib().gd_debug_force_bracket(self._h, int(mode))
        if st != 0:
            raise GDError(st, "gd_debug_force_bracket")

    SEG_FIELDS = ("lo", "hi", "clo", "miss", "d0", "r1", "p18", "r2", "thr", "need", "zero")

    def debug_state(self):
        """(per-segment state of the last call as a list of dicts, decomposition info dict)."""
        import numpy as np

        words = np.zeros((max(self.T, 1), 16), dtype=np.uint32)
        info = np.zeros(4, dtype=np.uint64)
        st = _lib().gd_debug_state(self._h, words.ctypes.data, self.T, info.ctypes.data)
        if st != 0:
            raise GDError(st, "gd_debug_state")
        segs = [dict(zip(self.SEG_FIELDS, (int(x) for x in row[:len(self.SEG_FIELDS)]))) for row in words]
        keys = ("unit_len", "units", "tile", "max_tiles")
        return segs, dict(zip(keys, (int(x) for x in info)))

    def profile_enable(self, every: int = 1) -> None:
        """Time dense launches 0, every, 2 * every, ... from now on (0: off)."""
        st = _lib().gd_profile_enable(self._h, int(every))
        if st != 0:
            raise GDError(st, "gd_profile_enable")

    def profile_read(self):
        """(summed milliseconds of the dense pass, number of timed launches)."""
        ms = ctypes.c_double(0.0)
        n = ctypes.c_uint64(0)
        st = _lib().gd_profile_read(self._h, ctypes.byref(ms), ctypes.byref(n))
        if st != 0:
            raise GDError(st, "gd_profile_read")
        return ms.value, n.value


def _check_pushes_ascending(idx: List[torch.Tensor]) -> None:
    """Raises GDError(GD_ERR_ARG) unless every push's indices (uint32 bits in
    int32 storage) are strictly ascending: the precondition gd_apply_sparse
    relies on and does not check.  Synchronises with the device."""
    for c, a in enumerate(idx):
        if a.numel() > 1:
            u = a.to(torch.int64) & 0xFFFFFFFF
            if not bool(torch.all(u[1:] > u[:-1])):
                raise GDError(1, f"apply: push {c} is not strictly ascending")


def apply_sparse(params: torch.Tensor, idx: List[torch.Tensor], val: List[torch.Tensor], lr: float = 1.0,
                 stream: Optional[torch.cuda.Stream] = None, validate: bool = False) -> None:
    """gd_apply_sparse: params[i] -= lr * (sum of pushed values at i, in push order).

    validate: first check that each push's indices are strictly ascending
    (unique and sorted), which the library assumes and does not check, and
    raise GDError(GD_ERR_ARG) otherwise.  This synchronises with the device.
    """
    if params.dtype != torch.float32 or not params.is_cuda or not params.is_contiguous():
        raise TypeError("params must be a contiguous float32 tensor on the GPU")
    C = len(idx)
    if len(val) != C:
        raise ValueError("idx and val must have the same number of pushes")
    for a, b in zip(idx, val):
        if a.dtype != torch.int32 or b.dtype != torch.float32 or a.numel() != b.numel():
            raise TypeError("each push is an int32 (uint32 bits) index tensor and a float32 value tensor")
        if not (a.is_cuda and b.is_cuda and a.is_contiguous() and b.is_contiguous()):
            raise TypeError("push tensors must be contiguous GPU tensors")
    if validate:
        _check_pushes_ascending(idx)
    ip = (ctypes.c_void_p * max(C, 1))(*[a.data_ptr() for a in idx])
    vp = (ctypes.c_void_p * max(C, 1))(*[b.data_ptr() for b in val])
    nz = (ctypes.c_uint64 * max(C, 1))(*[a.numel() for a in idx])
    st = _lib().gd_apply_sparse(params.data_ptr(), params.numel(), C, ctypes.cast(ip, ctypes.c_void_p),
                                ctypes.cast(vp, ctypes.c_void_p), ctypes.cast(nz, ctypes.c_void_p), float(lr),
                                _stream_handle(stream))
    if st != 0:
        raise GDError(st, "gd_apply_sparse")


def debug_apply_form(form: int) -> None:
    """gd_debug_apply_form: the form of later applies in this process (0 chosen per call, 1 scattered,
    2 streaming wherever the parameters are 16-byte aligned).  A test hook; results do not change."""
    st = _lib().gd_debug_apply_form(int(form))
    if st != 0:
        raise GDError(st, "gd_debug_apply_form")


STATIC_MAX_ELEMENTS = 1 << 21
STATIC_MAX_TENSORS = 64


def compress_static(offsets: Sequence[int], grad: torch.Tensor, residual: torch.Tensor, out: SparseOut,
                    drop_ratio: float = 0.99, per_tensor: bool = False, quant=False,
                    base: Optional[torch.Tensor] = None, stream: Optional[torch.cuda.Stream] = None) -> SparseOut:
    """gd_compress_static: gd_compress without a context and without any allocation, for layouts of at
    most STATIC_MAX_TENSORS tensors and STATIC_MAX_ELEMENTS elements.  ``out`` must be preallocated (for
    example by ``Compressor.alloc_out`` of the same layout); its ``k`` is set to the kept count."""
    n = int(offsets[-1])
    _check_f32(grad, "grad", n)
    _check_f32(residual, "residual", n)
    if base is not None:
        _check_f32(base, "base", n)
    off = (ctypes.c_uint64 * len(offsets))(*[int(o) for o in offsets])
    sp = _Sparse(out.idx.data_ptr(), out.val.data_ptr(),
                 out.sign_bits.data_ptr() if (quant and out.sign_bits is not None) else None,
                 out.means.data_ptr() if (quant and out.means is not None) else None,
                 out.tensor_counts.data_ptr(), out.idx.numel())
    st = _lib().gd_compress_static(off, len(offsets) - 1, grad.data_ptr(),
                                   None if base is None else base.data_ptr(), residual.data_ptr(),
                                   float(drop_ratio), GD_PER_TENSOR if per_tensor else GD_GLOBAL, int(quant),
                                   ctypes.byref(sp), _stream_handle(stream))
    if st != 0:
        raise GDError(st, "gd_compress_static")
    if per_tensor:
        out.k = sum(keep_count(int(offsets[t + 1]) - int(offsets[t]), drop_ratio) for t in range(len(offsets) - 1))
    else:
        out.k = keep_count(n, drop_ratio)
    return out
