"""Host sanitizer builds (CPU only, no GPU needed).

* The oracle, built with g++ -fsanitize=address,undefined, runs every pin of
  ``pins.py`` in a child process that preloads the sanitizer runtimes: any
  out-of-bounds access, use after free or undefined behaviour (shift, signed
  overflow, misaligned load...) in the oracle aborts the child.
* The HIP library, with its host code built under AddressSanitizer and
  UndefinedBehaviorSanitizer (device code is not instrumented), runs every
  entry point's host-side argument and layout checks that return before any
  HIP call: the key-count arithmetic, the layout validation of gd_create, the
  push checks of gd_apply_sparse, the status strings.
"""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TESTS = os.path.join(ROOT, "tests")


def _gcc_runtime(name):
    p = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


def _run_child(code, preload, timeout=900):
    env = dict(os.environ)
    env["LD_PRELOAD"] = ":".join(preload)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["PYTHONPATH"] = os.pathsep.join([ROOT, TESTS, env.get("PYTHONPATH", "")])
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=timeout)
    assert r.returncode == 0 and "SANITIZED_OK" in r.stdout, f"rc={r.returncode}\n{r.stdout[-3000:]}\n{r.stderr[-6000:]}"


def test_oracle_pins_under_asan_and_ubsan():
    asan, ubsan = _gcc_runtime("libasan.so"), _gcc_runtime("libubsan.so")
    if not (asan and ubsan):
        pytest.skip("g++ sanitizer runtimes not installed")
    import oracle

    d = tempfile.mkdtemp(prefix="gdo_san_")
    lib = oracle.build(os.path.join(d, "libgdoracle_san.so"),
                       extra_flags=["-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                                    "-fno-sanitize-recover=all"])
    code = f"""
import ctypes, oracle
from pins import ALL_PINS
lib = oracle.declare(ctypes.CDLL({lib!r}))
for pin in ALL_PINS:
    pin(lib)
print("SANITIZED_OK", len(ALL_PINS))
"""
    _run_child(code, [asan, ubsan])


def test_library_host_checks_under_asan_and_ubsan():
    clang_rt = None
    for root, _, files in os.walk("/opt/rocm/llvm/lib/clang"):
        if "libclang_rt.asan-x86_64.so" in files:
            clang_rt = os.path.join(root, "libclang_rt.asan-x86_64.so")
    if clang_rt is None:
        pytest.skip("clang AddressSanitizer runtime not installed")
    from paper_1704_05021_amd import build

    d = tempfile.mkdtemp(prefix="gd_san_")
    # sanitizers on the host side of every source only (device code is not instrumented)
    flags = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    lib = build.build(out=os.path.join(d, "libgd_san.so"), extra_flags=flags, objdir=os.path.join(d, "obj"))
    code = f"""
import ctypes
L = ctypes.CDLL({lib!r})
u64, u32, i32, dbl, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int, ctypes.c_double, ctypes.c_void_p
L.gd_keep_count.argtypes = [u64, dbl]; L.gd_keep_count.restype = u64
L.gd_keep_total.argtypes = [vp, dbl, i32]; L.gd_keep_total.restype = u64
L.gd_status_string.argtypes = [i32]; L.gd_status_string.restype = ctypes.c_char_p
L.gd_create.argtypes = [ctypes.POINTER(vp), vp, u32]; L.gd_create.restype = i32
L.gd_compress.argtypes = [vp, vp, vp, vp, dbl, i32, i32, vp, vp]; L.gd_compress.restype = i32
L.gd_apply_sparse.argtypes = [vp, u64, u32, vp, vp, vp, ctypes.c_float, vp]; L.gd_apply_sparse.restype = i32
assert L.gd_keep_count(669706, 0.99) == 6697
for n in (0, 1, 7, 2**32 - 2, 2**40):
    for r in (0.0, 0.5, 0.99, 1.0, -1.0, 2.0, float("nan")):
        L.gd_keep_count(n, r)
for c in (-2, -1, 0, 1, 2, 3, 4, 5, 6, 7, 8, 99, 2**31 - 1):
    assert L.gd_status_string(c)
assert L.gd_keep_total(None, 0.99, 0) == 0
h = vp()
def create(offs):
    a = (u64 * len(offs))(*offs)
    return L.gd_create(ctypes.byref(h), a, len(offs) - 1)
assert create([0, 2**32 - 1]) == 2            # N = 2^32 - 1: one index too many for uint32
assert create([0, 2**32]) == 2
assert create([0, 10, 5]) == 2                # decreasing
assert create([3, 10]) == 2                   # not starting at 0
assert L.gd_create(ctypes.byref(h), (u64 * 1)(0), 0) == 1   # no tensors
assert L.gd_create(None, (u64 * 2)(0, 1), 1) == 1
assert L.gd_create(ctypes.byref(h), None, 1) == 1
assert L.gd_compress(None, None, None, None, 0.99, 0, 0, None, None) == 1
ptrs = (vp * 65)(*([1] * 65)); nnz = (u64 * 65)(*([1] * 65))
assert L.gd_apply_sparse(vp(16), 10, 65, ptrs, ptrs, nnz, 1.0, None) == 1      # more than 64 pushes
assert L.gd_apply_sparse(vp(16), 2**32 - 1, 1, ptrs, ptrs, nnz, 1.0, None) == 1
assert L.gd_apply_sparse(vp(16), 10, 0, None, None, None, 1.0, None) == 0       # nothing to do
assert L.gd_apply_sparse(None, 10, 1, ptrs, ptrs, nnz, 1.0, None) == 1
big = (u64 * 1)(2**32 - 1)
assert L.gd_apply_sparse(vp(16), 10, 1, ptrs, ptrs, big, 1.0, None) == 1
null_push = (vp * 1)(None)
assert L.gd_apply_sparse(vp(16), 10, 1, null_push, ptrs, nnz, 1.0, None) == 1
print("SANITIZED_OK")
"""
    _run_child(code, [clang_rt])
