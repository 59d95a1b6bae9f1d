"""Host-side checks of the C ABI: the library loads and exports every entry
point that include/gd.h declares, and its host-only functions agree with the
oracle's closed forms.  No kernel is launched (no GPU needed)."""
import os
import re
import subprocess

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gd.h")
LIB = os.path.join(ROOT, "paper_1704_05021_amd", "libgd.so")


@pytest.fixture(scope="module")
def gd():
    if not os.path.exists(LIB):
        from paper_1704_05021_amd import build
        build.build()
    from paper_1704_05021_amd import gd as gdmod
    gdmod.load()
    return gdmod


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gd_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("gd_create", "gd_destroy", "gd_compress", "gd_apply_sparse", "gd_keep_count", "gd_keep_total"):
        assert required in names


def test_every_declared_symbol_is_exported(gd):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (gd_[a-z_]+)\b", out))
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    assert set(gd.EXPORTS) == set(declared_functions())


def test_keep_count_matches_oracle(gd):
    lib = oracle.load()
    for n in (0, 1, 6, 8, 100, 669_706, 20_037_642, 37_000_000, 42_500_000, 136_875_744):
        for r in (0.0, 1 / 3, 0.5, 0.625, 0.9, 0.99, 0.999, 1.0):
            assert gd.keep_count(n, r) == oracle.keep_count(n, r, lib), (n, r)
    assert gd.keep_count(669_706, 0.99) == 6_697
    # drop ratios outside [0, 1] keep nothing
    assert gd.keep_count(100, -0.5) == 0 and gd.keep_count(100, 1.5) == 0 and gd.keep_count(100, float("nan")) == 0


def test_status_strings(gd):
    lib = gd.load()
    seen = set()
    for code in range(7):
        s = lib.gd_status_string(code).decode()
        assert s and s not in seen
        seen.add(s)
    assert lib.gd_status_string(99).decode() == "unknown status"


def test_product_path_does_not_import_the_oracle():
    pkg = os.path.join(ROOT, "paper_1704_05021_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text and "oracle.cpp" not in text, f
                assert "gdo_" not in text, f


def test_create_refuses_layouts_past_uint32_indices(gd):
    """Indices are sent as uint32 and 2^32 - 1 is reserved, so gd_create takes N <= 2^32 - 2 and returns
    GD_ERR_LAYOUT for N = 2^32 - 1 and above, before touching any device (checked without a GPU)."""
    import ctypes

    lib = gd.load()
    h = ctypes.c_void_p()
    for n in (2 ** 32 - 1, 2 ** 32, 2 ** 40):
        offs = (ctypes.c_uint64 * 3)(0, 5, n)
        assert lib.gd_create(ctypes.byref(h), offs, 2) == 2, n
        assert h.value is None
    for bad in ((3, 10), (0, 10, 5)):
        offs = (ctypes.c_uint64 * len(bad))(*bad)
        assert lib.gd_create(ctypes.byref(h), offs, len(bad) - 1) == 2, bad


def test_static_entry_point_source_allocates_nothing():
    """gd_compress_static's file names no allocating or memset call, and host code reaches the scratch array
    only through the address hipGetSymbolAddress gives for the device."""
    src = open(os.path.join(ROOT, "paper_1704_05021_amd", "csrc", "gd_static.hip")).read()
    code = re.sub(r"//[^\n]*", "", src)
    for banned in ("hipMalloc", "hipFree", "hipMemset", "hipHostMalloc", "malloc(", " new ", "std::vector",
                   "torch"):
        assert banned not in code, banned
    assert "static __device__ __align__(256)" in code
    assert code.count("HIP_SYMBOL(scratch)") == 1 and "hipGetSymbolAddress" in code
    # the array's name appears only in its definition and in the symbol lookup
    assert len(re.findall(r"\bscratch\b(?!_)", code)) == 2
