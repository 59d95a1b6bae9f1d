"""GPU parity of pulls from the last pulled copy (Section 4, paragraph on pulls).

gd_compress_pull through the C ABI against the oracle's gdo_compress_pull on
the same bytes: sent indices and values, per-tensor counts and the updated
copy, all bit-exact, in every forced bracket mode.
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


def check_pull(comp, params, copy, offsets, drop, per, debug=0, what=""):
    p = torch.from_numpy(np.ascontiguousarray(params, np.float32)).cuda()
    c = torch.from_numpy(np.ascontiguousarray(copy, np.float32)).cuda()
    comp.debug_force_bracket(debug)
    try:
        out = comp.compress_pull(p, c, drop, per_tensor=per)
        torch.cuda.synchronize()
    finally:
        comp.debug_force_bracket(0)
    o, c_want = oracle.compress_pull(params, copy, offsets, drop, per_tensor=per)
    k = out.k
    g_idx = out.idx[:k].cpu().numpy().view(np.uint32)
    assert g_idx.shape == o.idx.shape and np.array_equal(g_idx, o.idx), what
    assert np.array_equal(bits(out.val[:k].cpu().numpy()), bits(o.val)), what
    assert np.array_equal(out.tensor_counts[:comp.T].cpu().numpy().view(np.uint32), o.tensor_counts), what
    c_got = c.cpu().numpy()
    if not np.array_equal(bits(c_got), bits(c_want)):
        bad = np.nonzero(bits(c_got) != bits(c_want))[0]
        raise AssertionError(f"{what}: {bad.size} copy words differ, first at {bad[0]}")
    return c_want


@pytest.mark.parametrize("debug", [0, 1, 3, 4], ids=["sampled", "fallback", "all_cands", "lo_at_hi"])
@pytest.mark.parametrize("seed", range(3))
def test_random_layouts(seed, debug):
    rng = np.random.default_rng(500 + seed)
    T = int(rng.integers(1, 7))
    sizes = rng.integers(0, 200_000, T)
    sizes[rng.random(T) < 0.2] = 0
    offsets = [0] + np.cumsum(sizes).tolist()
    if offsets[-1] == 0:
        offsets[-1] = 1
    N = offsets[-1]
    copy = rng.normal(0, 0.1, N).astype(np.float32)
    params = (copy + rng.standard_t(3, N) * 1e-3).astype(np.float32)
    # a few exact zeros and -0 deltas
    z = rng.random(N) < 0.01
    params[z] = copy[z]
    comp = gd.Compressor(offsets)
    for per in (False, True):
        check_pull(comp, params, copy, offsets, 0.99, per, debug, what=f"seed={seed} per={per} debug={debug}")


def test_full_shard_repeated_pulls():
    """The 37M shard after the four pushes, pulled three times (the copy carried, teacher-forced)."""
    cfg = wl.SHARD_FULL
    sh = wl.server_shard(**cfg)
    p1 = oracle.apply_sparse(sh.params, sh.idx, sh.val, 1.0)
    comp = gd.Compressor([0, cfg["n"]])
    copy = sh.params.copy()
    for step in range(3):
        copy = check_pull(comp, p1, copy, [0, cfg["n"]], 0.99, False, what=f"shard pull {step}")


def test_signed_zero_and_keep_all():
    comp = gd.Compressor([0, 4, 6])
    params = np.array([-0.0, 1.0, 2.0, -3.0, 0.5, -0.0], np.float32)
    copy = np.array([0.0, 1.0, 1.0, 1.0, 0.25, 0.0], np.float32)
    for per in (False, True):
        for drop in (0.0, 0.5, 1.0):
            check_pull(comp, params, copy, [0, 4, 6], drop, per, what=f"per={per} drop={drop}")


def test_errors():
    comp = gd.Compressor([0, 1000])
    p = torch.zeros(1000, device="cuda")
    c = torch.zeros(1000, device="cuda")
    with pytest.raises(gd.GDError):
        comp.compress_pull(torch.zeros(1001, device="cuda")[1:], c)
    with pytest.raises(gd.GDError):
        comp.compress_pull(p, c, 1.5)
    small = comp.alloc_out(0.99, capacity=5)
    with pytest.raises(gd.GDError):
        comp.compress_pull(p, c, 0.99, out=small)


def test_random_cases():
    """Seeded random cases of the pull from the last pulled copy: layouts of 1
    to 60 tensors, every drop ratio, both scopes, forced bracket modes, and
    parameters that equal their copy on a random share of entries."""
    for case in range(40):
        rng = np.random.default_rng(30_000 + case)
        T = int(rng.choice([1, 3, 60]))
        sizes = rng.integers(0, int(rng.choice([300, 30_000, 300_000])), T)
        offsets = [0] + np.cumsum(sizes).tolist()
        if offsets[-1] == 0:
            offsets[-1] = 1
        N = offsets[-1]
        copy = rng.normal(0, 0.1, N).astype(np.float32)
        params = (copy + rng.standard_t(3, N) * 1e-3).astype(np.float32)
        same = rng.random(N) < rng.random()
        params[same] = copy[same]
        drop = float(rng.choice([0.0, 0.5, 0.9, 0.99, 0.999, 1.0]))
        per = bool(rng.random() < 0.5)
        debug = int(rng.choice([0, 0, 1, 3, 4]))
        comp = gd.Compressor(offsets)
        check_pull(comp, params, copy, offsets, drop, per, debug,
                   what=f"case {case}: N={N} T={T} drop={drop} per={per} debug={debug}")
        comp.close()
