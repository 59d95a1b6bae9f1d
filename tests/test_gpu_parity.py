"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bar: bit-exact on kept indices, kept values, tensor counts, sign bits and
unquantised residuals; quantisation centres (fp64 sums in another order)
within 1e-6 relative, and every quantised residual bit-equal to
fl32(acc - the GPU's centre of its own group and sign).  Multi-step workloads are teacher-forced: every
GPU step starts from the oracle's residual, so one step's tolerance cannot
flip the next step's selection.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from paper_1704_05021_amd import gd, workloads as wl
from parity import assert_parity, bits, check_case, gpu_compress, oracle_compress

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "hand_examples.json")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gd.load()
    torch.cuda.set_device(0)


def test_hand_examples():
    gold = json.load(open(GOLDEN))
    for case in gold["compress"]:
        comp = gd.Compressor(case["offsets"])
        res = None
        for st in case["steps"]:
            r_in = res if st["residual_in"] == "previous" else np.array(st["residual_in"], np.float32)
            g = gpu_compress(comp, np.array(st["grad"], np.float32), r_in, case["drop"],
                             case.get("per_tensor", False), case.get("quant", False))
            assert g.idx.tolist() == st["idx"], case["name"]
            assert np.array_equal(bits(g.val), bits(np.array(st["val"], np.float32))), case["name"]
            assert np.array_equal(bits(g.residual), bits(np.array(st["residual_out"], np.float32))), case["name"]
            assert g.tensor_counts.tolist() == st["tensor_counts"], case["name"]
            if "sign_bits" in st:
                assert g.sign_bits.tolist() == st["sign_bits"]
                assert np.array_equal(bits(g.means), bits(np.array(st["means"], np.float32)))
            res = g.residual


def _tie_heavy(rng, n):
    levels = np.array([0.0, 0.25, 0.5, 1.0, 1.5, 3.0, 1e-3, 2.0 ** -130], np.float32)
    v = levels[rng.integers(0, levels.size, n)] * np.where(rng.random(n) < 0.5, -1, 1).astype(np.float32)
    return v.astype(np.float32)


@pytest.mark.parametrize("debug", [0, 1, 2, 3, 4], ids=["sampled", "fallback", "zero_all_cands", "all_cands", "lo_at_hi"])
@pytest.mark.parametrize("seed", range(6))
def test_random_layouts(seed, debug):
    rng = np.random.default_rng(100 + seed)
    T = int(rng.integers(1, 7))
    sizes = rng.integers(0, 30000, size=T)
    sizes[rng.integers(0, T)] = int(rng.choice([0, 1, 3, 17, 4095, 4096, 4097, 16385, 70001]))
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64).tolist()
    N = offsets[-1]
    if N == 0:
        offsets[-1] = N = 5
    for step, (drop, per, quant) in enumerate([(0.99, False, False), (0.99, True, False), (0.9, False, True),
                                               (0.5, True, True), (0.999, True, False)]):
        if seed % 2:
            g = _tie_heavy(rng, N)
            r = _tie_heavy(rng, N)
        else:
            g = (rng.standard_t(3, N) * 1e-3).astype(np.float32)
            r = (rng.normal(0, 1e-3, N) * (rng.random(N) < 0.7)).astype(np.float32)
        comp = gd.Compressor(offsets)
        check_case(g, r, offsets, drop, per, quant, comp=comp, debug_bracket=debug,
                   what=f"seed={seed} debug={debug} step={step} N={N} T={T}")


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 63, 64, 65, 1023, 1024, 1025, 4095, 4096, 4097, 16383, 16384, 16385,
                               65536, 65537, 300001])
def test_edge_sizes(n):
    rng = np.random.default_rng(n)
    g = rng.normal(0, 1, n).astype(np.float32)
    r = rng.normal(0, 1, n).astype(np.float32)
    comp = gd.Compressor([0, n])
    for drop in (0.0, 0.5, 0.99, 1.0):
        for debug in (0, 1):
            check_case(g, r, [0, n], drop, False, False, comp=comp, debug_bracket=debug,
                       what=f"n={n} drop={drop} debug={debug}")


def test_sparse_candidates_wide_windows():
    """Candidates so sparse that one tile of 1024 spans hundreds of units, up to
    one candidate per 1024-element unit: gather loads its whole window of
    non-empty units (past the first 192) and maps every position to the
    last unit start at or before it."""
    units = 3000
    n = 1024 * units
    rng = np.random.default_rng(11)
    u = np.arange(units)
    r = np.zeros(n, np.float32)
    comp = gd.Compressor([0, n])
    for noise in (0.0, 1e-6):  # no noise: the spikes are the only nonzero keys, one candidate per unit
        g = (rng.normal(0, 1, n) * noise).astype(np.float32)
        g[u * 1024 + (u * 37) % 1024] = (1.0 + u * 1e-4).astype(np.float32)  # one spike per unit
        for keep in (2900, 1024, 1025, 2048, 4000):
            drop = 1.0 - keep / n
            for per in (False, True):
                check_case(g, r, [0, n], drop, per, False, comp=comp, what=f"spikes noise={noise} keep={keep} per={per}")
                if noise == 0.0 and keep > units:
                    # fewer nonzero keys than k: every spike, and nothing else, is a
                    # candidate (one per unit, so a full tile's window holds 1024
                    # units), and the zero mode adds the lowest-index zeros
                    seg = comp.debug_state()[0][0]
                    assert seg["clo"] == units and seg["miss"] == 0 and seg["zero"] == 1, seg
    g2 = rng.normal(0, 1, n).astype(np.float32)
    r2 = (rng.normal(0, 1, n) * (rng.random(n) < 0.3)).astype(np.float32)
    offsets = [0, n // 3, n]
    comp2 = gd.Compressor(offsets)
    for drop, per, quant in ((0.9995, False, False), (0.9995, True, False), (0.999, False, True)):
        check_case(g2, r2, offsets, drop, per, quant, comp=comp2, what=f"sparse drop={drop} per={per} q={quant}")


def test_unaligned_tensor_offsets():
    # tensors whose offsets are not multiples of 4: vectors straddle tensor boundaries
    offsets = [0, 5, 6, 4103, 4103, 9001, 20003, 20010]
    rng = np.random.default_rng(7)
    N = offsets[-1]
    g = (rng.standard_t(3, N) * 1e-2).astype(np.float32)
    r = rng.normal(0, 1e-2, N).astype(np.float32)
    comp = gd.Compressor(offsets)
    for per in (False, True):
        for quant in (False, True):
            for debug in (0, 1, 2, 3, 4):
                check_case(g, r, offsets, 0.9, per, quant, comp=comp, debug_bracket=debug, what=f"per={per} q={quant}")


def test_special_values():
    v = np.array([1.0, np.inf, np.nan, -np.inf, 2.0, -0.0, 0.0, 2.0 ** -149, -(2.0 ** -148), 3.0], np.float32)
    z = np.array([0.0, 0.0, 0.0, 0.0, 0.0, -0.0, -0.0, 2.0 ** -149, 0.0, -3.0], np.float32)
    comp = gd.Compressor([0, v.size])
    for drop in (0.0, 0.3, 0.5, 0.8, 0.9, 1.0):
        for debug in (0, 1, 3):
            check_case(v, z, [0, v.size], drop, False, False, comp=comp, debug_bracket=debug, what=f"drop={drop}")


def test_all_zero_and_all_equal():
    n = 50000
    comp = gd.Compressor([0, 20000, n])
    z = np.zeros(n, np.float32)
    for per in (False, True):
        check_case(z, z, [0, 20000, n], 0.99, per, False, comp=comp, what="zeros")
        s = np.where(np.random.default_rng(1).random(n) < 0.5, -0.75, 0.75).astype(np.float32)
        check_case(s, z, [0, 20000, n], 0.99, per, True, comp=comp, what="equal magnitudes")


def _run_workload(name, steps=None, debug=0):
    w = wl.workload(name)
    off = w.layout.offsets.astype(np.int64).tolist()
    comp = gd.Compressor(off)
    comp.debug_force_bracket(debug)
    residual = np.zeros(w.layout.numel, np.float32)
    for step in range(steps or w.steps):
        grad = w.grad(step)
        g = gpu_compress(comp, grad, residual, w.drop, w.per_tensor, w.quant)
        o = oracle_compress(grad, residual, off, w.drop, w.per_tensor, w.quant)
        assert_parity(g, o, w.quant, f"{name} step {step}", offsets=off)
        residual = o.residual  # teacher forcing
    comp.close()


def test_mnist_mlp_full():
    _run_workload("mnist_mlp_784_512_512_10")


@pytest.mark.parametrize("name", ["mlp_784_256_256_10_t3_small", "nmt_small_per_tensor", "nmt_small_global_signmean"])
def test_small_workloads(name):
    _run_workload(name)
    _run_workload(name, steps=2, debug=1)
    _run_workload(name, steps=2, debug=4)


@pytest.mark.slow
@pytest.mark.parametrize("name", ["mlp_784_4096_4096_10_t3", "nmt_85k_per_tensor", "nmt_85k_global_signmean"])
def test_full_size_workloads_every_step(name):
    """Every step of the full-size configurations, at their full lengths (20
    carried steps for the 784-4096-4096-10 MLP, 10 for both NMT-shaped
    configurations), with the residual carried as Algorithm 1 carries it:
    each step's residual is the oracle's result of the step before (teacher
    forcing), so later steps, where residuals have filled in and the bracket
    sees another distribution, are compared too."""
    w = wl.workload(name)
    assert w.steps == {"mlp_784_4096_4096_10_t3": 20, "nmt_85k_per_tensor": 10, "nmt_85k_global_signmean": 10}[name]
    _run_workload(name)


def test_determinism():
    w = wl.workload("nmt_small_global_signmean")
    off = w.layout.offsets.astype(np.int64).tolist()
    comp = gd.Compressor(off)
    grad = w.grad(0)
    r0 = np.random.default_rng(3).normal(0, 1e-3, grad.size).astype(np.float32)
    a = gpu_compress(comp, grad, r0, 0.99, False, True)
    b = gpu_compress(comp, grad, r0, 0.99, False, True)
    assert np.array_equal(a.idx, b.idx) and np.array_equal(bits(a.residual), bits(b.residual))
    assert np.array_equal(bits(a.means), bits(b.means)) and np.array_equal(a.sign_bits, b.sign_bits)


def test_pull_delta_base():
    rng = np.random.default_rng(4)
    n = 200003
    p0 = rng.normal(0, 0.1, n).astype(np.float32)
    p1 = p0.copy()
    ix = rng.choice(n, 5000, replace=False)
    p1[ix] -= rng.normal(0, 1e-2, 5000).astype(np.float32)
    res = np.zeros(n, np.float32)
    comp = gd.Compressor([0, n])
    for debug in (0, 1):
        check_case(p1, res, [0, n], 0.99, False, False, base=p0, comp=comp, debug_bracket=debug, what="pull")


def _apply_case(n, C, nnz, dup, seed, lr=1.0):
    s = wl.server_shard(n=n, clients=C, nnz=nnz, dup_frac=dup, seed=seed)
    want = oracle.apply_sparse(s.params, s.idx, s.val, lr)
    p = torch.from_numpy(s.params).cuda()
    idx = [torch.from_numpy(a.view(np.int32)).cuda() for a in s.idx]
    val = [torch.from_numpy(a).cuda() for a in s.val]
    gd.apply_sparse(p, idx, val, lr)
    torch.cuda.synchronize()
    got = p.cpu().numpy()
    assert np.array_equal(bits(got), bits(want)), f"apply n={n} C={C}: {np.sum(bits(got) != bits(want))} differ"
    return s, got


@pytest.mark.parametrize("C,dup,lr", [(1, 0.0, 1.0), (2, 0.05, 1.0), (4, 0.05, 1.0), (4, 0.5, 0.25), (7, 0.3, 1.0)])
def test_apply_small(C, dup, lr, apply_form):
    _apply_case(60_000, C, 1500, dup, seed=C, lr=lr)


def test_apply_dense_buckets_and_many_clients(apply_form):
    # buckets too full for the staged (LDS) path: about 28,000 entries per bucket
    _apply_case(70_000, 4, 15_000, 0.3, seed=11)
    # the most clients one call takes, heavy sharing, a ragged last bucket
    _apply_case(100_003, 64, 40, 0.5, seed=12, lr=0.5)


def test_apply_random_cases(apply_form):
    """Seeded random server applies: shard sizes from a few hundred to millions
    of parameters (ragged last buckets), 1 to 64 clients, densities from a few
    entries to most of the shard, shared-index fractions from none to most, and
    several learning rates."""
    for case in range(40):
        rng = np.random.default_rng(40_000 + case)
        n = int(rng.choice([300, 33_333, 1 << 15, (1 << 15) + 1, 500_000, 3_000_001]))
        C = int(rng.choice([1, 2, 4, 9, 64]))
        # every client's fresh indices must fit outside the earlier clients' union
        nnz = max(1, min(int(n * float(rng.choice([0.0005, 0.01, 0.1, 0.6]))), n // (2 * C)))
        dup = float(rng.choice([0.0, 0.05, 0.5, 0.95]))
        lr = float(rng.choice([1.0, 0.5, 1e-3]))
        _apply_case(n, C, nnz, dup, seed=50_000 + case, lr=lr)


def test_apply_skips_out_of_range_and_empty_pushes(apply_form):
    rng = np.random.default_rng(13)
    n = 40_000
    p0 = rng.normal(0, 0.1, n).astype(np.float32)
    a = np.sort(rng.choice(n, 3000, replace=False)).astype(np.uint32)
    b = np.sort(np.concatenate([rng.choice(a, 500, replace=False),
                                rng.choice(np.setdiff1d(np.arange(n), a), 500, replace=False)])).astype(np.uint32)
    b_out = np.concatenate([b, np.array([n, n + 7, 2 ** 31], np.uint32)])  # entries past the shard are skipped
    va = rng.normal(0, 1e-3, a.size).astype(np.float32)
    vb = rng.normal(0, 1e-3, b_out.size).astype(np.float32)
    empty_i, empty_v = np.zeros(0, np.uint32), np.zeros(0, np.float32)
    want = oracle.apply_sparse(p0, [a, empty_i, b], [va, empty_v, vb[:b.size]], 1.0)
    p = torch.from_numpy(p0).cuda()
    idx = [torch.from_numpy(x.view(np.int32)).cuda() for x in (a, empty_i, b_out)]
    val = [torch.from_numpy(x).cuda() for x in (va, empty_v, vb)]
    gd.apply_sparse(p, idx, val, 1.0)
    torch.cuda.synchronize()
    assert np.array_equal(bits(p.cpu().numpy()), bits(want))


def test_apply_and_pull_full_shard(apply_form):
    cfg = wl.SHARD_FULL
    s, p1 = _apply_case(cfg["n"], cfg["clients"], cfg["nnz"], cfg["dup_frac"], cfg["seed"])
    comp = gd.Compressor([0, cfg["n"]])
    zeros = np.zeros(cfg["n"], np.float32)
    check_case(p1, zeros, [0, cfg["n"]], 0.99, False, False, base=s.params, comp=comp, what="pull of full shard")


def test_errors():
    comp = gd.Compressor([0, 1000])
    g = torch.zeros(1000, device="cuda")
    r = torch.zeros(1000, device="cuda")
    out = comp.alloc_out(0.99)
    small = comp.alloc_out(0.99, capacity=5)
    with pytest.raises(gd.GDError) as e:
        comp.compress(g, r, 0.99, out=small)
    assert e.value.status == 3
    big = torch.zeros(1001, device="cuda")
    with pytest.raises(gd.GDError) as e:
        comp.compress(big[1:], r, 0.99, out=out)
    assert e.value.status == 4
    with pytest.raises(gd.GDError) as e:
        comp.compress(g, r, 1.5, out=out)
    assert e.value.status == 1
    with pytest.raises(gd.GDError) as e:
        gd.Compressor([0, 10, 5])
    assert e.value.status == 2
    with pytest.raises(gd.GDError) as e:
        gd.Compressor([3, 10])
    assert e.value.status == 2
    p = torch.zeros(10, device="cuda")
    ix = [torch.zeros(1, dtype=torch.int32, device="cuda")] * 65
    vx = [torch.zeros(1, device="cuda")] * 65
    with pytest.raises(gd.GDError) as e:
        gd.apply_sparse(p, ix, vx)
    assert e.value.status == 1
    # failed calls leave buffers untouched
    r.fill_(1.5)
    with pytest.raises(gd.GDError):
        comp.compress(g, r, 0.99, out=small)
    torch.cuda.synchronize()
    assert torch.all(r == 1.5)


def test_non_default_stream():
    w = wl.workload("nmt_small_per_tensor")
    off = w.layout.offsets.astype(np.int64).tolist()
    comp = gd.Compressor(off)
    grad = w.grad(0)
    o = oracle_compress(grad, np.zeros_like(grad), off, 0.99, True, False)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        gt = torch.from_numpy(grad).cuda()
        rt = torch.zeros_like(gt)
        out = comp.compress(gt, rt, 0.99, per_tensor=True)
    s.synchronize()
    assert np.array_equal(out.idx[:out.k].cpu().numpy().view(np.uint32), o.idx)
    assert np.array_equal(bits(rt.cpu().numpy()), bits(o.residual))


def test_dense_timing_every_nth_launch():
    """Timing every third dense launch over seven calls times launches 0, 3 and 6; results are unchanged."""
    w = wl.workload("nmt_small_per_tensor")
    off = w.layout.offsets.astype(np.int64).tolist()
    comp = gd.Compressor(off)
    grad = w.grad(0)
    o = oracle_compress(grad, np.zeros_like(grad), off, 0.99, True, False)
    gt = torch.from_numpy(grad).cuda()
    comp.profile_enable(3)
    for _ in range(7):
        rt = torch.zeros_like(gt)
        out = comp.compress(gt, rt, 0.99, per_tensor=True)
    ms, n = comp.profile_read()
    assert n == 3 and ms > 0.0
    assert np.array_equal(out.idx[:out.k].cpu().numpy().view(np.uint32), o.idx)
    assert np.array_equal(bits(rt.cpu().numpy()), bits(o.residual))
    comp.profile_enable(0)
    comp.compress(gt, torch.zeros_like(gt), 0.99, per_tensor=True)
    assert comp.profile_read() == (0.0, 0)
    with pytest.raises(gd.GDError):
        comp.profile_enable(-1)


@pytest.mark.parametrize("T", [3000, 70_000])
def test_many_tensors(T):
    """Thousands of small tensors (empty ones among them): every per-segment loop and grid runs past one block."""
    rng = np.random.default_rng(T)
    sizes = rng.integers(0, 40, T)
    sizes[rng.random(T) < 0.1] = 0
    sizes[rng.integers(0, T, 3)] = [5000, 1025, 4096]
    offsets = [0] + np.cumsum(sizes).tolist()
    N = offsets[-1]
    g = (rng.standard_t(3, N) * 1e-3).astype(np.float32)
    r = rng.normal(0, 1e-3, N).astype(np.float32)
    comp = gd.Compressor(offsets)
    for per, quant, drop in ((True, False, 0.9), (False, False, 0.99), (True, True, 0.5)):
        check_case(g, r, offsets, drop, per, quant, comp=comp, what=f"T={T} per={per} quant={quant}")


def test_empty_layout():
    """Every tensor empty (N = 0): each compress form succeeds and sends nothing."""
    comp = gd.Compressor([0, 0, 0])
    e = torch.zeros(0, device="cuda")
    for quant in (False, True):
        out = comp.compress(e, e, 0.99, per_tensor=True, quant=quant)
        torch.cuda.synchronize()
        assert out.k == 0 and out.tensor_counts[:2].cpu().tolist() == [0, 0]
    out = comp.compress_pull(e, e, 0.99)
    s = comp.compress_sampled(e, e, 0.99, per_tensor=True, capacity=4, quant=gd.GD_QUANT_THRESHOLD)
    torch.cuda.synchronize()
    assert out.tensor_counts[:2].cpu().tolist() == [0, 0] and s.tensor_counts[:2].cpu().tolist() == [0, 0]


def test_apply_unaligned_parameters(apply_form):
    """A parameter buffer that is not 16-byte aligned (a view one float in) is updated exactly like an
    aligned one: results equal the oracle's bit for bit.  With validate=True the binding refuses a push
    whose indices are not ascending."""
    s = wl.server_shard(n=100_001, clients=3, nnz=4_000, dup_frac=0.1, seed=21)
    want = oracle.apply_sparse(s.params, s.idx, s.val, 1.0)
    buf = torch.zeros(s.params.size + 1, device="cuda")
    buf[1:] = torch.from_numpy(s.params).cuda()
    p = buf[1:]
    assert p.data_ptr() % 16 != 0
    gd.apply_sparse(p, [torch.from_numpy(a.view(np.int32)).cuda() for a in s.idx],
                    [torch.from_numpy(a).cuda() for a in s.val], 1.0, validate=True)
    torch.cuda.synchronize()
    assert np.array_equal(bits(p.cpu().numpy()), bits(want))
    with pytest.raises(gd.GDError) as e:  # a push out of order is refused when asked to check
        bad = torch.from_numpy(s.idx[0][::-1].copy().view(np.int32)).cuda()
        gd.apply_sparse(p, [bad], [torch.from_numpy(s.val[0]).cuda()], 1.0, validate=True)
    assert e.value.status == 1


def test_apply_streams_keep_their_own_tables(apply_form):
    """Applies on two streams, interleaved: each stream reuses the streaming form's bounds table of its
    own stream, so calls in flight on the other stream cannot disturb it; every result equals the
    oracle's bit for bit."""
    shards = [wl.server_shard(n=300_001 + 4096 * j, clients=2 + j, nnz=9_000, dup_frac=0.2, seed=60 + j)
              for j in range(2)]
    want = [oracle.apply_sparse(s.params, s.idx, s.val, 1.0) for s in shards]
    streams = [torch.cuda.Stream() for _ in shards]
    dev = []
    for s, st in zip(shards, streams):
        with torch.cuda.stream(st):
            dev.append((torch.from_numpy(s.params).cuda(), [torch.from_numpy(a.view(np.int32)).cuda() for a in s.idx],
                        [torch.from_numpy(a).cuda() for a in s.val]))
    torch.cuda.synchronize()
    for rep in range(4):
        ps = []
        for (p0, ii, vv), st in zip(dev, streams):
            with torch.cuda.stream(st):
                p = p0.clone()
                gd.apply_sparse(p, ii, vv, 1.0, stream=st)
                ps.append(p)
        torch.cuda.synchronize()
        for p, w in zip(ps, want):
            assert np.array_equal(p.cpu().numpy().view(np.uint32), w.view(np.uint32)), f"repeat {rep}"


def test_apply_per_thread_default_streams(apply_form):
    """Applies from two host threads on the per-thread default stream (one HIP stream per thread behind
    one handle): the streaming form keeps a bounds table per thread for it, and every result equals the
    oracle's bit for bit."""
    import ctypes
    import threading

    per_thread_stream = ctypes.c_void_p(2)  # hipStreamPerThread
    shards = [wl.server_shard(n=250_003 + 8192 * j, clients=3, nnz=8_000, dup_frac=0.3, seed=70 + j)
              for j in range(2)]
    want = [oracle.apply_sparse(s.params, s.idx, s.val, 1.0) for s in shards]
    dev = [(torch.from_numpy(s.params).cuda(), [torch.from_numpy(a.view(np.int32)).cuda() for a in s.idx],
            [torch.from_numpy(a).cuda() for a in s.val]) for s in shards]
    outs = [[None] * 4 for _ in shards]
    torch.cuda.synchronize()
    lib = gd.load()

    errors = []

    def run(j):
        try:
            apply_all(j)
        except BaseException as e:  # reported by the main thread
            errors.append((j, e))

    def apply_all(j):
        p0, ii, vv = dev[j]
        ptr_i = (ctypes.c_void_p * len(ii))(*[a.data_ptr() for a in ii])
        ptr_v = (ctypes.c_void_p * len(vv))(*[b.data_ptr() for b in vv])
        nnz = (ctypes.c_uint64 * len(ii))(*[a.numel() for a in ii])
        for rep in range(4):
            p = outs[j][rep]
            st = lib.gd_apply_sparse(p.data_ptr(), p.numel(), len(ii), ctypes.cast(ptr_i, ctypes.c_void_p),
                                     ctypes.cast(ptr_v, ctypes.c_void_p), ctypes.cast(nnz, ctypes.c_void_p),
                                     1.0, per_thread_stream)
            assert st == 0

    for j in range(len(shards)):
        for rep in range(4):
            outs[j][rep] = dev[j][0].clone()
    torch.cuda.synchronize()
    threads = [threading.Thread(target=run, args=(j,)) for j in range(len(shards))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for j, w in enumerate(want):
        for rep in range(4):
            assert np.array_equal(outs[j][rep].cpu().numpy().view(np.uint32), w.view(np.uint32)), (j, rep)
