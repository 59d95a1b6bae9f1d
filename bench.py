#!/usr/bin/env python3
"""Throughput of the gradient-dropping compressor on one MI355X.

A step is one gd_compress call (residual add, exact k-th largest |acc|
selection, ordered compaction, residual write-back) over one NMT-shaped
gradient set of 136,875,744 fp32 elements in 27 tensors (three 85000x500
embeddings with Zipf-sparse rows plus GRU-shaped dense tensors), per-tensor
threshold, 99% drop.  Ten seeded gradient steps are staged in HBM before
timing; timed steps cycle through them with the residual carried.

Timing protocol: after the warm-up calls, each of the K timed calls is
preceded by a read of a 1 GiB scrub buffer (four times the 256 MB Infinity
Cache), so that no input is served from the cache, and is bracketed by HIP
events on the stream it runs on.  ``ms_per_step`` is the
median of those cold calls (p10 and p90 beside it); K more calls without the
scrub are reported as ``warm`` for information.

Prints one JSON line.  ``value`` is gradient elements compressed per second
(whole job, inputs resident in HBM), from the cold median.  ``roofline``
reports the dense pass (the kernel that streams grad and residual) against
the 8 TB/s HBM peak under the 12-bytes-per-element model; ``cpu_baseline``
times the CPU oracle on a bounded sample of the same workload.  On the
NMT-shaped per-tensor workload the same staged gradients are also run with a
global threshold and per-tensor sign-mean 1-bit centres (Section 5.4), and
that row is reported under ``nmt_85k_global_signmean``.
"""
import argparse
import json
import os
import platform
import statistics
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "G grad-elements/s compressed at 99% drop; % of HBM peak (1 GPU)"
SAMPLED_CAPACITY_PCT = 4  # output room of the sampled mode, in percent of the elements
SCRUB_BYTES = 1 << 30  # read and written before every cold call: four times the 256 MB Infinity Cache
QUANT_KINDS = {"none": 0, "sign_mean": 1, "threshold": 2, "global_mean": 3, "column_mean": 4}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="nmt_85k_per_tensor",
                    help="a compress workload, or shard_apply_pull for the server side (apply + pull delta)")
    ap.add_argument("--selection", choices=("exact", "sampled"), default="exact",
                    help="exact k-th largest threshold (gd_compress, the default), or the paper's threshold "
                         "selected on a sample (gd_compress_sampled, Section 4)")
    ap.add_argument("--quant", choices=("workload",) + tuple(QUANT_KINDS), default="workload",
                    help="1-bit centres of Section 5.4 (default: the workload's own)")
    ap.add_argument("--pull", choices=("residual", "copy"), default="residual",
                    help="shard_apply_pull: the pull delta with a residual (gd_compress with a base) or from "
                         "the last pulled copy (gd_compress_pull)")
    ap.add_argument("--sample-ppm", type=int, default=1000,
                    help="sample size per million entries for --selection sampled (1000 = 0.1%%)")
    ap.add_argument("--cpu-baseline-seconds", type=float, default=12.0,
                    help="rough bound on oracle CPU time for the cpu_baseline leg (0 disables it)")
    ap.add_argument("--scrub", choices=("read", "rw"), default="read",
                    help="what runs before each cold call: a 1 GiB read (default) or read-modify-write")
    ap.add_argument("--with-global-signmean", type=int, default=1,
                    help="on nmt_85k_per_tensor, also time the global threshold with sign-mean centres on the "
                         "same gradients (1, the default) or not (0)")
    ap.add_argument("--with-shard", type=int, default=1,
                    help="with the default NMT-shaped workload, also time the server step on the 37M shard "
                         "(apply of four pushes, then the pull delta) and add it to the line")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB five times (the known-size "
                         "kernel that scales the HBM byte counters), then exit")
    return ap.parse_args()


def cpu_baseline(w, grads_host, budget_s, sample_ppm=0, quant=0):
    """The oracle, single-threaded, on consecutive steps of the same workload.

    Steps cycle through the staged gradients with the residual carried, as
    the GPU steps do, until about budget_s seconds of oracle time.
    """
    import numpy as np

    import oracle

    off = w.layout.offsets.astype(np.int64).tolist()
    residual = np.zeros(w.layout.numel, np.float32)
    done, elapsed, first = 0, 0.0, None
    lib = oracle.load()
    while done == 0 or elapsed < budget_s:
        t0 = time.perf_counter()
        g = grads_host[done % len(grads_host)]
        if sample_ppm:
            o = oracle.compress_sampled(g, residual, off, w.drop, per_tensor=w.per_tensor, sample_ppm=sample_ppm,
                                        seed=done, capacity=SAMPLED_CAPACITY_PCT * w.layout.numel // 100, lib=lib,
                                        quant=quant, columns=w.layout.columns if quant == 4 else None)
        else:
            o = oracle.compress(g, residual, off, w.drop, per_tensor=w.per_tensor, quant=quant, lib=lib,
                                columns=w.layout.columns if quant == 4 else None)
        elapsed += time.perf_counter() - t0
        if first is None:
            first = o
        residual = o.residual
        done += 1
    return {
        "value": w.layout.numel * done / elapsed / 1e9,
        "unit": "G grad-elements/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"{done} consecutive steps of {w.name} from zero residual, cycling its {len(grads_host)} "
                  f"staged gradients ({elapsed:.1f} s of single-threaded oracle time)",
        **host_info(),
    }, first


def host_info():
    """The host the oracle ran on: logical CPUs, those this process may use, and the CPU model."""
    model = None
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.lower().startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except (OSError, subprocess.SubprocessError):
        pass
    if model is None:
        try:
            with open("/proc/cpuinfo") as fh:
                for line in fh:
                    if line.lower().startswith("model name"):
                        model = line.split(":", 1)[1].strip()
                        break
        except OSError:
            model = platform.processor() or None
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = None
    return {"host_cpus": os.cpu_count(), "host_cpus_usable": usable, "cpu_model": model}


def make_scrub(torch, kind="read"):
    """A callable that streams SCRUB_BYTES of device memory through the caches on the current stream:
    a read (a sum into one float; the default) evicts the inputs and leaves only clean lines behind, a
    read-modify-write (``rw``) also leaves the caches full of dirty lines that get written back while
    the next call runs."""
    buf = torch.ones(SCRUB_BYTES // 4, dtype=torch.float32, device="cuda")
    acc = torch.zeros((), dtype=torch.float32, device="cuda")

    def scrub_read():
        torch.sum(buf, dim=0, out=acc)

    def scrub_rw():
        buf.add_(1.0)

    return scrub_rw if kind == "rw" else scrub_read


def time_calls(torch, step, first, count, scrub=None):
    """Per-call times (ms) of step(first) .. step(first + count - 1), each bracketed by HIP events on
    the current stream (the stream the calls are enqueued on); with ``scrub``, it runs before each
    call, outside the events."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(count)]
    for i in range(count):
        if scrub is not None:
            scrub()
        ev[i][0].record()
        step(first + i)
        ev[i][1].record()
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ev]


def written_elements(torch, step, first, count, residual):
    """Elements per call in the 16-byte vectors of the residual that a call changes (the dense pass stores
    only those), averaged over ``count`` calls after the timed ones."""
    n = residual.numel()
    n4 = n - n % 4
    total = 0
    for i in range(count):
        before = residual.clone()
        step(first + i)
        torch.cuda.synchronize()
        a, b = before.view(torch.int32), residual.view(torch.int32)
        total += 4 * int((a[:n4].view(-1, 4) != b[:n4].view(-1, 4)).any(dim=1).sum())
        total += int((a[n4:] != b[n4:]).sum())
        del before
    return total / count


def pct(xs, q):
    """q-th percentile (0..100) of xs by linear interpolation."""
    ys = sorted(xs)
    if len(ys) == 1:
        return ys[0]
    x = (len(ys) - 1) * q / 100.0
    i = int(x)
    j = min(i + 1, len(ys) - 1)
    return ys[i] + (ys[j] - ys[i]) * (x - i)


def spread(ms):
    return {"ms_median": round(statistics.median(ms), 4), "ms_p10": round(pct(ms, 10), 4),
            "ms_p90": round(pct(ms, 90), 4)}


def quant_residuals_ok(np, idx, val, sign_bits, means, residual, offsets, quant, columns=None):
    """Each kept entry's residual is one binary32 subtraction, acc - centre: bit-equal to it, taken
    with this call's own centre of the entry's group (tensor, or column) and sign."""
    off = np.asarray(offsets, np.int64)
    i = idx.astype(np.int64)
    t = np.searchsorted(off, i, side="right") - 1
    if quant == 4:
        cols = np.asarray(columns, np.int64)
        grp = np.concatenate([[0], np.cumsum(cols)])[t] + (i - off[t]) % cols[t]
    else:
        grp = t
    j = np.arange(idx.size, dtype=np.int64)
    bit = (sign_bits[j >> 5].astype(np.int64) >> (j & 31)) & 1
    want = val.astype(np.float32) - means.astype(np.float32)[2 * grp + bit]
    return bool(np.array_equal(residual[idx].view(np.uint32), want.view(np.uint32)))


TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "k_dense_nmt_85k_per_tensor_traffic.md")
# The dense pass is timed with HIP events on every fourth step of the timed
# region: each timed dispatch delays the next kernel by a few microseconds,
# and timing a quarter of the launches keeps that out of the step time while
# still averaging 10 launches of a 40-step run.
DENSE_TIMING_EVERY = 4
DENSE_SOURCES = [os.path.join(ROOT, "paper_1704_05021_amd", "csrc", f)
                 for f in ("gd_dense.hip", "gd_kernels.h", "gd_device.hpp")]


def dense_source_digest():
    import hashlib

    h = hashlib.sha256()
    for f in DENSE_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per k_dense launch from the committed counter summary, or None.

    The summary records the digest of the dense kernel's sources when the
    counters were taken; a changed kernel makes the figure stale (None).
    """
    try:
        with open(TRAFFIC_SUMMARY) as fh:
            text = fh.read()
    except OSError:
        return None
    fields = {}
    for line in text.splitlines():
        if line.startswith("- ") and ": " in line:
            key, val = line[2:].split(": ", 1)
            fields[key.strip()] = val.strip().strip("`")
    if fields.get("workload") != workload or fields.get("source_sha256") != dense_source_digest():
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(mib):
    import torch

    n = mib * (1 << 20) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(5):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": 4 * n, "launches": 5}), flush=True)


def main_shard(args, torch, np, gd, wl, emit=True):
    """The server side at one GPU's shard (37M parameters, 4 clients x 370,000 pushes,
    about 5% shared): per step, apply the four pushes (gd_apply_sparse), then compress the
    pull delta p - p_last with a global threshold and a carried pull residual (or, with
    --pull copy, from the last pulled copy).  Prints the JSON line (emit) and returns it."""
    sh = wl.server_shard(**wl.SHARD_FULL)
    N = sh.params.size
    print(f"[bench] shard of {N} parameters, {len(sh.idx)} pushes", file=sys.stderr, flush=True)
    p = torch.from_numpy(sh.params).cuda()
    p_last = p.clone()
    pull_res = torch.zeros_like(p)
    idx = [torch.from_numpy(a.view(np.int32)).cuda() for a in sh.idx]
    val = [torch.from_numpy(a).cuda() for a in sh.val]
    comp = gd.Compressor([0, N])
    drop = 0.99
    k = comp.keep_total(drop, False)
    out = comp.alloc_out(drop, False)
    entries = sum(int(a.size) for a in sh.idx)

    use_copy = args.pull == "copy"

    def step(i):
        gd.apply_sparse(p, idx, val, lr=1.0)
        if use_copy:
            comp.compress_pull(p, p_last, drop, per_tensor=False, out=out)
        else:
            comp.compress(p, pull_res, drop, per_tensor=False, base=p_last, out=out)

    # parity of step 0 (apply, then the pull) against the oracle
    step(0)
    torch.cuda.synchronize()
    first_p = p.cpu().numpy().copy()
    first_idx = out.idx[:k].cpu().numpy().view(np.uint32).copy()
    first_res = (p_last if use_copy else pull_res).cpu().numpy().copy()
    p0 = torch.from_numpy(sh.params).cuda()
    p.copy_(p0)
    p_last.copy_(p0)
    pull_res.zero_()
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    scrub = make_scrub(torch, args.scrub)
    comp.profile_enable(DENSE_TIMING_EVERY)
    torch.cuda.synchronize()
    # cold calls, with the apply's share timed by an event between its two parts
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        scrub()
        ev[i][0].record()
        gd.apply_sparse(p, idx, val, lr=1.0)
        ev[i][1].record()
        if use_copy:
            comp.compress_pull(p, p_last, drop, per_tensor=False, out=out)
        else:
            comp.compress(p, pull_res, drop, per_tensor=False, base=p_last, out=out)
        ev[i][2].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    cold = [a.elapsed_time(c) for a, _, c in ev]
    cold_apply = [a.elapsed_time(b) for a, b, _ in ev]
    dense_ms, dense_n = comp.profile_read()
    comp.profile_enable(0)
    warm = time_calls(torch, step, args.warmup + args.steps, args.steps)
    sec = statistics.median(cold) / 1e3
    dense_avg_s = dense_ms / 1e3 / max(dense_n, 1)
    # params and copy read; or params, base and residual read and the changed residual vectors written
    written = 0 if use_copy else written_elements(torch, step, args.warmup + 2 * args.steps, 4, pull_res)
    per_elem = 8 if use_copy else 16
    dense_alg = (8 * N) if use_copy else (12 * N + 4 * written)
    achieved = dense_alg / dense_avg_s / 1e9
    model_bytes = 16 * entries + per_elem * N + 8 * k
    line = {
        "metric": METRIC,
        "value": round(N / sec / 1e9, 3),
        "unit": "G grad-elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(sec * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "hbm_model_frac": round(model_bytes / sec / 1e9 / HBM_PEAK_GBPS, 4),
        "timing": {
            "cold": spread(cold),
            "warm": spread(warm),
            "apply_cold": spread(cold_apply),
            "per_call": "HIP events around each step (apply, then the pull) on its stream; cold calls follow "
                        f"a {'read' if args.scrub == 'read' else 'read-modify-write'} of a {SCRUB_BYTES >> 20} "
                        "MiB scrub buffer; ms_per_step is the cold median",
            "timed_region_s": round(t1 - t0, 4),
        },
        "config": {
            "workload": "shard_apply_pull",
            "elements": N,
            "pushes": len(sh.idx),
            "push_entries": entries,
            "kept_per_step": k,
            "threshold": "global",
            "drop": drop,
            "pull": "from the last pulled copy" if use_copy else "delta with a carried residual",
            "byte_model": f"16 B/push entry + {per_elem} B/element + 8 B/kept element",
        },
        "roofline": {
            "kernel": "k_dense<2>" if use_copy else "k_dense<1>",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": None,
            "algorithmic_bytes": round(dense_alg),
            "bytes_rule": "8 B/element read (params, copy)" if use_copy else
                          "12 B/element read (params, base, residual) + 4 B/element of the 16-byte residual "
                          "vectors the call changes",
            "dense_us": round(dense_avg_s * 1e6, 2),
            "dense_launches": dense_n,
            "dense_timed_every": DENSE_TIMING_EVERY,
        },
    }
    if args.cpu_baseline_seconds > 0:
        import oracle

        lib = oracle.load()
        t0 = time.perf_counter()
        p1 = oracle.apply_sparse(sh.params, sh.idx, sh.val, 1.0, lib=lib)
        if use_copy:
            o, want_state = oracle.compress_pull(p1, sh.params, [0, N], drop, lib=lib)
        else:
            o = oracle.compress(p1, np.zeros(N, np.float32), [0, N], drop, base=sh.params, lib=lib)
            want_state = o.residual
        el = time.perf_counter() - t0
        line["cpu_baseline"] = {
            "value": N / el / 1e9, "unit": "G grad-elements/s", "cores": 1, "kind": "oracle",
            "sample": f"one step (apply of {len(sh.idx)} pushes, then the pull delta) of the 37M shard "
                      f"({el:.1f} s of single-threaded oracle time)",
            **host_info(),
        }
        line["parity_step0"] = bool(np.array_equal(p1.view(np.uint32), first_p.view(np.uint32)) and
                                    np.array_equal(o.idx, first_idx) and
                                    np.array_equal(want_state.view(np.uint32), first_res.view(np.uint32)))
    if emit:
        print(json.dumps(line), flush=True)
    return line


def oracle_quant_step_ok(np, o, idx, val, res, sign_bits, means, offsets, quant, columns=None):
    """One quantised call against the oracle's: sent indices and values and sign bits bit-exact, centres
    within 1e-6 relative (fp64 sums in another order), dropped residuals bit-exact, and every kept
    residual bit-equal to fl32(acc - its own centre) with the GPU's centres."""
    kept = np.zeros(res.size, bool)
    kept[o.idx] = True
    m_o = o.means.astype(np.float64)
    return bool(np.array_equal(o.idx, idx) and np.array_equal(o.val.view(np.uint32), val.view(np.uint32)) and
                np.array_equal(o.sign_bits, sign_bits) and
                np.all(np.abs(means.astype(np.float64) - m_o) <= 1e-6 * np.abs(m_o)) and
                np.array_equal(o.residual[~kept].view(np.uint32), res[~kept].view(np.uint32)) and
                quant_residuals_ok(np, idx, val, sign_bits, means, res, offsets, quant, columns))


def bench_global_signmean(args, torch, np, gd, wl, comp, grads, scrub):
    """The global threshold with per-tensor sign-mean centres (Section 5.4) on the same staged NMT-shaped
    gradients and the same context: its own carried residual, the same cold/warm protocol."""
    N = comp.N
    drop = 0.99
    residual = torch.zeros(N, dtype=torch.float32, device="cuda")
    k = comp.keep_total(drop, False)
    out = comp.alloc_out(drop, False, 1)

    def step(i):
        comp.compress(grads[i % len(grads)], residual, drop, per_tensor=False, quant=1, out=out)

    step(0)
    torch.cuda.synchronize()
    rec = {"idx": out.idx[:k].cpu().numpy().view(np.uint32).copy(), "val": out.val[:k].cpu().numpy().copy(),
           "res": residual.cpu().numpy().copy(),
           "bits": out.sign_bits[:(k + 31) // 32].cpu().numpy().view(np.uint32).copy(),
           "means": out.means[:2 * comp.T].cpu().numpy().copy()}
    residual.zero_()
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    cold = time_calls(torch, step, args.warmup, args.steps, scrub)
    warm = time_calls(torch, step, args.warmup + args.steps, args.steps)
    sec = statistics.median(cold) / 1e3
    rec["line"] = {
        "value": round(N / sec / 1e9, 3),
        "unit": "G grad-elements/s",
        "ms_per_step": round(sec * 1e3, 4),
        "hbm_model_frac": round((12 * N + 8 * k) / sec / 1e9 / HBM_PEAK_GBPS, 4),
        "timing": {"cold": spread(cold), "warm": spread(warm)},
        "config": {"workload": "nmt_85k_global_signmean", "elements": N, "kept_per_step": k,
                   "threshold": "global", "quant": "sign_mean", "drop": drop,
                   "byte_model": "12 B/element + 8 B/kept element"},
    }
    return rec


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the compressor runs per worker and needs no collective)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1704_05021_amd import gd, workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    if args.copy_calibration_mib:
        copy_calibration(args.copy_calibration_mib)
        return
    if args.workload == "shard_apply_pull":
        main_shard(args, torch, np, gd, wl)
        return
    w = wl.workload(args.workload)
    N = w.layout.numel
    off = w.layout.offsets.astype(np.int64).tolist()
    print(f"[bench] generating {w.steps} steps of {w.name} (N={N})", file=sys.stderr, flush=True)
    grads_host = [w.grad(s) for s in range(w.steps)]
    grads = [torch.from_numpy(g).cuda() for g in grads_host]
    residual = torch.zeros(N, dtype=torch.float32, device="cuda")
    comp = gd.Compressor(off)
    sampled = args.selection == "sampled"
    quant = int(w.quant) if args.quant == "workload" else QUANT_KINDS[args.quant]
    if quant == 4:
        comp.set_columns(w.layout.columns)
    if sampled:
        cap = SAMPLED_CAPACITY_PCT * N // 100
        out = comp.alloc_out(1.0, w.per_tensor, quant, capacity=cap)

        def step(i):
            comp.compress_sampled(grads[i % len(grads)], residual, w.drop, per_tensor=w.per_tensor,
                                  sample_ppm=args.sample_ppm, seed=i, out=out, capacity=cap, quant=quant)

        def kept_now():
            return int(out.tensor_counts[:comp.T].cpu().numpy().view(np.uint32).astype(np.int64).sum())
    else:
        k = comp.keep_total(w.drop, w.per_tensor)
        out = comp.alloc_out(w.drop, w.per_tensor, quant)

        def step(i):
            comp.compress(grads[i % len(grads)], residual, w.drop, per_tensor=w.per_tensor, quant=quant,
                          out=out)

        def kept_now():
            return k

    # parity of the benchmarked configuration: step 0 from zero residual vs the oracle
    step(0)
    torch.cuda.synchronize()
    k0 = kept_now()
    first_idx = out.idx[:k0].cpu().numpy().view(np.uint32).copy()
    first_val = out.val[:k0].cpu().numpy().copy()
    first_res = residual.cpu().numpy().copy()
    first_bits = out.sign_bits[:(k0 + 31) // 32].cpu().numpy().view(np.uint32).copy() if quant else None
    first_means = out.means[:comp.quant_centres(quant)].cpu().numpy().copy() if quant else None
    residual.zero_()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    scrub = make_scrub(torch, args.scrub)
    comp.profile_enable(DENSE_TIMING_EVERY)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    cold = time_calls(torch, step, args.warmup, args.steps, scrub)
    t1 = time.perf_counter()
    dense_ms, dense_n = comp.profile_read()
    comp.profile_enable(0)
    warm = time_calls(torch, step, args.warmup + args.steps, args.steps)
    written = written_elements(torch, step, args.warmup + 2 * args.steps, len(grads), residual)

    sec = statistics.median(cold) / 1e3
    value = N / sec / 1e9
    k = kept_now()  # the sampled mode's count varies: the last timed step's
    model_bytes = 12 * N + 8 * k
    dense_avg_s = dense_ms / 1e3 / max(dense_n, 1)
    dense_bytes = 8 * N + 4 * written  # grad and residual read, the changed residual vectors written
    achieved = dense_bytes / dense_avg_s / 1e9
    line = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "G grad-elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(sec * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "hbm_model_frac": round(model_bytes / sec / 1e9 / HBM_PEAK_GBPS, 4),
        "timing": {
            "cold": spread(cold),
            "warm": spread(warm),
            "per_call": "HIP events around each call on its stream; cold calls follow a "
                        f"{'read' if args.scrub == 'read' else 'read-modify-write'} of a {SCRUB_BYTES >> 20} MiB "
                        "scrub buffer; ms_per_step is the cold median",
            "timed_region_s": round(t1 - t0, 4),
        },
        "config": {
            "workload": w.name,
            "elements": N,
            "tensors": w.layout.num_tensors,
            "kept_per_step": k,
            "selection": f"sampled, {args.sample_ppm} ppm sample, count of the last step" if sampled
                         else "exact k-th largest",
            "threshold": "per_tensor" if w.per_tensor else "global",
            "quant": {v: k for k, v in QUANT_KINDS.items()}[quant],
            "drop": w.drop,
            "gradient_steps_cycled": len(grads),
            "byte_model": "12 B/element + 8 B/kept element",
        },
        "roofline": {
            "kernel": "k_dense",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": None if sampled else measured_traffic(w.name),
            "algorithmic_bytes": round(dense_bytes),
            "bytes_rule": "8 B/element read (grad, residual) + 4 B/element of the 16-byte residual vectors "
                          "the call changes",
            "written_fraction": round(written / N, 4),
            "dense_us": round(dense_avg_s * 1e6, 2),
            "dense_launches": dense_n,
            "dense_timed_every": DENSE_TIMING_EVERY,
        },
    }
    extra = None
    if w.name == "nmt_85k_per_tensor" and not sampled and args.quant == "workload" and args.with_global_signmean:
        extra = bench_global_signmean(args, torch, np, gd, wl, comp, grads, scrub)
        line["nmt_85k_global_signmean"] = extra["line"]
    if w.name == "nmt_85k_per_tensor" and not sampled and args.quant == "workload" and args.with_shard:
        # the server step (a7, a8) under the same protocol: its own JSON record, nested
        sl = main_shard(args, torch, np, gd, wl, emit=False)
        line["shard_37m_apply_pull"] = {key: sl[key] for key in ("value", "unit", "ms_per_step", "hbm_model_frac",
                                                                  "timing", "config", "parity_step0") if key in sl}
    if args.cpu_baseline_seconds > 0:
        cb, first = cpu_baseline(w, grads_host, args.cpu_baseline_seconds, args.sample_ppm if sampled else 0, quant)
        line["cpu_baseline"] = cb
        if quant in (0,):  # no float reduction: bit-exact everywhere
            res_ok = np.array_equal(first.residual.view(np.uint32), first_res.view(np.uint32))
        else:
            res_ok = oracle_quant_step_ok(np, first, first_idx, first_val, first_res, first_bits, first_means,
                                          off, quant, w.layout.columns)
        line["parity_step0"] = bool(np.array_equal(first.idx, first_idx) and res_ok)
        if extra is not None:
            import oracle

            o = oracle.compress(grads_host[0], np.zeros(N, np.float32), off, w.drop, per_tensor=False, quant=1)
            line["nmt_85k_global_signmean"]["parity_step0"] = bool(
                np.array_equal(o.idx, extra["idx"]) and
                oracle_quant_step_ok(np, o, extra["idx"], extra["val"], extra["res"], extra["bits"],
                                     extra["means"], off, 1))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
