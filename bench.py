#!/usr/bin/env python3
"""Throughput of the gradient-dropping compressor on one MI355X.

A step is one gd_compress call (residual add, exact k-th largest |acc|
selection, ordered compaction, residual write-back) over one NMT-shaped
gradient set of 136,875,744 fp32 elements in 27 tensors (three 85000x500
embeddings with Zipf-sparse rows plus GRU-shaped dense tensors), per-tensor
threshold, 99% drop.  Ten seeded gradient steps are staged in HBM before
timing; timed steps cycle through them with the residual carried.

Prints one JSON line.  ``value`` is gradient elements compressed per second
(whole job, inputs resident in HBM).  ``roofline`` reports the dense pass
(the kernel that streams grad and residual) against the 8 TB/s HBM peak under
the 12-bytes-per-element model; ``cpu_baseline`` times the CPU oracle on a
bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "G grad-elements/s compressed at 99% drop; % of HBM peak (1 GPU)"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="nmt_85k_per_tensor")
    ap.add_argument("--cpu-baseline-seconds", type=float, default=12.0,
                    help="rough bound on oracle CPU time for the cpu_baseline leg (0 disables it)")
    return ap.parse_args()


def cpu_baseline(w, grads_host, budget_s):
    """The oracle, single-threaded, on the first steps of the same workload."""
    import numpy as np

    import oracle

    off = w.layout.offsets.astype(np.int64).tolist()
    residual = np.zeros(w.layout.numel, np.float32)
    done, elapsed, first = 0, 0.0, None
    lib = oracle.load()
    while done < len(grads_host) and (done == 0 or elapsed < budget_s * 0.6):
        t0 = time.perf_counter()
        o = oracle.compress(grads_host[done], residual, off, w.drop, per_tensor=w.per_tensor, quant=w.quant, lib=lib)
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
        "sample": f"{done} consecutive steps of {w.name} from zero residual ({elapsed:.1f} s of oracle time)",
    }, first


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
    w = wl.workload(args.workload)
    N = w.layout.numel
    off = w.layout.offsets.astype(np.int64).tolist()
    print(f"[bench] generating {w.steps} steps of {w.name} (N={N})", file=sys.stderr, flush=True)
    grads_host = [w.grad(s) for s in range(w.steps)]
    grads = [torch.from_numpy(g).cuda() for g in grads_host]
    residual = torch.zeros(N, dtype=torch.float32, device="cuda")
    comp = gd.Compressor(off)
    k = comp.keep_total(w.drop, w.per_tensor)
    out = comp.alloc_out(w.drop, w.per_tensor, w.quant)

    def step(i):
        comp.compress(grads[i % len(grads)], residual, w.drop, per_tensor=w.per_tensor, quant=w.quant, out=out)

    # parity of the benchmarked configuration: step 0 from zero residual vs the oracle
    step(0)
    torch.cuda.synchronize()
    first_idx = out.idx[:k].cpu().numpy().view(np.uint32).copy()
    first_res = residual.cpu().numpy().copy()
    residual.zero_()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    comp.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    dense_ms, dense_n = comp.profile_read()
    comp.profile_enable(False)

    sec = (t1 - t0) / args.steps
    value = N / sec / 1e9
    model_bytes = 12 * N + 8 * k
    dense_avg_s = dense_ms / 1e3 / max(dense_n, 1)
    achieved = 12 * N / dense_avg_s / 1e9
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
        "config": {
            "workload": w.name,
            "elements": N,
            "tensors": w.layout.num_tensors,
            "kept_per_step": k,
            "threshold": "per_tensor" if w.per_tensor else "global",
            "quant": "sign_mean" if w.quant else "none",
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
            "traffic": None,
            "dense_us": round(dense_avg_s * 1e6, 2),
            "dense_launches": dense_n,
        },
    }
    if args.cpu_baseline_seconds > 0:
        cb, first = cpu_baseline(w, grads_host, args.cpu_baseline_seconds)
        line["cpu_baseline"] = cb
        line["parity_step0"] = bool(np.array_equal(first.idx, first_idx) and
                                    np.array_equal(first.residual.view(np.uint32), first_res.view(np.uint32)))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
