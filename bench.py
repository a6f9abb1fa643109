#!/usr/bin/env python3
"""Benchmark: the sparse 1x1 convolution on the headline layer.

Workload: Cin = Cout = 512, 14x14, batch 256, 90% sparse weights, fp32, ReLU
epilogue -- the 512x512 layer of the sparsity sweep.  The unstructured mask is
the headline (``value``); the 1x4 output-channel-blocked mask of the same
sweep point is reported beside it.  Inputs are seeded synthetic tensors with
the paper's layer shapes (no trained weights or images are used).

One step = one spconv_run over the whole batch (bias and activation fused).
Inputs are resident in HBM before timing starts; three (X, Y) buffer sets,
616 MB in all, rotate so no step finds its operands in the 256 MB
last-level cache.  Kernel durations come from HIP events recorded on the
launch stream around every launch.

Prints one JSON line.  ``--gpus`` above 1 is refused: this build measures one GPU.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E peak
FP32_VECTOR_PEAK_TFS = 157.3  # MI355X fp32 vector peak (packed FMA)
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_spmm_strip_512_14_b256.json")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_1911_09723_amd", "csrc", f)
                  for f in ("spmm_kernels.hip", "planner.cpp", "planner.hpp")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """Per-launch HBM bytes from the committed rocprofv3 counter runs, if they
    were taken on the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_hash") != kernel_source_hash():
        return None
    return t


def time_variant(layer, steps, warmup, sets):
    import torch
    from paper_1911_09723_amd import Plan, spconv_run

    dev = torch.device("cuda:0")
    plan = Plan.from_layer(layer)
    n, c, h, w = layer.x.shape
    x0 = torch.from_numpy(layer.x).to(dev)
    xs = [x0] + [x0.clone() for _ in range(sets - 1)]
    ys = [torch.empty((n, layer.cout, h, w), dtype=x0.dtype, device=dev) for _ in range(sets)]
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        spconv_run(plan.handle, xs[i % sets], ys[i % sets], n, h, w, stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for i in range(steps):
        ev[i][0].record(stream)
        spconv_run(plan.handle, xs[i % sets], ys[i % sets], n, h, w, stream)
        ev[i][1].record(stream)
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    region_ms = t_start.elapsed_time(t_end)
    kern_ms = [a.elapsed_time(b) for a, b in ev]
    info = plan.info()
    plan.close()
    del xs, ys
    torch.cuda.empty_cache()
    return dict(region_ms=region_ms, wall_s=wall, kernel_ms=kern_ms, info=info)


def cpu_baseline(layer, budget_s=12.0):
    """The oracle on the first images of the batch, timed on this host."""
    import numpy as np
    import oracle

    oracle.build(force=False)
    t0 = time.perf_counter()
    oracle.spconv_ref_layer(layer, x=layer.x[:1], with_scale=False)
    t1 = time.perf_counter() - t0
    n_s = int(max(1, min(layer.n, budget_s / max(t1, 1e-6))))
    t0 = time.perf_counter()
    oracle.spconv_ref_layer(layer, x=np.ascontiguousarray(layer.x[:n_s]), with_scale=False)
    dt = time.perf_counter() - t0
    return {
        "value": round(layer.flops(n_s) / dt / 1e9, 3),
        "unit": "effective GFLOP/s",
        "cores": oracle.threads(),
        "kind": "oracle",
        "sample": "%d of %d images of the same layer (fp64 accumulation, OpenMP over images x rows), %.1f s"
                  % (n_s, layer.n, dt),
    }


def summarize(layer, r):
    import numpy as np
    steps = len(r["kernel_ms"])
    t_step = r["region_ms"] / steps / 1e3
    t_kern = float(np.mean(r["kernel_ms"])) / 1e3
    flops = layer.flops()
    b_alg = layer.alg_bytes()
    t_roof = max(b_alg / (HBM_PEAK_GBS * 1e9), flops / (FP32_VECTOR_PEAK_TFS * 1e12))
    return {
        "gflops_effective": round(flops / t_step / 1e9, 1),
        "ms_per_step": round(t_step * 1e3, 5),
        "kernel_us_mean": round(t_kern * 1e6, 3),
        "kernel_us_min": round(min(r["kernel_ms"]) * 1e3, 3),
        "hbm_gbs_algorithmic": round(b_alg / t_kern / 1e9, 1),
        "roofline_us": round(t_roof * 1e6, 3),
        "roofline_frac": round(t_roof / t_kern, 4),
        "bound": "hbm" if b_alg / (HBM_PEAK_GBS * 1e9) >= flops / (FP32_VECTOR_PEAK_TFS * 1e12) else "fp32",
        "nnz": layer.nnz,
        "alg_bytes": b_alg,
        "flops": flops,
        "plan": {k: r["info"][k] for k in ("kernel", "lanes_per_row", "tile_cols", "waves", "lds_bytes",
                                           "slots")},
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--sets", type=int, default=3, help="rotating (X, Y) buffer sets")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (got --gpus %d)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import torch
    from synth.configs import TARGET, config_layers, build

    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a ROCm GPU")
    specs = [s for s in config_layers(TARGET["config"]) if s["layer"] == TARGET["layer"]]
    results = {}
    layers = {}
    for spec in specs:
        tag = "1x%d" % spec["block_rows"]
        log("bench: generating %s" % spec["name"])
        layer = build(TARGET["config"], spec)
        layers[tag] = layer
        log("bench: timing %s (%d warmup, %d steps, %d buffer sets)" % (tag, args.warmup, args.steps, args.sets))
        r = time_variant(layer, args.steps, args.warmup, args.sets)
        results[tag] = summarize(layer, r)
        log("bench: %s %s" % (tag, json.dumps(results[tag])))

    head = results["1x1"]
    layer = layers["1x1"]
    traffic = measured_traffic()
    achieved = head["hbm_gbs_algorithmic"]
    line = {
        "metric": "effective GFLOP/s (2*nnz*HW*N) + HBM GB/s % peak, sparse 1x1 conv",
        "value": head["gflops_effective"],
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "sparse 1x1 conv 512->512 @14x14, batch 256, 90% unstructured sparsity, fp32, ReLU",
            "cin": 512, "cout": 512, "h": 14, "w": 14, "batch": 256, "sparsity": 0.9, "block_rows": 1,
            "nnz": layer.nnz, "buffer_sets": args.sets,
        },
        "hbm_gbs": achieved,
        "hbm_pct_peak": round(100 * achieved / HBM_PEAK_GBS, 2),
        "roofline": {
            "bound": head["bound"],
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None if traffic is None else traffic["bytes_per_launch"],
        },
        "variants": results,
        "device": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle")
        line["cpu_baseline"] = cpu_baseline(layer, args.cpu_budget)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
