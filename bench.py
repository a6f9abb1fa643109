#!/usr/bin/env python3
"""Benchmark: the sparse 1x1 convolution on the headline layer.

Workload: Cin = Cout = 512, 14x14, batch 256, 90% sparse weights, fp32, ReLU
epilogue -- the 512x512 layer of the sparsity sweep.  The unstructured mask is
the headline (``value``); the 1x4 output-channel-blocked mask of the same
sweep point is reported beside it, and so are blocks of 4 input channels
("4x1 in") and of 2 x 2 channels ("2x2 in").  Inputs are seeded synthetic tensors with
the paper's layer shapes (no trained weights or images are used).

One step = one spconv_run over the whole batch (bias and activation fused).
The "1x1 indexed" and "1x4 indexed" variants run the same layers on the
register-indexed kernel (kernel=3) instead of the automatic choice.
A third variant runs the same 1x1 behind a fused depthwise 3x3 (stride 1,
ReLU6): one MobileNet v1 block at 512 channels.  The ``network`` entries time
a whole synthetic MobileNet v1 forward pass (one graph replay) at batch 1
and 64.
Inputs are resident in HBM before timing starts; three (X, Y) buffer sets,
616 MB in all, rotate so no step finds its operands in the 256 MB
last-level cache.  The kernel's mean duration is one pair of HIP events on
the launch stream around the timed region of back-to-back launches, divided
by the launch count; a second pass with an event pair around every launch
gives the minimum and ``event_pair_us_mean`` (each event pair adds its own
cost, a few microseconds).

The ``configs`` list times every layer of every workload configuration (c0
.. c4: the small parity layer, MobileNet v1's pointwise layers at batch 1
and 64, the 512x512 sparsity sweep, the MobileNet v2-like heavy-tail
layers, and the fp16 layers), each on the automatic kernel and, for fp32,
on the register-indexed kernel, with kernel time, effective GFLOP/s,
algorithmic GB/s, bound and roofline fraction (the per-layer view of paper
Sec. 4.1 / Fig. 4).  ``--config C`` runs only configuration C's sweep (for
rocprofv3 kernel traces).

The CPU baseline is the oracle, built for this host (gcc -O3 -march=native,
no floating-point contraction), timed in child processes: the median of 3
runs on the headline layer with all threads (``value``), and 1-thread runs on
the headline layer and on c0, each also the median of 3.

Prints one JSON line.  ``--gpus`` above 1 is refused: this build measures one GPU.

Two more modes produce the HBM-traffic figures of the ``roofline`` object:
  --profile-run            a few launches of each variant, then a plain copy
                           kernel of known size (run under rocprofv3 --pmc)
  --traffic-summary F W    read the FETCH_SIZE (F) and WRITE_SIZE (W) counter
                           directories of two such runs, scale each counter by
                           what it read for the copy, and write
                           profiles/traffic_spmm_pipe_512x512_14x14_b256.{json,md}
"""

from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0         # MI355X HBM3E peak
FP32_VECTOR_PEAK_TFS = 157.3  # MI355X fp32 vector peak (packed FMA)
TRAFFIC_BASE = os.path.join(ROOT, "profiles", "traffic_spmm_pipe_512x512_14x14_b256")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_1911_09723_amd", "csrc", f)
                  for f in ("spmm_kernels.hip", "spmm_indexed.hip", "spmm_outer.hip", "planner.cpp", "planner.hpp")]
COPY_BYTES = 256 << 20        # calibration copy: 256 MiB read + 256 MiB written
CALIBRATION_KERNEL = "neg_kernel"  # torch.neg(a, out=b): a plain elementwise copy
METRIC = "effective GFLOP/s (2*nnz*HW*N) + HBM GB/s % peak, sparse 1x1 conv"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """Per-launch HBM bytes from the committed counter runs, if they were taken
    on the current kernel source; else None."""
    try:
        with open(TRAFFIC_BASE + ".json") as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_hash") != kernel_source_hash():
        return None
    return t


def headline_layers(input_blocks=True):
    """The headline layer, unstructured and 1x4 (output-channel blocks), and
    with input-channel blocks of 4 (4x1) and 2 x 2 at the same sparsity, same
    seed recipe."""
    from synth import make_layer
    from synth.configs import TARGET, config_layers, build, layer_seed
    specs = [s for s in config_layers(TARGET["config"]) if s["layer"] == TARGET["layer"]]
    out = {}
    for spec in specs:
        tag = "1x%d" % spec["block_rows"]
        log("bench: generating %s" % spec["name"])
        out[tag] = build(TARGET["config"], spec)
    if input_blocks:
        spec = specs[0]
        for vi, (kr, kc) in enumerate(((1, 4), (2, 2)), start=2):
            tag = "%dx%d in" % (kc, kr)
            log("bench: generating %s with %d x %d blocks (output x input channels)" % (spec["name"], kr, kc))
            out[tag] = make_layer(spec["cin"], spec["cout"], spec["h"], spec["w"], spec["n"], spec["sparsity"],
                                  block_rows=kr, block_cols=kc, act=spec["act"],
                                  seed=layer_seed(TARGET["config"], TARGET["layer"], vi))
    return out


def fused_layer(layer):
    """The headline layer's 1x1 weights and input with a depthwise 3x3 stage
    (stride 1, ReLU6) in front: one MobileNet v1 block at 512 channels."""
    from synth import make_depthwise
    kw, kb = make_depthwise(layer.cin, 2021)
    return kw, kb


def time_variant(layer, steps, warmup, sets, dw=None, **options):
    import torch
    from paper_1911_09723_amd import Plan, spconv_run

    dev = torch.device("cuda:0")
    if dw is None:
        plan = Plan.from_layer(layer, **options)
    else:
        plan = Plan.fused(layer.cout, layer.cin, layer.block_rows, layer.row_ptr, layer.col_idx, layer.values,
                          layer.bias, layer.act, dw[0], dw[1], "relu6", 1)
    n, c, h, w = layer.x.shape
    x0 = torch.from_numpy(layer.x).to(dev)
    xs = [x0] + [x0.clone() for _ in range(sets - 1)]
    ys = [torch.empty((n, layer.cout) + plan.out_hw(h, w), dtype=x0.dtype, device=dev) for _ in range(sets)]
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        spconv_run(plan.handle, xs[i % sets], ys[i % sets], n, h, w, stream)
    # The timed region: `steps` launches back to back between one pair of
    # HIP events on the launch stream (its mean is the kernel's average
    # duration plus the launch gaps; an event pair around every launch would
    # add each event's own cost), then a second pass with an event pair per
    # launch for the spread (min, and the per-launch mean it reports).
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for i in range(steps):
        spconv_run(plan.handle, xs[i % sets], ys[i % sets], n, h, w, stream)
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    region_ms = t_start.elapsed_time(t_end)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for i in range(steps):
        ev[i][0].record(stream)
        spconv_run(plan.handle, xs[i % sets], ys[i % sets], n, h, w, stream)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    kern_ms = [a.elapsed_time(b) for a, b in ev]
    info = plan.info()
    flags = plan.check(clear=True)
    plan.close()
    if flags:
        raise RuntimeError("a bounded wait gave up during the timed launches (error word %d)" % flags)
    del xs, ys
    torch.cuda.empty_cache()
    return dict(region_ms=region_ms, wall_s=wall, kernel_ms=kern_ms, info=info, forced_kernel=options.get("kernel"))


def time_network(batch, steps, warmup, graph=True):
    """Whole MobileNet v1 forward passes (synthetic 90%-sparse weights,
    224 x 224 images) replayed as one captured graph; per-replay time from
    HIP events on the replay stream."""
    import numpy as np
    import torch
    from paper_1911_09723_amd.mobilenet import MobileNetV1Engine
    from synth import make_mobilenet_v1, make_image

    net = make_mobilenet_v1(seed=0)
    eng = MobileNetV1Engine(net, batch)
    eng.x.copy_(torch.from_numpy(make_image(batch, seed=0)).to(eng.x.device))
    if graph:
        eng.capture()
    run = eng.replay if graph else eng.forward
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        run()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        ev[i][0].record(stream)
        run()
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    launches = eng.launches()
    layers = list(eng.layers)
    fused = eng.fused_blocks
    fusion_times = list(eng.fusion_times)
    eng.close()
    torch.cuda.empty_cache()
    b_alg = network_alg_bytes(net, batch)
    t = float(ms.mean()) / 1e3
    return {
        "model": "MobileNet v1 1.0 224x224, 90%-sparse pointwise layers, synthetic weights",
        "batch": batch, "graph": graph, "launches": launches, "layers": layers,
        "ms_per_batch_mean": round(float(ms.mean()), 4), "ms_per_batch_min": round(float(ms.min()), 4),
        "images_per_s": round(batch / t, 1), "fused_blocks": fused,
        "fusion_times_ms": fusion_times,
        "alg_bytes": b_alg, "hbm_gbs_algorithmic": round(b_alg / t / 1e9, 1),
        "roofline_frac": round(b_alg / (HBM_PEAK_GBS * 1e9) / t, 4),
    }


def network_alg_bytes(net, batch, h=224):
    """HBM bytes a forward pass must move at least, fp32: the image, the
    stem's output, every block's input and output once (the depthwise output
    counted as staying on chip, as in a fused block, whether or not the
    engine fuses it) and every weight once."""
    e = 4
    hs = (h - 1) // 2 + 1
    c0 = net.stem_w.shape[0]
    total = batch * (h * h * 3 + c0 * hs * hs) + net.stem_w.size + net.stem_b.size
    hh = hs
    for i, blk in enumerate(net.blocks):
        ho = (hh - 1) // blk.stride + 1
        total += batch * (blk.cin * hh * hh + blk.cout * ho * ho)
        pw = blk.pw
        total += blk.dw_k.size + blk.dw_b.size + pw.nnz + pw.nnzb + pw.row_ptr.size + pw.bias.size
        hh = ho
    cl = net.blocks[-1].cout
    total += batch * (cl * hh * hh + cl) + batch * (cl + net.fc_w.shape[0]) + net.fc_w.size + net.fc_b.size
    return float(total * e)


def sweep_configs(configs, steps, warmup, indexed=True):
    """Every layer of the given workload configurations on the automatic
    kernel, on the register-indexed kernel (fp32) and on the outer-product
    kernel (1x4 blocks)."""
    from synth import config_layers
    from synth.configs import build

    out = []
    for c in configs:
        for spec in config_layers(c):
            layer = build(c, spec)
            entry = {"config": "c%d" % c, "layer": spec["name"], "cin": layer.cin, "cout": layer.cout,
                     "h": layer.h, "w": layer.w, "batch": layer.n, "sparsity": spec["sparsity"],
                     "block_rows": layer.block_rows, "pattern": spec["pattern"], "storage": layer.storage}
            kinds = [("auto", {})]
            if indexed and layer.storage == "f32":
                kinds.append(("indexed", {"kernel": 3}))
            if indexed and layer.block_rows == 4 and layer.cin <= 632:
                kinds.append(("outer", {"kernel": 4}))
            for kind, opts in kinds:
                r = time_variant(layer, steps, warmup, 2, **opts)
                sm = summarize(layer, r)
                entry[kind] = {k: sm[k] for k in ("kernel_us_mean", "kernel_us_min", "gflops_effective",
                                                   "hbm_gbs_algorithmic", "bound", "roofline_us", "roofline_frac")}
                entry[kind]["ms"] = round(sm["kernel_us_mean"] / 1e3, 5)
                entry[kind]["kernel"] = sm["plan"]["kernel_run"]
                if "device_weight_extra_bytes" in sm:
                    entry[kind]["device_weight_extra_bytes"] = sm["device_weight_extra_bytes"]
            entry["alg_bytes"] = layer.alg_bytes()
            entry["flops"] = layer.flops()
            out.append(entry)
            log("bench: %s %s auto %.1f us (%s, frac %.3f)%s%s" % (
                entry["config"], spec["name"], entry["auto"]["kernel_us_mean"], entry["auto"]["kernel"],
                entry["auto"]["roofline_frac"],
                "  indexed %.1f us" % entry["indexed"]["kernel_us_mean"] if "indexed" in entry else "",
                "  outer %.1f us" % entry["outer"]["kernel_us_mean"] if "outer" in entry else ""))
            del layer
    return out


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def native_oracle(path):
    """The oracle's C source built for this host: -O3 -march=native, OpenMP,
    no floating-point contraction (the same arithmetic as the tests' build)."""
    import subprocess
    import oracle
    src = os.path.join(os.path.dirname(oracle.__file__), "spconv_ref.c")
    cmd = ["gcc", "-O3", "-march=native", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared", "-o", path, src, "-lm"]
    subprocess.check_call(cmd)
    return " ".join(cmd[:6])


def cpu_leg(lib_path, budget_s):
    """Child process of the CPU baseline: time the oracle (the library at
    lib_path) on the headline layer and on c0, 3 runs each, with the threads
    OMP_NUM_THREADS gives; print one JSON line."""
    import numpy as np
    import oracle
    from synth import config_layers
    from synth.configs import TARGET, build

    lib = oracle.load_library(lib_path)

    def run(layer, x):
        oracle.spconv_ref(layer.cout, layer.cin, layer.block_rows, layer.row_ptr, layer.col_idx, layer.values,
                          layer.bias, layer.act, x, storage=layer.storage, with_scale=False, lib=lib)

    spec_t = [sp for sp in config_layers(TARGET["config"]) if sp["layer"] == TARGET["layer"]][0]
    layers = {"target": build(TARGET["config"], spec_t), "c0": build(0, config_layers(0)[0])}
    out = {"threads": int(lib.spconv_ref_threads())}
    for name, layer in layers.items():
        # a warm-up pass sizes the runs: each run is `reps` passes over n_s
        # images, about budget_s / 3 seconds of work
        n_w = min(layer.n, 8)
        run(layer, layer.x[:n_w])
        t0 = time.perf_counter()
        run(layer, layer.x[:n_w])
        t_img = max(time.perf_counter() - t0, 1e-6) / n_w
        n_s = int(max(1, min(layer.n, budget_s / 3.0 / t_img)))
        reps = int(max(1, min(1000, budget_s / 3.0 / (t_img * n_s))))
        xs = np.ascontiguousarray(layer.x[:n_s])
        runs = []
        for _ in range(3):
            t0 = time.perf_counter()
            for _ in range(reps):
                run(layer, xs)
            runs.append(reps * layer.flops(n_s) / (time.perf_counter() - t0) / 1e9)
        out[name] = {"gflops_runs": [round(v, 3) for v in runs], "gflops_median": round(float(np.median(runs)), 3),
                     "images": n_s, "of": layer.n, "passes": reps}
    print(json.dumps(out), flush=True)


def cpu_baseline(budget_s=8.0):
    """The oracle as it stands, built for this host, timed in child processes
    with all threads and with one (see the module docstring)."""
    import subprocess
    import tempfile
    d = tempfile.mkdtemp(prefix="spconv_oracle_")
    lib = os.path.join(d, "libspconv_ref_native.so")
    build_cmd = native_oracle(lib)
    res = {}
    for threads in (None, 1):
        env = dict(os.environ)
        if threads:
            env["OMP_NUM_THREADS"] = str(threads)
        out = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-leg", lib, "--cpu-budget",
                              str(budget_s)], env=env, capture_output=True, text=True, check=True)
        res[threads or "all"] = json.loads(out.stdout.strip().splitlines()[-1])
    a, one = res["all"], res[1]
    return {
        "value": a["target"]["gflops_median"],
        "unit": "GFLOP/s",
        "cores": a["threads"],
        "kind": "oracle",
        "sample": "median of 3 runs, each %d pass(es) over %d of %d images of the headline layer (fp64 "
                  "accumulation, OpenMP over images x rows)" % (a["target"]["passes"], a["target"]["images"],
                                                                a["target"]["of"]),
        "runs": a["target"]["gflops_runs"],
        "one_thread": {"target": one["target"], "c0": one["c0"]},
        "c0_all_threads": a["c0"],
        "cpu_model": cpu_model(),
        "build": build_cmd,
    }


def summarize(layer, r, dw=False):
    import numpy as np
    steps = len(r["kernel_ms"])
    t_step = r["region_ms"] / steps / 1e3
    t_kern = t_step  # back-to-back launches in the timed region
    t_launch = float(np.mean(r["kernel_ms"])) / 1e3  # the per-launch event pairs
    flops = layer.flops()
    b_alg = layer.alg_bytes()
    if dw:
        # stride 1: the depthwise input has the output's size, so X and Y
        # traffic are as for the 1x1 alone; add the 3x3 taps (2 flops each)
        # and the depthwise parameters
        flops += 2.0 * 9 * layer.cin * layer.hw * layer.n
        b_alg += 4.0 * 10 * layer.cin
    t_hbm = b_alg / (HBM_PEAK_GBS * 1e9)
    t_alu = flops / (FP32_VECTOR_PEAK_TFS * 1e12)
    t_roof = max(t_hbm, t_alu)
    out = {
        "gflops_effective": round(flops / t_step / 1e9, 1),
        "ms_per_step": round(t_step * 1e3, 5),
        "kernel_us_mean": round(t_kern * 1e6, 3),
        "kernel_us_min": round(min(r["kernel_ms"]) * 1e3, 3),
        "event_pair_us_mean": round(t_launch * 1e6, 3),
        "hbm_gbs_algorithmic": round(b_alg / t_kern / 1e9, 1),
        "roofline_us": round(t_roof * 1e6, 3),
        "roofline_frac": round(t_roof / t_kern, 4),
        "bound": "hbm" if t_hbm >= t_alu else "alu",
        "nnz": layer.nnz,
        "alg_bytes": b_alg,
        # strip reads from LDS: every packed slot reads one 256-byte strip row
        # per tile (the on-chip traffic that bounds the unstructured kernel)
        "lds_strip_read_bytes": r["info"]["slots"] * 256 * -(-layer.n * layer.hw // r["info"]["tile_cols"]),
        "flops": flops,
        "plan": {k: r["info"][k] for k in ("kernel", "group_lanes", "tile_cols", "waves", "lds_bytes", "slots",
                                           "max_parts", "indexed_min_cols")},
    }
    # the kernel the runs took, as spconv_run chooses it: outer-product, then
    # register-indexed (forced, or automatic for this many columns), else the
    # plan's LDS-strip or direct-load kernel
    cols = layer.n * layer.hw
    imc = r["info"]["indexed_min_cols"]
    omc = r["info"]["outer_min_cols"]
    forced = r.get("forced_kernel")
    if forced == 4 or (forced in (None, 0) and omc > 0 and cols >= omc):
        run = "outer"
    elif forced == 3 or (forced in (None, 0) and imc > 0 and cols >= imc):
        run = "indexed"
    else:
        run = "direct" if r["info"]["kernel"] == 1 else "strip"
    out["plan"]["kernel_run"] = run
    out["plan"]["outer_min_cols"] = omc
    if layer.storage == "f16":
        # fp16 plans round W to fp16 but keep it as fp32 in device memory: the
        # weights move 4 bytes per value, not the 2 alg_bytes counts
        out["device_weight_extra_bytes"] = 2.0 * layer.nnz
    return out


def profile_run(reps: int):
    """A few launches of each variant (the unstructured layer first), then the
    calibration copy (for rocprofv3)."""
    import torch
    from paper_1911_09723_amd import Plan, spconv_run

    dev = torch.device("cuda:0")
    layers = headline_layers(input_blocks=False)
    runs = [(tag, layer, None) for tag, layer in layers.items()]
    runs.append(("dw3x3+1x1", layers["1x1"], fused_layer(layers["1x1"])))
    for tag, layer, dw in runs:
        if dw is None:
            plan = Plan.from_layer(layer)
        else:
            plan = Plan.fused(layer.cout, layer.cin, layer.block_rows, layer.row_ptr, layer.col_idx, layer.values,
                              layer.bias, layer.act, dw[0], dw[1], "relu6", 1)
        n, c, h, w = layer.x.shape
        x0 = torch.from_numpy(layer.x).to(dev)
        xs = [x0, x0.clone(), x0.clone()]  # the bench's three rotating buffer sets
        ys = [torch.empty((n, layer.cout, h, w), dtype=x0.dtype, device=dev) for _ in range(3)]
        for i in range(reps):
            spconv_run(plan.handle, xs[i % 3], ys[i % 3], n, h, w)
        torch.cuda.synchronize()
        plan.close()
        del xs, ys, x0
        torch.cuda.empty_cache()
        log("profile-run: %s done" % tag)
    a = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    for _ in range(reps):
        torch.neg(a, out=b)  # a plain copy: reads and writes COPY_BYTES once each
    torch.cuda.synchronize()
    log("profile-run: copy of %d bytes done" % COPY_BYTES)


def _read_counter_dir(d, counter):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit("no counter_collection.csv under %s" % d)
    per = {}
    for f in files:
        for row in csv.DictReader(open(f)):
            if row["Counter_Name"] != counter:
                continue
            key = (row["Kernel_Name"], int(row["Dispatch_Id"]))
            per[key] = per.get(key, 0.0) + float(row["Counter_Value"])
    return per


def _layer_kernel(name):
    """A kernel of the sparse 1x1 (strip, direct, register-indexed or outer-product)."""
    return "spmm" in name or "outer_kernel" in name


def traffic_summary(fetch_dir, write_dir, commands, out_base):
    """Scale FETCH_SIZE / WRITE_SIZE (KiB per dispatch) by the copy kernel's
    reading and write the per-launch HBM traffic of the headline kernel."""
    import numpy as np
    out = {"kernel_source_hash": kernel_source_hash(), "copy_bytes": COPY_BYTES, "commands": commands}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        per = _read_counter_dir(d, counter)
        copy = [v for (k, _), v in per.items() if CALIBRATION_KERNEL in k]
        if not copy:
            raise SystemExit("no calibration copy dispatch found in %s" % d)
        copy_kib = float(np.median(copy))
        factor = COPY_BYTES / (copy_kib * 1024.0)
        out[counter] = {"copy_kib_per_dispatch": copy_kib, "factor": factor, "kernels": {}}
        kinds = sorted({k for (k, _) in per if _layer_kernel(k)})
        for k in kinds:
            vals = [v for (kk, _), v in per.items() if kk == k]
            out[counter]["kernels"][k] = {"kib_per_dispatch": float(np.median(vals)), "dispatches": len(vals),
                                          "bytes_scaled": float(np.median(vals)) * 1024.0 * factor}
    # the headline kernel: --profile-run launches the unstructured layer first,
    # so its kernel is the spmm kernel of the lowest dispatch id
    firsts = sorted((d, k) for (k, d) in _read_counter_dir(fetch_dir, "FETCH_SIZE") if _layer_kernel(k))
    if firsts:
        k = firsts[0][1]
        out["headline_kernel"] = k
        out["bytes_per_launch"] = round(out["FETCH_SIZE"]["kernels"][k]["bytes_scaled"] +
                                        out["WRITE_SIZE"]["kernels"].get(k, {}).get("bytes_scaled", 0.0))
    os.makedirs(os.path.dirname(out_base), exist_ok=True)
    with open(out_base + ".json", "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
    lines = ["# HBM traffic per launch: sparse 1x1 conv 512->512 @14x14, batch 256, 90%", "",
             "Counters FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each from its own rocprofv3 run, "
             "scaled by the factor that maps the same counter's reading for a plain copy of %d bytes "
             "(read once, written once) to that size." % COPY_BYTES, "", "Commands:", ""]
    lines += ["    " + c for c in commands]
    lines += ["", "| counter | copy KiB/dispatch | factor |", "|---|---|---|"]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        lines.append("| %s | %.0f | %.4f |" % (c, out[c]["copy_kib_per_dispatch"], out[c]["factor"]))
    lines += ["", "| kernel | counter | KiB/dispatch | scaled MB |", "|---|---|---|---|"]
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        for k, v in out[c]["kernels"].items():
            m = re.search(r"(spmm_\w+|outer_kernel)<[^>]*>", k)
            lines.append("| `%s` | %s | %.0f | %.2f |" % (m.group(0) if m else k, c, v["kib_per_dispatch"],
                                                          v["bytes_scaled"] / 1e6))
    if "bytes_per_launch" in out:
        lines += ["", "Headline kernel: %.2f MB per launch (fetch + write, scaled)." % (out["bytes_per_launch"] / 1e6)]
    lines += ["", "kernel source hash: %s" % out["kernel_source_hash"]]
    with open(out_base + ".md", "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps({k: out[k] for k in ("bytes_per_launch", "headline_kernel") if k in out}))


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--sets", type=int, default=3, help="rotating (X, Y) buffer sets")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=8.0, help="seconds of oracle work per layer and thread count")
    ap.add_argument("--profile-run", action="store_true", help="launches for rocprofv3 counter passes")
    ap.add_argument("--reps", type=int, default=5, help="launches per variant in --profile-run")
    ap.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--no-network", action="store_true", help="skip the MobileNet v1 timing")
    ap.add_argument("--network-run", action="store_true",
                    help="only the MobileNet v1 graph replays (batch 64), for rocprofv3 kernel traces")
    ap.add_argument("--command", action="append", default=[], help="command lines recorded in the summary")
    ap.add_argument("--out", default=TRAFFIC_BASE, help="output path (without extension) of --traffic-summary")
    ap.add_argument("--config", type=int, help="only the per-layer sweep of workload configuration C (0 .. 4)")
    ap.add_argument("--no-sweep", action="store_true", help="skip the per-configuration layer sweep")
    ap.add_argument("--sweep-steps", type=int, default=20, help="timed launches per layer in the sweep")
    ap.add_argument("--cpu-leg", metavar="LIB", help=argparse.SUPPRESS)
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (got --gpus %d)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    if args.traffic_summary:
        traffic_summary(args.traffic_summary[0], args.traffic_summary[1], args.command, args.out)
        return
    if args.cpu_leg:
        cpu_leg(args.cpu_leg, args.cpu_budget)
        return

    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a ROCm GPU")
    if args.profile_run:
        profile_run(args.reps)
        return
    if args.network_run:
        print(json.dumps(time_network(64, args.steps, args.warmup)), flush=True)
        return
    if args.config is not None:
        print(json.dumps(sweep_configs([args.config], args.sweep_steps, 3)), flush=True)
        return

    layers = headline_layers()
    results = {}
    for tag, layer in layers.items():
        log("bench: timing %s (%d warmup, %d steps, %d buffer sets)" % (tag, args.warmup, args.steps, args.sets))
        r = time_variant(layer, args.steps, args.warmup, args.sets)
        results[tag] = summarize(layer, r)
        log("bench: %s %s" % (tag, json.dumps(results[tag])))
    # the same 1x1 behind a fused depthwise 3x3 (stride 1, ReLU6)
    tag = "dw3x3+1x1"
    log("bench: timing %s" % tag)
    r = time_variant(layers["1x1"], args.steps, args.warmup, args.sets, dw=fused_layer(layers["1x1"]))
    results[tag] = summarize(layers["1x1"], r, dw=True)
    log("bench: %s %s" % (tag, json.dumps(results[tag])))
    # the headline layers on the register-indexed kernel, and 1x4 on the outer-product kernel
    for base, kern, name in (("1x1", 3, "indexed"), ("1x4", 3, "indexed"), ("1x4", 4, "outer")):
        tag = base + " " + name
        log("bench: timing %s" % tag)
        r = time_variant(layers[base], args.steps, args.warmup, args.sets, kernel=kern)
        results[tag] = summarize(layers[base], r)
        log("bench: %s %s" % (tag, json.dumps(results[tag])))

    configs = []
    if not args.no_sweep:
        log("bench: per-layer sweep of configurations c0 .. c4 (%d launches each)" % args.sweep_steps)
        configs = sweep_configs(range(5), args.sweep_steps, 3)

    network = []
    for batch in (() if args.no_network else (1, 64)):
        log("bench: MobileNet v1 forward, batch %d, graph replays" % batch)
        network.append(time_network(batch, 50, 5))
        log("bench: network %s" % json.dumps({k: v for k, v in network[-1].items() if k != "layers"}))

    head = results["1x1"]
    layer = layers["1x1"]
    traffic = measured_traffic()
    achieved = head["hbm_gbs_algorithmic"]
    line = {
        "metric": METRIC,
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
            "traffic": None if traffic is None else traffic.get("bytes_per_launch"),
        },
        "variants": results,
        "configs": configs,
        "network": network,
        "device": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle")
        line["cpu_baseline"] = cpu_baseline(args.cpu_budget)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
