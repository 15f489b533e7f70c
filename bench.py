#!/usr/bin/env python3
"""Benchmark: effective TFLOP/s (structural non-zero MACs) of the phase-
decomposed transposed / dilated convolution on one MI355X.

One step = one pass of every layer of the workload over one batch of seeded
synthetic input already resident in HBM (default: the DCGAN generator's four
ConvTranspose layers, bf16 NCHW, batch 64, chained on the device; the z ->
linear layer is input generation and is not timed).  Each layer is one
kernel launch (huge2_plan_execute); the plans (weight packing) are built
before the timed region.

Prints ONE JSON line.  Fields beyond the standard ones:
  roofline      the dominant layer's GEMM kernel: algorithmic FLOP per launch /
                its mean duration from HIP events on the launch stream, vs the
                dense MFMA peak of its dtype.
  cpu_baseline  the CPU oracle (Algorithm 1 zero insertion / Algorithm 2
                gather, float64) timed on a bounded sample of the workload.
  layers        per-layer mean time, effective TFLOP/s, issued-MAC utilisation.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--no-cpu-baseline]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective TFLOP/s (non-zero MACs) per layer + MFMA util vs peak, 1 MI355X"
# MI355X dense peaks at 2.4 GHz (256 CUs): TFLOP/s
PEAK = {"bf16": 2516.6, "f32": 157.3}
HBM_PEAK_GBS = 8000.0

DESCRIPTIONS = {
    "dcgan": "DCGAN generator deconv stack, bf16 NCHW, batch 64: ConvT k4 s2 p1 "
             "1024->512 (4->8), 512->256 (8->16), 256->128 (16->32), 128->3 (32->64)",
    "dcgan_f32": "DCGAN generator deconv stack, fp32 NCHW, batch 64 (same layers)",
    "convt_small": "ConvT 64->32 k4 s2 p1, 8x8->16x16, fp32 NCHW, batch 1",
    "convt_odd": "ConvT 256->128 k3 s2 p1 op1, 32x32->64x64, bf16 NHWC, batch 16",
    "aspp": "ASPP: four 3x3 dilated convs 2048->256 (d=6,12,18,24, same pad), 64x64, "
            "bf16 NHWC, batch 8",
    "fcn_upsample": "ConvT 21->21 k64 s32 p16, 16x16->512x512, bf16 NCHW, batch 4",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="dcgan", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle sample")
    return ap.parse_args()


def layer_flops(plans):
    return [2 * p.macs()[0] for p in plans]


def build_workload(name, dev):
    import torch
    from paper_1907_11210_amd import huge2 as h2
    from paper_1907_11210_amd import workloads as wl

    items = wl.generate(name, seed=0)
    plans, inputs = [], []
    for layer, x, w in items:
        dt = wl.torch_dtype(layer.dtype)
        w_dev = w.to(dt).contiguous().to(dev)
        x_shape = ((layer.n, layer.c_in, layer.h, layer.w) if layer.layout == "NCHW"
                   else (layer.n, layer.h, layer.w, layer.c_in))
        plans.append(h2.Plan(w_dev, x_shape, layer.transposed, layer.stride, layer.pad,
                             layer.out_pad, layer.dil, layer.layout))
        inputs.append(None if x is None else wl.to_layout(x.to(dt), layer.layout).to(dev))
        del w_dev
    chained = name in ("dcgan", "dcgan_f32")
    outs = [torch.empty(p.out_shape, dtype=wl.torch_dtype(l.dtype), device=dev)
            for p, (l, _, _) in zip(plans, items)]

    def step(events=None):
        for i, p in enumerate(plans):
            x = inputs[i] if (not chained or i == 0) else outs[i - 1]
            if events is not None:
                events[i].record()
            p(x, out=outs[i])
        if events is not None:
            events[len(plans)].record()

    return items, plans, step


def cpu_baseline(name, target_s):
    """Time the oracle on a bounded sample of the workload (float64, all host threads)."""
    import numpy as np

    import oracle
    from paper_1907_11210_amd import huge2 as h2
    from paper_1907_11210_amd import workloads as wl

    oracle.build()
    threads = os.cpu_count() or 1

    def run(batch):
        items = wl.generate(name, seed=0, batch=batch) if name != "aspp" else None
        if name == "aspp":
            layers = [l.with_(n=batch) for l in wl.WORKLOADS["aspp"]]
            g = wl.layer_input(layers[0], seed=0)
            items = [(l, g.clamp(min=0), wl.random_weight(l, seed=1 + i, std=0.01))
                     for i, l in enumerate(layers)]
        flops = 0
        t0 = time.perf_counter()
        prev = None
        for layer, x, w in items:
            dt = wl.torch_dtype(layer.dtype)
            xin = x if x is not None else prev
            xd = xin.to(dt).double().numpy()
            wd = w.to(dt).double().numpy()
            if layer.transposed:
                y = oracle.conv2d_transpose_alg1(xd, wd, None, layer.stride, layer.pad,
                                                 layer.out_pad, layer.dil, nthreads=threads)
            else:
                y = oracle.conv2d_dilated_alg2(xd, wd, None, layer.stride, layer.pad, layer.dil,
                                               nthreads=threads)
            prev = __import__("torch").from_numpy(y).float()
            d = h2.make_desc(layer.n, layer.c_in, layer.h, layer.w, layer.c_out, layer.r,
                             layer.s, layer.stride, layer.pad, layer.out_pad, layer.dil,
                             h2.HUGE2_NCHW, h2.HUGE2_F32)
            flops += 2 * h2.huge2_plan_macs(d, layer.transposed)[0]
        return flops, time.perf_counter() - t0, len(items)

    full_batch = wl.WORKLOADS[name][0].n
    flops, secs, nl = run(1)
    batch = 1
    if secs < target_s and full_batch > 1:
        batch = int(min(full_batch, max(1, target_s / max(secs, 1e-3))))
        if batch > 1:
            flops, secs, nl = run(batch)
    return {
        "value": flops / secs / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "%s at batch %d of %d (all %d layers, same shapes and distributions, bf16/fp32 "
                  "inputs widened to float64), %.1f s" % (name, batch, full_batch, nl, secs),
        "seconds": secs,
    }


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the kernels shard by batch, output channel or "
              "phase without communication, and no multi-GPU run is part of this build "
              "(asked for --gpus %d, WORLD_SIZE %d)" % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_1907_11210_amd import huge2 as h2

    if not os.path.exists(h2.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    dev = torch.device("cuda", 0)
    items, plans, step = build_workload(args.workload, dev)
    flops = layer_flops(plans)
    issued = [2 * p.macs()[1] for p in plans]
    total_flops = sum(flops)
    dtype = items[0][0].dtype

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    nl = len(plans)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(nl + 1)] for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record()
    for k in range(args.steps):
        step(ev[k])
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(stop) / args.steps

    per_layer_ms = np.array([[ev[k][i].elapsed_time(ev[k][i + 1]) for i in range(nl)]
                             for k in range(args.steps)]).mean(axis=0)
    layers = []
    for i, ((layer, _, _), p) in enumerate(zip(items, plans)):
        t = per_layer_ms[i] * 1e-3
        layers.append({
            "layer": layer.name, "ms": round(per_layer_ms[i], 5),
            "eff_tflops": round(flops[i] / t / 1e12, 2),
            "mfma_issued_util": round(issued[i] / t / 1e12 / PEAK[layer.dtype], 4),
            "nz_gflop": round(flops[i] / 1e9, 3),
        })
    dom = int(np.argmax(per_layer_ms))
    dom_t = per_layer_ms[dom] * 1e-3
    achieved = flops[dom] / dom_t / 1e12
    roofline = {
        "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK[dtype], "unit": "TFLOP/s",
        "frac": round(achieved / PEAK[dtype], 4), "traffic": None,
        "kernel": "phase_gemm_kernel (%s)" % items[dom][0].name,
        "algorithmic_flop_per_launch": flops[dom],
    }
    out = {
        "metric": METRIC,
        "value": round(total_flops / (ms_step * 1e-3) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic (seeded; random-init weights of the workload's shapes)",
        "config": {"workload": args.workload, "description": DESCRIPTIONS[args.workload],
                   "batch": items[0][0].n, "layout": items[0][0].layout},
        "roofline": roofline,
        "layers": layers,
        "wall_s_timed": round(wall, 3),
    }
    for p in plans:
        p.close()
    if not args.no_cpu_baseline:
        cb = cpu_baseline(args.workload, args.cpu_seconds)
        cb["speedup_gpu_over_oracle"] = round(out["value"] / cb["value"], 1)
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
