#!/usr/bin/env python3
"""Benchmark: effective TFLOP/s (structural non-zero MACs) of the phase-
decomposed transposed / dilated convolution on one MI355X.

One step = one pass of every layer of the workload over one batch of seeded
synthetic input already resident in HBM.  The default workload is the
largest single-GPU one: the atrous spatial pyramid (four 3x3 dilated convs
2048 -> 256 channels, dilations 6/12/18/24, bf16 NHWC, batch 8, 886.6 GFLOP
of structural work per step).  The DCGAN generator's four ConvTranspose
layers (bf16 NCHW, batch 64, chained on the device) are timed the same way
in the same run and reported under "also".  Each layer is an input-staging
launch where the layout needs one (NCHW, or channels not a multiple of the
vector width) followed by one GEMM launch (and the split-K reduce where the
plan has one), all from one huge2_plan_execute call; the plans (weight
packing) are built before the timed region.  Before the warmup steps,
untimed steps run for about --settle-ms of GPU time, so that the timed steps
see settled clocks.  Kernels are launched eagerly from the host (measured faster here
than replaying the step as one captured HIP graph, which --launch graph
does after checking a replay bitwise against the eager step).  Per-layer
times come from a separate eager pass with HIP events around each kernel
(huge2_plan_stage_input and huge2_plan_run_gemm, the two halves of
huge2_plan_execute, called separately there).

Prints ONE JSON line.  Fields beyond the standard ones:
  roofline      the dominant layer's main kernel (the layer with the most
                structural FLOPs; the longest mean launch on a tie), timed over
                back-to-back launches of that kernel
                alone between two HIP events on the launch stream:
                algorithmic FLOP (or bytes, when its arithmetic intensity is below
                the MI355X ridge) per launch / mean duration, vs the dense MFMA peak
                of its dtype (or HBM bandwidth); traffic from the committed
                rocprofv3 counter summary when it matches the kernel source.
  cpu_baseline  the CPU oracle (Algorithm 1 zero insertion / Algorithm 2
                gather, float64) timed on a bounded sample of the workload.
  layers        per-layer mean time, effective TFLOP/s, issued-MAC utilisation and
                achieved algorithmic HBM GB/s (|x| + |w| + |y| per launch / time).
  library_reference
                context for roofline.frac, not part of the path: the vendor
                library's dense GEMM (torch.matmul -> hipBLASLt) of the same
                M x N x K as the dominant layer's phase GEMMs (M output pixels,
                N output channels, K = input channels x taps per phase), timed
                the same way on random operands of the layer's dtype.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--also NAMES|none] [--no-cpu-baseline]
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
    "table1_dcgan": "the paper's Table 1 DCGAN deconvolutions: ConvT k5 s2 (p2 op1) 1024->512 "
                    "(4->8), 512->256, 256->128, 128->3 (32->64), bf16 NCHW, batch 1",
    "table1_cgan": "the paper's Table 1 cGAN deconvolutions: ConvT k4 s2 p1 256->128 (8->16), "
                   "128->3 (16->32), bf16 NCHW, batch 1",
    "dcgan_generator": "the whole DCGAN generator, bf16 NCHW, batch 64: z (100) -> ConvT k4 s1 "
                       "p0 to 4x4x1024, then ConvT k4 s2 p1 1024->512->256->128->3 (64x64); "
                       "ReLU fused after each layer, tanh after the last",
    "dcgan_generator_b1": "the whole DCGAN generator at batch 1 (latency): z (100) -> ConvT k4 "
                          "s1 p0 to 4x4x1024, then ConvT k4 s2 p1 1024->512->256->128->3 "
                          "(64x64), bf16 NCHW; ReLU fused after each layer, tanh after the last",
    "dcgan_generator_nhwc": "the whole DCGAN generator in NHWC (channel-contiguous from z to "
                            "the image), bf16, batch 64: z (100) -> ConvT k4 s1 p0 to 4x4x1024, "
                            "then ConvT k4 s2 p1 1024->512->256->128->3 (64x64); ReLU fused "
                            "after each layer, tanh after the last",
    "dcgan_generator_nhwc_b1": "the whole DCGAN generator in NHWC at batch 1 (latency): z (100) "
                               "-> ConvT k4 s1 p0 to 4x4x1024, then ConvT k4 s2 p1 "
                               "1024->512->256->128->3 (64x64), bf16; ReLU fused after each "
                               "layer, tanh after the last",
    "dcgan_dgrad": "training (section 3.2.3): data gradients of the DCGAN generator's four ConvT "
                   "layers, back to front, as stride-2 convs of the output errors with the same "
                   "weights: 3->128 (64->32), 128->256, 256->512, 512->1024 (8->4), bf16 NCHW, "
                   "batch 64",
    "dcgan_wgrad": "training (section 3.2.3): weight gradients of the DCGAN generator's four "
                   "ConvT layers (k4 s2 p1, 1024->512->256->128->3, bf16 NCHW, batch 64) from "
                   "their inputs and seeded output errors",
}
WGRAD_WORKLOADS = {"dcgan_wgrad": "dcgan"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    # about 30 ms of untimed steps: a cold MI355X needs some 20 ms of load
    # before its clocks settle (the first 200 timed DCGAN steps after 10
    # warmup steps averaged 93 us, every later 200 averaged 85.6 us)
    ap.add_argument("--warmup", type=int, default=300)
    # the largest single-GPU workload (886.6 GFLOP of structural work per step)
    ap.add_argument("--workload", default="aspp", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--also", default="dcgan",
                    help="comma-separated further forward workloads timed the same way in the "
                         "same run and reported under 'also' (empty: none)")
    ap.add_argument("--settle-ms", type=float, default=100.0,
                    help="untimed load (GPU milliseconds of steps) run before the warmup steps, "
                         "so that the timed steps see settled clocks")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-library-reference", action="store_true",
                    help="skip the dense-GEMM library timing reported as context")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 256 MiB device copy (to scale HBM traffic counters)")
    ap.add_argument("--launch", choices=["graph", "eager"], default="eager",
                    help="replay each timed step as one captured HIP graph, or launch eagerly")
    ap.add_argument("--summarize-profiles", metavar="DIR",
                    help="no GPU: turn the rocprofv3 CSVs of PROFILE_COMMANDS under DIR into "
                         "the summaries under profiles/")
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
                             layer.out_pad, layer.dil, layer.layout, layer.act))
        inputs.append(None if x is None else wl.to_layout(x.to(dt), layer.layout).to(dev))
        del w_dev
    chained = name in wl.CHAINED
    outs = [torch.empty(p.out_shape, dtype=wl.torch_dtype(l.dtype), device=dev)
            for p, (l, _, _) in zip(plans, items)]
    # layers of one input (the pyramid's branches) run as one grouped launch
    group = h2.Group(plans) if name in wl.GROUPED else None

    def step(events=None):
        # events[3*i]: before the layer's input staging, events[3*i+1]: before its
        # GEMM kernel, events[3*i+2]: after it (all on the launch stream).  The
        # per-layer pass (events given) runs a grouped workload layer by layer.
        if group is not None and events is None:
            group(inputs[0], outs=outs)
            return
        for i, p in enumerate(plans):
            x = inputs[i] if (not chained or i == 0) else outs[i - 1]
            if events is None:
                p(x, out=outs[i])  # staging (if any) and GEMM in one library call
                continue
            events[3 * i].record()
            p.stage(x)
            events[3 * i + 1].record()
            p.gemm(x, outs[i])
            events[3 * i + 2].record()

    def step_input(i):
        return inputs[i] if (not chained or i == 0) else outs[i - 1]

    return items, plans, step, lambda: outs, step_input, group


def kernel_source_sha():
    import hashlib
    h = hashlib.sha256()
    for f in ("kernels.hip", "kernels.hpp", "capi.cpp", "plan.cpp"):
        with open(os.path.join(ROOT, "paper_1907_11210_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, layer_name):
    """HBM bytes per launch of the layer's GEMM kernel, from the committed
    rocprofv3 counter summary, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "layer_kernels_%s_traffic.json" % workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_sha") != kernel_source_sha():
        return None
    entry = t.get("layers", {}).get(layer_name)
    return None if entry is None else entry.get("traffic_bytes")


COPY_MIB = 256


def copy_calibration(dev, mib=COPY_MIB, reps=10):
    """A plain elementwise copy kernel (y = x * 1) of known size, to scale the
    FETCH_SIZE / WRITE_SIZE counters: it reads and writes mib MiB per launch."""
    import torch
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    for _ in range(reps):
        torch.mul(a, 1.0, out=b)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n * 4, "reps": reps}), flush=True)


# The rocprofv3 runs whose CSVs --summarize-profiles reads ($R = repository root,
# $O = output directory).  Each line is run on its own, after
# `cd /tmp && export TMPDIR=/tmp`.
PROFILE_COMMANDS = [
    ("trace", "rocprofv3 --kernel-trace --stats -f csv -d $O -o trace -- "
              "python3 $R/bench.py --workload {w} --also none --no-cpu-baseline --no-library-reference"),
    ("fetch", "timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE -f csv -d $O -o fetch -- "
              "python3 $R/bench.py --workload {w} --also none --no-cpu-baseline "
              "--no-library-reference --steps 3 --warmup 1 --settle-ms 0"),
    ("write", "timeout -s KILL 120 rocprofv3 --pmc WRITE_SIZE -f csv -d $O -o write -- "
              "python3 $R/bench.py --workload {w} --also none --no-cpu-baseline "
              "--no-library-reference --steps 3 --warmup 1 --settle-ms 0"),
    ("copy_fetch", "timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE -f csv -d $O -o copy_fetch -- "
                   "python3 $R/bench.py --copy-calibration"),
    ("copy_write", "timeout -s KILL 120 rocprofv3 --pmc WRITE_SIZE -f csv -d $O -o copy_write -- "
                   "python3 $R/bench.py --copy-calibration"),
    ("mfma", "timeout -s KILL 120 rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_VALU_MFMA_BF16 "
             "-f csv -d $O -o mfma -- python3 $R/bench.py --workload {w} --also none "
             "--no-cpu-baseline --no-library-reference --steps 3 --warmup 1 --settle-ms 0"),
]
# one bf16 MFMA "MOP" is 512 flops (a 32x32x16 bf16 MFMA, 32768 flops, counts 64)
MFMA_FLOPS_PER_MOP_BF16 = 512


def _csv_rows(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def _counter_per_dispatch(path, counter):
    """{dispatch id: (kernel name and grid size, counter value summed over instances)}"""
    out = {}
    for r in _csv_rows(path):
        if r["Counter_Name"] != counter:
            continue
        d = int(r["Dispatch_Id"])
        name, v = out.get(d, ("%s grid %s" % (r["Kernel_Name"], r["Grid_Size"]), 0.0))
        out[d] = (name, v + float(r["Counter_Value"]))
    return out


MAIN_KERNELS = ("phase_gemm_kernel", "phase_gemm2_kernel", "phase_gemm3_kernel", "ztile_kernel",
                "rowphase_kernel", "colphase_kernel", "quad_kernel", "grouped_kernel")


def _is_main(name):
    return any("::" + k + "<" in name or "::" + k + "(" in name for k in MAIN_KERNELS)


def _layer_dispatches(per_dispatch, nl, trailing):
    """Assign each layer's main-kernel dispatches (in launch order) to it.
    bench.py launches every layer in order once per step, then the dominant
    layer's kernel alone, back to back (`trailing` = the --steps of the
    profiled command): that trailing run (same kernel name and grid, at most
    `trailing` long, since several layers may share a kernel instance) is left
    out, except for the dispatches that complete the last step."""
    ids = sorted(d for d, (name, _) in per_dispatch.items() if _is_main(name))
    run = 1
    while (run < min(len(ids), trailing) and
           per_dispatch[ids[-run - 1]][0] == per_dispatch[ids[-1]][0]):
        run += 1
    if nl > 1 and run > 1:
        keep = len(ids) - run
        keep += (-keep) % nl
        ids = ids[:keep]
    by_layer = [[] for _ in range(nl)]
    for k, d in enumerate(ids):
        by_layer[k % nl].append(d)
    return by_layer


def _split_group(per):
    """Separate the grouped launches (the main-kernel dispatches with the
    largest grid) from the per-layer ones: returns (the rest, [(name, value)]
    of the grouped launches in dispatch order)."""
    def grid(name):
        return int(name[name.rfind(" grid ") + 6:].split("x")[0])
    mains = [i for i, (name, _) in per.items() if _is_main(name)]
    if not mains:
        return per, []
    top = max(grid(per[i][0]) for i in mains)
    gids = sorted(i for i in mains if grid(per[i][0]) == top)
    rest = {i: v for i, v in per.items() if i not in set(gids)}
    return rest, [per[i] for i in gids]


def summarize_profiles(d, workload):
    import numpy as np
    from paper_1907_11210_amd import workloads as wl

    layers = wl.WORKLOADS[workload]
    nl = len(layers)
    grouped = workload in wl.GROUPED
    cmds = ["cd /tmp && export TMPDIR=/tmp"] + [c.format(w=workload) for _, c in PROFILE_COMMANDS]
    lines = ["# Main kernel of each layer (phase GEMM or all-taps form) on workload `%s`: "
             "rocprofv3 kernel trace" % workload, "",
             "Kernel source sha256[:16]: `%s`" % kernel_source_sha(), "",
             "Commands (R = repository root, O = output directory):", "", "```"] + cmds + ["```", ""]

    stats = _csv_rows(os.path.join(d, "trace_kernel_stats.csv"))
    lines += ["## --stats (all kernels of the process)", "",
              "| kernel | calls | average ns | total ns | % |", "|---|---|---|---|---|"]
    for r in stats[:10]:
        lines.append("| %s | %s | %.0f | %s | %.2f |" % (r["Name"][:110], r["Calls"],
                                                       float(r["AverageNs"]), r["TotalDurationNs"],
                                                       float(r["Percentage"])))
    trace = _csv_rows(os.path.join(d, "trace_kernel_trace.csv"))
    per = {int(r["Dispatch_Id"]): ("%s grid %sx%s" % (r["Kernel_Name"], r["Grid_Size_X"], r["Grid_Size_Y"]),
                                   int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
           for r in trace}
    group_ids = []
    if grouped:
        # the grouped launches (every layer's works: the largest grid) run the
        # steps; the layers' own launches come from the per-layer pass
        per, group_ids = _split_group(per)
        gt = np.array([per_group[1] for per_group in group_ids]) / 1e3
        lines += ["", "## Grouped launch of the %d layers (one kernel per step)" % nl, "",
                  "| launches | mean us | min us | kernel instance |", "|---|---|---|---|",
                  "| %d | %.2f | %.2f | %s |" % (len(gt), gt.mean(), gt.min(),
                                               group_ids[0][0].split("(")[0].split("::")[-1] +
                                               group_ids[0][0][group_ids[0][0].rfind(" grid "):])]
        avg_group_us = float(gt.mean())
    by_layer = _layer_dispatches(per, nl, 50)
    lines += ["", "## Main kernel per layer (dispatches in launch order, layer = k mod %d)" % nl,
              "", "| layer | dispatches | mean us | min us | kernel instance |", "|---|---|---|---|---|"]
    avg_us = {}
    for l, ids in zip(layers, by_layer):
        t = np.array([per[i][1] for i in ids]) / 1e3
        avg_us[l.name] = float(t.mean())
        name = per[ids[0]][0]
        kname = name.split("(")[0].split("::")[-1]
        inst = kname + (name[name.find("<"):name.find(">") + 1] if "<" in name and "<" not in kname else "")
        inst += name[name.rfind(" grid "):]
        lines.append("| %s | %d | %.2f | %.2f | %s |" % (l.name, len(ids), t.mean(), t.min(), inst))

    # the trailing back-to-back run of the dominant layer's kernel: what the
    # benchmark's roofline.mean_launch_ms times
    ids_all = sorted(i for i, (name, _) in per.items() if _is_main(name))
    run = 1
    while run < min(len(ids_all), 50) and per[ids_all[-run - 1]][0] == per[ids_all[-1]][0]:
        run += 1
    tail = [per[i][1] for i in ids_all[-run:]][-50:] if ids_all else []
    if tail:
        name = per[ids_all[-1]][0]
        lines += ["", "Back-to-back launches of the dominant layer's kernel (the benchmark's roofline "
                  "timing; the last %d dispatches): mean %.2f us, min %.2f us, `%s`" % (
                      len(tail), float(np.mean(tail)) / 1e3, float(np.min(tail)) / 1e3,
                      name.split("(")[0].split("::")[-1] + name[name.rfind(" grid "):])]

    traffic = None
    if os.path.exists(os.path.join(d, "fetch_counter_collection.csv")):
        cf = _counter_per_dispatch(os.path.join(d, "copy_fetch_counter_collection.csv"), "FETCH_SIZE")
        cw = _counter_per_dispatch(os.path.join(d, "copy_write_counter_collection.csv"), "WRITE_SIZE")
        copy_name = max(cf.values(), key=lambda t: t[1])[0]
        known_kib = COPY_MIB * 1024.0
        f_fetch = known_kib / np.mean([v for n, v in cf.values() if n == copy_name])
        f_write = known_kib / np.mean([v for n, v in cw.values() if n == copy_name])
        fe = _counter_per_dispatch(os.path.join(d, "fetch_counter_collection.csv"), "FETCH_SIZE")
        wr = _counter_per_dispatch(os.path.join(d, "write_counter_collection.csv"), "WRITE_SIZE")
        traffic = {"kernel_source_sha": kernel_source_sha(), "workload": workload,
                   "copy_kernel": copy_name[:120], "copy_bytes": COPY_MIB << 20,
                   "scale_fetch": round(float(f_fetch), 4), "scale_write": round(float(f_write), 4),
                   "layers": {}}
        lines += ["", "## HBM traffic of each layer's main kernel (FETCH_SIZE, WRITE_SIZE; KiB per dispatch)",
                  "", "Calibration: a %d MiB elementwise copy reads FETCH_SIZE x %.4f and writes "
                  "WRITE_SIZE x %.4f of its known size." % (COPY_MIB, f_fetch, f_write), "",
                  "| layer | FETCH_SIZE KiB | WRITE_SIZE KiB | scaled traffic MB | algorithmic MB |",
                  "|---|---|---|---|---|"]
        if grouped:
            fe, gfe = _split_group(fe)
            wr, gwr = _split_group(wr)
            fk = float(np.mean([v for _, v in gfe]))
            wk = float(np.mean([v for _, v in gwr]))
            tb = 1024.0 * (fk * f_fetch + wk * f_write)
            l0 = layers[0]
            esz = 2 if l0.dtype == "bf16" else 4
            algo = esz * l0.n * l0.c_in * l0.h * l0.w
            for l in layers:
                ho, wo = l.out_hw()
                algo += esz * (l.c_in * l.c_out * l.r * l.s + l.n * l.c_out * ho * wo)
            traffic["layers"]["group"] = {"fetch_kib": round(fk, 1), "write_kib": round(wk, 1),
                                          "traffic_bytes": int(round(tb)), "algorithmic_bytes": algo}
            lines.append("| grouped launch | %.1f | %.1f | %.2f | %.2f |" % (fk, wk, tb / 1e6, algo / 1e6))
        for l, fids, wids in zip(layers, _layer_dispatches(fe, nl, 3), _layer_dispatches(wr, nl, 3)):
            fk = float(np.mean([fe[i][1] for i in fids]))
            wk = float(np.mean([wr[i][1] for i in wids]))
            tb = 1024.0 * (fk * f_fetch + wk * f_write)
            ho, wo = l.out_hw()
            esz = 2 if l.dtype == "bf16" else 4
            algo = esz * (l.n * l.c_in * l.h * l.w + l.c_in * l.c_out * l.r * l.s + l.n * l.c_out * ho * wo)
            traffic["layers"][l.name] = {"fetch_kib": round(fk, 1), "write_kib": round(wk, 1),
                                         "traffic_bytes": int(round(tb)), "algorithmic_bytes": algo}
            lines.append("| %s | %.1f | %.1f | %.2f | %.2f |" % (l.name, fk, wk, tb / 1e6, algo / 1e6))
    mfma_csv = os.path.join(d, "mfma_counter_collection.csv")
    if os.path.exists(mfma_csv):
        from paper_1907_11210_amd import huge2 as h2
        mops = _counter_per_dispatch(mfma_csv, "SQ_INSTS_VALU_MFMA_MOPS_BF16")
        lines += ["", "## MFMA work of each layer's main kernel (SQ_INSTS_VALU_MFMA_MOPS_BF16)", "",
                  "Counted MFMA flops = %d x MOPs per dispatch. Utilisation = counted flops / mean "
                  "duration (kernel trace above) / %.1f TFLOP/s (the published dense bf16 peak); "
                  "structural = the non-zero MACs of the layer, the same numerator as the "
                  "benchmark's effective TFLOP/s." % (MFMA_FLOPS_PER_MOP_BF16, PEAK["bf16"]), "",
                  "| layer | counted MFMA GFLOP | issued (plan) GFLOP | structural GFLOP | "
                  "MFMA utilisation | structural / peak |", "|---|---|---|---|---|---|"]
        if grouped:
            mops, gm = _split_group(mops)
            cf = MFMA_FLOPS_PER_MOP_BF16 * float(np.mean([v for _, v in gm]))
            nz = issued = 0.0
            for l in layers:
                desc = h2.make_desc(l.n, l.c_in, l.h, l.w, l.c_out, l.r, l.s, l.stride, l.pad,
                                    l.out_pad, l.dil,
                                    h2.HUGE2_NCHW if l.layout == "NCHW" else h2.HUGE2_NHWC,
                                    h2.HUGE2_BF16)
                m = h2.huge2_plan_macs(desc, l.transposed)
                nz += 2.0 * m[0]
                issued += 2.0 * m[1]
            t = avg_group_us * 1e-6
            lines.append("| grouped launch | %.2f | %.2f | %.2f | %.3f | %.3f |" % (
                cf / 1e9, issued / 1e9, nz / 1e9, cf / t / (PEAK["bf16"] * 1e12),
                nz / t / (PEAK["bf16"] * 1e12)))
        for l, ids in zip(layers, _layer_dispatches(mops, nl, 3)):
            if l.dtype != "bf16":
                continue
            cf = MFMA_FLOPS_PER_MOP_BF16 * float(np.mean([mops[i][1] for i in ids]))
            desc = h2.make_desc(l.n, l.c_in, l.h, l.w, l.c_out, l.r, l.s, l.stride, l.pad,
                                l.out_pad, l.dil,
                                h2.HUGE2_NCHW if l.layout == "NCHW" else h2.HUGE2_NHWC,
                                h2.HUGE2_BF16)
            nz = 2.0 * h2.huge2_plan_macs(desc, l.transposed)[0]
            issued = 2.0 * h2.huge2_plan_macs(desc, l.transposed)[1]
            t = avg_us[l.name] * 1e-6
            lines.append("| %s | %.2f | %.2f | %.2f | %.3f | %.3f |" % (
                l.name, cf / 1e9, issued / 1e9, nz / 1e9, cf / t / (PEAK["bf16"] * 1e12),
                nz / t / (PEAK["bf16"] * 1e12)))
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", "layer_kernels_%s.md" % workload), "w") as f:
        f.write("\n".join(lines) + "\n")
    if traffic is not None:
        with open(os.path.join(ROOT, "profiles", "layer_kernels_%s_traffic.json" % workload), "w") as f:
            json.dump(traffic, f, indent=1)
            f.write("\n")
    print(json.dumps({"layer_mean_us": avg_us}))


def run_wgrad(args, dev):
    """The weight-gradient workload: one step = the weight gradient of every
    layer (huge2_wgrad_execute: staging, MFMA GEMM, store), inputs and output
    errors resident in HBM; FLOP = 2 x the layers' structural non-zero MACs
    (each product of the forward pass appears once in the gradient)."""
    import numpy as np
    import torch
    from paper_1907_11210_amd import huge2 as h2
    from paper_1907_11210_amd import workloads as wl

    layers = wl.WORKLOADS[WGRAD_WORKLOADS[args.workload]]
    g = torch.Generator().manual_seed(0)
    plans, xs, dys, dws, flops = [], [], [], [], []
    for layer in layers:
        dt = wl.torch_dtype(layer.dtype)
        ho, wo = layer.out_hw()
        xs.append(torch.randn(layer.n, layer.c_in, layer.h, layer.w, generator=g).to(dt).to(dev))
        dys.append(torch.randn(layer.n, layer.c_out, ho, wo, generator=g).to(dt).to(dev))
        desc = h2.make_desc(layer.n, layer.c_in, layer.h, layer.w, layer.c_out, layer.r, layer.s,
                            layer.stride, layer.pad, layer.out_pad, layer.dil, h2.HUGE2_NCHW,
                            h2.HUGE2_BF16 if layer.dtype == "bf16" else h2.HUGE2_F32)
        plans.append(h2.huge2_wgrad_plan_create(desc, 1 if layer.transposed else 0))
        dws.append(torch.empty(layer.c_in, layer.c_out, layer.r, layer.s, dtype=dt, device=dev))
        flops.append(2 * h2.huge2_plan_macs(desc, layer.transposed)[0])
    stream = torch.cuda.current_stream(dev).cuda_stream

    def run_layer(i):
        h2.huge2_wgrad_execute(plans[i], xs[i].data_ptr(), dys[i].data_ptr(), dws[i].data_ptr(),
                               stream)

    def step():
        for i in range(len(layers)):
            run_layer(i)

    for _ in range(args.warmup):
        step()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record()
    for _ in range(args.steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(stop) / args.steps
    per = []
    for i in range(len(layers)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            run_layer(i)
        e1.record()
        torch.cuda.synchronize()
        per.append(e0.elapsed_time(e1) / args.steps)
    dom = int(np.argmax(per))
    peak = PEAK[layers[0].dtype]
    achieved = flops[dom] / (per[dom] * 1e-3) / 1e12
    out = {
        "metric": METRIC, "value": round(sum(flops) / (ms_step * 1e-3) / 1e12, 3), "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": layers[0].dtype,
        "data": "synthetic (seeded inputs and output errors of the layers' shapes)",
        "config": {"workload": args.workload, "description": DESCRIPTIONS[args.workload],
                   "batch": layers[0].n, "layout": "NCHW", "launch": "eager launches"},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": None,
                     "kernel": "wgrad_stage + wgrad_gemm + wgrad_store (%s)" % layers[dom].name,
                     "mean_launch_ms": round(per[dom], 5), "algorithmic_flop_per_launch": flops[dom]},
        "layers": [{"layer": l.name, "ms": round(t, 5), "eff_tflops": round(f / (t * 1e-3) / 1e12, 2),
                    "nz_gflop": round(f / 1e9, 3)} for l, t, f in zip(layers, per, flops)],
        "kernel_source_sha": kernel_source_sha(), "wall_s_timed": round(wall, 3),
    }
    for p in plans:
        h2.huge2_wgrad_plan_destroy(p)
    if not args.no_cpu_baseline:
        cb = cpu_baseline_wgrad(layers, args.cpu_seconds)
        cb["speedup_gpu_over_oracle"] = round(out["value"] / cb["value"], 1)
        out["cpu_baseline"] = cb
    return out


def cpu_baseline_wgrad(layers, target_s):
    """The oracle's weight gradients on a batch-reduced sample of the layers."""
    import numpy as np

    import oracle
    from paper_1907_11210_amd import huge2 as h2

    oracle.build()
    threads = os.cpu_count() or 1
    rng = np.random.default_rng(0)

    def run(batch):
        flops, t0 = 0, time.perf_counter()
        for l in layers:
            ho, wo = l.out_hw()
            x = rng.standard_normal((batch, l.c_in, l.h, l.w))
            dy = rng.standard_normal((batch, l.c_out, ho, wo))
            oracle.conv2d_transpose_wgrad(x, dy, (l.c_in, l.c_out, l.r, l.s), l.stride, l.pad,
                                          l.out_pad, l.dil, nthreads=threads)
            d = h2.make_desc(batch, l.c_in, l.h, l.w, l.c_out, l.r, l.s, l.stride, l.pad, l.out_pad,
                             l.dil, h2.HUGE2_NCHW, h2.HUGE2_F32)
            flops += 2 * h2.huge2_plan_macs(d, 1)[0]
        return flops, time.perf_counter() - t0

    full = layers[0].n
    flops, secs = run(1)
    batch = 1
    if secs < target_s and full > 1:
        batch = int(min(full, max(1, target_s / max(secs, 1e-3))))
        if batch > 1:
            flops, secs = run(batch)
    return {"value": flops / secs / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": "the %d layers' weight gradients at batch %d of %d (float64), %.1f s"
                      % (len(layers), batch, full, secs), "seconds": secs}


def library_reference(layer, steps, dev):
    """The vendor library's dense GEMM with the M x N x K of the layer's phase
    GEMMs: a calibration of what this GPU reaches on that contraction size."""
    import torch
    ho, wo = layer.out_hw()
    m, n = layer.n * ho * wo, layer.c_out
    k = layer.c_in * layer.r * layer.s
    if layer.transposed:
        k //= layer.stride ** 2  # taps per phase
    dt = torch.bfloat16 if layer.dtype == "bf16" else torch.float32
    g = torch.Generator(device=dev).manual_seed(0)
    a = torch.randn(m, k, device=dev, generator=g).to(dt)
    b = torch.randn(k, n, device=dev, generator=g).to(dt)
    for _ in range(3):
        c = a @ b
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        c = a @ b
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    tf = 2.0 * m * n * k / (ms * 1e-3) / 1e12
    del a, b, c
    return {"op": "torch.matmul %s (hipBLASLt), %d x %d x %d" % (layer.dtype, m, n, k),
            "layer": layer.name, "ms": round(ms, 5), "tflops": round(tf, 1),
            "frac_of_peak": round(tf / PEAK[layer.dtype], 4)}


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
            y = oracle.activate(y, layer.act)
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


def settle(step, ms):
    """Run untimed steps until about `ms` milliseconds of GPU time have passed
    (at least one step): a cold MI355X raises its clocks over the first tens
    of milliseconds of load.  Returns the GPU time spent."""
    import torch
    if ms <= 0:
        return 0.0
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    step()
    e1.record()
    torch.cuda.synchronize()
    one = max(e0.elapsed_time(e1), 1e-3)
    reps = int(min(10000, max(0, ms / one - 1)))
    e0.record()
    for _ in range(reps):
        step()
    e1.record()
    torch.cuda.synchronize()
    return one + (e0.elapsed_time(e1) if reps else 0.0)


def bench_forward(name, args, dev):
    """Time one forward workload: returns its JSON record and the dominant layer."""
    import numpy as np
    import torch

    items, plans, step, step_outputs, step_input, group = build_workload(name, dev)
    flops = layer_flops(plans)
    issued = [2 * p.macs()[1] for p in plans]
    total_flops = sum(flops)
    dtype = items[0][0].dtype
    esz = 2 if dtype == "bf16" else 4

    settled_ms = settle(step, args.settle_ms)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # The whole step as one HIP graph (the library's launches are captured on
    # torch's capture stream); replays must reproduce the eager outputs bitwise.
    graph = None
    if args.launch == "graph":
        eager_out = [o.clone() for o in step_outputs()]
        s_side = torch.cuda.Stream()
        s_side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s_side):
            step()
        torch.cuda.current_stream().wait_stream(s_side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        for _ in range(3):
            for o in step_outputs():
                o.fill_(float("nan"))
            graph.replay()
            torch.cuda.synchronize()
            for o, e in zip(step_outputs(), eager_out):
                iv = torch.int16 if o.dtype == torch.bfloat16 else torch.int32
                if not torch.equal(o.view(iv), e.view(iv)):
                    raise RuntimeError("graph replay differs from the eager step")
        del eager_out

    def run_once():
        if graph is not None:
            graph.replay()
        else:
            step()

    for _ in range(args.warmup):
        run_once()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record()
    for _ in range(args.steps):
        run_once()
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(stop) / args.steps

    # Per-layer breakdown: a separate eager pass with events around each kernel.
    nl = len(plans)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3 * nl)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for k in range(args.steps):
        step(ev[k])
    torch.cuda.synchronize()
    stage_ms = np.array([[ev[k][3 * i].elapsed_time(ev[k][3 * i + 1]) for i in range(nl)]
                         for k in range(args.steps)]).mean(axis=0)
    gemm_ms = np.array([[ev[k][3 * i + 1].elapsed_time(ev[k][3 * i + 2]) for i in range(nl)]
                        for k in range(args.steps)]).mean(axis=0)
    layers = []
    algo_bytes = []
    for i, ((layer, _, _), p) in enumerate(zip(items, plans)):
        ho, wo = layer.out_hw()
        nbytes = esz * (layer.n * layer.c_in * layer.h * layer.w +
                        layer.c_in * layer.c_out * layer.r * layer.s +
                        layer.n * layer.c_out * ho * wo)
        algo_bytes.append(nbytes)
        t = (stage_ms[i] + gemm_ms[i]) * 1e-3
        layers.append({
            "layer": layer.name, "kernel": p.kernel, "ms": round(stage_ms[i] + gemm_ms[i], 5),
            "gemm_ms": round(gemm_ms[i], 5), "stage_ms": round(stage_ms[i], 5),
            "eff_tflops": round(flops[i] / t / 1e12, 2),
            "gemm_eff_tflops": round(flops[i] / (gemm_ms[i] * 1e-3) / 1e12, 2),
            "mfma_issued_util": round(issued[i] / (gemm_ms[i] * 1e-3) / 1e12 / PEAK[layer.dtype], 4),
            "nz_gflop": round(flops[i] / 1e9, 3),
            "algorithmic_mb": round(nbytes / 1e6, 2),
            "gemm_alg_gbs": round(nbytes / (gemm_ms[i] * 1e-3) / 1e9, 1),
        })
    # the layer with the most work: chosen by FLOPs, not by the per-layer
    # times, whose order flips between layers of near-equal time from run to
    # run (and under the profiler)
    dom = max(range(len(plans)), key=lambda i: (flops[i], gemm_ms[i]))
    # The dominant layer's main kernel alone: its input staged once, then
    # `steps` back-to-back launches between two events on the launch stream
    # (the same input every time), so that per-launch event overhead does
    # not enter the mean launch duration.
    # A grouped workload's kernel is the one launch of all its layers: its
    # algorithmic work is every layer's FLOPs, its bytes the shared input once
    # plus every layer's weights and output.
    x_dom = step_input(dom)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if group is not None:
        l0 = items[0][0]
        dom_flops = total_flops
        dom_bytes = sum(algo_bytes) - (len(items) - 1) * esz * l0.n * l0.c_in * l0.h * l0.w
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            group(x_dom, outs=step_outputs())
        e1.record()
    else:
        dom_flops, dom_bytes = flops[dom], algo_bytes[dom]
        plans[dom].stage(x_dom)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            plans[dom].gemm(x_dom, step_outputs()[dom])
        e1.record()
    torch.cuda.synchronize()
    dom_ms = e0.elapsed_time(e1) / args.steps
    dom_t = dom_ms * 1e-3
    intensity = dom_flops / dom_bytes
    ridge = PEAK[dtype] * 1e12 / (HBM_PEAK_GBS * 1e9)
    if intensity >= ridge:
        achieved = dom_flops / dom_t / 1e12
        roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK[dtype],
                    "unit": "TFLOP/s", "frac": round(achieved / PEAK[dtype], 4)}
        per_launch = {"algorithmic_flop_per_launch": dom_flops}
    else:
        achieved = dom_bytes / dom_t / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4)}
        per_launch = {"algorithmic_bytes_per_launch": dom_bytes}
    dom_layer = items[dom][0]
    dom_name = "group" if group is not None else items[dom][0].name
    roofline["traffic"] = measured_traffic(name, dom_name)
    roofline.update({"kernel": ("grouped launch of %d layers: %s (%s)" % (len(plans), group.kernel, name)
                                if group is not None else
                                "%s (%s)" % (plans[dom].kernel, items[dom][0].name)),
                     "mean_launch_ms": round(dom_ms, 5),
                     "arithmetic_intensity_flop_per_byte": round(intensity, 1)})
    roofline.update(per_launch)
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
        "config": {"workload": name, "description": DESCRIPTIONS[name],
                   "batch": items[0][0].n, "layout": items[0][0].layout,
                   "launch": "one HIP graph per step" if graph is not None else "eager launches"},
        "roofline": roofline,
        "layers": layers,
        "kernel_source_sha": kernel_source_sha(),
        "wall_s_timed": round(wall, 3),
        "settle_ms": round(settled_ms, 1),
    }
    if group is not None:
        group.close()
    for p in plans:
        p.close()
    del plans, step, items, group
    torch.cuda.synchronize()
    return out, dom_layer




def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the kernels shard by batch, output channel or "
              "phase without communication, and there is no multi-GPU path "
              "(asked for --gpus %d, WORLD_SIZE %d)" % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    if args.summarize_profiles:
        summarize_profiles(args.summarize_profiles, args.workload)
        return

    import numpy as np
    import torch
    from paper_1907_11210_amd import huge2 as h2

    if not os.path.exists(h2.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    dev = torch.device("cuda", 0)
    if args.copy_calibration:
        copy_calibration(dev)
        return
    if args.workload in WGRAD_WORKLOADS:
        print(json.dumps(run_wgrad(args, dev)), flush=True)
        return
    out, dom_layer = bench_forward(args.workload, args, dev)
    if not args.no_library_reference:
        out["library_reference"] = library_reference(dom_layer, args.steps, dev)
    also = [w for w in args.also.split(",") if w and w not in ("none", args.workload)]
    if also:
        out["also"] = {}
    for w in also:
        o, _ = bench_forward(w, args, dev)
        torch.cuda.empty_cache()
        out["also"][w] = {k: o[k] for k in ("value", "unit", "ms_per_step", "dtype", "config",
                                             "roofline", "layers")}
    if not args.no_cpu_baseline:
        cb = cpu_baseline(args.workload, args.cpu_seconds)
        cb["speedup_gpu_over_oracle"] = round(out["value"] / cb["value"], 1)
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
