"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Every case feeds both sides the same dtype-rounded inputs and compares element
by element (see tests/parity.py for the criterion).  Small cases are checked in
full; the five benchmark workloads are checked in full at reduced size and on
sampled outputs at full size, in the plan configuration the benchmark times.
"""
import zlib

import numpy as np
import pytest
import torch

from paper_1907_11210_amd import huge2 as h2
from paper_1907_11210_amd import workloads as wl
from paper_1907_11210_amd.workloads import Layer

import parity as P

pytestmark = pytest.mark.gpu


def L(name, tr, n, ci, h, w, co, r, s, st, pd, op, dl, layout, dtype):
    return Layer(name, tr, n, ci, h, w, co, r, s, st, pd, op, dl, layout, dtype)


SMALL = [
    L("ct_ragged_f32_nchw", True, 2, 40, 9, 9, 136, 4, 4, 2, 1, 0, 1, "NCHW", "f32"),
    L("ct_ragged_bf16_nhwc", True, 2, 40, 9, 9, 136, 4, 4, 2, 1, 0, 1, "NHWC", "bf16"),
    L("ct_ragged_bf16_nchw", True, 3, 72, 6, 7, 200, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_ragged_f32_nhwc", True, 1, 20, 10, 6, 36, 4, 4, 2, 1, 0, 1, "NHWC", "f32"),
    L("ct_odd_op_bf16_nhwc", True, 2, 24, 7, 7, 40, 3, 3, 2, 1, 1, 1, "NHWC", "bf16"),
    L("ct_zero_tap_phases", True, 1, 16, 5, 5, 16, 1, 1, 2, 0, 1, 1, "NHWC", "f32"),
    L("ct_crop", True, 1, 8, 6, 6, 8, 3, 3, 2, 2, 0, 1, "NCHW", "f32"),
    L("ct_c21_staged", True, 2, 21, 6, 6, 21, 8, 8, 4, 2, 0, 1, "NHWC", "bf16"),
    L("ct_stride32", True, 1, 3, 3, 3, 3, 64, 64, 32, 16, 0, 1, "NCHW", "bf16"),
    L("ct_dilated_kernel", True, 2, 16, 5, 6, 24, 3, 3, 2, 1, 1, 2, "NCHW", "f32"),
    L("ct_stride1", True, 1, 32, 8, 8, 32, 3, 3, 1, 1, 0, 1, "NHWC", "bf16"),
    L("ct_h1", True, 2, 32, 1, 9, 48, 4, 4, 2, 1, 0, 1, "NCHW", "f32"),
    L("ct_cout1", True, 2, 64, 8, 8, 1, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_big_k", True, 1, 256, 4, 4, 160, 4, 4, 2, 1, 0, 1, "NHWC", "bf16"),
    L("dil_aspp_d6", False, 1, 64, 64, 64, 48, 3, 3, 1, 6, 0, 6, "NHWC", "bf16"),
    L("dil_aspp_d24", False, 1, 64, 64, 64, 48, 3, 3, 1, 24, 0, 24, "NHWC", "bf16"),
    L("dil_f32_nchw", False, 2, 12, 13, 11, 20, 3, 3, 1, 2, 0, 2, "NCHW", "f32"),
    L("dil_valid", False, 1, 16, 12, 12, 16, 3, 3, 1, 0, 0, 3, "NHWC", "f32"),
    L("conv_strided_dilated", False, 2, 8, 11, 11, 40, 3, 3, 2, 2, 0, 2, "NHWC", "f32"),
    L("conv_plain", False, 2, 48, 9, 9, 136, 3, 3, 1, 1, 0, 1, "NCHW", "bf16"),
    L("conv_1x1", False, 1, 64, 5, 5, 64, 1, 1, 1, 0, 0, 1, "NHWC", "bf16"),
    L("ct_vecstage_bf16", True, 2, 72, 4, 6, 40, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_vecstage_f32", True, 2, 70, 3, 4, 24, 3, 3, 2, 1, 1, 1, "NCHW", "f32"),
    # few output channels, NCHW: the all-taps form
    L("ct_fewout_bf16", True, 2, 40, 6, 16, 3, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_fewout_f32_op", True, 2, 24, 5, 8, 2, 3, 3, 2, 1, 1, 1, "NCHW", "f32"),
    L("ct_fewout_s3d2", True, 1, 16, 7, 8, 4, 3, 3, 3, 2, 1, 2, "NCHW", "bf16"),
    L("ct_fewout_tall", True, 3, 130, 37, 8, 1, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_fewout_wide", True, 1, 8, 3, 64, 2, 5, 5, 2, 2, 1, 1, "NCHW", "f32"),
    # large stride, few channels, NCHW bf16: the output-stationary form
    L("ct_rowphase_s8", True, 2, 5, 6, 6, 7, 16, 16, 8, 4, 0, 1, "NCHW", "bf16"),
    L("ct_rowphase_s4", True, 2, 20, 5, 8, 9, 6, 6, 4, 1, 0, 1, "NCHW", "bf16"),
    L("ct_rowphase_zerotap", True, 1, 4, 3, 8, 3, 6, 6, 8, 3, 0, 1, "NCHW", "bf16"),
    L("ct_rowphase_c32", True, 1, 32, 4, 4, 32, 8, 8, 4, 2, 0, 1, "NCHW", "bf16"),
    # stride 2, 4x4, padding 1, NCHW bf16: the all-phase form
    L("ct_quad_img8", True, 2, 64, 8, 8, 64, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_quad_img4_ragged", True, 5, 64, 4, 4, 40, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_quad_two_kgroups", True, 3, 128, 8, 8, 32, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_quad_rows16", True, 2, 192, 16, 16, 96, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_quad_w32", True, 1, 64, 8, 32, 32, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_quad_w64", True, 1, 64, 4, 64, 32, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_quad_np4_rows", True, 2, 128, 16, 16, 64, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ct_quad_np4_ragged", True, 3, 128, 8, 8, 48, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    # a 1x1 input (the generator's projection of z): one dense GEMM
    L("ct_1x1_proj", True, 3, 20, 1, 1, 24, 4, 4, 1, 0, 0, 1, "NCHW", "bf16"),
    L("ct_1x1_proj_f32", True, 2, 16, 1, 1, 8, 3, 5, 2, 0, 0, 1, "NCHW", "f32"),
    L("ct_1x1_nhwc", True, 2, 16, 1, 1, 8, 3, 3, 1, 0, 0, 1, "NHWC", "bf16"),
    # the projection on the 32 x 256 tile: two row tiles (the second ragged), a
    # ragged last channel tile (800 GEMM columns) and a K of 100 (ragged K block)
    L("ct_1x1_proj_rag", True, 45, 100, 1, 1, 50, 4, 4, 1, 0, 0, 1, "NCHW", "bf16"),
]


def _inputs(layer, seed):
    x = wl.layer_input(layer, seed=seed)
    w = wl.random_weight(layer, seed=seed + 1, std=0.1)
    return P.quantise(x, layer.dtype), P.quantise(w, layer.dtype)


@pytest.mark.parametrize("layer", SMALL, ids=lambda l: l.name)
def test_small_case(layer):
    P.say("case", layer)
    xq, wq = _inputs(layer, seed=zlib.crc32(layer.name.encode()) % 1000)
    bias = torch.linspace(-0.5, 0.5, layer.c_out)
    ref = P.oracle_full(layer, xq, wq, bias)
    absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
    y = P.run_gpu(layer, xq, wq, bias)
    P.check(y, ref, absref, layer.dtype, layer.name)


def _random_layers(count, seed):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        tr = bool(rng.integers(0, 2))
        n = int(rng.integers(1, 3))
        ci, co = int(rng.integers(1, 41)), int(rng.integers(1, 70))
        h, w = int(rng.integers(1, 10)), int(rng.integers(1, 10))
        r = int(rng.integers(1, 6))
        st = int(rng.integers(1, 4)) if tr else int(rng.choice([1, 1, 2]))
        dl = int(rng.integers(1, 3))
        pd = int(rng.integers(0, dl * (r - 1) + 1))
        op = int(rng.integers(0, max(st, dl))) if tr else 0
        layout = str(rng.choice(["NCHW", "NHWC"]))
        dtype = str(rng.choice(["f32", "bf16"]))
        lay = L("rand%d" % len(out), tr, n, ci, h, w, co, r, r, st, pd, op, dl, layout, dtype)
        ho, wo = lay.out_hw()
        if ho < 1 or wo < 1:
            continue
        out.append(lay)
    return out


def test_random_sweep():
    for i, layer in enumerate(_random_layers(30, 2024)):
        P.say("case", layer)
        xq, wq = _inputs(layer, seed=500 + i)
        ref = P.oracle_full(layer, xq, wq)
        absref = P.oracle_full(layer, xq, wq, absolute=True)
        y = P.run_gpu(layer, xq, wq)
        P.check(y, ref, absref, layer.dtype, layer.name)


@pytest.mark.parametrize("layer", [SMALL[1], SMALL[4], SMALL[14], SMALL[18]],
                         ids=lambda l: l.name)
def test_one_shot_entry_points(layer):
    P.say("case", layer)
    xq, wq = _inputs(layer, seed=77)
    bias = torch.linspace(1.0, -1.0, layer.c_out)
    ref = P.oracle_full(layer, xq, wq, bias)
    absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
    y = P.run_gpu(layer, xq, wq, bias, one_shot=True)
    P.check(y, ref, absref, layer.dtype, layer.name + " one-shot")


def test_coverage_and_determinism():
    """Every output element is written (a NaN-prefilled output keeps no NaN) and
    two executions of one plan agree bitwise."""
    dev = torch.device("cuda", 0)
    for layer in [SMALL[2], SMALL[4], SMALL[7], SMALL[8], SMALL[15]]:
        P.say("case", layer)
        xq, wq = _inputs(layer, seed=5)
        x_dev = wl.to_layout(xq, layer.layout).to(dev)
        plan = P.make_plan(layer, wq.contiguous().to(dev))
        y1 = torch.full(plan.out_shape, float("nan"), dtype=xq.dtype, device=dev)
        y2 = torch.full(plan.out_shape, float("nan"), dtype=xq.dtype, device=dev)
        plan(x_dev, out=y1)
        plan(x_dev, out=y2)
        torch.cuda.synchronize()
        plan.close()
        assert not torch.isnan(y1).any(), layer.name
        assert torch.equal(y1.view(torch.int16) if y1.dtype == torch.bfloat16 else y1.view(torch.int32),
                           y2.view(torch.int16) if y2.dtype == torch.bfloat16 else y2.view(torch.int32))


# ---- the benchmark workloads ------------------------------------------------

def test_dcgan_chain_reduced_batch():
    """DCGAN generator at batch 2: each layer gets the oracle's output of the
    previous layer (rounded to the dtype), so errors do not compound."""
    for wname in ("dcgan_f32", "dcgan", "dcgan_dgrad", "dcgan_generator"):
        items = wl.generate(wname, seed=0, batch=2)
        x_prev = None
        for layer, x, w in items:
            P.say("case", wname, layer)
            xin = x if x is not None else x_prev
            xq = P.quantise(xin, layer.dtype)
            wq = P.quantise(w, layer.dtype)
            ref = P.oracle_full(layer, xq, wq)
            absref = P.oracle_full(layer, xq, wq, absolute=True)
            y = P.run_gpu(layer, xq, wq)
            P.check(y, ref, absref, layer.dtype, layer.name)
            x_prev = torch.from_numpy(ref).to(torch.float32)


@pytest.mark.parametrize("wname", ["table1_dcgan", "table1_cgan", "dcgan_generator_b1",
                                   "dcgan_generator_nhwc_b1"])
def test_batch1_workloads_full(wname):
    """The paper's own Table 1 deconvolution layers (5x5 DCGAN with unequal
    phases, 4x4 cGAN) and the whole generator with its fused activations, at
    batch 1 (the plan path the benchmark times), checked in full; each layer
    gets the oracle's output of the previous one."""
    items = wl.generate(wname, seed=0)
    x_prev = None
    for layer, x, w in items:
        P.say("case", wname, layer)
        xin = x if x is not None else x_prev
        xq, wq = P.quantise(xin, layer.dtype), P.quantise(w, layer.dtype)
        ref = P.oracle_full(layer, xq, wq)
        absref = P.oracle_full(layer, xq, wq, absolute=True)
        y = P.run_gpu(layer, xq, wq)
        P.check(y, ref, absref, layer.dtype, layer.name)
        x_prev = torch.from_numpy(ref).to(torch.float32)


def test_batch1_form_choice():
    """At batch 1 the long-K DCGAN L1 (16 all-phase workgroups over 1024
    channels) runs on the phase GEMM with its K split across workgroups and
    one K group per workgroup; L2 (512 channels) keeps the all-phase kernel;
    at batch 64 L1 keeps it too."""
    kinds = {}
    for l in wl.WORKLOADS["dcgan_generator_b1"][1:3] + wl.WORKLOADS["dcgan"][:1]:
        P.say("case", l)
        w = wl.random_weight(l, seed=3).to(torch.bfloat16).cuda()
        p = P.make_plan(l, w)
        kinds[(l.name, l.n)] = p.kernel
        p.close()
    assert kinds[("gen_l1", 1)].startswith("phase_gemm2_kernel 64x128 w4 k1"), kinds
    assert kinds[("gen_l2", 1)].startswith("quad_kernel"), kinds
    assert kinds[("dcgan_l1", 64)].startswith("quad_kernel"), kinds


@pytest.mark.parametrize("wname", ["dcgan_generator_nhwc_b1", "dcgan_generator_b1"])
def test_generator_end_to_end(wname):
    """The whole generator as the benchmark runs it: each layer reads the
    previous layer's output where it lies on the device, in the workload's
    layout (no host round trip).  Every layer's output matches the oracle
    applied to that same device input, and the image is written in full."""
    dev = torch.device("cuda", 0)
    items = wl.generate(wname, seed=0)
    layout = items[0][0].layout
    x_dev = None
    plans = []
    try:
        for i, (layer, x, w) in enumerate(items):
            P.say("case", wname, layer)
            if x_dev is None:
                x_dev = wl.to_layout(P.quantise(x, layer.dtype), layout).to(dev)
            wq = P.quantise(w, layer.dtype)
            plans.append(P.make_plan(layer, wq.contiguous().to(dev)))
            y_dev = torch.full(plans[-1].out_shape, float("nan"), dtype=x_dev.dtype, device=dev)
            plans[-1](x_dev, out=y_dev)
            torch.cuda.synchronize()
            xin = wl.from_layout(x_dev.cpu(), layout).float()
            ref = P.oracle_full(layer, xin, wq)
            absref = P.oracle_full(layer, xin, wq, absolute=True)
            y = wl.from_layout(y_dev.cpu(), layout).double().numpy()
            P.check(y, ref, absref, layer.dtype, layer.name)
            x_dev = y_dev
        assert tuple(x_dev.shape) == ((1, 3, 64, 64) if layout == "NCHW" else (1, 64, 64, 3))
    finally:
        for p in plans:
            p.close()


REDUCED = [
    ("convt_small", {}),
    ("convt_odd", dict(n=1)),
    ("aspp", dict(n=1, c_in=256, c_out=64)),
    ("fcn_upsample", dict(n=1, c_in=5, c_out=5, h=3, w=3)),
]


@pytest.mark.parametrize("wname,over", REDUCED, ids=[r[0] for r in REDUCED])
def test_workload_reduced_full_check(wname, over):
    for i, layer in enumerate(wl.WORKLOADS[wname]):
        layer = layer.with_(**over)
        P.say("case", layer)
        g = torch.Generator("cpu").manual_seed(i)
        x = wl.layer_input(layer, seed=10 + i)
        if wname == "aspp":
            x = torch.relu(x)
        w = wl.random_weight(layer, seed=20 + i, std=0.02)
        if wname == "fcn_upsample":
            f = wl.bilinear_kernel(layer.r).to(torch.float32)
            w = w * 0.05
            for c in range(layer.c_in):
                w[c, c] += torch.outer(f, f)
        del g
        xq, wq = P.quantise(x, layer.dtype), P.quantise(w, layer.dtype)
        ref = P.oracle_full(layer, xq, wq)
        absref = P.oracle_full(layer, xq, wq, absolute=True)
        y = P.run_gpu(layer, xq, wq)
        P.check(y, ref, absref, layer.dtype, layer.name)


FULL = ["convt_small", "dcgan_f32", "dcgan", "convt_odd", "aspp", "fcn_upsample", "dcgan_dgrad",
        "dcgan_generator", "dcgan_generator_nhwc"]


@pytest.mark.parametrize("wname", FULL)
def test_workload_full_size_sampled(wname):
    """Full-size workloads, plan path (as timed by the benchmark), checked on
    sampled outputs that cover every phase, border and first/last channel;
    the output starts as NaN, so the finiteness check over the whole tensor
    shows that every element was written."""
    items = wl.generate(wname, seed=0)
    for i, (layer, x, w) in enumerate(items):
        if x is None:  # chained layers 2-4: standalone input of the chained shape
            x = wl.layer_input(layer, seed=100 + i, std=0.25)
        P.say("case", wname, layer)
        xq, wq = P.quantise(x, layer.dtype), P.quantise(w, layer.dtype)
        y = P.run_gpu(layer, xq, wq, prefill_nan=True)
        idx = P.sample_indices(layer, 3000, seed=i)
        ref = P.oracle_points(layer, xq, wq, idx)
        absref = P.oracle_points(layer, xq, wq, idx, absolute=True)
        P.check(y.ravel()[idx], ref, absref, layer.dtype, layer.name)
        assert np.all(np.isfinite(y))


TILE_CONFIGS = list(range(P.tile_count()))  # every GEMM tile configuration


@pytest.mark.parametrize("tile", TILE_CONFIGS)
def test_every_tile_configuration(tile, monkeypatch):
    """Each tile shape (forced through HUGE2_TILE at plan creation) matches the
    oracle on ragged transposed and dilated cases in both layouts and dtypes."""
    monkeypatch.setenv("HUGE2_TILE", str(tile))
    for layer in [SMALL[0], SMALL[2], SMALL[4], SMALL[7], SMALL[14], SMALL[19]]:
        P.say("case tile", tile, layer)
        xq, wq = _inputs(layer, seed=31 + tile)
        bias = torch.linspace(-0.25, 0.75, layer.c_out)
        ref = P.oracle_full(layer, xq, wq, bias)
        absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
        y = P.run_gpu(layer, xq, wq, bias)
        P.check(y, ref, absref, layer.dtype, "%s tile %d" % (layer.name, tile))


@pytest.mark.parametrize("layer", [SMALL[2], SMALL[1], SMALL[7], SMALL[14]], ids=lambda l: l.name)
def test_stage_then_gemm_equals_execute(layer):
    """huge2_plan_stage_input followed by huge2_plan_run_gemm writes the same
    bits as huge2_plan_execute, whether or not the plan stages its input."""
    P.say("case", layer)
    dev = torch.device("cuda", 0)
    xq, wq = _inputs(layer, seed=9)
    x_dev = wl.to_layout(xq, layer.layout).to(dev)
    bias = torch.linspace(-1.0, 1.0, layer.c_out).to(dev)
    plan = P.make_plan(layer, wq.contiguous().to(dev))
    y1 = torch.full(plan.out_shape, float("nan"), dtype=xq.dtype, device=dev)
    y2 = torch.full(plan.out_shape, float("nan"), dtype=xq.dtype, device=dev)
    plan(x_dev, bias=bias, out=y1)
    plan.stage(x_dev)
    plan.gemm(x_dev, y2, bias=bias)
    torch.cuda.synchronize()
    staged = plan.stages_input
    plan.close()
    assert staged == (layer.layout == "NCHW" or layer.c_in % (8 if layer.dtype == "bf16" else 4) != 0)
    assert not torch.isnan(y2).any()
    iv = torch.int16 if y1.dtype == torch.bfloat16 else torch.int32
    assert torch.equal(y1.view(iv), y2.view(iv)), layer.name


@pytest.mark.parametrize("split", [0, 1, 2])
def test_border_class_forms(split, monkeypatch):
    """Both forms of a phase's border handling (one masked segment, or border
    classes that read only in-range inputs) and the per-group choice agree
    with the oracle."""
    monkeypatch.setenv("HUGE2_CLASS_SPLIT", str(split))
    for layer in [SMALL[0], SMALL[4], SMALL[9], SMALL[15], SMALL[16], SMALL[18]]:
        P.say("case split", split, layer)
        xq, wq = _inputs(layer, seed=50 + split)
        bias = torch.linspace(-0.5, 0.25, layer.c_out)
        ref = P.oracle_full(layer, xq, wq, bias)
        absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
        y = P.run_gpu(layer, xq, wq, bias)
        P.check(y, ref, absref, layer.dtype, "%s split %d" % (layer.name, split))


def test_plan_execute_in_hip_graph():
    """A plan's launches captured in a HIP graph reproduce the eager result on
    every replay, with other eager work on the device between replays."""
    dev = torch.device("cuda", 0)
    layer = SMALL[2]  # NCHW bf16: staging kernel + GEMM
    P.say("case graph", layer)
    xq, wq = _inputs(layer, seed=3)
    x_dev = wl.to_layout(xq, layer.layout).to(dev)
    bias = torch.linspace(-1.0, 1.0, layer.c_out).to(dev)
    plan = P.make_plan(layer, wq.contiguous().to(dev))
    y_eager = torch.empty(plan.out_shape, dtype=xq.dtype, device=dev)
    plan(x_dev, bias=bias, out=y_eager)
    y = torch.empty_like(y_eager)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        plan(x_dev, bias=bias, out=y)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        plan(x_dev, bias=bias, out=y)
    scratch = torch.empty(1 << 20, device=dev)
    for k in range(4):
        y.fill_(float("nan"))
        scratch.normal_()  # unrelated eager work between replays
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), y_eager.view(torch.int16)), "replay %d" % k
    del g
    plan.close()


FEWOUT_NHWC = [
    # NHWC input and output (16-byte channel groups per pixel)
    L("ct_fewout_nhwc", True, 2, 40, 6, 8, 3, 4, 4, 2, 1, 0, 1, "NHWC", "bf16"),
    # stride 3, dilation 2: phases with different tap counts
    L("ct_fewout_nhwc_s3d2", True, 1, 16, 5, 6, 4, 3, 3, 3, 2, 0, 2, "NHWC", "bf16"),
    # three 64-channel passes, the last one ragged (136 channels)
    L("ct_fewout_nhwc_tall", True, 1, 136, 4, 4, 1, 4, 4, 2, 1, 0, 1, "NHWC", "bf16"),
]


@pytest.mark.parametrize("ztile", [0, 1])
def test_few_output_channel_forms(ztile, monkeypatch):
    """Few-output-channel transposed convs (NCHW, and NHWC with 8-channel
    groups) through the all-taps form and, with it switched off, through the
    phase GEMM: both match the oracle."""
    monkeypatch.setenv("HUGE2_ZTILE", str(ztile))
    for layer in [l for l in SMALL if l.name.startswith("ct_fewout")] + [SMALL[12]] + FEWOUT_NHWC:
        P.say("case ztile", ztile, layer)
        xq, wq = _inputs(layer, seed=70 + ztile)
        bias = torch.linspace(-0.3, 0.6, layer.c_out)
        ref = P.oracle_full(layer, xq, wq, bias)
        absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
        y = P.run_gpu(layer, xq, wq, bias, prefill_nan=True)
        P.check(y, ref, absref, layer.dtype, "%s ztile %d" % (layer.name, ztile))
        if layer in FEWOUT_NHWC:
            plan = P.make_plan(layer, wq.contiguous().to(torch.device("cuda", 0)))
            try:
                assert plan.kernel.startswith("ztile_kernel") == bool(ztile), plan.kernel
            finally:
                plan.close()


def test_plan_reports_its_kernel():
    """huge2_plan_kernel names the kernel family the planner chose."""
    dev = torch.device("cuda", 0)
    for layer, family in [(SMALL[23], "ztile_kernel"), (SMALL[1], "phase_gemm"),
                          (SMALL[14], "phase_gemm")]:
        P.say("case kernel name", layer)
        wq = P.quantise(wl.random_weight(layer, seed=1, std=0.1), layer.dtype)
        plan = P.make_plan(layer, wq.contiguous().to(dev))
        name = plan.kernel
        plan.close()
        assert name.startswith(family), (layer.name, name)


@pytest.mark.parametrize("rowphase", [0, 1])
def test_large_stride_forms(rowphase, monkeypatch):
    """Large-stride few-channel NCHW transposed convs through the output-
    stationary form and, with it switched off, through the phase GEMM."""
    monkeypatch.setenv("HUGE2_ROWPHASE", str(rowphase))
    dev = torch.device("cuda", 0)
    for layer in [l for l in SMALL if l.name.startswith("ct_rowphase")]:
        P.say("case rowphase", rowphase, layer)
        xq, wq = _inputs(layer, seed=90 + rowphase)
        bias = torch.linspace(-0.4, 0.4, layer.c_out)
        ref = P.oracle_full(layer, xq, wq, bias)
        absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
        y = P.run_gpu(layer, xq, wq, bias)
        P.check(y, ref, absref, layer.dtype, "%s rowphase %d" % (layer.name, rowphase))
        plan = P.make_plan(layer, wq.contiguous().to(dev))
        name = plan.kernel
        plan.close()
        assert name.startswith("rowphase_kernel") == bool(rowphase), (layer.name, name)



QUAD = [l for l in SMALL if l.name.startswith("ct_quad")]
# the same layers in NHWC (16-byte channel groups in, pixel runs of channels out)
QUAD += [l.with_(name=l.name + "_nhwc", layout="NHWC") for l in QUAD]


# (layer, K groups) pairs that tile 128 positions per workgroup
QUAD_NP4 = {("ct_quad_img8", 1), ("ct_quad_two_kgroups", 1), ("ct_quad_two_kgroups", 2),
            ("ct_quad_rows16", 1), ("ct_quad_np4_rows", 1), ("ct_quad_np4_ragged", 1),
            ("ct_quad_np4_ragged", 2)}


@pytest.mark.parametrize("quad,wch,np_,ks", [(0, 1, 0, 0), (1, 1, 2, 0), (1, 2, 2, 0), (1, 1, 4, 1),
                                             (1, 1, 4, 2)])
@pytest.mark.parametrize("layer", QUAD, ids=lambda l: l.name)
def test_all_phase_forms(layer, quad, wch, np_, ks, monkeypatch):
    """The all-phase kernel (64 positions per workgroup in both wave layouts,
    128 positions in one or two K groups) and the phase GEMM it replaces all
    match the oracle."""
    monkeypatch.setenv("HUGE2_QUAD", str(quad))
    monkeypatch.setenv("HUGE2_QUAD_WCH", str(wch))
    monkeypatch.setenv("HUGE2_QUAD_NP", str(np_))
    monkeypatch.setenv("HUGE2_QUAD_KS", str(ks))
    P.say("case", layer, "HUGE2_QUAD", quad, "HUGE2_QUAD_WCH", wch, "HUGE2_QUAD_NP", np_,
          "HUGE2_QUAD_KS", ks)
    xq, wq = _inputs(layer, seed=11)
    bias = torch.linspace(-1.0, 1.0, layer.c_out)
    y = P.run_gpu(layer, xq, wq, bias, prefill_nan=True)
    P.check(y, P.oracle_full(layer, xq, wq, bias), P.oracle_full(layer, xq, wq, bias, absolute=True),
            layer.dtype, layer.name)
    plan = P.make_plan(layer, wq.contiguous().to(torch.device("cuda", 0)))
    try:
        expect = bool(quad) and (np_ != 4 or (layer.name.replace("_nhwc", ""), ks) in QUAD_NP4)
        assert ("quad_kernel" in plan.kernel) == expect, plan.kernel
        if expect and np_ == 4:
            dims = plan.kernel.split()[1].split("x")
            assert int(dims[0]) * int(dims[1]) * int(dims[2]) == 128, plan.kernel
    finally:
        plan.close()


# one layer per kernel form: phase GEMM (NHWC bf16, NCHW fp32, a zero-tap
# phase), all-taps, row-phase and all-phase
ACT_LAYERS = [SMALL[i] for i in range(len(SMALL)) if SMALL[i].name in (
    "ct_fewout_bf16", "ct_rowphase_zerotap", "ct_rowphase_s4", "ct_quad_img8", "ct_quad_np4_rows",
    "dil_f32_nchw", "conv_plain", "dil_aspp_d6", "ct_1x1_proj")]


@pytest.mark.parametrize("act", ["relu", "tanh"])
@pytest.mark.parametrize("layer", ACT_LAYERS, ids=lambda l: l.name)
def test_fused_activation(layer, act):
    """y = act(op(x) + bias) from every kernel's epilogue, plan and one-shot
    entry points, against the oracle followed by the same function."""
    layer = layer.with_(act=act)
    P.say("case", layer)
    xq, wq = _inputs(layer, seed=13)
    bias = torch.linspace(-0.5, 0.5, layer.c_out)
    ref = P.oracle_full(layer, xq, wq, bias)
    absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
    P.check(P.run_gpu(layer, xq, wq, bias), ref, absref, layer.dtype, layer.name)
    P.check(P.run_gpu(layer, xq, wq, bias, one_shot=True), ref, absref, layer.dtype, layer.name)
    if act == "relu":
        assert np.all(P.run_gpu(layer, xq, wq, bias) >= 0)


# phase-GEMM layers of every output layout and dtype, with ragged channels
SPLITK_LAYERS = [l for l in SMALL if l.name in ("ct_vecstage_bf16", "ct_ragged_bf16_nhwc")] + [
    L("sk_conv_nchw", False, 2, 200, 9, 7, 40, 3, 3, 2, 1, 0, 1, "NCHW", "bf16"),
    L("sk_ct_nhwc_f32", True, 1, 150, 5, 6, 24, 3, 3, 2, 1, 1, 1, "NHWC", "f32"),
    L("sk_dgrad_nchw", False, 2, 256, 8, 8, 64, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("sk_proj_nchw", True, 2, 300, 1, 1, 16, 4, 4, 1, 0, 0, 1, "NCHW", "bf16"),
    L("sk_proj_nhwc", True, 2, 300, 1, 1, 24, 3, 4, 1, 0, 0, 1, "NHWC", "bf16"),
]


@pytest.mark.parametrize("ksplit", [2, 3, 4])
@pytest.mark.parametrize("layer", SPLITK_LAYERS, ids=lambda l: l.name)
def test_split_k(layer, ksplit, monkeypatch):
    """K split across workgroups (fp32 partials added in order by a second
    kernel, with bias and activation) matches the oracle and is bitwise
    reproducible."""
    monkeypatch.setenv("HUGE2_SPLITK", str(ksplit))
    layer = layer.with_(act="relu")
    P.say("case", layer, "HUGE2_SPLITK", ksplit)
    xq, wq = _inputs(layer, seed=17)
    bias = torch.linspace(-0.5, 0.5, layer.c_out)
    ref = P.oracle_full(layer, xq, wq, bias)
    absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
    y1 = P.run_gpu(layer, xq, wq, bias)
    P.check(y1, ref, absref, layer.dtype, layer.name)
    assert np.array_equal(y1, P.run_gpu(layer, xq, wq, bias))


PRODUCT_NHWC_LAYERS = [
    # the generator's projection of z in NHWC: ragged row tile and channels
    L("pn_proj_rag", True, 45, 100, 1, 1, 50, 4, 4, 1, 0, 0, 1, "NHWC", "bf16"),
    # fp32, a 3 x 5 kernel, a stride (irrelevant for one input pixel)
    L("pn_f32_3x5", True, 2, 16, 1, 1, 8, 3, 5, 2, 0, 0, 1, "NHWC", "f32"),
    # many columns (the generator's 1024 channels x 16 taps) at batch 1
    L("pn_wide_b1", True, 1, 100, 1, 1, 1024, 4, 4, 1, 0, 0, 1, "NHWC", "bf16"),
]


@pytest.mark.parametrize("product", [1, 0])
@pytest.mark.parametrize("layer", PRODUCT_NHWC_LAYERS, ids=lambda l: l.name)
def test_product_form_nhwc(layer, product, monkeypatch):
    """A 1x1 NHWC input as one dense GEMM whose columns are the output's own
    order (tap-major weight packing, bias repeating every C_out columns),
    and with the form switched off the phase GEMM: both match the oracle,
    with bias and ReLU, and write every output element."""
    monkeypatch.setenv("HUGE2_PRODUCT_NHWC", str(product))
    layer = layer.with_(act="relu")
    P.say("case", layer, "HUGE2_PRODUCT_NHWC", product)
    xq, wq = _inputs(layer, seed=23)
    bias = torch.linspace(-0.5, 0.5, layer.c_out)
    ref = P.oracle_full(layer, xq, wq, bias)
    absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
    y = P.run_gpu(layer, xq, wq, bias, prefill_nan=True)
    P.check(y, ref, absref, layer.dtype, layer.name)


TWO_PASS_LAYERS = [l for l in SMALL if l.name in ("ct_fewout_f32_op", "ct_fewout_wide")] + [
    L("tp_rgb_f32", True, 2, 128, 8, 8, 3, 4, 4, 2, 1, 0, 1, "NCHW", "f32"),
    L("tp_dil_f32", True, 1, 40, 6, 7, 4, 3, 3, 3, 2, 1, 2, "NCHW", "f32"),
]


@pytest.mark.parametrize("two_pass", [1, 0])
@pytest.mark.parametrize("layer", TWO_PASS_LAYERS, ids=lambda l: l.name)
def test_two_pass_forms(layer, two_pass, monkeypatch):
    """fp32 transposed convs with few output channels: the two-pass form
    (pointwise GEMM to per-tap maps, then the ordered gather) and the phase
    GEMM it replaces both match the oracle, bias and activation included."""
    monkeypatch.setenv("HUGE2_TWOPASS", str(two_pass))
    layer = layer.with_(act="tanh")
    P.say("case", layer, "HUGE2_TWOPASS", two_pass)
    xq, wq = _inputs(layer, seed=19)
    bias = torch.linspace(-0.5, 0.5, layer.c_out)
    ref = P.oracle_full(layer, xq, wq, bias)
    absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
    y = P.run_gpu(layer, xq, wq, bias)
    P.check(y, ref, absref, layer.dtype, layer.name)
    assert np.array_equal(y, P.run_gpu(layer, xq, wq, bias))
    P.check(P.run_gpu(layer, xq, wq, bias, one_shot=True), ref, absref, layer.dtype, layer.name)
    plan = P.make_plan(layer, wq.contiguous().to(torch.device("cuda", 0)))
    try:
        assert plan.kernel.startswith("two-pass") == bool(two_pass), plan.kernel
    finally:
        plan.close()


GATHER_LAYERS = [
    L("ga_rgb_s2", False, 2, 3, 16, 16, 40, 4, 4, 2, 1, 0, 1, "NCHW", "bf16"),
    L("ga_rgb_f32", False, 2, 3, 11, 9, 24, 3, 3, 1, 1, 0, 1, "NCHW", "f32"),
    L("ga_dil", False, 1, 5, 13, 12, 16, 3, 3, 1, 2, 0, 2, "NCHW", "bf16"),
    L("ga_valid_odd", False, 3, 7, 10, 14, 8, 3, 3, 2, 0, 0, 1, "NCHW", "bf16"),
]


@pytest.mark.parametrize("gather", [1, 0])
@pytest.mark.parametrize("layer", GATHER_LAYERS, ids=lambda l: l.name)
def test_gather_forms(layer, gather, monkeypatch):
    """Convs with few input channels: the receptive-field gather into a
    pointwise GEMM and the phase GEMM it replaces both match the oracle."""
    monkeypatch.setenv("HUGE2_GATHER", str(gather))
    layer = layer.with_(act="relu")
    P.say("case", layer, "HUGE2_GATHER", gather)
    xq, wq = _inputs(layer, seed=23)
    bias = torch.linspace(-0.5, 0.5, layer.c_out)
    ref = P.oracle_full(layer, xq, wq, bias)
    absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
    y = P.run_gpu(layer, xq, wq, bias)
    P.check(y, ref, absref, layer.dtype, layer.name)
    assert np.array_equal(y, P.run_gpu(layer, xq, wq, bias))
    P.check(P.run_gpu(layer, xq, wq, bias, one_shot=True), ref, absref, layer.dtype, layer.name)
    plan = P.make_plan(layer, wq.contiguous().to(torch.device("cuda", 0)))
    try:
        assert plan.kernel.startswith("gather_taps") == bool(gather), plan.kernel
        assert plan.stages_input
    finally:
        plan.close()


LISTED_LAYERS = [
    L("li_aspp_d6", False, 2, 64, 64, 64, 48, 3, 3, 1, 6, 0, 6, "NHWC", "bf16"),
    L("li_aspp_d24", False, 1, 64, 64, 64, 48, 3, 3, 1, 24, 0, 24, "NHWC", "bf16"),
    # an image whose pixel count is no multiple of the tile height: the last
    # tile of each image is partial and must not touch the next image
    L("li_ragged_img", False, 3, 40, 13, 11, 72, 3, 3, 1, 3, 0, 3, "NHWC", "bf16"),
    # dilation larger than half the image: a band with only the centre tap
    L("li_wide_dil", False, 2, 24, 9, 10, 40, 3, 3, 1, 7, 0, 7, "NHWC", "bf16"),
    L("li_aniso_5x3", False, 2, 16, 12, 17, 36, 5, 3, 1, 2, 0, 2, "NCHW", "f32"),
    L("li_valid_pad0", False, 1, 32, 15, 15, 64, 3, 3, 1, 0, 0, 3, "NHWC", "f32"),
    L("li_c300", False, 1, 300, 20, 20, 260, 3, 3, 1, 4, 0, 4, "NHWC", "bf16"),
]


@pytest.mark.parametrize("listed", [0, 1])
@pytest.mark.parametrize("layer", LISTED_LAYERS, ids=lambda l: l.name)
def test_listed_form(layer, listed, monkeypatch):
    """Stride-1 dilated convs through the listed form (per-image pixel list in
    border-cell and phase-view order, each tile with the union of its pixels'
    taps) and through the phase-view segments: both match the oracle and write
    every output element."""
    monkeypatch.setenv("HUGE2_LISTED", str(listed))
    layer = layer.with_(act="relu")
    P.say("case", layer, "HUGE2_LISTED", listed)
    xq, wq = _inputs(layer, seed=29)
    bias = torch.linspace(-0.5, 0.5, layer.c_out)
    ref = P.oracle_full(layer, xq, wq, bias)
    absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
    y = P.run_gpu(layer, xq, wq, bias, prefill_nan=True)
    P.check(y, ref, absref, layer.dtype, layer.name)
    plan = P.make_plan(layer, wq.contiguous().to(torch.device("cuda", 0)))
    try:
        assert plan.kernel.endswith("listed") == bool(listed), plan.kernel
    finally:
        plan.close()


GROUP_SETS = [
    # the pyramid's four branches at reduced size (listed form)
    [L("gr_d%d" % d, False, 2, 96, 24, 24, 64, 3, 3, 1, d, 0, d, "NHWC", "bf16") for d in (2, 3, 5, 8)],
    # branches of different kinds and paddings on one input, fp32
    [L("gr_f32_a", False, 1, 24, 13, 11, 40, 3, 3, 1, 1, 0, 1, "NHWC", "f32"),
     L("gr_f32_b", False, 1, 24, 13, 11, 40, 3, 3, 1, 2, 0, 2, "NHWC", "f32"),
     L("gr_f32_c", False, 1, 24, 13, 11, 40, 3, 3, 1, 3, 0, 3, "NHWC", "f32")],
]


# four branches of 256 works each (the single plans take the 8-wave
# pipelined tile) whose 1024 works make the group run the 4-wave form
GROUP_UPGRADE = [L("gu_d%d" % d, False, 2, 64, 128, 128, 256, 3, 3, 1, d, 0, d, "NHWC", "bf16")
                 for d in (2, 6, 12, 24)]


def test_grouped_launch_two_per_cu():
    """A group long enough for two workgroups per compute unit runs the
    4-wave pipelined tile: its outputs match the oracle on sampled points,
    are written in full, and equal each plan's own output to rounding."""
    dev = torch.device("cuda", 0)
    layers = GROUP_UPGRADE
    x = P.quantise(wl.layer_input(layers[0], seed=43), "bf16")
    x_dev = wl.to_layout(x, "NHWC").to(dev)
    plans, ws = [], []
    for i, layer in enumerate(layers):
        P.say("case group", layer)
        wq = P.quantise(wl.random_weight(layer, seed=44 + i, std=0.05), "bf16")
        ws.append(wq)
        plans.append(P.make_plan(layer, wq.contiguous().to(dev)))
        assert "w8" in plans[-1].kernel, plans[-1].kernel
    group = h2.Group(plans)
    try:
        assert "phase_gemm3_kernel 128x256 w4" in group.kernel, group.kernel
        outs = [torch.full(p.out_shape, float("nan"), dtype=x.dtype, device=dev) for p in plans]
        group(x_dev, None, outs)
        single = [p(x_dev) for p in plans]
        torch.cuda.synchronize()
        for k, (layer, wq, y, y1) in enumerate(zip(layers, ws, outs, single)):
            yf, y1f = y.float(), y1.float()
            assert bool(torch.isfinite(yf).all()), layer.name
            scale = float(y1f.abs().max())
            assert float((yf - y1f).abs().max()) <= 2e-2 * scale, layer.name
            idx = P.sample_indices(layer, 3000, seed=50 + k)
            yn = wl.from_layout(y.cpu(), "NHWC").double().numpy().reshape(-1)[idx]
            ref = P.oracle_points(layer, x, wq, idx)
            absref = P.oracle_points(layer, x, wq, idx, absolute=True)
            P.check(yn, ref, absref, "bf16", layer.name + " grouped w4")
    finally:
        group.close()
        for p in plans:
            p.close()


@pytest.mark.parametrize("layers", GROUP_SETS, ids=["aspp_reduced", "mixed_f32"])
def test_grouped_launch(layers):
    """Several plans of one input in one launch (huge2_group): every output
    matches the oracle, equals its own plan's output bitwise, and is written
    in full (NaN-prefilled outputs keep no NaN)."""
    dev = torch.device("cuda", 0)
    x = P.quantise(wl.layer_input(layers[0], seed=41), layers[0].dtype)
    x_dev = wl.to_layout(x, layers[0].layout).to(dev)
    plans, ws, biases = [], [], []
    for i, layer in enumerate(layers):
        P.say("case group", layer)
        wq = P.quantise(wl.random_weight(layer, seed=42 + i, std=0.05), layer.dtype)
        ws.append(wq)
        plans.append(P.make_plan(layer, wq.contiguous().to(dev)))
        biases.append(torch.linspace(-0.5, 0.5 + i, layer.c_out).to(dev))
    group = h2.Group(plans)
    try:
        outs = [torch.full(p.out_shape, float("nan"), dtype=x.dtype, device=dev) for p in plans]
        group(x_dev, biases, outs)
        single = [p(x_dev, b) for p, b in zip(plans, biases)]
        torch.cuda.synchronize()
        for layer, wq, b, y, y1 in zip(layers, ws, biases, outs, single):
            iv = torch.int16 if y.dtype == torch.bfloat16 else torch.int32
            assert torch.equal(y.view(iv), y1.view(iv)), layer.name
            yn = wl.from_layout(y.cpu(), layer.layout).double().numpy()
            ref = P.oracle_full(layer, x, wq, b.cpu())
            absref = P.oracle_full(layer, x, wq, b.cpu(), absolute=True)
            P.check(yn, ref, absref, layer.dtype, layer.name + " grouped")
    finally:
        group.close()
        for p in plans:
            p.close()


def test_group_rejects_unlike_plans():
    """Plans of different input shapes cannot share a launch."""
    dev = torch.device("cuda", 0)
    a = L("ga", False, 1, 16, 8, 8, 32, 3, 3, 1, 1, 0, 1, "NHWC", "bf16")
    b = a.with_(name="gb", h=9)
    pa = P.make_plan(a, P.quantise(wl.random_weight(a, seed=1), "bf16").to(dev))
    pb = P.make_plan(b, P.quantise(wl.random_weight(b, seed=2), "bf16").to(dev))
    try:
        with pytest.raises(h2.Huge2Error) as e:
            h2.Group([pa, pb])
        assert e.value.status == h2.HUGE2_ERR_UNSUPPORTED
    finally:
        pa.close()
        pb.close()


COLPHASE_LAYERS = [
    L("cp_fcn_reduced", True, 2, 21, 5, 6, 21, 64, 64, 32, 16, 0, 1, "NCHW", "bf16"),
    # 32 input channels, a short kernel (phases with one tap or none per axis)
    L("cp_c32_short", True, 1, 32, 3, 4, 8, 36, 40, 32, 8, 0, 1, "NCHW", "bf16"),
    # output padding, a kernel shorter than two row strides
    L("cp_outpad", True, 3, 5, 4, 3, 6, 30, 64, 32, 8, 8, 1, "NCHW", "bf16"),
    # no padding: the first and last column blocks are whole
    L("cp_pad0", True, 1, 12, 2, 2, 33, 64, 64, 32, 0, 0, 1, "NCHW", "bf16"),
    # input rows of 8 and 16 pixels: the 16-byte staging pieces, fewer pieces
    # than threads (15) and more than four rounds of them (1056)
    L("cp_w8_few", True, 1, 5, 3, 8, 7, 64, 64, 32, 16, 0, 1, "NCHW", "bf16"),
    L("cp_w8_many", True, 1, 32, 33, 8, 2, 32, 32, 32, 0, 0, 1, "NCHW", "bf16"),
]


_COLPHASE_REF = {}


def _colphase_reference(layer):
    # the oracle's result for a layer, computed once for both forms
    if layer.name not in _COLPHASE_REF:
        xq, wq = _inputs(layer, seed=37)
        bias = torch.linspace(-0.5, 0.5, layer.c_out)
        _COLPHASE_REF[layer.name] = (xq, wq, bias, P.oracle_full(layer, xq, wq, bias),
                                     P.oracle_full(layer, xq, wq, bias, absolute=True))
    return _COLPHASE_REF[layer.name]


@pytest.mark.parametrize("colphase", [1, 0])
@pytest.mark.parametrize("layer", COLPHASE_LAYERS, ids=lambda l: l.name)
def test_colphase_form(layer, colphase, monkeypatch):
    """Column stride 32: the column-phase form (the 32 column phases as MFMA
    rows, 16-byte row pieces) and, with it switched off, the other forms all
    match the oracle and write every output element."""
    monkeypatch.setenv("HUGE2_COLPHASE", str(colphase))
    layer = layer.with_(act="relu")
    P.say("case", layer, "HUGE2_COLPHASE", colphase)
    xq, wq, bias, ref, absref = _colphase_reference(layer)
    y = P.run_gpu(layer, xq, wq, bias, prefill_nan=True)
    P.check(y, ref, absref, layer.dtype, layer.name)
    plan = P.make_plan(layer, wq.contiguous().to(torch.device("cuda", 0)))
    try:
        assert plan.kernel.startswith("colphase_kernel") == bool(colphase), plan.kernel
    finally:
        plan.close()


def LG(name, tr, n, ci, h, w, co, r, s, st, pd, op, dl, layout, dtype, groups):
    return Layer(name, tr, n, ci, h, w, co, r, s, st, pd, op, dl, layout, dtype, "none", groups)


GROUPED_LAYERS = [
    # depthwise transposed upsampling (groups = C_in = C_out)
    LG("gp_dw_ct_nhwc", True, 2, 64, 8, 8, 64, 4, 4, 2, 1, 0, 1, "NHWC", "bf16", 64),
    # depthwise with channel multiplier 2 and output padding
    LG("gp_dw_mult2_f32", True, 2, 8, 5, 6, 16, 3, 3, 2, 1, 1, 1, "NCHW", "f32", 8),
    LG("gp_ct_g4", True, 1, 32, 6, 5, 48, 3, 3, 2, 1, 0, 1, "NHWC", "bf16", 4),
    LG("gp_dil_g3", False, 2, 24, 9, 10, 36, 3, 3, 1, 2, 0, 2, "NCHW", "bf16", 3),
    LG("gp_dw_strided_dil", False, 1, 16, 11, 9, 16, 3, 3, 2, 2, 0, 2, "NHWC", "f32", 16),
]


@pytest.mark.parametrize("layer", GROUPED_LAYERS, ids=lambda l: l.name)
def test_grouped_and_depthwise(layer):
    """Grouped and depthwise transposed / dilated convs (the descriptor's
    groups) against the grouped oracle, plan and one-shot entry points, every
    output element written."""
    layer = layer.with_(act="relu")
    P.say("case", layer)
    xq, wq = _inputs(layer, seed=43)
    bias = torch.linspace(-0.5, 0.5, layer.c_out)
    ref = P.oracle_full(layer, xq, wq, bias)
    absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
    P.check(P.run_gpu(layer, xq, wq, bias, prefill_nan=True), ref, absref, layer.dtype, layer.name)
    P.check(P.run_gpu(layer, xq, wq, bias, one_shot=True), ref, absref, layer.dtype, layer.name)
    plan = P.make_plan(layer, wq.contiguous().to(torch.device("cuda", 0)))
    try:
        assert plan.kernel.startswith("grouped_kernel"), plan.kernel
        nz, issued = plan.macs()
        assert nz == issued
    finally:
        plan.close()


def test_launch_fault_is_reported(monkeypatch):
    """HUGE2_FAULT=launch (set from the host) makes every enqueueing entry
    point report HUGE2_ERR_HIP without touching its output."""
    dev = torch.device("cuda", 0)
    layer = SMALL[1]  # NHWC bf16 phase GEMM
    xq, wq = _inputs(layer, seed=5)
    x_dev = wl.to_layout(xq, layer.layout).to(dev)
    w_dev = wq.contiguous().to(dev)
    plan = P.make_plan(layer, w_dev)
    try:
        y = torch.full(plan.out_shape, 3.0, dtype=xq.dtype, device=dev)
        monkeypatch.setenv("HUGE2_FAULT", "launch")
        for call in (lambda: plan(x_dev, out=y), lambda: plan.gemm(x_dev, y),
                     lambda: h2.conv2d_transpose(x_dev, w_dev, None, layer.stride, layer.pad,
                                                 layer.out_pad, layer.dil, layer.layout, out=y)):
            with pytest.raises(h2.Huge2Error) as e:
                call()
            assert e.value.status == h2.HUGE2_ERR_HIP
        monkeypatch.delenv("HUGE2_FAULT")
        torch.cuda.synchronize()
        assert bool((y == 3.0).all())
    finally:
        plan.close()
