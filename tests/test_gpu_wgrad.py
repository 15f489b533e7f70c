"""GPU parity of the weight gradients (section 3.2.3, GAN training) through
the C ABI, against the CPU oracle's chain-rule definitions, element by
element with the dot-product error bound (tests/parity.py): the bound uses
the oracle on |x| and |dy|.  Also the data gradients, which are the forward
entry points with the roles exchanged."""
import numpy as np
import pytest
import torch

import oracle
from paper_1907_11210_amd import huge2 as h2
from paper_1907_11210_amd import workloads as wl

import parity as P

pytestmark = pytest.mark.gpu

# (name, transposed, n, c_in, h, w, c_out, r, s, stride, pad, out_pad, dil, dtype)
CASES = [
    ("ct_dcgan_like", True, 3, 64, 8, 8, 40, 4, 4, 2, 1, 0, 1, "bf16"),
    ("ct_op_dil_f32", True, 2, 12, 5, 6, 20, 3, 3, 2, 1, 1, 2, "f32"),
    ("ct_ragged", True, 5, 70, 4, 4, 130, 4, 4, 2, 1, 0, 1, "bf16"),
    ("ct_table1_5x5", True, 2, 32, 4, 4, 24, 5, 5, 2, 2, 1, 1, "bf16"),
    ("ct_stride1", True, 1, 16, 7, 9, 8, 3, 3, 1, 1, 0, 1, "f32"),
    ("conv_discriminator", False, 3, 24, 16, 16, 48, 4, 4, 2, 1, 0, 1, "bf16"),
    ("conv_dilated_f32", False, 2, 16, 12, 12, 20, 3, 3, 1, 2, 0, 2, "f32"),
    ("conv_1x1", False, 2, 33, 5, 7, 17, 1, 1, 1, 0, 0, 1, "bf16"),
    ("conv_aspp_like", False, 1, 64, 24, 24, 32, 3, 3, 1, 6, 0, 6, "bf16"),
    # 128 x 128 GEMM tiles (both channel counts >= 128), ragged in both
    ("ct_tile128_ragged", True, 2, 130, 4, 4, 200, 4, 4, 2, 1, 0, 1, "bf16"),
    ("conv_tile128_f32", False, 2, 136, 8, 8, 144, 3, 3, 2, 1, 0, 1, "f32"),
    # small grids with rows of 2 and 1 pixels (staging pieces of whole rows)
    ("ct_rows2", True, 2, 16, 4, 2, 24, 4, 4, 2, 1, 0, 1, "f32"),
    ("ct_rows1", True, 1, 8, 8, 1, 8, 3, 3, 2, 1, 1, 1, "bf16"),
    # 128 x 128 tiles on wider grids: ragged channels, dilation with output
    # padding, and strided convs (small grid = their output)
    ("ct_wide_ragged", True, 3, 136, 8, 16, 130, 4, 4, 2, 1, 0, 1, "bf16"),
    ("ct_wide_dil_op", True, 2, 128, 8, 8, 128, 3, 3, 2, 2, 1, 2, "bf16"),
    ("conv_wide", False, 2, 144, 16, 16, 136, 4, 4, 2, 1, 0, 1, "bf16"),
    ("conv_wide_pad0", False, 1, 128, 18, 34, 128, 3, 3, 2, 0, 0, 1, "bf16"),
    # fp32 on the phase planes (8x8 small grid, planes of 10 rows) with the
    # GEMM writing dw itself
    ("ct_f32_phase", True, 2, 32, 8, 8, 24, 4, 4, 2, 1, 0, 1, "f32"),
]


def _w_shape(c):
    _, tr, n, ci, h, w, co, r, s = c[:9]
    return (ci, co, r, s) if tr else (co, ci, r, s)


def _inputs(c, seed):
    name, tr, n, ci, h, w, co, r, s, st, pd, op, dl, dt = c
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(n, ci, h, w, generator=g)
    if tr:
        ho = (h - 1) * st - 2 * pd + dl * (r - 1) + op + 1
        wo = (w - 1) * st - 2 * pd + dl * (s - 1) + op + 1
    else:
        ho = (h + 2 * pd - dl * (r - 1) - 1) // st + 1
        wo = (w + 2 * pd - dl * (s - 1) - 1) // st + 1
    dy = torch.randn(n, co, ho, wo, generator=g)
    dtype = wl.torch_dtype(dt)
    return x.to(dtype), dy.to(dtype)


def _oracle(c, xq, dyq, absolute=False):
    name, tr, n, ci, h, w, co, r, s, st, pd, op, dl, dt = c
    x, dy = xq.double().numpy(), dyq.double().numpy()
    if absolute:
        x, dy = np.abs(x), np.abs(dy)
    if tr:
        return oracle.conv2d_transpose_wgrad(x, dy, _w_shape(c), st, pd, op, dl)
    return oracle.conv2d_dilated_wgrad(x, dy, _w_shape(c), st, pd, dl)


def _gpu(c, xq, dyq):
    name, tr, n, ci, h, w, co, r, s, st, pd, op, dl, dt = c
    dev = torch.device("cuda", 0)
    x, dy = xq.to(dev), dyq.to(dev)
    if tr:
        dw = h2.conv2d_transpose_wgrad(x, dy, _w_shape(c), st, pd, op, dl)
    else:
        dw = h2.conv2d_dilated_wgrad(x, dy, _w_shape(c), st, pd, dl)
    torch.cuda.synchronize()
    return dw.cpu().double().numpy()


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0])
def test_weight_gradient(case):
    P.say("case", case)
    xq, dyq = _inputs(case, seed=5)
    ref, absref = _oracle(case, xq, dyq), _oracle(case, xq, dyq, absolute=True)
    got = _gpu(case, xq, dyq)
    P.check(got, ref, absref, case[-1], case[0])


@pytest.mark.parametrize("case", [CASES[0], CASES[5], CASES[9]], ids=lambda c: c[0])
def test_weight_gradient_chunks(case, monkeypatch):
    """Images split into chunks (one per image here): the fp32 gradient is
    accumulated over the chunks in order; same bar, and deterministic."""
    monkeypatch.setenv("HUGE2_WGRAD_CHUNK", "1")
    P.say("case", case, "one image per chunk")
    xq, dyq = _inputs(case, seed=6)
    ref, absref = _oracle(case, xq, dyq), _oracle(case, xq, dyq, absolute=True)
    got = _gpu(case, xq, dyq)
    P.check(got, ref, absref, case[-1], case[0])
    again = _gpu(case, xq, dyq)
    assert np.array_equal(got, again)


@pytest.mark.parametrize("case", [CASES[0], CASES[5], CASES[9], CASES[12]], ids=lambda c: c[0])
def test_weight_gradient_gather_forms(case, monkeypatch):
    """The per-tap copies of the large tensor built through LDS (whole planes
    per workgroup) and by the plain staging kernel (HUGE2_WGRAD_GATHER=0):
    both match the oracle, and bitwise each other (the same copies)."""
    P.say("case", case, "LDS gather and plain staging")
    xq, dyq = _inputs(case, seed=12)
    ref, absref = _oracle(case, xq, dyq), _oracle(case, xq, dyq, absolute=True)
    got = _gpu(case, xq, dyq)
    P.check(got, ref, absref, case[-1], case[0])
    monkeypatch.setenv("HUGE2_WGRAD_GATHER", "0")
    plain = _gpu(case, xq, dyq)
    assert np.array_equal(got, plain)


@pytest.mark.parametrize("case", [CASES[0], CASES[5], CASES[8], CASES[13], CASES[1]],
                         ids=lambda c: c[0])
def test_weight_gradient_in_place_and_direct_out_forms(case, monkeypatch):
    """The small tensor read in place (channel planes of a multiple of 64
    pixels) or staged first (HUGE2_WGRAD_DIRECT=0), and, with one K slice,
    the GEMM writing the gradient itself or through the fp32 slices and the
    store (HUGE2_WGRAD_DIRECT_OUT=0): every form matches the oracle, and all
    give the same values (same products, same order, one rounding)."""
    P.say("case", case, "in-place / direct-out forms")
    xq, dyq = _inputs(case, seed=13)
    ref, absref = _oracle(case, xq, dyq), _oracle(case, xq, dyq, absolute=True)
    outs = []
    for direct in ("1", "0"):
        for direct_out in ("1", "0"):
            monkeypatch.setenv("HUGE2_WGRAD_DIRECT", direct)
            monkeypatch.setenv("HUGE2_WGRAD_DIRECT_OUT", direct_out)
            got = _gpu(case, xq, dyq)
            P.check(got, ref, absref, case[-1],
                    "%s direct=%s direct_out=%s" % (case[0], direct, direct_out))
            outs.append(got)
    for o in outs[1:]:
        assert np.array_equal(outs[0], o)


@pytest.mark.parametrize("case", [CASES[0], CASES[5], CASES[8], CASES[13], CASES[14], CASES[15],
                                  CASES[17]], ids=lambda c: c[0])
def test_weight_gradient_phase_planes(case, monkeypatch):
    """The large tensor's copies as phase planes with halo rows (the taps
    that differ only in their row shift read one plane at different row
    offsets) or one copy per tap (HUGE2_WGRAD_PHASE=0): both match the
    oracle and give the same bits (the same values in the same K order)."""
    P.say("case", case, "phase planes / per-tap copies")
    xq, dyq = _inputs(case, seed=15)
    ref, absref = _oracle(case, xq, dyq), _oracle(case, xq, dyq, absolute=True)
    got = _gpu(case, xq, dyq)
    P.check(got, ref, absref, case[-1], case[0] + " phase planes")
    monkeypatch.setenv("HUGE2_WGRAD_PHASE", "0")
    per_tap = _gpu(case, xq, dyq)
    P.check(per_tap, ref, absref, case[-1], case[0] + " per-tap copies")
    assert np.array_equal(got, per_tap)


def test_weight_gradient_plan_reuse():
    """One plan, two calls on different data: each matches the oracle."""
    case = CASES[2]
    name, tr, n, ci, h, w, co, r, s, st, pd, op, dl, dt = case
    desc = h2.make_desc(n, ci, h, w, co, r, s, st, pd, op, dl, h2.HUGE2_NCHW, h2.HUGE2_BF16)
    plan = h2.huge2_wgrad_plan_create(desc, 1)
    dev = torch.device("cuda", 0)
    try:
        for seed in (7, 8):
            xq, dyq = _inputs(case, seed)
            x, dy = xq.to(dev), dyq.to(dev)
            dw = torch.empty(_w_shape(case), dtype=x.dtype, device=dev)
            h2.huge2_wgrad_execute(plan, x.data_ptr(), dy.data_ptr(), dw.data_ptr(),
                                   torch.cuda.current_stream().cuda_stream)
            torch.cuda.synchronize()
            P.check(dw.cpu().double().numpy(), _oracle(case, xq, dyq),
                    _oracle(case, xq, dyq, absolute=True), dt, name)
    finally:
        h2.huge2_wgrad_plan_destroy(plan)


def test_dcgan_layer_weight_gradient_full_size():
    """The generator's second layer (512 -> 256, 8x8 -> 16x16, batch 64) in
    full, checked element by element against the oracle."""
    case = ("dcgan_l2_wgrad", True, 64, 512, 8, 8, 256, 4, 4, 2, 1, 0, 1, "bf16")
    P.say("case", case)
    xq, dyq = _inputs(case, seed=9)
    got = _gpu(case, xq, dyq)
    P.check(got, _oracle(case, xq, dyq), _oracle(case, xq, dyq, absolute=True), "bf16", case[0])


def test_dcgan_last_layer_weight_gradient_full_size():
    """The generator's last layer (128 -> 3, 32x32 -> 64x64, batch 64) in
    full: three big-tensor channels (48 GEMM columns with the taps), the
    small tensor read in place, and more than a hundred K slices added by
    the split store."""
    case = ("dcgan_l4_wgrad", True, 64, 128, 32, 32, 3, 4, 4, 2, 1, 0, 1, "bf16")
    P.say("case", case)
    xq, dyq = _inputs(case, seed=14)
    got = _gpu(case, xq, dyq)
    P.check(got, _oracle(case, xq, dyq), _oracle(case, xq, dyq, absolute=True), "bf16", case[0])


def test_data_gradients_are_the_exchanged_forward_forms():
    """dx of the transposed conv = strided conv of dy with the same w; dx of
    the strided conv = transposed conv of dy; both against the oracle."""
    dev = torch.device("cuda", 0)
    g = torch.Generator().manual_seed(10)
    # transposed conv 64 -> 32, k4 s2 p1, 6x6 -> 12x12
    w = (torch.randn(64, 32, 4, 4, generator=g) * 0.1).to(torch.bfloat16)
    dy = torch.randn(2, 32, 12, 12, generator=g).to(torch.bfloat16)
    dx = h2.conv2d_transpose_dgrad(dy.to(dev), w.to(dev), 2, 1, 1).cpu().double().numpy()
    assert dx.shape == (2, 64, 6, 6)
    ref = oracle.conv2d_dilated_alg2(dy.double().numpy(), w.double().numpy(), None, 2, 1, 1)
    absref = oracle.conv2d_dilated_alg2(np.abs(dy.double().numpy()), np.abs(w.double().numpy()),
                                        None, 2, 1, 1)
    P.check(dx, ref, absref, "bf16", "transpose dgrad")
    # strided conv 16 -> 24, k3 s2 p1, 11x11 -> 6x6: dx back to 11x11
    w2 = (torch.randn(24, 16, 3, 3, generator=g) * 0.1).to(torch.bfloat16)
    dy2 = torch.randn(2, 24, 6, 6, generator=g).to(torch.bfloat16)
    dx2 = h2.conv2d_dilated_dgrad(dy2.to(dev), w2.to(dev), (11, 11), 2, 1, 1).cpu().double().numpy()
    assert dx2.shape == (2, 16, 11, 11)
    ref2 = oracle.conv2d_transpose_alg1(dy2.double().numpy(), w2.double().numpy(), None, 2, 1, 0, 1)
    absref2 = oracle.conv2d_transpose_alg1(np.abs(dy2.double().numpy()), np.abs(w2.double().numpy()),
                                           None, 2, 1, 0, 1)
    P.check(dx2, ref2, absref2, "bf16", "dilated dgrad")
    # and the adjoint relation the data gradient must satisfy, in float64
    x2 = np.random.default_rng(3).standard_normal((2, 16, 11, 11))
    y2 = oracle.conv2d_dilated_alg2(x2, w2.double().numpy(), None, 2, 1, 1)
    assert abs(np.sum(y2 * dy2.double().numpy()) - np.sum(x2 * ref2)) < 1e-9 * np.sum(np.abs(y2 * dy2.double().numpy()))


# grouped and depthwise layers: (name, transposed, n, c_in, h, w, c_out, r, s,
# stride, pad, out_pad, dil, dtype, groups)
GROUPED_CASES = [
    # depthwise transposed upsampling (the generator-side depthwise layer)
    ("ct_depthwise", True, 3, 32, 8, 8, 32, 4, 4, 2, 1, 0, 1, "bf16", 32),
    # channel multiplier 2, output padding and dilation, fp32
    ("ct_dw_mult2_f32", True, 2, 6, 5, 7, 12, 3, 3, 2, 1, 1, 2, "f32", 6),
    # four groups of 8 -> 6 channels, a 5x5 kernel (two runs of 16 taps)
    ("ct_groups4_k5", True, 2, 32, 6, 5, 24, 5, 5, 2, 2, 1, 1, "bf16", 4),
    # the discriminator's depthwise strided conv (section 3.2.3's C = 1 case)
    ("conv_depthwise", False, 4, 24, 16, 16, 24, 4, 4, 2, 1, 0, 1, "bf16", 24),
    # dilated grouped conv, 3 groups of 4 -> 5 channels
    ("conv_groups3_dil", False, 2, 12, 13, 11, 15, 3, 3, 1, 2, 0, 2, "f32", 3),
    # many pixels per plane (more than one pass of the workgroup's threads)
    ("conv_dw_large", False, 2, 8, 40, 36, 8, 3, 3, 1, 1, 0, 1, "bf16", 8),
]


def _g_w_shape(c):
    _, tr, n, ci, h, w, co, r, s = c[:9]
    g = c[14]
    return (ci, co // g, r, s) if tr else (co, ci // g, r, s)


def _g_oracle(c, xq, dyq, absolute=False):
    name, tr, n, ci, h, w, co, r, s, st, pd, op, dl, dt, g = c
    x, dy = xq.double().numpy(), dyq.double().numpy()
    if absolute:
        x, dy = np.abs(x), np.abs(dy)
    if tr:
        return oracle.conv2d_transpose_wgrad(x, dy, _g_w_shape(c), st, pd, op, dl, groups=g)
    return oracle.conv2d_dilated_wgrad(x, dy, _g_w_shape(c), st, pd, dl, groups=g)


@pytest.mark.parametrize("case", GROUPED_CASES, ids=lambda c: c[0])
def test_grouped_weight_gradient(case):
    """Grouped and depthwise weight gradients (each weight plane joins one
    input map to one error map) against the grouped oracle, element by
    element, deterministic across calls, through the plan entry points too."""
    P.say("case", case)
    name, tr, n, ci, h, w, co, r, s, st, pd, op, dl, dt, g = case
    xq, dyq = _inputs(case[:14], seed=11)
    ref, absref = _g_oracle(case, xq, dyq), _g_oracle(case, xq, dyq, absolute=True)
    dev = torch.device("cuda", 0)
    x, dy = xq.to(dev), dyq.to(dev)
    if tr:
        got = h2.conv2d_transpose_wgrad(x, dy, _g_w_shape(case), st, pd, op, dl, groups=g)
    else:
        got = h2.conv2d_dilated_wgrad(x, dy, _g_w_shape(case), st, pd, dl, groups=g)
    torch.cuda.synchronize()
    got = got.cpu().double().numpy()
    P.check(got, ref, absref, dt, name)
    desc = h2.make_desc(n, ci, h, w, co, r, s, st, pd, op, dl, h2.HUGE2_NCHW,
                        h2.HUGE2_BF16 if dt == "bf16" else h2.HUGE2_F32, groups=g)
    plan = h2.huge2_wgrad_plan_create(desc, int(tr))
    try:
        dw = torch.full(_g_w_shape(case), float("nan"), dtype=x.dtype, device=dev)
        h2.huge2_wgrad_execute(plan, x.data_ptr(), dy.data_ptr(), dw.data_ptr(),
                               torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        assert np.array_equal(dw.cpu().double().numpy(), got)
    finally:
        h2.huge2_wgrad_plan_destroy(plan)
