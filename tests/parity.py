"""Helpers for the GPU parity tests: run a layer through the C ABI and compare
it with the CPU oracle on the same (dtype-rounded) bytes.

Pass criterion (the tolerance of the method's stated parity bar, read as a
norm-wise relative error per output tensor):
    max|y - y*| / max|y*|  <=  1e-4 (fp32)  or  2e-2 (bf16 in, fp32 accumulate)
and, element by element, the error bound of a dot product:
    |y - y*| <= tol * (|x| conv |w|)
where |x| conv |w| is the oracle applied to the absolute values.
"""
import sys

import numpy as np
import torch

import oracle
from paper_1907_11210_amd import huge2 as h2
from paper_1907_11210_amd import workloads as wl

TOL = {"f32": 1e-4, "bf16": 2e-2}


def tile_count():
    """Number of GEMM tile configurations (entries of kTiles in kernels.hpp)."""
    import os
    import re
    src = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                       "paper_1907_11210_amd", "csrc", "kernels.hpp")
    text = open(src).read()
    body = text[text.index("kTiles[] = {"):]
    body = body[:body.index("};")]
    return len(re.findall(r"\{\s*\d+\s*,", body))


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def quantise(t, dtype):
    return t.to(wl.torch_dtype(dtype))


def oracle_full(layer, xq, wq, bias=None, absolute=False):
    x = xq.double().numpy()
    w = wq.double().numpy()
    b = None if bias is None else bias.double().numpy()
    if absolute:
        x, w, b = np.abs(x), np.abs(w), None if b is None else np.abs(b)
    if layer.transposed:
        y = oracle.conv2d_transpose_alg1(x, w, b, layer.stride, layer.pad, layer.out_pad,
                                         layer.dil, groups=layer.groups)
    else:
        y = oracle.conv2d_dilated_alg2(x, w, b, layer.stride, layer.pad, layer.dil,
                                       groups=layer.groups)
    # |act(u) - act(v)| <= |u - v| for both functions: the bound of the
    # absolute-value run still holds after the activation
    return y if absolute else oracle.activate(y, layer.act)


def oracle_points(layer, xq, wq, idx, bias=None, absolute=False):
    x = xq.double().numpy()
    w = wq.double().numpy()
    b = None if bias is None else bias.double().numpy()
    if absolute:
        x, w, b = np.abs(x), np.abs(w), None if b is None else np.abs(b)
    if layer.transposed:
        y = oracle.conv2d_transpose_points(x, w, idx, b, layer.stride, layer.pad,
                                           layer.out_pad, layer.dil, groups=layer.groups)
    else:
        y = oracle.conv2d_dilated_points(x, w, idx, b, layer.stride, layer.pad, layer.dil,
                                         groups=layer.groups)
    return y if absolute else oracle.activate(y, layer.act)


def make_plan(layer, w_dev):
    return h2.Plan(w_dev, _x_shape(layer), layer.transposed, layer.stride, layer.pad,
                   layer.out_pad, layer.dil, layer.layout, layer.act, layer.groups)


def _x_shape(layer):
    if layer.layout == "NCHW":
        return (layer.n, layer.c_in, layer.h, layer.w)
    return (layer.n, layer.h, layer.w, layer.c_in)


def run_gpu(layer, xq, wq, bias=None, one_shot=False, plan=None, prefill_nan=False):
    """Run the layer on the GPU; returns the output as a float64 NCHW array.
    prefill_nan: the plan path writes into an output filled with NaN first, so
    that an element the kernels never write stays NaN."""
    dev = torch.device("cuda", 0)
    x_dev = wl.to_layout(xq, layer.layout).to(dev)
    w_dev = wq.contiguous().to(dev)
    b_dev = None if bias is None else bias.to(torch.float32).to(dev)
    if prefill_nan and not one_shot:
        p = plan if plan is not None else make_plan(layer, w_dev)
        y = torch.full(p.out_shape, float("nan"), dtype=xq.dtype, device=dev)
        p(x_dev, b_dev, out=y)
        if plan is None:
            torch.cuda.synchronize()
            p.close()
        torch.cuda.synchronize()
        return wl.from_layout(y.cpu(), layer.layout).double().numpy()
    if one_shot:
        if layer.transposed:
            y = h2.conv2d_transpose(x_dev, w_dev, b_dev, layer.stride, layer.pad, layer.out_pad,
                                    layer.dil, layer.layout, activation=layer.act,
                                    groups=layer.groups)
        else:
            y = h2.conv2d_dilated(x_dev, w_dev, b_dev, layer.stride, layer.pad, layer.dil,
                                  layer.layout, activation=layer.act, groups=layer.groups)
    else:
        p = plan if plan is not None else make_plan(layer, w_dev)
        y = p(x_dev, b_dev)
        if plan is None:
            torch.cuda.synchronize()
            p.close()
    torch.cuda.synchronize()
    return wl.from_layout(y.cpu(), layer.layout).double().numpy()


def check(y, ref, absref, dtype, what=""):
    tol = TOL[dtype]
    scale = float(np.max(np.abs(ref))) if ref.size else 0.0
    err = np.abs(y - ref)
    assert np.all(np.isfinite(y)), "non-finite output " + what
    if ref.size == 0:
        return 0.0
    normwise = float(err.max()) / max(scale, 1e-300)
    assert normwise <= tol, "%s: max|y-y*|/max|y*| = %.3e > %.1e" % (what, normwise, tol)
    bound = tol * absref + 1e-30
    worst = float(np.max(err / bound))
    assert worst <= 1.0, "%s: elementwise error exceeds tol*(|x|*|w|) by %.3f" % (what, worst)
    return normwise


def sample_indices(layer, count, seed):
    """Flat NCHW output indices: uniform picks plus every output phase, the
    borders and the first/last channel, so that every phase and border class
    of the decomposition is hit."""
    ho, wo = layer.out_hw()
    n, co = layer.n, layer.c_out
    rng = np.random.default_rng(seed)
    picks = [rng.integers(0, n * co * ho * wo, size=count)]
    step = layer.stride if layer.transposed else max(layer.dil, 1)
    rows = sorted({0, 1, 2, ho // 2, ho - 3, ho - 2, ho - 1} | set(range(min(step, ho))) |
                  {ho - 1 - i for i in range(min(step, ho))})
    cols = sorted({0, 1, 2, wo // 2, wo - 3, wo - 2, wo - 1} | set(range(min(step, wo))) |
                  {wo - 1 - i for i in range(min(step, wo))})
    rows = [r for r in rows if 0 <= r < ho]
    cols = [c for c in cols if 0 <= c < wo]
    for k in {0, co - 1, co // 2}:
        for img in {0, n - 1}:
            rr = rng.choice(rows, size=min(len(rows), 12), replace=False)
            for r in rr:
                for c in cols[:24]:
                    picks.append(np.array([((img * co + k) * ho + r) * wo + c]))
    return np.unique(np.concatenate(picks)).astype(np.int64)
