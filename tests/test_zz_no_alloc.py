"""The no-allocation transposed conv (huge2_conv2d_transpose_noalloc, its
buffers in the library's static per-GPU scratch array) against the one-shot
entry point it varies (huge2_conv2d_transpose), through the C ABI: two calls
in a row, the second with a smaller input, each compared with the oracle and
with the allocating entry point on the same inputs."""
import ctypes

import numpy as np
import pytest
import torch

from paper_1907_11210_amd import huge2 as h2
from paper_1907_11210_amd import workloads as wl
from paper_1907_11210_amd.workloads import Layer

import parity as P

pytestmark = pytest.mark.gpu

# two calls in a row, the second smaller; the first stages its NCHW input and
# splits K across workgroups (few output tiles), so the scratch array holds
# packed weights, work list, staging buffer and K-slice partials; the second
# reuses the array with a different plan on top of the first one's contents
PAIRS = [
    (Layer("na_big", True, 2, 256, 6, 6, 96, 3, 3, 2, 1, 1, 1, "NCHW", "bf16", "relu"),
     Layer("na_small", True, 1, 40, 5, 7, 24, 3, 3, 2, 1, 1, 1, "NHWC", "bf16")),
    # the second call of this pair takes the fp32 two-pass form (an inner
    # pointwise GEMM plan and its per-tap buffer in the array too)
    (Layer("na_f32_big", True, 1, 64, 9, 9, 48, 4, 4, 2, 1, 0, 1, "NCHW", "f32"),
     Layer("na_f32_small", True, 1, 16, 4, 4, 3, 4, 4, 2, 1, 0, 1, "NCHW", "f32", "tanh")),
]


def _desc(layer):
    return h2.make_desc(layer.n, layer.c_in, layer.h, layer.w, layer.c_out, layer.r, layer.s,
                        layer.stride, layer.pad, layer.out_pad, layer.dil,
                        h2.HUGE2_NCHW if layer.layout == "NCHW" else h2.HUGE2_NHWC,
                        h2.HUGE2_BF16 if layer.dtype == "bf16" else h2.HUGE2_F32,
                        h2.ACTIVATIONS[layer.act])


def _run(layer, xq, wq, bias, entry):
    dev = torch.device("cuda", 0)
    x = wl.to_layout(xq, layer.layout).to(dev)
    w = wq.contiguous().to(dev)
    b = bias.to(torch.float32).to(dev)
    desc = _desc(layer)
    ho, wo = h2.huge2_output_shape(desc, 1)
    shape = (layer.n, layer.c_out, ho, wo) if layer.layout == "NCHW" else (layer.n, ho, wo, layer.c_out)
    y = torch.full(shape, float("nan"), dtype=xq.dtype, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    entry(desc, x.data_ptr(), w.data_ptr(), b.data_ptr(), y.data_ptr(), stream)
    torch.cuda.synchronize()
    return wl.from_layout(y.cpu(), layer.layout).double().numpy()


@pytest.mark.parametrize("pair", PAIRS, ids=[p[0].name for p in PAIRS])
def test_noalloc_matches_one_shot(pair):
    for i, layer in enumerate(pair):
        P.say("case no-alloc", layer)
        xq = P.quantise(wl.layer_input(layer, seed=61 + i), layer.dtype)
        wq = P.quantise(wl.random_weight(layer, seed=71 + i, std=0.05), layer.dtype)
        bias = torch.linspace(-0.5, 0.5, layer.c_out)
        y_na = _run(layer, xq, wq, bias, h2.huge2_conv2d_transpose_noalloc)
        y_os = _run(layer, xq, wq, bias, h2.huge2_conv2d_transpose)
        ref = P.oracle_full(layer, xq, wq, bias)
        absref = P.oracle_full(layer, xq, wq, bias, absolute=True)
        P.check(y_na, ref, absref, layer.dtype, layer.name + " no-alloc")
        # the same plan and kernels over a different memory region: equal bits
        assert np.array_equal(y_na, y_os), layer.name


def test_noalloc_rejects_too_large():
    """A layer whose packed weights alone exceed the 64 MiB region is refused
    before anything is written."""
    layer = Layer("na_huge", True, 1, 4096, 2, 2, 2048, 4, 4, 2, 1, 0, 1, "NHWC", "bf16")
    dev = torch.device("cuda", 0)
    desc = _desc(layer)
    x = torch.zeros(1, 2, 2, 4096, dtype=torch.bfloat16, device=dev)
    w = torch.zeros(4096, 2048, 4, 4, dtype=torch.bfloat16, device=dev)  # 256 MiB packed
    y = torch.full((1, 4, 4, 2048), 7.0, dtype=torch.bfloat16, device=dev)
    with pytest.raises(h2.Huge2Error) as e:
        h2.huge2_conv2d_transpose_noalloc(desc, x.data_ptr(), w.data_ptr(), 0, y.data_ptr(),
                                          torch.cuda.current_stream(dev).cuda_stream)
    assert e.value.status == h2.HUGE2_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())
