"""Seeded synthetic inputs for the five benchmark workloads (CPU tensors).

Input generation only -- no convolution arithmetic lives here.  Both the GPU
path and the CPU oracle are fed from these generators, so they see the same
bytes.  All draws use ``torch.Generator('cpu').manual_seed(seed)`` in a fixed
order; bf16 tensors are the float32 draws rounded to nearest even
(``.to(torch.bfloat16)``).

The paper evaluates DCGAN / cGAN generators pretrained on CIFAR100 (section 4);
neither the weights nor the dataset are available, so random-init weights and
random activations of the same shapes stand in, following the distributions
named per workload below.

Workloads (``name``: layers):
  convt_small  single ConvTranspose 64->32, 8x8 -> 16x16, k4 s2 p1, fp32 NCHW, batch 1.
  dcgan        z(100) -> linear -> 4x4x1024, then ConvTranspose k4 s2 p1:
               1024->512 (8x8), 512->256 (16x16), 256->128 (32x32), 128->3 (64x64);
               batch 64, NCHW, fp32 and bf16.
  convt_odd    ConvTranspose 256->128, 32x32 -> 64x64, k3 s2 p1 op1, bf16 NHWC, batch 16.
  aspp         four 3x3 dilated convs 2048->256 on 64x64, dilations 6/12/18/24, 'same'
               padding, bf16 NHWC, batch 8, input ReLU(N(0,1)).
  fcn_upsample ConvTranspose 21->21, 16x16 -> 512x512, k64 s32 p16, bilinear kernel plus
               N(0, 1e-3) noise, bf16 NCHW, batch 4.
  table1_dcgan the DCGAN deconvolution layers of the paper's Table 1: 5x5 kernels, stride
               2, 4x4x1024 -> 8x8x512 -> 16x16x256 -> 32x32x128 -> 64x64x3, batch 1
               (inference), bf16 NCHW.  The table gives no padding; the output doubles
               the input, which symmetric padding reaches with pad 2 and output
               padding 1 (the same taps per phase as TensorFlow's 'SAME' deconvolution,
               with the phase roles mirrored).  Input N(0,1), weights N(0,0.02), chained.
  table1_cgan  the cGAN layers of Table 1: 4x4 kernels, stride 2, pad 1,
               8x8x256 -> 16x16x128 -> 32x32x3, batch 1, bf16 NCHW, chained.
  dcgan_generator
               the whole DCGAN generator on the library, bf16 NCHW, batch 64: the projection
               of z (100-d, N(0,1)) to 4x4x1024 as a ConvTranspose k4 s1 p0 of the 1x1 input,
               then the four dcgan layers; ReLU after every layer but the last, tanh after
               the last, fused into the epilogues (batch normalisation, which a trained
               generator folds into weights and bias, is left out: no bias).  Weights
               N(0,0.02), chained.
  dcgan_generator_b1
               the same generator at batch 1 (one image: the latency case).
  dcgan_generator_nhwc, dcgan_generator_nhwc_b1
               the same generator with every activation in NHWC (channel-contiguous
               pixels from z to the image), batch 64 and batch 1; the same draws.
  dcgan_dgrad  training (section 3.2.3): the data gradients of the dcgan generator's
               four ConvTranspose layers, back to front.  The gradient of a stride-2
               transposed conv with respect to its input is the stride-2 conv of the
               output error with the same weight array, read as [C_out_conv = C_in,
               C_in_conv = C_out, 4, 4]: 3->128 (64x64 -> 32x32), 128->256 (32 -> 16),
               256->512 (16 -> 8), 512->1024 (8 -> 4), batch 64, bf16 NCHW.  The
               generator has no activations between its layers, so each layer's input
               gradient is the previous one's output error (chained).  The first error
               is N(0,1); the weights are the dcgan draws.
"""
from __future__ import annotations

import dataclasses

import torch


@dataclasses.dataclass(frozen=True)
class Layer:
    name: str
    transposed: bool
    n: int
    c_in: int
    h: int
    w: int
    c_out: int
    r: int
    s: int
    stride: int
    pad: int
    out_pad: int
    dil: int
    layout: str  # "NCHW" or "NHWC"
    dtype: str   # "f32" or "bf16"
    act: str = "none"  # epilogue function after the bias: "none", "relu" or "tanh"
    groups: int = 1    # grouped convolution (groups = c_in: depthwise)

    def out_hw(self):
        if self.transposed:
            ho = (self.h - 1) * self.stride - 2 * self.pad + self.dil * (self.r - 1) + self.out_pad + 1
            wo = (self.w - 1) * self.stride - 2 * self.pad + self.dil * (self.s - 1) + self.out_pad + 1
        else:
            ho = (self.h + 2 * self.pad - self.dil * (self.r - 1) - 1) // self.stride + 1
            wo = (self.w + 2 * self.pad - self.dil * (self.s - 1) - 1) // self.stride + 1
        return ho, wo

    def w_shape(self):
        return ((self.c_in, self.c_out // self.groups, self.r, self.s) if self.transposed
                else (self.c_out, self.c_in // self.groups, self.r, self.s))

    def with_(self, **kw):
        return dataclasses.replace(self, **kw)


def dcgan_layers(dtype="bf16", batch=64):
    chans = [(1024, 512), (512, 256), (256, 128), (128, 3)]
    out = []
    for i, (ci, co) in enumerate(chans):
        hw = 4 << i
        out.append(Layer("dcgan_l%d" % (i + 1), True, batch, ci, hw, hw, co, 4, 4, 2, 1, 0, 1,
                         "NCHW", dtype))
    return out


def dcgan_dgrad_layers(dtype="bf16", batch=64):
    fwd = dcgan_layers(dtype, batch)
    return [Layer("dcgan_dgrad_l%d" % (4 - i), False, batch, l.c_out, 2 * l.h, 2 * l.w, l.c_in,
                  l.r, l.s, l.stride, l.pad, 0, l.dil, l.layout, dtype)
            for i, l in enumerate(reversed(fwd))]


def generator_layers(dtype="bf16", batch=64, layout="NCHW"):
    proj = Layer("gen_proj", True, batch, 100, 1, 1, 1024, 4, 4, 1, 0, 0, 1, layout, dtype, "relu")
    body = [l.with_(name=l.name.replace("dcgan", "gen"), act="relu" if i < 3 else "tanh",
                    layout=layout)
            for i, l in enumerate(dcgan_layers(dtype, batch))]
    return [proj] + body


def table1_layers(kind, batch=1, dtype="bf16"):
    if kind == "dcgan":
        chans, k, pad, op, hw0 = [(1024, 512), (512, 256), (256, 128), (128, 3)], 5, 2, 1, 4
    else:
        chans, k, pad, op, hw0 = [(256, 128), (128, 3)], 4, 1, 0, 8
    return [Layer("t1_%s_dc%d" % (kind, i + 1), True, batch, ci, hw0 << i, hw0 << i, co, k, k, 2,
                  pad, op, 1, "NCHW", dtype) for i, (ci, co) in enumerate(chans)]


def aspp_layers(batch=8, c_in=2048, c_out=256, hw=64):
    return [Layer("aspp_d%d" % d, False, batch, c_in, hw, hw, c_out, 3, 3, 1, d, 0, d, "NHWC",
                  "bf16") for d in (6, 12, 18, 24)]


WORKLOADS = {
    "convt_small": [Layer("convt_small", True, 1, 64, 8, 8, 32, 4, 4, 2, 1, 0, 1, "NCHW", "f32")],
    "dcgan": dcgan_layers("bf16"),
    "dcgan_f32": dcgan_layers("f32"),
    "convt_odd": [Layer("convt_odd", True, 16, 256, 32, 32, 128, 3, 3, 2, 1, 1, 1, "NHWC", "bf16")],
    "aspp": aspp_layers(),
    "fcn_upsample": [Layer("fcn_upsample", True, 4, 21, 16, 16, 21, 64, 64, 32, 16, 0, 1, "NCHW",
                           "bf16")],
    "table1_dcgan": table1_layers("dcgan"),
    "table1_cgan": table1_layers("cgan"),
    "dcgan_dgrad": dcgan_dgrad_layers("bf16"),
    "dcgan_generator": generator_layers("bf16"),
    "dcgan_generator_b1": generator_layers("bf16", batch=1),
    "dcgan_generator_nhwc": generator_layers("bf16", layout="NHWC"),
    "dcgan_generator_nhwc_b1": generator_layers("bf16", batch=1, layout="NHWC"),
}
GENERATORS = ("dcgan_generator", "dcgan_generator_b1", "dcgan_generator_nhwc",
              "dcgan_generator_nhwc_b1")
# layers that read one input and run as one grouped launch (huge2_group)
GROUPED = ("aspp",)
CHAINED = ("dcgan", "dcgan_f32", "table1_dcgan", "table1_cgan", "dcgan_dgrad") + GENERATORS


def torch_dtype(name):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def bilinear_kernel(size):
    """FCN-style bilinear upsampling taps: f[m] = (2*min(m, size-1-m) + 1) / size."""
    m = torch.arange(size, dtype=torch.float64)
    f = (2 * torch.minimum(m, size - 1 - m) + 1) / size
    return f


def _normal(g, shape, std=1.0):
    return torch.randn(shape, generator=g, dtype=torch.float32) * std


def generate(workload, seed=0, batch=None):
    """Inputs of a workload: list of (Layer, x NCHW float32, w float32).

    ``batch`` overrides the batch size (the draws are then made at that size).
    For ``dcgan`` only the first layer has a drawn input (the linear layer of
    the generator); the others are chained on the device by the benchmark.
    Use :func:`layer_input` for a standalone input of any layer.
    """
    g = torch.Generator("cpu").manual_seed(seed)
    layers = WORKLOADS[workload]
    if batch is not None:
        layers = [l.with_(n=batch) for l in layers]
    if workload in ("dcgan", "dcgan_f32"):
        n = layers[0].n
        z = _normal(g, (n, 100))
        lin_w = _normal(g, (1024 * 4 * 4, 100), 0.02)
        x1 = (z @ lin_w.t()).reshape(n, 1024, 4, 4)  # linear layer, bias 0
        ws = [_normal(g, l.w_shape(), 0.02) for l in layers]
        out = [(layers[0], x1, ws[0])]
        out += [(l, None, w) for l, w in zip(layers[1:], ws[1:])]
        return out
    if workload in GENERATORS:
        l0 = layers[0]
        z = _normal(g, (l0.n, 100, 1, 1))
        ws = [_normal(g, l.w_shape(), 0.02) for l in layers]
        return [(layers[0], z, ws[0])] + [(l, None, w) for l, w in zip(layers[1:], ws[1:])]
    if workload == "dcgan_dgrad":
        # the dcgan draws (z, linear weight, w1..w4), then the output error
        n = layers[0].n
        _normal(g, (n, 100))
        _normal(g, (1024 * 4 * 4, 100), 0.02)
        ws = [_normal(g, l.w_shape(), 0.02) for l in dcgan_layers("bf16", n)]
        l0 = layers[0]
        dy = _normal(g, (n, l0.c_in, l0.h, l0.w))
        ws = ws[::-1]  # back to front; [C_in_T, C_out_T, 4, 4] = [C_out_conv, C_in_conv, 4, 4]
        return [(layers[0], dy, ws[0])] + [(l, None, w) for l, w in zip(layers[1:], ws[1:])]
    if workload in ("table1_dcgan", "table1_cgan"):
        l0 = layers[0]
        x1 = _normal(g, (l0.n, l0.c_in, l0.h, l0.w))
        ws = [_normal(g, l.w_shape(), 0.02) for l in layers]
        return [(layers[0], x1, ws[0])] + [(l, None, w) for l, w in zip(layers[1:], ws[1:])]
    if workload == "aspp":
        l0 = layers[0]
        x = torch.relu(_normal(g, (l0.n, l0.c_in, l0.h, l0.w)))
        return [(l, x, _normal(g, l.w_shape(), 0.01)) for l in layers]
    l0 = layers[0]
    if workload == "convt_small":
        x = _normal(g, (l0.n, l0.c_in, l0.h, l0.w))
        return [(l0, x, _normal(g, l0.w_shape(), 0.02))]
    if workload == "convt_odd":
        x = torch.rand((l0.n, l0.c_in, l0.h, l0.w), generator=g, dtype=torch.float32) * 2 - 1
        return [(l0, x, _normal(g, l0.w_shape(), 0.02))]
    if workload == "fcn_upsample":
        x = _normal(g, (l0.n, l0.c_in, l0.h, l0.w))
        f = bilinear_kernel(l0.r).to(torch.float32)
        w = _normal(g, l0.w_shape(), 1e-3)
        for c in range(l0.c_in):
            w[c, c] += torch.outer(f, f)
        return [(l0, x, w)]
    raise KeyError(workload)


def layer_input(layer, seed=0, std=1.0):
    """A standalone N(0, std^2) NCHW float32 input for one layer."""
    g = torch.Generator("cpu").manual_seed(seed)
    return _normal(g, (layer.n, layer.c_in, layer.h, layer.w), std)


def random_weight(layer, seed=0, std=0.02):
    g = torch.Generator("cpu").manual_seed(seed)
    return _normal(g, layer.w_shape(), std)


def to_layout(x_nchw, layout):
    """NCHW tensor -> contiguous tensor in ``layout`` (a permutation, no arithmetic)."""
    if layout == "NCHW":
        return x_nchw.contiguous()
    return x_nchw.permute(0, 2, 3, 1).contiguous()


def from_layout(x, layout):
    """Tensor in ``layout`` -> NCHW view."""
    if layout == "NCHW":
        return x
    return x.permute(0, 3, 1, 2)
