"""CPU oracle for HUGE^2's transposed and dilated 2-D convolution (arXiv 1907.11210).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The product library
(``paper_1907_11210_amd``) never imports it and shares no code with it.

The arithmetic lives in ``huge2_oracle.c`` (plain C, float64).  This module only
marshals numpy arrays into it:

* :func:`conv2d_transpose_alg1` -- Algorithm 1 (section 2.1.1) read as the
  zero-insertion emulation the paper describes right after Algorithm 2:
  materialise the zero-inserted input, then a stride-1 convolution with the
  rotated, in/out-swapped kernel, multiplying every inserted zero.
* :func:`conv2d_dilated_alg2` -- Algorithm 2 (section 2.1.1) as a direct gather,
  extended with zero padding and stride.
* ``*_points`` -- the same definitions for selected output elements only.
* ``*_wgrad`` -- the weight gradients of both (section 3.2.3, GAN training),
  written out from the definitions by the chain rule.
* :func:`activate` -- the generator's elementwise functions applied after the
  bias (ReLU between deconvolution layers, tanh after the last one), by their
  definitions, in float64 (numpy).

All arrays are float64 NCHW; transposed weights are ``[C_in, C_out, R, S]`` (the
paper's C x N x R x S of section 4.2), conv weights ``[C_out, C_in, R, S]``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "huge2_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")


def build(force: bool = False) -> str:
    """Compile the oracle with gcc into ``oracle/liboracle.so``."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-pthread", "-Wall", "-Werror",
             "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Conv(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int) for name in (
        "n", "c_in", "h", "w", "c_out", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w",
        "out_pad_h", "out_pad_w", "dil_h", "dil_w", "groups")]


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        dp = ctypes.POINTER(ctypes.c_double)
        cp = ctypes.POINTER(_Conv)
        ip = ctypes.POINTER(ctypes.c_int)
        i64p = ctypes.POINTER(ctypes.c_int64)
        lib.oracle_transpose_out_dims.argtypes = [cp, ip, ip]
        lib.oracle_conv_out_dims.argtypes = [cp, ip, ip]
        for f in (lib.oracle_conv2d_transpose_alg1, lib.oracle_conv2d_dilated_alg2):
            f.argtypes = [cp, dp, dp, dp, dp, ctypes.c_int]
        for f in (lib.oracle_conv2d_transpose_points, lib.oracle_conv2d_dilated_points):
            f.argtypes = [cp, dp, dp, dp, i64p, ctypes.c_int64, dp, ctypes.c_int]
        for f in (lib.oracle_conv2d_transpose_wgrad, lib.oracle_conv2d_dilated_wgrad):
            f.argtypes = [cp, dp, dp, dp, ctypes.c_int]
        _lib = lib
    return _lib


def _pair(v):
    return (int(v), int(v)) if np.isscalar(v) else (int(v[0]), int(v[1]))


def _desc(x_shape, w_shape, transposed, stride, padding, output_padding, dilation, groups=1):
    n, c_in, h, w = x_shape
    g = int(groups)
    if transposed:
        wc_in, cog, r, s = w_shape
        c_out = cog * g
    else:
        c_out, cig, r, s = w_shape
        wc_in = cig * g
    if wc_in != c_in:
        raise ValueError("weight C_in %d does not match input C_in %d" % (wc_in, c_in))
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    oph, opw = _pair(output_padding)
    dh, dw = _pair(dilation)
    return _Conv(n, c_in, h, w, c_out, r, s, sh, sw, ph, pw, oph, opw, dh, dw, g)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _threads(nthreads):
    return int(nthreads) if nthreads else (os.cpu_count() or 1)


def transpose_out_dims(x_shape, w_shape, stride, padding, output_padding=0, dilation=1, groups=1):
    d = _desc(x_shape, w_shape, True, stride, padding, output_padding, dilation, groups)
    ho, wo = ctypes.c_int(), ctypes.c_int()
    if _load().oracle_transpose_out_dims(ctypes.byref(d), ctypes.byref(ho), ctypes.byref(wo)):
        raise ValueError("invalid transposed-conv descriptor")
    return ho.value, wo.value


def conv_out_dims(x_shape, w_shape, stride, padding, dilation=1, groups=1):
    d = _desc(x_shape, w_shape, False, stride, padding, 0, dilation, groups)
    ho, wo = ctypes.c_int(), ctypes.c_int()
    if _load().oracle_conv_out_dims(ctypes.byref(d), ctypes.byref(ho), ctypes.byref(wo)):
        raise ValueError("invalid conv descriptor")
    return ho.value, wo.value


def conv2d_transpose_alg1(x, w, bias=None, stride=1, padding=0, output_padding=0, dilation=1,
                          nthreads=None, groups=1):
    """Transposed conv by zero insertion (Algorithm 1); float64 NCHW in and out.
    groups > 1: w is [C_in, C_out/groups, R, S] and each output channel sums
    over its group's input channels only."""
    x, w, bias = _f64(x), _f64(w), _f64(bias)
    d = _desc(x.shape, w.shape, True, stride, padding, output_padding, dilation, groups)
    ho, wo = transpose_out_dims(x.shape, w.shape, stride, padding, output_padding, dilation, groups)
    y = np.empty((d.n, d.c_out, ho, wo), dtype=np.float64)
    rc = _load().oracle_conv2d_transpose_alg1(ctypes.byref(d), _ptr(x), _ptr(w), _ptr(bias),
                                              _ptr(y), _threads(nthreads))
    if rc:
        raise ValueError("oracle_conv2d_transpose_alg1 rejected its arguments")
    return y


def conv2d_dilated_alg2(x, w, bias=None, stride=1, padding=0, dilation=1, nthreads=None,
                        groups=1):
    """Dilated / strided conv by direct gather (Algorithm 2); float64 NCHW in and out.
    groups > 1: w is [C_out, C_in/groups, R, S]."""
    x, w, bias = _f64(x), _f64(w), _f64(bias)
    d = _desc(x.shape, w.shape, False, stride, padding, 0, dilation, groups)
    ho, wo = conv_out_dims(x.shape, w.shape, stride, padding, dilation, groups)
    y = np.empty((d.n, d.c_out, ho, wo), dtype=np.float64)
    rc = _load().oracle_conv2d_dilated_alg2(ctypes.byref(d), _ptr(x), _ptr(w), _ptr(bias),
                                            _ptr(y), _threads(nthreads))
    if rc:
        raise ValueError("oracle_conv2d_dilated_alg2 rejected its arguments")
    return y


def _points(fn, d, x, w, bias, flat_idx, nthreads):
    idx = np.ascontiguousarray(flat_idx, dtype=np.int64)
    out = np.empty(idx.shape, dtype=np.float64)
    rc = fn(ctypes.byref(d), _ptr(x), _ptr(w), _ptr(bias),
            idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), idx.size, _ptr(out),
            _threads(nthreads))
    if rc:
        raise ValueError("oracle point evaluation rejected its arguments")
    return out


def conv2d_transpose_points(x, w, flat_idx, bias=None, stride=1, padding=0, output_padding=0,
                            dilation=1, nthreads=None, groups=1):
    """Algorithm 1 evaluated at flat NCHW output indices ``flat_idx``."""
    x, w, bias = _f64(x), _f64(w), _f64(bias)
    d = _desc(x.shape, w.shape, True, stride, padding, output_padding, dilation, groups)
    return _points(_load().oracle_conv2d_transpose_points, d, x, w, bias, flat_idx, nthreads)


def conv2d_dilated_points(x, w, flat_idx, bias=None, stride=1, padding=0, dilation=1,
                          nthreads=None, groups=1):
    """Algorithm 2 evaluated at flat NCHW output indices ``flat_idx``."""
    x, w, bias = _f64(x), _f64(w), _f64(bias)
    d = _desc(x.shape, w.shape, False, stride, padding, 0, dilation, groups)
    return _points(_load().oracle_conv2d_dilated_points, d, x, w, bias, flat_idx, nthreads)


def conv2d_transpose_wgrad(x, dy, w_shape, stride=1, padding=0, output_padding=0, dilation=1,
                           nthreads=None, groups=1):
    """Weight gradient of the transposed conv: dw [C_in, C_out/groups, R, S]
    from the input x and the output error dy; float64."""
    x, dy = _f64(x), _f64(dy)
    d = _desc(x.shape, tuple(w_shape), True, stride, padding, output_padding, dilation, groups)
    ho, wo = transpose_out_dims(x.shape, w_shape, stride, padding, output_padding, dilation,
                                groups)
    if dy.shape != (d.n, d.c_out, ho, wo):
        raise ValueError("dy shape %s does not match the output %s" % (dy.shape, (d.n, d.c_out, ho, wo)))
    dw = np.empty(tuple(w_shape), dtype=np.float64)
    if _load().oracle_conv2d_transpose_wgrad(ctypes.byref(d), _ptr(x), _ptr(dy), _ptr(dw),
                                             _threads(nthreads)):
        raise ValueError("oracle_conv2d_transpose_wgrad rejected its arguments")
    return dw


def conv2d_dilated_wgrad(x, dy, w_shape, stride=1, padding=0, dilation=1, nthreads=None,
                         groups=1):
    """Weight gradient of the dilated / strided conv: dw [C_out, C_in/groups,
    R, S] from the input x and the output error dy; float64."""
    x, dy = _f64(x), _f64(dy)
    d = _desc(x.shape, tuple(w_shape), False, stride, padding, 0, dilation, groups)
    ho, wo = conv_out_dims(x.shape, w_shape, stride, padding, dilation, groups)
    if dy.shape != (d.n, d.c_out, ho, wo):
        raise ValueError("dy shape %s does not match the output %s" % (dy.shape, (d.n, d.c_out, ho, wo)))
    dw = np.empty(tuple(w_shape), dtype=np.float64)
    if _load().oracle_conv2d_dilated_wgrad(ctypes.byref(d), _ptr(x), _ptr(dy), _ptr(dw),
                                           _threads(nthreads)):
        raise ValueError("oracle_conv2d_dilated_wgrad rejected its arguments")
    return dw


def activate(y, act):
    """The generator's nonlinearity applied to an oracle output: "none" (or
    None) leaves y, "relu" is max(y, 0) and "tanh" the hyperbolic tangent,
    elementwise in float64."""
    if act in (None, "none"):
        return y
    y = _f64(y)
    if act == "relu":
        return np.maximum(y, 0.0)
    if act == "tanh":
        return np.tanh(y)
    raise ValueError("unknown activation %r" % (act,))
