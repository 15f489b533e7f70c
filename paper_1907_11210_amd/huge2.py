"""Python binding of libhuge2 (the C ABI in include/huge2.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libhuge2.so``.  PyTorch supplies device memory and the current
HIP stream; nothing here computes a convolution, and there is no CPU
fallback: if the library is missing, every entry point raises.

The ``huge2_*`` functions mirror the C entry points one to one and take raw
device pointers (ints).  :func:`conv2d_transpose`, :func:`conv2d_dilated` and
:class:`Plan` are thin torch conveniences on top of them.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhuge2.so")

HUGE2_OK, HUGE2_ERR_INVALID_ARG, HUGE2_ERR_UNSUPPORTED, HUGE2_ERR_ALLOC, HUGE2_ERR_HIP = range(5)
HUGE2_F32, HUGE2_BF16 = 0, 1
HUGE2_NCHW, HUGE2_NHWC = 0, 1
HUGE2_ACT_NONE, HUGE2_ACT_RELU, HUGE2_ACT_TANH = 0, 1, 2
ACTIVATIONS = {None: HUGE2_ACT_NONE, "none": HUGE2_ACT_NONE, "relu": HUGE2_ACT_RELU,
               "tanh": HUGE2_ACT_TANH}

EXPORTED = (
    "huge2_status_str", "huge2_output_shape", "huge2_plan_create", "huge2_plan_execute",
    "huge2_plan_stage_input", "huge2_plan_run_gemm", "huge2_plan_stages_input",
    "huge2_plan_kernel",
    "huge2_plan_destroy", "huge2_conv2d_transpose", "huge2_conv2d_dilated",
    "huge2_plan_describe", "huge2_plan_macs",
    "huge2_wgrad_plan_create", "huge2_wgrad_execute", "huge2_wgrad_plan_destroy",
    "huge2_conv2d_transpose_wgrad", "huge2_conv2d_dilated_wgrad",
    "huge2_group_create", "huge2_group_execute", "huge2_group_destroy", "huge2_group_kernel",
    "huge2_conv2d_transpose_noalloc", "huge2_dgrad_output_padding",
)
MAX_GROUP = 8


class Huge2Error(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s failed: %s" % (where, status_str(status)))


class ConvDesc(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in (
        "n", "c_in", "h", "w", "c_out", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w",
        "out_pad_h", "out_pad_w", "dil_h", "dil_w", "layout", "dtype", "activation", "groups")]


class Segment(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in (
        "phase0_h", "phase0_w", "nphase_h", "nphase_w", "out_step_h", "out_step_w",
        "q0_h", "q0_w", "qn_h", "qn_w", "in0_h", "in0_w", "in_dphase_h", "in_dphase_w",
        "in_step_h", "in_step_w", "tap_begin", "tap_count")]


class Tap(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in ("kh", "kw", "off_h", "off_w")]


_lib = None


def lib():
    """The loaded libhuge2.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                "libhuge2.so is not built (%s); run __graft_entry__.build() or "
                "python -m paper_1907_11210_amd._build" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64p = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64)
        dp = ctypes.POINTER(ConvDesc)
        i32p = ctypes.POINTER(ctypes.c_int32)
        L.huge2_status_str.restype = ctypes.c_char_p
        L.huge2_status_str.argtypes = [ctypes.c_int]
        L.huge2_output_shape.argtypes = [dp, i32, i32p, i32p]
        L.huge2_plan_create.argtypes = [ctypes.POINTER(vp), dp, i32, vp, vp]
        L.huge2_plan_execute.argtypes = [vp, vp, vp, vp, vp]
        L.huge2_plan_stage_input.argtypes = [vp, vp, vp]
        L.huge2_plan_run_gemm.argtypes = [vp, vp, vp, vp, vp]
        L.huge2_plan_stages_input.argtypes = [vp]
        L.huge2_plan_kernel.argtypes = [vp]
        L.huge2_plan_destroy.argtypes = [vp]
        L.huge2_conv2d_transpose.argtypes = [dp, vp, vp, vp, vp, vp]
        L.huge2_conv2d_dilated.argtypes = [dp, vp, vp, vp, vp, vp]
        L.huge2_plan_describe.argtypes = [dp, i32, i32, ctypes.POINTER(Segment), i32, i32p,
                                          ctypes.POINTER(Tap), i32, i32p]
        L.huge2_plan_macs.argtypes = [dp, i32, i64p, i64p]
        L.huge2_wgrad_plan_create.argtypes = [ctypes.POINTER(vp), dp, i32]
        L.huge2_wgrad_execute.argtypes = [vp, vp, vp, vp, vp]
        L.huge2_wgrad_plan_destroy.argtypes = [vp]
        L.huge2_conv2d_transpose_wgrad.argtypes = [dp, vp, vp, vp, vp]
        L.huge2_conv2d_dilated_wgrad.argtypes = [dp, vp, vp, vp, vp]
        L.huge2_group_create.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(vp), i32, vp]
        L.huge2_group_execute.argtypes = [vp, vp, ctypes.POINTER(vp), ctypes.POINTER(vp), vp]
        L.huge2_group_destroy.argtypes = [vp]
        L.huge2_group_kernel.argtypes = [vp]
        L.huge2_conv2d_transpose_noalloc.argtypes = [dp, vp, vp, vp, vp, vp]
        L.huge2_dgrad_output_padding.argtypes = [dp, i32p, i32p]
        for name in EXPORTED[1:]:
            getattr(L, name).restype = ctypes.c_int
        L.huge2_plan_kernel.restype = ctypes.c_char_p
        L.huge2_group_kernel.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_str(status):
    return lib().huge2_status_str(int(status)).decode()


def _check(status, where):
    if status != HUGE2_OK:
        raise Huge2Error(status, where)


def _pair(v):
    if isinstance(v, (tuple, list)):
        return int(v[0]), int(v[1])
    return int(v), int(v)


def make_desc(n, c_in, h, w, c_out, r, s, stride=1, padding=0, output_padding=0, dilation=1,
              layout=HUGE2_NCHW, dtype=HUGE2_F32, activation=HUGE2_ACT_NONE, groups=1):
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    oph, opw = _pair(output_padding)
    dh, dw = _pair(dilation)
    return ConvDesc(n, c_in, h, w, c_out, r, s, sh, sw, ph, pw, oph, opw, dh, dw, layout, dtype,
                    activation, groups)


# ---- the C entry points ---------------------------------------------------

def huge2_output_shape(desc, transposed):
    ho, wo = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().huge2_output_shape(ctypes.byref(desc), int(transposed), ctypes.byref(ho),
                                    ctypes.byref(wo)), "huge2_output_shape")
    return ho.value, wo.value


def huge2_dgrad_output_padding(conv_desc):
    oph, opw = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().huge2_dgrad_output_padding(ctypes.byref(conv_desc), ctypes.byref(oph),
                                            ctypes.byref(opw)), "huge2_dgrad_output_padding")
    return oph.value, opw.value


def huge2_plan_create(desc, transposed, w_ptr, stream=0):
    plan = ctypes.c_void_p()
    _check(lib().huge2_plan_create(ctypes.byref(plan), ctypes.byref(desc), int(transposed),
                                   ctypes.c_void_p(w_ptr), ctypes.c_void_p(stream)),
           "huge2_plan_create")
    return plan


def huge2_plan_execute(plan, x_ptr, bias_ptr, y_ptr, stream=0):
    _check(lib().huge2_plan_execute(plan, ctypes.c_void_p(x_ptr), ctypes.c_void_p(bias_ptr),
                                    ctypes.c_void_p(y_ptr), ctypes.c_void_p(stream)),
           "huge2_plan_execute")


def huge2_plan_stage_input(plan, x_ptr, stream=0):
    _check(lib().huge2_plan_stage_input(plan, ctypes.c_void_p(x_ptr), ctypes.c_void_p(stream)),
           "huge2_plan_stage_input")


def huge2_plan_run_gemm(plan, x_ptr, bias_ptr, y_ptr, stream=0):
    _check(lib().huge2_plan_run_gemm(plan, ctypes.c_void_p(x_ptr), ctypes.c_void_p(bias_ptr),
                                     ctypes.c_void_p(y_ptr), ctypes.c_void_p(stream)),
           "huge2_plan_run_gemm")


def huge2_plan_stages_input(plan):
    return int(lib().huge2_plan_stages_input(plan))


def huge2_plan_kernel(plan):
    return lib().huge2_plan_kernel(plan).decode()


def huge2_plan_destroy(plan):
    _check(lib().huge2_plan_destroy(plan), "huge2_plan_destroy")


def huge2_conv2d_transpose(desc, x_ptr, w_ptr, bias_ptr, y_ptr, stream=0):
    _check(lib().huge2_conv2d_transpose(ctypes.byref(desc), ctypes.c_void_p(x_ptr),
                                        ctypes.c_void_p(w_ptr), ctypes.c_void_p(bias_ptr),
                                        ctypes.c_void_p(y_ptr), ctypes.c_void_p(stream)),
           "huge2_conv2d_transpose")


def huge2_conv2d_transpose_noalloc(desc, x_ptr, w_ptr, bias_ptr, y_ptr, stream=0):
    _check(lib().huge2_conv2d_transpose_noalloc(ctypes.byref(desc), ctypes.c_void_p(x_ptr),
                                                ctypes.c_void_p(w_ptr), ctypes.c_void_p(bias_ptr),
                                                ctypes.c_void_p(y_ptr), ctypes.c_void_p(stream)),
           "huge2_conv2d_transpose_noalloc")


def huge2_conv2d_dilated(desc, x_ptr, w_ptr, bias_ptr, y_ptr, stream=0):
    _check(lib().huge2_conv2d_dilated(ctypes.byref(desc), ctypes.c_void_p(x_ptr),
                                      ctypes.c_void_p(w_ptr), ctypes.c_void_p(bias_ptr),
                                      ctypes.c_void_p(y_ptr), ctypes.c_void_p(stream)),
           "huge2_conv2d_dilated")


def huge2_plan_describe(desc, transposed, class_split=2):
    """(segments, taps) as lists of dicts."""
    ns, nt = ctypes.c_int32(), ctypes.c_int32()
    L = lib()
    _check(L.huge2_plan_describe(ctypes.byref(desc), int(transposed), int(class_split), None, 0,
                                 ctypes.byref(ns), None, 0, ctypes.byref(nt)),
           "huge2_plan_describe")
    segs = (Segment * max(ns.value, 1))()
    taps = (Tap * max(nt.value, 1))()
    _check(L.huge2_plan_describe(ctypes.byref(desc), int(transposed), int(class_split), segs,
                                 ns.value, ctypes.byref(ns), taps, nt.value, ctypes.byref(nt)),
           "huge2_plan_describe")
    seg_list = [{f: getattr(segs[i], f) for f, _ in Segment._fields_} for i in range(ns.value)]
    tap_list = [{f: getattr(taps[i], f) for f, _ in Tap._fields_} for i in range(nt.value)]
    return seg_list, tap_list


def huge2_plan_macs(desc, transposed):
    nz, issued = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().huge2_plan_macs(ctypes.byref(desc), int(transposed), ctypes.byref(nz),
                                 ctypes.byref(issued)), "huge2_plan_macs")
    return nz.value, issued.value

def huge2_wgrad_plan_create(desc, transposed):
    plan = ctypes.c_void_p()
    _check(lib().huge2_wgrad_plan_create(ctypes.byref(plan), ctypes.byref(desc), int(transposed)),
           "huge2_wgrad_plan_create")
    return plan


def huge2_wgrad_execute(plan, x_ptr, dy_ptr, dw_ptr, stream=0):
    _check(lib().huge2_wgrad_execute(plan, ctypes.c_void_p(x_ptr), ctypes.c_void_p(dy_ptr),
                                     ctypes.c_void_p(dw_ptr), ctypes.c_void_p(stream)),
           "huge2_wgrad_execute")


def huge2_wgrad_plan_destroy(plan):
    _check(lib().huge2_wgrad_plan_destroy(plan), "huge2_wgrad_plan_destroy")


def huge2_conv2d_transpose_wgrad(desc, x_ptr, dy_ptr, dw_ptr, stream=0):
    _check(lib().huge2_conv2d_transpose_wgrad(ctypes.byref(desc), ctypes.c_void_p(x_ptr),
                                              ctypes.c_void_p(dy_ptr), ctypes.c_void_p(dw_ptr),
                                              ctypes.c_void_p(stream)),
           "huge2_conv2d_transpose_wgrad")


def huge2_conv2d_dilated_wgrad(desc, x_ptr, dy_ptr, dw_ptr, stream=0):
    _check(lib().huge2_conv2d_dilated_wgrad(ctypes.byref(desc), ctypes.c_void_p(x_ptr),
                                            ctypes.c_void_p(dy_ptr), ctypes.c_void_p(dw_ptr),
                                            ctypes.c_void_p(stream)),
           "huge2_conv2d_dilated_wgrad")


# ---- torch conveniences -----------------------------------------------------

def huge2_group_create(plans, stream=0):
    arr = (ctypes.c_void_p * len(plans))(*plans)
    out = ctypes.c_void_p()
    _check(lib().huge2_group_create(ctypes.byref(out), arr, len(plans), stream),
           "huge2_group_create")
    return out.value


def huge2_group_execute(group, x_ptr, bias_ptrs, y_ptrs, stream=0):
    ys = (ctypes.c_void_p * len(y_ptrs))(*y_ptrs)
    bs = None if bias_ptrs is None else (ctypes.c_void_p * len(bias_ptrs))(*bias_ptrs)
    _check(lib().huge2_group_execute(group, x_ptr, bs, ys, stream), "huge2_group_execute")


def huge2_group_kernel(group):
    return lib().huge2_group_kernel(group).decode()


def huge2_group_destroy(group):
    _check(lib().huge2_group_destroy(group), "huge2_group_destroy")


def _torch():
    import torch
    return torch


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return HUGE2_F32
    if t.dtype == torch.bfloat16:
        return HUGE2_BF16
    raise TypeError("unsupported dtype %s (float32 or bfloat16)" % t.dtype)


def _layout_code(layout):
    if layout in ("NCHW", HUGE2_NCHW):
        return HUGE2_NCHW
    if layout in ("NHWC", HUGE2_NHWC):
        return HUGE2_NHWC
    raise ValueError("layout must be NCHW or NHWC")


def _check_tensor(t, name, device=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if t.data_ptr() % 16:
        raise ValueError("%s must be 16-byte aligned" % name)
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))


def _act_code(activation):
    if activation not in ACTIVATIONS:
        raise ValueError("unknown activation %r (none, relu, tanh)" % (activation,))
    return ACTIVATIONS[activation]


def _desc_for(x, w, transposed, stride, padding, output_padding, dilation, layout,
              activation=None, groups=1):
    lay = _layout_code(layout)
    if x.dim() != 4 or w.dim() != 4:
        raise ValueError("x and w must be 4-D")
    if lay == HUGE2_NCHW:
        n, c_in, h, wd = x.shape
    else:
        n, h, wd, c_in = x.shape
    g = int(groups)
    if transposed:
        wc_in, cog, r, s = w.shape
        c_out = cog * g
    else:
        c_out, cig, r, s = w.shape
        wc_in = cig * g
    if wc_in != c_in:
        raise ValueError("weight has %d input channels, x has %d" % (wc_in, c_in))
    if w.dtype != x.dtype:
        raise ValueError("x and w must share a dtype")
    return make_desc(n, c_in, h, wd, c_out, r, s, stride, padding, output_padding, dilation,
                     lay, _dtype_code(x), _act_code(activation), g)


def _out_shape(desc, transposed):
    ho, wo = huge2_output_shape(desc, transposed)
    if desc.layout == HUGE2_NCHW:
        return (desc.n, desc.c_out, ho, wo)
    return (desc.n, ho, wo, desc.c_out)


def _bias_ptr(bias, x):
    torch = _torch()
    if bias is None:
        return 0
    _check_tensor(bias, "bias", x.device)
    if bias.dtype != torch.float32 or bias.dim() != 1:
        raise ValueError("bias must be a 1-D float32 tensor")
    return bias.data_ptr()


def _stream(x):
    return _torch().cuda.current_stream(x.device).cuda_stream


def conv2d_transpose(x, w, bias=None, stride=1, padding=0, output_padding=0, dilation=1,
                     layout="NCHW", out=None, activation=None, groups=1):
    """Transposed conv on the GPU (w: [C_in, C_out/groups, R, S]); returns
    y = activation(op(x) + bias), activation None, "relu" or "tanh"."""
    torch = _torch()
    _check_tensor(x, "x")
    _check_tensor(w, "w", x.device)
    desc = _desc_for(x, w, True, stride, padding, output_padding, dilation, layout, activation,
                     groups)
    shape = _out_shape(desc, True)
    if bias is not None and bias.numel() != desc.c_out:
        raise ValueError("bias size does not match C_out")
    y = out if out is not None else torch.empty(shape, dtype=x.dtype, device=x.device)
    _check_tensor(y, "out", x.device)
    if tuple(y.shape) != shape or y.dtype != x.dtype:
        raise ValueError("out has the wrong shape or dtype")
    huge2_conv2d_transpose(desc, x.data_ptr(), w.data_ptr(), _bias_ptr(bias, x), y.data_ptr(),
                           _stream(x))
    return y


def conv2d_dilated(x, w, bias=None, stride=1, padding=0, dilation=1, layout="NCHW", out=None,
                   activation=None, groups=1):
    """Dilated / strided conv on the GPU (w: [C_out, C_in/groups, R, S]); returns
    y = activation(op(x) + bias)."""
    torch = _torch()
    _check_tensor(x, "x")
    _check_tensor(w, "w", x.device)
    desc = _desc_for(x, w, False, stride, padding, 0, dilation, layout, activation, groups)
    shape = _out_shape(desc, False)
    if bias is not None and bias.numel() != desc.c_out:
        raise ValueError("bias size does not match C_out")
    y = out if out is not None else torch.empty(shape, dtype=x.dtype, device=x.device)
    _check_tensor(y, "out", x.device)
    if tuple(y.shape) != shape or y.dtype != x.dtype:
        raise ValueError("out has the wrong shape or dtype")
    huge2_conv2d_dilated(desc, x.data_ptr(), w.data_ptr(), _bias_ptr(bias, x), y.data_ptr(),
                         _stream(x))
    return y


def _wgrad(x, dy, w_shape, transposed, stride, padding, output_padding, dilation, out,
           groups=1):
    torch = _torch()
    _check_tensor(x, "x")
    _check_tensor(dy, "dy", x.device)
    if dy.dtype != x.dtype:
        raise ValueError("x and dy must share a dtype")
    w_shape = tuple(int(v) for v in w_shape)
    if x.dim() != 4 or len(w_shape) != 4:
        raise ValueError("x and the weight shape must be 4-D")
    n, c_in, h, wd = x.shape
    g = int(groups)
    if transposed:
        wc_in, cog, r, s = w_shape
        c_out = cog * g
    else:
        c_out, cig, r, s = w_shape
        wc_in = cig * g
    if wc_in != c_in:
        raise ValueError("weight has %d input channels, x has %d" % (wc_in, c_in))
    desc = make_desc(n, c_in, h, wd, c_out, r, s, stride, padding, output_padding, dilation,
                     HUGE2_NCHW, _dtype_code(x), groups=g)
    if tuple(dy.shape) != _out_shape(desc, transposed):
        raise ValueError("dy has shape %s, the layer's output is %s"
                         % (tuple(dy.shape), _out_shape(desc, transposed)))
    dw = out if out is not None else torch.empty(w_shape, dtype=x.dtype, device=x.device)
    _check_tensor(dw, "out", x.device)
    if tuple(dw.shape) != w_shape or dw.dtype != x.dtype:
        raise ValueError("out has the wrong shape or dtype")
    fn = huge2_conv2d_transpose_wgrad if transposed else huge2_conv2d_dilated_wgrad
    fn(desc, x.data_ptr(), dy.data_ptr(), dw.data_ptr(), _stream(x))
    return dw


def conv2d_transpose_wgrad(x, dy, w_shape, stride=1, padding=0, output_padding=0, dilation=1,
                           out=None, groups=1):
    """Weight gradient of the transposed conv (NCHW): dw [C_in, C_out/groups,
    R, S] from the input x and the output error dy."""
    return _wgrad(x, dy, w_shape, True, stride, padding, output_padding, dilation, out, groups)


def conv2d_dilated_wgrad(x, dy, w_shape, stride=1, padding=0, dilation=1, out=None, groups=1):
    """Weight gradient of the dilated / strided conv (NCHW): dw [C_out,
    C_in/groups, R, S] from the input x and the output error dy."""
    return _wgrad(x, dy, w_shape, False, stride, padding, 0, dilation, out, groups)


def conv2d_transpose_dgrad(dy, w, stride=1, padding=0, dilation=1, layout="NCHW"):
    """Data gradient of the transposed conv: the strided conv of dy with the
    same w ([C_in, C_out, R, S] is the strided conv's [C_out, C_in, R, S])."""
    return conv2d_dilated(dy, w, None, stride, padding, dilation, layout)


def conv2d_dilated_dgrad(dy, w, x_hw, stride=1, padding=0, dilation=1, layout="NCHW"):
    """Data gradient of the dilated / strided conv: the transposed conv of dy
    with the same w, output padding chosen so that the result is x_hw."""
    lay = _layout_code(layout)
    n, c_y = (dy.shape[0], dy.shape[1]) if lay == HUGE2_NCHW else (dy.shape[0], dy.shape[3])
    # the forward strided conv: input x_hw with w.shape[1] channels, c_y outputs
    fwd = make_desc(n, w.shape[1], x_hw[0], x_hw[1], c_y, w.shape[2], w.shape[3], stride,
                    padding, 0, dilation, lay, _dtype_code(dy))
    op = huge2_dgrad_output_padding(fwd)
    return conv2d_transpose(dy, w, None, stride, padding, op, dilation, layout)


class Plan:
    """A reusable plan: weights packed once (huge2_plan_create), then
    :meth:`__call__` enqueues huge2_plan_execute on the current stream."""

    def __init__(self, w, x_shape, transposed, stride=1, padding=0, output_padding=0,
                 dilation=1, layout="NCHW", activation=None, groups=1):
        torch = _torch()
        _check_tensor(w, "w")
        dummy = torch.empty(0, dtype=w.dtype)
        lay = _layout_code(layout)
        if lay == HUGE2_NCHW:
            n, c_in, h, wd = x_shape
        else:
            n, h, wd, c_in = x_shape
        g = int(groups)
        if transposed:
            wc_in, cog, r, s = w.shape
            c_out = cog * g
        else:
            c_out, cig, r, s = w.shape
            wc_in = cig * g
        if wc_in != c_in:
            raise ValueError("weight has %d input channels, x has %d" % (wc_in, c_in))
        self.desc = make_desc(n, c_in, h, wd, c_out, r, s, stride, padding, output_padding,
                              dilation, lay, _dtype_code(dummy), _act_code(activation), g)
        self.transposed = bool(transposed)
        self.device = w.device
        self.dtype = w.dtype
        self.x_shape = tuple(x_shape)
        self.out_shape = _out_shape(self.desc, self.transposed)
        self._plan = None
        self._plan = huge2_plan_create(self.desc, self.transposed, w.data_ptr(),
                                       torch.cuda.current_stream(w.device).cuda_stream)

    def __call__(self, x, bias=None, out=None):
        torch = _torch()
        _check_tensor(x, "x", self.device)
        if tuple(x.shape) != self.x_shape or x.dtype != self.dtype:
            raise ValueError("x does not match the plan")
        y = out if out is not None else torch.empty(self.out_shape, dtype=x.dtype,
                                                    device=x.device)
        _check_tensor(y, "out", self.device)
        if tuple(y.shape) != self.out_shape or y.dtype != self.dtype:
            raise ValueError("out does not match the plan")
        if bias is not None and bias.numel() != self.desc.c_out:
            raise ValueError("bias size does not match C_out")
        huge2_plan_execute(self._plan, x.data_ptr(), _bias_ptr(bias, x), y.data_ptr(),
                           _stream(x))
        return y

    def stage(self, x):
        """Enqueue only the input re-layout (no-op for plans that need none)."""
        _check_tensor(x, "x", self.device)
        if tuple(x.shape) != self.x_shape or x.dtype != self.dtype:
            raise ValueError("x does not match the plan")
        huge2_plan_stage_input(self._plan, x.data_ptr(), _stream(x))

    def gemm(self, x, out, bias=None):
        """Enqueue only the phase GEMM (after :meth:`stage` when the plan stages)."""
        _check_tensor(x, "x", self.device)
        _check_tensor(out, "out", self.device)
        if tuple(out.shape) != self.out_shape or out.dtype != self.dtype:
            raise ValueError("out does not match the plan")
        huge2_plan_run_gemm(self._plan, x.data_ptr(), _bias_ptr(bias, x), out.data_ptr(),
                            _stream(x))
        return out

    @property
    def stages_input(self):
        return huge2_plan_stages_input(self._plan) == 1

    @property
    def kernel(self):
        """Name and tile shape of the main kernel this plan launches."""
        return huge2_plan_kernel(self._plan)

    def macs(self):
        return huge2_plan_macs(self.desc, self.transposed)

    def close(self):
        if self._plan is not None:
            huge2_plan_destroy(self._plan)
            self._plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Group:
    """Several :class:`Plan` objects of one input run as one launch
    (huge2_group_create); :meth:`__call__` enqueues huge2_group_execute on the
    current stream.  The plans must stay open while the group is used."""

    def __init__(self, plans):
        torch = _torch()
        self.plans = list(plans)
        self._group = None
        self._group = huge2_group_create([p._plan for p in self.plans],
                                         torch.cuda.current_stream(self.plans[0].device).cuda_stream)

    def __call__(self, x, biases=None, outs=None):
        torch = _torch()
        p0 = self.plans[0]
        _check_tensor(x, "x", p0.device)
        if tuple(x.shape) != p0.x_shape or x.dtype != p0.dtype:
            raise ValueError("x does not match the plans")
        if outs is None:
            outs = [torch.empty(p.out_shape, dtype=x.dtype, device=x.device) for p in self.plans]
        for p, y in zip(self.plans, outs):
            _check_tensor(y, "out", p0.device)
            if tuple(y.shape) != p.out_shape or y.dtype != p.dtype:
                raise ValueError("out does not match its plan")
        bias_ptrs = None
        if biases is not None:
            bias_ptrs = [_bias_ptr(b, x) for b in biases]
        huge2_group_execute(self._group, x.data_ptr(), bias_ptrs, [y.data_ptr() for y in outs],
                            _stream(x))
        return outs

    @property
    def kernel(self):
        """Name and tile shape of the kernel the group launches."""
        return huge2_group_kernel(self._group)

    def close(self):
        if self._group is not None:
            huge2_group_destroy(self._group)
            self._group = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
