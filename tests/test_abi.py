"""The C ABI on the CPU: the library loads, exports every symbol the header
declares, and rejects invalid arguments before any HIP call (no GPU needed)."""
import ctypes
import os
import re
import subprocess

import pytest

h2 = pytest.importorskip("paper_1907_11210_amd.huge2")
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(h2.LIB_PATH):
        from paper_1907_11210_amd import _build
        _build.build()
    return h2.lib()


def _declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(huge2_\w+)\s*\(", text))
    return names


def test_every_declared_symbol_is_exported(L):
    declared = _declared_functions()
    assert declared >= set(h2.EXPORTED)
    for name in declared:
        assert hasattr(L, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", h2.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (huge2_\w+)", out))
    assert declared <= exported


def test_status_strings(L):
    for code, name in enumerate(["HUGE2_OK", "HUGE2_ERR_INVALID_ARG", "HUGE2_ERR_UNSUPPORTED",
                                 "HUGE2_ERR_ALLOC", "HUGE2_ERR_HIP"]):
        assert h2.status_str(code) == name
    assert h2.status_str(99) == "HUGE2_ERR_UNKNOWN"


def _good():
    return h2.make_desc(2, 8, 5, 5, 4, 4, 4, 2, 1, 0, 1, h2.HUGE2_NCHW, h2.HUGE2_F32)


@pytest.mark.parametrize("field,value", [
    ("n", 0), ("c_in", 0), ("h", -1), ("c_out", 0), ("r", 0), ("stride_h", 0), ("dil_w", 0),
    ("pad_h", -1), ("out_pad_w", 2), ("layout", 2), ("dtype", 7), ("pad_h", 40),
    ("activation", 3), ("activation", -1),
])
def test_invalid_descriptor_rejected_without_gpu(L, field, value):
    d = _good()
    setattr(d, field, value)
    ho, wo = ctypes.c_int32(-5), ctypes.c_int32(-5)
    st = L.huge2_output_shape(ctypes.byref(d), 1, ctypes.byref(ho), ctypes.byref(wo))
    assert st == h2.HUGE2_ERR_INVALID_ARG
    assert ho.value == -5  # untouched
    fake = ctypes.c_void_p(4096)
    assert L.huge2_conv2d_transpose(ctypes.byref(d), fake, fake, None, ctypes.c_void_p(8192),
                                    None) == h2.HUGE2_ERR_INVALID_ARG
    plan = ctypes.c_void_p(1234)
    assert L.huge2_plan_create(ctypes.byref(plan), ctypes.byref(d), 1, fake,
                               None) == h2.HUGE2_ERR_INVALID_ARG
    assert plan.value is None


def test_dilated_rejects_output_padding(L):
    d = h2.make_desc(1, 4, 8, 8, 4, 3, 3, 1, 2, 1, 2, h2.HUGE2_NHWC, h2.HUGE2_BF16)
    ho, wo = ctypes.c_int32(), ctypes.c_int32()
    assert L.huge2_output_shape(ctypes.byref(d), 0, ctypes.byref(ho),
                                ctypes.byref(wo)) == h2.HUGE2_ERR_INVALID_ARG
    # the same descriptor is valid as a transposed conv (out_pad < dilation)
    assert L.huge2_output_shape(ctypes.byref(d), 1, ctypes.byref(ho), ctypes.byref(wo)) == 0


def test_null_and_aliased_pointers_rejected(L):
    d = _good()
    fake = ctypes.c_void_p(4096)
    assert L.huge2_conv2d_transpose(ctypes.byref(d), None, fake, None, fake,
                                    None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_conv2d_transpose(ctypes.byref(d), fake, None, None, ctypes.c_void_p(8192),
                                    None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_conv2d_transpose(ctypes.byref(d), fake, fake, None, fake,
                                    None) == h2.HUGE2_ERR_INVALID_ARG  # x == y
    assert L.huge2_conv2d_dilated(None, fake, fake, None, ctypes.c_void_p(8192),
                                  None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_plan_execute(None, fake, None, ctypes.c_void_p(8192),
                                None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_plan_stage_input(None, fake, None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_plan_run_gemm(None, fake, None, ctypes.c_void_p(8192),
                                 None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_plan_stages_input(None) == -1
    assert h2.huge2_plan_kernel(None) == ""
    assert L.huge2_plan_destroy(None) == h2.HUGE2_OK
    assert L.huge2_plan_create(None, ctypes.byref(d), 1, fake, None) == h2.HUGE2_ERR_INVALID_ARG
    plan = ctypes.c_void_p()
    assert L.huge2_plan_create(ctypes.byref(plan), ctypes.byref(d), 2, fake,
                               None) == h2.HUGE2_ERR_INVALID_ARG


def test_too_large_is_unsupported(L):
    d = h2.make_desc(64, 4096, 512, 512, 16, 3, 3, 1, 1, 0, 1, h2.HUGE2_NHWC, h2.HUGE2_BF16)
    ho, wo = ctypes.c_int32(), ctypes.c_int32()
    assert L.huge2_output_shape(ctypes.byref(d), 0, ctypes.byref(ho), ctypes.byref(wo)) == 0
    plan = ctypes.c_void_p()
    assert L.huge2_plan_create(ctypes.byref(plan), ctypes.byref(d), 0, ctypes.c_void_p(4096),
                               None) == h2.HUGE2_ERR_UNSUPPORTED


def test_allocation_failure_is_reported(L, monkeypatch):
    monkeypatch.setenv("HUGE2_FAULT", "alloc")
    d = _good()
    plan = ctypes.c_void_p(77)
    assert L.huge2_plan_create(ctypes.byref(plan), ctypes.byref(d), 1, ctypes.c_void_p(4096),
                               None) == h2.HUGE2_ERR_ALLOC
    assert plan.value is None


def test_describe_sizes_and_caps(L):
    d = _good()
    ns, nt = ctypes.c_int32(), ctypes.c_int32()
    assert L.huge2_plan_describe(ctypes.byref(d), 1, 2, None, 0, ctypes.byref(ns), None, 0,
                                 ctypes.byref(nt)) == 0
    assert ns.value > 0 and nt.value > 0
    assert L.huge2_plan_describe(ctypes.byref(d), 1, 3, None, 0, ctypes.byref(ns), None, 0,
                                 ctypes.byref(nt)) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_plan_describe(ctypes.byref(d), 1, 1, None, 5, ctypes.byref(ns), None, 0,
                                 ctypes.byref(nt)) == h2.HUGE2_ERR_INVALID_ARG


def test_product_path_has_no_cpu_fallback():
    """The binding never imports the oracle and raises if the library is missing."""
    src = open(os.path.join(ROOT, "paper_1907_11210_amd", "huge2.py")).read()
    assert "oracle" not in src
    for fn in os.listdir(os.path.join(ROOT, "paper_1907_11210_amd")):
        if fn.endswith(".py"):
            assert "import oracle" not in open(os.path.join(ROOT, "paper_1907_11210_amd", fn)).read()


def test_weight_gradient_entry_points_validate_without_gpu(L, monkeypatch):
    d = _good()
    fake, other = ctypes.c_void_p(4096), ctypes.c_void_p(8192)
    plan = ctypes.c_void_p(55)
    assert L.huge2_wgrad_plan_create(None, ctypes.byref(d), 1) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_wgrad_plan_create(ctypes.byref(plan), None, 1) == h2.HUGE2_ERR_INVALID_ARG
    assert plan.value is None
    assert L.huge2_wgrad_plan_create(ctypes.byref(plan), ctypes.byref(d), 3) == h2.HUGE2_ERR_INVALID_ARG
    bad = _good()
    bad.stride_h = 0
    assert L.huge2_wgrad_plan_create(ctypes.byref(plan), ctypes.byref(bad), 1) == h2.HUGE2_ERR_INVALID_ARG
    nhwc = _good()
    nhwc.layout = h2.HUGE2_NHWC
    assert L.huge2_wgrad_plan_create(ctypes.byref(plan), ctypes.byref(nhwc), 1) == h2.HUGE2_ERR_UNSUPPORTED
    fused = _good()
    fused.activation = h2.HUGE2_ACT_RELU  # the gradient of a fused activation is not built
    assert L.huge2_wgrad_plan_create(ctypes.byref(plan), ctypes.byref(fused), 1) == h2.HUGE2_ERR_UNSUPPORTED
    assert L.huge2_wgrad_execute(None, fake, fake, other, None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_wgrad_plan_destroy(None) == h2.HUGE2_OK
    # one-shot forms: NULL and aliased pointers, before any allocation
    assert L.huge2_conv2d_transpose_wgrad(ctypes.byref(d), None, fake, other, None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_conv2d_transpose_wgrad(ctypes.byref(d), fake, other, fake, None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_conv2d_dilated_wgrad(ctypes.byref(d), fake, other, other, None) == h2.HUGE2_ERR_INVALID_ARG
    monkeypatch.setenv("HUGE2_FAULT", "alloc")
    assert L.huge2_wgrad_plan_create(ctypes.byref(plan), ctypes.byref(d), 1) == h2.HUGE2_ERR_ALLOC
    assert plan.value is None


def test_group_entry_points_validate_without_gpu(L):
    """Grouped launches reject NULL and out-of-range arguments before any HIP call."""
    import ctypes
    out = ctypes.c_void_p()
    assert L.huge2_group_create(None, None, 1, None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_group_create(ctypes.byref(out), None, 1, None) == h2.HUGE2_ERR_INVALID_ARG
    arr = (ctypes.c_void_p * 1)(None)
    assert L.huge2_group_create(ctypes.byref(out), arr, 1, None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_group_create(ctypes.byref(out), arr, 0, None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_group_create(ctypes.byref(out), arr, 9, None) == h2.HUGE2_ERR_INVALID_ARG
    assert out.value is None
    assert L.huge2_group_execute(None, None, None, None, None) == h2.HUGE2_ERR_INVALID_ARG
    assert L.huge2_group_destroy(None) == h2.HUGE2_OK
    assert h2.huge2_group_kernel(None) == ""


def test_groups_validated_without_gpu(L):
    """groups must divide both channel counts; grouped layers have no weight
    gradient and their MAC count is the ungrouped one over groups."""
    import ctypes
    d = h2.make_desc(1, 6, 5, 5, 4, 3, 3, 2, 1, 0, 1, h2.HUGE2_NHWC, h2.HUGE2_BF16)
    full = h2.huge2_plan_macs(d, 1)[0]
    d.groups = 2
    assert h2.huge2_plan_macs(d, 1) == (full // 2, full // 2)
    for bad in (4, -1):
        d.groups = bad
        nz, iss = ctypes.c_int64(), ctypes.c_int64()
        assert L.huge2_plan_macs(ctypes.byref(d), 1, ctypes.byref(nz), ctypes.byref(iss)) == \
            h2.HUGE2_ERR_INVALID_ARG
    d.groups = 2
    p = ctypes.c_void_p()
    assert L.huge2_wgrad_plan_create(ctypes.byref(p), ctypes.byref(d), 1) in (
        h2.HUGE2_ERR_UNSUPPORTED, h2.HUGE2_ERR_INVALID_ARG)


def test_dgrad_output_padding_without_gpu(L):
    """The output padding that carries a strided conv's output size back to
    its input size: the transposed conv with it has exactly the input's size,
    and it is a valid output padding, over a sweep of shapes."""
    import numpy as np
    rng = np.random.default_rng(3)
    checked = 0
    for _ in range(300):
        h, w = int(rng.integers(1, 40)), int(rng.integers(1, 40))
        r, s = int(rng.integers(1, 6)), int(rng.integers(1, 6))
        st, dl = int(rng.integers(1, 5)), int(rng.integers(1, 4))
        pd = int(rng.integers(0, dl * (r - 1) + 1))
        conv = h2.make_desc(2, 8, h, w, 4, r, s, st, pd, 0, dl)
        try:
            ho, wo = h2.huge2_output_shape(conv, 0)
        except h2.Huge2Error:
            continue
        oph, opw = h2.huge2_dgrad_output_padding(conv)
        assert 0 <= oph < max(st, dl) and 0 <= opw < max(st, dl), (h, w, r, s, st, pd, dl)
        tr = h2.make_desc(2, 4, ho, wo, 8, r, s, st, pd, (oph, opw), dl)
        assert h2.huge2_output_shape(tr, 1) == (h, w)
        checked += 1
    assert checked > 100


def test_pyramid_plans_take_the_listed_form(L):
    """The atrous pyramid's four branches plan the listed form: the tiles'
    issued multiply-adds stay within 6% of the structural ones (the masked
    phase views issue 14% / 30% / 51% / 78% more for d = 6 / 12 / 18 / 24)."""
    for d in (6, 12, 18, 24):
        desc = h2.make_desc(8, 2048, 64, 64, 256, 3, 3, 1, d, 0, d, h2.HUGE2_NHWC, h2.HUGE2_BF16)
        nz, issued = h2.huge2_plan_macs(desc, 0)
        assert nz <= issued <= 1.06 * nz, (d, nz, issued)
