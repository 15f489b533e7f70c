"""Pins for the CPU oracle (CPU only).

The oracle is the parity authority for the GPU path, so it is pinned here to
things other than itself:

* hand-worked 1-channel examples derived from the definitions (tests/golden/);
* an independent library routine (torch CPU, float64) over a seeded sweep;
* the adjoint identity <T x, z> = <x, C z> between the zero-insertion code
  (transposed conv) and the gather code (strided conv);
* the dense-matrix identity A_T == A_C^T, bitwise;
* closed forms: the sum invariant, stride 1 = full convolution (scipy),
  dilation 1 = correlation (scipy), dilation = zero-inserted kernel,
  bilinear partition of unity;
* per-element evaluation against the full tensor.
"""
import glob
import json
import os

import numpy as np
import pytest
import scipy.signal
import torch

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_cases():
    return sorted(glob.glob(os.path.join(GOLDEN, "*.json")))


def _golden_of(kind):
    out = []
    for path in _golden_cases():
        with open(path) as f:
            op = json.load(f)["op"]
        k = "wgrad" if op.endswith("_wgrad") else "grouped" if op.endswith("_grouped") else "forward"
        if k == kind:
            out.append(path)
    return out


@pytest.mark.parametrize("path", _golden_of("forward"), ids=lambda p: os.path.basename(p)[:-5])
def test_golden_examples(oracle_mod, path):
    with open(path) as f:
        g = json.load(f)
    assert g["citation"]
    x = np.array(g["x"], dtype=np.float64)[None, None]
    w = np.array(g["w"], dtype=np.float64)[None, None]
    exp = np.array(g["expected"], dtype=np.float64)
    if g["op"] == "transpose":
        y = oracle_mod.conv2d_transpose_alg1(x, w, None, g["stride"], g["padding"],
                                             g["output_padding"], g["dilation"], nthreads=1)
    else:
        y = oracle_mod.conv2d_dilated_alg2(x, w, None, g["stride"], g["padding"], g["dilation"],
                                           nthreads=1)
    assert y.shape[2:] == exp.shape
    np.testing.assert_array_equal(y[0, 0], exp)


@pytest.mark.parametrize("path", _golden_of("grouped"), ids=lambda p: os.path.basename(p)[:-5])
def test_golden_grouped(oracle_mod, path):
    """Hand-worked grouped and depthwise cases: multi-channel fixtures whose
    expected outputs fail if a group reads another group's channels or the
    weight of the wrong in-group channel."""
    with open(path) as f:
        g = json.load(f)
    assert g["citation"]
    x = np.array(g["x"], dtype=np.float64)[None]
    w = np.array(g["w"], dtype=np.float64)
    exp = np.array(g["expected"], dtype=np.float64)
    if g["op"] == "transpose_grouped":
        y = oracle_mod.conv2d_transpose_alg1(x, w, None, g["stride"], g["padding"],
                                             g["output_padding"], g["dilation"], nthreads=1,
                                             groups=g["groups"])
    else:
        y = oracle_mod.conv2d_dilated_alg2(x, w, None, g["stride"], g["padding"], g["dilation"],
                                           nthreads=1, groups=g["groups"])
    np.testing.assert_array_equal(y[0], exp)


def _block_diagonal(w, groups, transposed):
    """The ungrouped weight array equal to a grouped one: zero wherever the
    input and output channel lie in different groups."""
    if transposed:
        c_in, cog = w.shape[:2]
        full = np.zeros((c_in, cog * groups) + w.shape[2:])
        cig = c_in // groups
        for c in range(c_in):
            g = c // cig
            full[c, g * cog:(g + 1) * cog] = w[c]
    else:
        c_out, cig = w.shape[:2]
        full = np.zeros((c_out, cig * groups) + w.shape[2:])
        cog = c_out // groups
        for k in range(c_out):
            g = k // cog
            full[k, g * cig:(g + 1) * cig] = w[k]
    return full


@pytest.mark.parametrize("transposed", [True, False])
def test_grouped_equals_block_diagonal(oracle_mod, transposed):
    """A grouped conv is the ungrouped conv whose weight is block diagonal
    over the groups (the ungrouped loops check the grouped indexing), over
    random shapes, strides, paddings and dilations, depthwise included."""
    rng = np.random.default_rng(7 if transposed else 8)
    for _ in range(12):
        groups = int(rng.choice([2, 3, 4]))
        cig, cog = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        n, h, w = int(rng.integers(1, 3)), int(rng.integers(2, 7)), int(rng.integers(2, 7))
        r = int(rng.integers(1, 5))
        st, dl = int(rng.integers(1, 4)), int(rng.integers(1, 3))
        pd = int(rng.integers(0, dl * (r - 1) + 1))
        x = rng.standard_normal((n, cig * groups, h, w))
        b = rng.standard_normal(cog * groups)
        if transposed:
            op = int(rng.integers(0, max(st, dl)))
            wt = rng.standard_normal((cig * groups, cog, r, r))
            y = oracle_mod.conv2d_transpose_alg1(x, wt, b, st, pd, op, dl, groups=groups)
            y0 = oracle_mod.conv2d_transpose_alg1(x, _block_diagonal(wt, groups, True), b, st, pd,
                                                  op, dl)
        else:
            if h + 2 * pd - dl * (r - 1) - 1 < 0 or w + 2 * pd - dl * (r - 1) - 1 < 0:
                continue
            wt = rng.standard_normal((cog * groups, cig, r, r))
            y = oracle_mod.conv2d_dilated_alg2(x, wt, b, st, pd, dl, groups=groups)
            y0 = oracle_mod.conv2d_dilated_alg2(x, _block_diagonal(wt, groups, False), b, st, pd, dl)
        np.testing.assert_allclose(y, y0, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("transposed", [True, False])
def test_grouped_matches_torch(oracle_mod, transposed):
    """torch.nn.functional.conv_transpose2d / conv2d with groups=, float64 on
    the CPU, over a sweep that includes depthwise layers with multipliers."""
    rng = np.random.default_rng(9 if transposed else 10)
    cases = [(2, 3, 2), (4, 1, 1), (3, 2, 4), (6, 1, 3)]  # (groups, C_in/groups, C_out/groups)
    for groups, cig, cog in cases:
        x = rng.standard_normal((2, cig * groups, 6, 5))
        if transposed:
            w = rng.standard_normal((cig * groups, cog, 3, 4))
            y = oracle_mod.conv2d_transpose_alg1(x, w, None, (2, 3), (1, 2), (1, 0), (1, 1),
                                                 groups=groups)
            t = torch.nn.functional.conv_transpose2d(torch.from_numpy(x), torch.from_numpy(w), None,
                                                     (2, 3), (1, 2), (1, 0), groups, (1, 1))
        else:
            w = rng.standard_normal((cog * groups, cig, 3, 3))
            y = oracle_mod.conv2d_dilated_alg2(x, w, None, (1, 2), (2, 1), (2, 1), groups=groups)
            t = torch.nn.functional.conv2d(torch.from_numpy(x), torch.from_numpy(w), None, (1, 2),
                                           (2, 1), (2, 1), groups)
        np.testing.assert_allclose(y, t.numpy(), rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("path", _golden_of("wgrad"), ids=lambda p: os.path.basename(p)[:-5])
def test_golden_weight_gradients(oracle_mod, path):
    with open(path) as f:
        g = json.load(f)
    assert g["citation"]
    groups = g.get("groups", 1)
    if groups > 1:  # multi-channel fixtures: [C][H][W] maps, the whole gradient
        x = np.array(g["x"], dtype=np.float64)[None]
        dy = np.array(g["dy"], dtype=np.float64)[None]
    else:
        x = np.array(g["x"], dtype=np.float64)[None, None]
        dy = np.array(g["dy"], dtype=np.float64)[None, None]
    if g["op"].startswith("transpose"):
        dw = oracle_mod.conv2d_transpose_wgrad(x, dy, g["w_shape"], g["stride"], g["padding"],
                                               g["output_padding"], g["dilation"], nthreads=1,
                                               groups=groups)
    else:
        dw = oracle_mod.conv2d_dilated_wgrad(x, dy, g["w_shape"], g["stride"], g["padding"],
                                             g["dilation"], nthreads=1, groups=groups)
    exp = np.array(g["expected"], dtype=np.float64)
    np.testing.assert_array_equal(dw if groups > 1 else dw[0, 0], exp)


def _random_case(rng, transposed):
    n = int(rng.integers(1, 3))
    ci, co = int(rng.integers(1, 5)), int(rng.integers(1, 5))
    h, w = int(rng.integers(1, 8)), int(rng.integers(1, 8))
    r, s = int(rng.integers(1, 7)), int(rng.integers(1, 7))
    sh, sw = int(rng.integers(1, 5)), int(rng.integers(1, 5))
    dh, dw = int(rng.integers(1, 4)), int(rng.integers(1, 4))
    ph, pw = int(rng.integers(0, dh * (r - 1) + 1)), int(rng.integers(0, dw * (s - 1) + 1))
    if transposed:
        oph, opw = int(rng.integers(0, max(sh, dh))), int(rng.integers(0, max(sw, dw)))
    else:
        oph = opw = 0
    return dict(n=n, ci=ci, co=co, h=h, w=w, r=r, s=s, stride=(sh, sw), pad=(ph, pw),
                op=(oph, opw), dil=(dh, dw))


def test_transpose_matches_torch_sweep(oracle_mod):
    rng = np.random.default_rng(1234)
    checked = 0
    for _ in range(400):
        c = _random_case(rng, True)
        x = rng.standard_normal((c["n"], c["ci"], c["h"], c["w"]))
        w = rng.standard_normal((c["ci"], c["co"], c["r"], c["s"]))
        b = rng.standard_normal(c["co"])
        try:
            ref = torch.nn.functional.conv_transpose2d(
                torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b), stride=c["stride"],
                padding=c["pad"], output_padding=c["op"], dilation=c["dil"]).numpy()
        except RuntimeError:
            continue  # torch rejects (e.g. empty output); the oracle must reject too
        got = oracle_mod.conv2d_transpose_alg1(x, w, b, c["stride"], c["pad"], c["op"], c["dil"],
                                               nthreads=2)
        assert got.shape == ref.shape, c
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12 * max(1.0, np.abs(ref).max()))
        checked += 1
    assert checked > 300


def test_dilated_matches_torch_sweep(oracle_mod):
    rng = np.random.default_rng(4321)
    checked = 0
    for _ in range(400):
        c = _random_case(rng, False)
        x = rng.standard_normal((c["n"], c["ci"], c["h"], c["w"]))
        w = rng.standard_normal((c["co"], c["ci"], c["r"], c["s"]))
        b = rng.standard_normal(c["co"])
        try:
            ref = torch.nn.functional.conv2d(
                torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b), stride=c["stride"],
                padding=c["pad"], dilation=c["dil"]).numpy()
        except RuntimeError:
            with pytest.raises(ValueError):
                oracle_mod.conv2d_dilated_alg2(x, w, b, c["stride"], c["pad"], c["dil"])
            continue
        got = oracle_mod.conv2d_dilated_alg2(x, w, b, c["stride"], c["pad"], c["dil"], nthreads=2)
        assert got.shape == ref.shape, c
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12 * max(1.0, np.abs(ref).max()))
        checked += 1
    assert checked > 150


ADJOINT_CASES = [
    # (n, ci, co, h, w, r, s, stride, pad, out_pad, dil)
    (1, 2, 3, 4, 5, 3, 3, (2, 2), (1, 1), (1, 1), (1, 1)),
    (2, 3, 2, 5, 4, 5, 5, (2, 2), (2, 1), (1, 0), (2, 2)),
    (1, 1, 2, 3, 3, 8, 8, (4, 4), (2, 2), (0, 0), (1, 1)),
    (1, 2, 2, 6, 3, 4, 4, (2, 3), (1, 1), (0, 2), (1, 1)),
    (2, 2, 3, 4, 4, 3, 2, (1, 1), (0, 1), (0, 0), (3, 2)),
]


@pytest.mark.parametrize("case", ADJOINT_CASES)
def test_adjoint_identity(oracle_mod, case):
    """<T x, z> == <x, C z>: the zero-insertion transposed conv (Algorithm 1) is
    the adjoint of the strided conv computed by direct gather (Algorithm 2 code).
    The same weight array serves as the conv's [C_out=C_in_T, C_in=C_out_T, R, S]."""
    n, ci, co, h, w_, r, s, st, pd, op, dl = case
    rng = np.random.default_rng(7)
    x = rng.standard_normal((n, ci, h, w_))
    w = rng.standard_normal((ci, co, r, s))
    tx = oracle_mod.conv2d_transpose_alg1(x, w, None, st, pd, op, dl)
    z = rng.standard_normal(tx.shape)
    cz = oracle_mod.conv2d_dilated_alg2(z, w, None, st, pd, dl)
    assert cz.shape == x.shape
    lhs, rhs = float(np.sum(tx * z)), float(np.sum(x * cz))
    assert abs(lhs - rhs) <= 1e-12 * (np.abs(tx).sum() * np.abs(z).max() + 1.0)


@pytest.mark.parametrize("case", ADJOINT_CASES[:4])
def test_dense_matrix_transpose_bitwise(oracle_mod, case):
    """Build both operators' dense matrices from basis vectors: A_T == A_C^T
    exactly, because each (input, output) pair meets at most one kernel tap."""
    n, ci, co, h, w_, r, s, st, pd, op, dl = case
    n = 1
    rng = np.random.default_rng(11)
    w = rng.integers(-8, 9, size=(ci, co, r, s)).astype(np.float64) + 0.25
    ho, wo = oracle_mod.transpose_out_dims((n, ci, h, w_), w.shape, st, pd, op, dl)
    nin, nout = ci * h * w_, co * ho * wo
    eye_in = np.eye(nin).reshape(nin, 1, ci, h, w_)
    a_t = np.stack([oracle_mod.conv2d_transpose_alg1(e, w, None, st, pd, op, dl).ravel()
                    for e in eye_in], axis=1)  # [nout, nin]
    eye_out = np.eye(nout).reshape(nout, 1, co, ho, wo)
    a_c = np.stack([oracle_mod.conv2d_dilated_alg2(e, w, None, st, pd, dl).ravel()
                    for e in eye_out], axis=1)  # [nin, nout]
    assert a_t.shape == (nout, nin) and a_c.shape == (nin, nout)
    np.testing.assert_array_equal(a_t, a_c.T)
    assert np.count_nonzero(a_t) > 0


def test_sum_invariant(oracle_mod):
    """With no padding and no output padding every product lands inside the
    output, so sum(y) = sum_{c,k} (sum x[:,c]) * (sum w[c,k])."""
    rng = np.random.default_rng(3)
    for st, r, dl in [((2, 2), 4, 1), ((3, 2), 5, 2), ((1, 1), 3, 1), ((32, 32), 64, 1)]:
        x = rng.standard_normal((2, 3, 3, 4))
        w = rng.standard_normal((3, 2, r, r))
        y = oracle_mod.conv2d_transpose_alg1(x, w, None, st, 0, 0, dl)
        expect = np.einsum("c,ck->", x.sum(axis=(0, 2, 3)), w.sum(axis=(2, 3)))
        assert abs(y.sum() - expect) <= 1e-10 * (1 + abs(expect))


def test_stride1_is_full_convolution(oracle_mod):
    rng = np.random.default_rng(5)
    x = rng.standard_normal((1, 3, 5, 6))
    w = rng.standard_normal((3, 2, 3, 4))
    y = oracle_mod.conv2d_transpose_alg1(x, w, None, 1, 0, 0, 1)
    for k in range(2):
        ref = sum(scipy.signal.convolve2d(x[0, c], w[c, k], mode="full") for c in range(3))
        np.testing.assert_allclose(y[0, k], ref, rtol=1e-12, atol=1e-12)


def test_dilation1_is_correlation_and_dilation_is_zero_inserted_kernel(oracle_mod):
    rng = np.random.default_rng(6)
    x = rng.standard_normal((1, 2, 9, 8))
    w = rng.standard_normal((3, 2, 3, 3))
    y1 = oracle_mod.conv2d_dilated_alg2(x, w, None, 1, 0, 1)
    for k in range(3):
        ref = sum(scipy.signal.correlate2d(x[0, c], w[k, c], mode="valid") for c in range(2))
        np.testing.assert_allclose(y1[0, k], ref, rtol=1e-12, atol=1e-12)
    # dilation d == dilation 1 with a kernel that has d-1 zeros inserted between taps
    d = 3
    wz = np.zeros((3, 2, 1 + d * 2, 1 + d * 2))
    wz[:, :, ::d, ::d] = w
    yd = oracle_mod.conv2d_dilated_alg2(x, w, None, 1, 3, d)
    yz = oracle_mod.conv2d_dilated_alg2(x, wz, None, 1, 3, 1)
    np.testing.assert_allclose(yd, yz, rtol=1e-12, atol=1e-12)


def test_points_match_full(oracle_mod):
    rng = np.random.default_rng(8)
    x = rng.standard_normal((2, 3, 5, 4))
    w = rng.standard_normal((3, 4, 5, 3))
    b = rng.standard_normal(4)
    y = oracle_mod.conv2d_transpose_alg1(x, w, b, (2, 3), (2, 1), (1, 2), (1, 1))
    idx = rng.choice(y.size, size=60, replace=False)
    pts = oracle_mod.conv2d_transpose_points(x, w, idx, b, (2, 3), (2, 1), (1, 2), (1, 1))
    np.testing.assert_array_equal(pts, y.ravel()[idx])
    wc = rng.standard_normal((4, 3, 3, 3))
    yc = oracle_mod.conv2d_dilated_alg2(x, wc, b, 1, 2, 2)
    idx = rng.choice(yc.size, size=40, replace=False)
    pts = oracle_mod.conv2d_dilated_points(x, wc, idx, b, 1, 2, 2)
    np.testing.assert_array_equal(pts, yc.ravel()[idx])
    with pytest.raises(ValueError):
        oracle_mod.conv2d_dilated_points(x, wc, np.array([yc.size]), b, 1, 2, 2)


def test_bilinear_partition_of_unity(oracle_mod):
    """FCN-style bilinear upsampling (kernel 2s, stride s, pad s/2): with
    f[m] = (2 min(m, 2s-1-m) + 1) / (2s), f[r] + f[r+s] = 1, so a constant input
    reproduces itself exactly on the interior of the output."""
    s = 8
    f = (2 * np.minimum(np.arange(2 * s), 2 * s - 1 - np.arange(2 * s)) + 1) / (2.0 * s)
    np.testing.assert_array_equal(f[:s] + f[s:], np.ones(s))
    w = np.zeros((2, 2, 2 * s, 2 * s))
    for c in range(2):
        w[c, c] = np.outer(f, f)
    x = np.full((1, 2, 4, 4), 3.0)
    y = oracle_mod.conv2d_transpose_alg1(x, w, None, s, s // 2, 0, 1)
    assert y.shape == (1, 2, 4 * s, 4 * s)
    inner = y[:, :, s // 2: 4 * s - s // 2, s // 2: 4 * s - s // 2]
    np.testing.assert_array_equal(inner, np.full(inner.shape, 3.0))


@pytest.mark.parametrize("bad", [
    dict(stride=0), dict(dilation=0), dict(padding=-1), dict(output_padding=2),
    dict(padding=9),
])
def test_invalid_descriptors_rejected(oracle_mod, bad):
    x = np.ones((1, 1, 2, 2))
    w = np.ones((1, 1, 3, 3))
    kw = dict(stride=2, padding=0, output_padding=0, dilation=1)
    kw.update(bad)
    with pytest.raises(ValueError):
        oracle_mod.conv2d_transpose_alg1(x, w, None, **kw)


# ---------------------------------------------------------------------------
# Weight gradients (section 3.2.3)

@pytest.mark.parametrize("transposed", [True, False])
def test_wgrad_inner_product_identity(oracle_mod, transposed):
    """y is linear in the weights, so the gradient of <dy, y(x; w)> is dw
    with <dw, v> = <dy, y(x; v)> for every v: pins the weight gradient to the
    (separately pinned) forward definitions."""
    rng = np.random.default_rng(77 if transposed else 78)
    checked = 0
    for _ in range(60):
        c = _random_case(rng, transposed)
        x = rng.standard_normal((c["n"], c["ci"], c["h"], c["w"]))
        wshape = (c["ci"], c["co"], c["r"], c["s"]) if transposed else (c["co"], c["ci"], c["r"], c["s"])
        v = rng.standard_normal(wshape)
        try:
            if transposed:
                yv = oracle_mod.conv2d_transpose_alg1(x, v, None, c["stride"], c["pad"], c["op"], c["dil"],
                                                      nthreads=2)
            else:
                yv = oracle_mod.conv2d_dilated_alg2(x, v, None, c["stride"], c["pad"], c["dil"], nthreads=2)
        except ValueError:
            continue
        dy = rng.standard_normal(yv.shape)
        if transposed:
            dw = oracle_mod.conv2d_transpose_wgrad(x, dy, wshape, c["stride"], c["pad"], c["op"], c["dil"],
                                                   nthreads=2)
        else:
            dw = oracle_mod.conv2d_dilated_wgrad(x, dy, wshape, c["stride"], c["pad"], c["dil"], nthreads=2)
        lhs, rhs = float(np.sum(dw * v)), float(np.sum(dy * yv))
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, np.sum(np.abs(dw * v)), np.sum(np.abs(dy * yv))), c
        checked += 1
    assert checked >= 30


@pytest.mark.parametrize("transposed", [True, False])
def test_wgrad_matches_torch_autograd(oracle_mod, transposed):
    """An independent library routine: torch CPU autograd in float64."""
    rng = np.random.default_rng(91 if transposed else 92)
    checked = 0
    for _ in range(60):
        c = _random_case(rng, transposed)
        x = rng.standard_normal((c["n"], c["ci"], c["h"], c["w"]))
        wshape = (c["ci"], c["co"], c["r"], c["s"]) if transposed else (c["co"], c["ci"], c["r"], c["s"])
        w = torch.tensor(rng.standard_normal(wshape), requires_grad=True)
        try:
            if transposed:
                y = torch.nn.functional.conv_transpose2d(torch.from_numpy(x), w, stride=c["stride"],
                                                         padding=c["pad"], output_padding=c["op"],
                                                         dilation=c["dil"])
            else:
                y = torch.nn.functional.conv2d(torch.from_numpy(x), w, stride=c["stride"], padding=c["pad"],
                                               dilation=c["dil"])
        except RuntimeError:
            continue
        if y.numel() == 0:
            continue
        dy = rng.standard_normal(tuple(y.shape))
        (y * torch.from_numpy(dy)).sum().backward()
        if transposed:
            got = oracle_mod.conv2d_transpose_wgrad(x, dy, wshape, c["stride"], c["pad"], c["op"], c["dil"],
                                                    nthreads=2)
        else:
            got = oracle_mod.conv2d_dilated_wgrad(x, dy, wshape, c["stride"], c["pad"], c["dil"], nthreads=2)
        np.testing.assert_allclose(got, w.grad.numpy(), rtol=1e-10, atol=1e-10)
        checked += 1
    assert checked >= 30


@pytest.mark.parametrize("transposed", [True, False])
def test_grouped_wgrad_matches_torch_autograd(oracle_mod, transposed):
    """Grouped and depthwise weight gradients against torch CPU autograd in
    float64 (an independent routine), and the inner-product identity with
    the separately pinned grouped forward definitions."""
    rng = np.random.default_rng(93 if transposed else 94)
    checked = depthwise = 0
    for _ in range(80):
        c = _random_case(rng, transposed)
        g = int(rng.integers(2, 5))
        cig, cog = int(rng.integers(1, 4)), int(rng.integers(1, 4))
        if rng.random() < 0.4:
            cig = 1  # depthwise (with a channel multiplier cog)
        ci, co = g * cig, g * cog
        x = rng.standard_normal((c["n"], ci, c["h"], c["w"]))
        wshape = (ci, cog, c["r"], c["s"]) if transposed else (co, cig, c["r"], c["s"])
        w = torch.tensor(rng.standard_normal(wshape), requires_grad=True)
        try:
            if transposed:
                y = torch.nn.functional.conv_transpose2d(torch.from_numpy(x), w, stride=c["stride"],
                                                         padding=c["pad"], output_padding=c["op"],
                                                         dilation=c["dil"], groups=g)
            else:
                y = torch.nn.functional.conv2d(torch.from_numpy(x), w, stride=c["stride"],
                                               padding=c["pad"], dilation=c["dil"], groups=g)
        except RuntimeError:
            continue
        if y.numel() == 0:
            continue
        dy = rng.standard_normal(tuple(y.shape))
        (y * torch.from_numpy(dy)).sum().backward()
        v = rng.standard_normal(wshape)
        if transposed:
            got = oracle_mod.conv2d_transpose_wgrad(x, dy, wshape, c["stride"], c["pad"], c["op"],
                                                    c["dil"], nthreads=2, groups=g)
            yv = oracle_mod.conv2d_transpose_alg1(x, v, None, c["stride"], c["pad"], c["op"],
                                                  c["dil"], nthreads=2, groups=g)
        else:
            got = oracle_mod.conv2d_dilated_wgrad(x, dy, wshape, c["stride"], c["pad"], c["dil"],
                                                  nthreads=2, groups=g)
            yv = oracle_mod.conv2d_dilated_alg2(x, v, None, c["stride"], c["pad"], c["dil"],
                                                nthreads=2, groups=g)
        np.testing.assert_allclose(got, w.grad.numpy(), rtol=1e-10, atol=1e-10)
        lhs, rhs = float(np.sum(got * v)), float(np.sum(dy * yv))
        assert abs(lhs - rhs) <= 1e-12 * max(1.0, np.sum(np.abs(got * v)), np.sum(np.abs(dy * yv)))
        checked += 1
        depthwise += cig == 1
    assert checked >= 30 and depthwise >= 8


@pytest.mark.parametrize("act", ["relu", "tanh"])
def test_activation_matches_torch(oracle_mod, act):
    """The generator's fused activations against torch's own functions on a
    transposed conv (bias included) in float64, and the identity for none."""
    rng = np.random.default_rng(7)
    x = rng.standard_normal((2, 5, 6, 7))
    w = rng.standard_normal((5, 3, 4, 4)) * 0.3
    b = rng.standard_normal(3)
    y = oracle_mod.conv2d_transpose_alg1(x, w, b, 2, 1, 0, 1)
    ref = torch.nn.functional.conv_transpose2d(torch.from_numpy(x), torch.from_numpy(w),
                                               torch.from_numpy(b), stride=2, padding=1)
    ref = torch.relu(ref) if act == "relu" else torch.tanh(ref)
    got = oracle_mod.activate(y, act)
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-12, atol=1e-12)
    assert (got >= 0).all() if act == "relu" else (np.abs(got) < 1).all()
    assert oracle_mod.activate(y, "none") is y
    with pytest.raises(ValueError):
        oracle_mod.activate(y, "gelu")
