"""Pins of the CPU oracle against things other than itself (CPU only).

Each test compares the oracle with a result the mathematics fixes independently:
library routines for the special cases (scipy correlation for a depthwise plane,
numpy matmul for a 1x1 conv, torch's dense/grouped conv2d in float64 for the
compositions), hand-worked values, exact invariants (identity kernels, power-of-two
homogeneity, layout/batch independence), and exact integer/rational arithmetic for
requantisation. Shapes are non-square with C != C_out so that a transposed operand or a
swapped index fails at least one test.
"""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.signal
import torch
import torch.nn.functional as F

import oracle
from paper_2404_19331_amd.workloads import Case, make_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _nchw(a, layout):
    return a if layout == "nchw" else np.transpose(a, (0, 3, 1, 2))


def _to_layout(a, layout):
    a = np.ascontiguousarray(a)
    return a if layout == "nchw" else np.ascontiguousarray(np.transpose(a, (0, 2, 3, 1)))


def _rand(rng, shape):
    return rng.standard_normal(shape)


def _bf16_np(a):
    t = torch.from_numpy(np.asarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def _bf16_to_f32(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------------------
# Depthwise and pointwise layers against library routines (float64, exact mode)
# --------------------------------------------------------------------------------------

DW_GEOMS = [(3, 1, 1), (3, 2, 1), (3, 1, 0), (5, 1, 2), (5, 2, 2), (5, 2, 1), (2, 1, 0), (1, 1, 0), (7, 2, 3)]


@pytest.mark.parametrize("k,s,p", DW_GEOMS)
@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
def test_dw_matches_scipy_correlate(k, s, p, layout):
    rng = np.random.default_rng(100 + 10 * k + s + p)
    n, c, h, w = 2, 3, 9, 7
    if h + 2 * p < k:
        pytest.skip("degenerate")
    x = _rand(rng, (n, c, h, w))
    wd = _rand(rng, (c, k, k))
    bd = _rand(rng, (c,))
    case = dict(n=n, h=h, w=w, c_in=c, c_mid=c, c_out=c, k=k, stride=s, pad=p, dtype="f64",
                layout=layout, act=["none"] * 3)
    y = _nchw(oracle.dw(case, _to_layout(x, layout), wd, bd), layout)
    for b in range(n):
        for ch in range(c):
            xp = np.pad(x[b, ch], p)
            ref = scipy.signal.correlate2d(xp, wd[ch], mode="valid")[::s, ::s] + bd[ch]
            np.testing.assert_allclose(y[b, ch], ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
def test_pw_matches_matmul(layout):
    rng = np.random.default_rng(7)
    n, c, co, h, w = 2, 5, 3, 4, 6
    x = _rand(rng, (n, c, h, w))
    wp = _rand(rng, (co, c))
    bp = _rand(rng, (co,))
    case = dict(n=n, h=h, w=w, c_in=c, c_mid=c, c_out=co, k=1, stride=1, pad=0, dtype="f64",
                layout=layout)
    y = _nchw(oracle.pw(case, _to_layout(x, layout), wp, bp), layout)
    ref = np.matmul(wp, x.reshape(n, c, h * w)).reshape(n, co, h, w) + bp[None, :, None, None]
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------------------
# Compositions against torch's dense / grouped conv2d in float64
# --------------------------------------------------------------------------------------

@pytest.mark.parametrize("k,s,p", [(3, 1, 1), (3, 2, 1), (5, 2, 2), (5, 1, 2)])
def test_dw_pw_equals_dense_conv(k, s, p):
    """With no activation between them, DW then PW equals one standard convolution
    with W[o,c,u,v] = P[o,c] * Wd[c,u,v]; a DW bias folds into the PW bias."""
    rng = np.random.default_rng(11 + k + s)
    n, c, co, h, w = 2, 4, 6, 10, 8
    x = _rand(rng, (n, c, h, w))
    wd, bd = _rand(rng, (c, k, k)), _rand(rng, (c,))
    wp, bp = _rand(rng, (co, c)), _rand(rng, (co,))
    case = dict(n=n, h=h, w=w, c_in=c, c_mid=c, c_out=co, k=k, stride=s, pad=p, dtype="f64",
                layout="nchw", act=["none"] * 3)
    y = oracle.dw_pw(case, x, wd, bd, wp, bp)
    wdense = torch.from_numpy(wp[:, :, None, None] * wd[None, :, :, :])
    beff = torch.from_numpy(bp + wp @ bd)
    ref = F.conv2d(torch.from_numpy(x), wdense, beff, stride=s, padding=p).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("act", [("relu", "relu"), ("relu6", "none"), ("none", "relu6")])
def test_dw_pw_with_activation_matches_torch(act):
    rng = np.random.default_rng(12)
    n, c, co, h, w, k, s, p = 1, 4, 5, 7, 9, 3, 2, 1
    x = _rand(rng, (n, c, h, w)) * 4
    wd, bd = _rand(rng, (c, k, k)), _rand(rng, (c,))
    wp, bp = _rand(rng, (co, c)), _rand(rng, (co,))
    case = dict(n=n, h=h, w=w, c_in=c, c_mid=c, c_out=co, k=k, stride=s, pad=p, dtype="f64",
                layout="nchw", act=list(act) + ["none"])
    y = oracle.dw_pw(case, x, wd, bd, wp, bp)
    acts = {"none": lambda t: t, "relu": F.relu, "relu6": F.relu6}
    t = F.conv2d(torch.from_numpy(x), torch.from_numpy(wd[:, None]), torch.from_numpy(bd),
                 stride=s, padding=p, groups=c)
    t = acts[act[0]](t)
    t = F.conv2d(t, torch.from_numpy(wp[:, :, None, None]), torch.from_numpy(bp))
    t = acts[act[1]](t)
    np.testing.assert_allclose(y, t.numpy(), rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("k,s,p", [(3, 1, 1), (3, 2, 1), (5, 2, 2)])
def test_pw_dw_border_is_zero_not_activated_bias(k, s, p):
    """PW->DW: the DW zero-pads its own input, so intermediate positions outside the
    image are 0 even when act(PW bias) != 0 (ReLU6 with positive biases)."""
    rng = np.random.default_rng(13)
    n, ci, cm, h, w = 2, 3, 5, 8, 6
    x = _rand(rng, (n, ci, h, w))
    wp, bp = _rand(rng, (cm, ci)), np.abs(_rand(rng, (cm,))) + 0.5
    wd, bd = _rand(rng, (cm, k, k)), _rand(rng, (cm,))
    case = dict(n=n, h=h, w=w, c_in=ci, c_mid=cm, c_out=cm, k=k, stride=s, pad=p, dtype="f64",
                layout="nchw", act=["relu6", "relu", "none"])
    y = oracle.pw_dw(case, x, wp, bp, wd, bd)
    e = F.relu6(F.conv2d(torch.from_numpy(x), torch.from_numpy(wp[:, :, None, None]), torch.from_numpy(bp)))
    ref = F.relu(F.conv2d(e, torch.from_numpy(wd[:, None]), torch.from_numpy(bd), stride=s,
                          padding=p, groups=cm)).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-11)
    # the wrong reading (pad with act(bias)) differs at the border
    e_wrong = F.pad(e, (p, p, p, p), value=0.0)
    e_wrong[:, :, :p, :] = F.relu6(torch.from_numpy(bp))[None, :, None, None]
    wrong = F.relu(F.conv2d(e_wrong, torch.from_numpy(wd[:, None]), torch.from_numpy(bd), stride=s,
                            groups=cm)).numpy()
    assert np.max(np.abs(wrong - y)) > 1e-3


def test_pw_dw_equals_dense_conv_without_activation():
    rng = np.random.default_rng(14)
    n, ci, cm, h, w, k, s, p = 1, 4, 6, 7, 8, 3, 2, 1
    x = _rand(rng, (n, ci, h, w))
    wp, wd = _rand(rng, (cm, ci)), _rand(rng, (cm, k, k))
    case = dict(n=n, h=h, w=w, c_in=ci, c_mid=cm, c_out=cm, k=k, stride=s, pad=p, dtype="f64",
                layout="nchw", act=["none"] * 3)
    y = oracle.pw_dw(case, x, wp, None, wd, None)
    wdense = torch.from_numpy(wd[:, None, :, :] * wp[:, :, None, None])  # [cm, ci, k, k]
    ref = F.conv2d(torch.from_numpy(x), wdense, stride=s, padding=p).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
def test_pw_pw_without_activation_is_one_pw_with_composed_weights(layout):
    """Two linear 1x1 convolutions compose into one: W = W2 W1, b = W2 b1 + b2 (float64
    exact mode, torch's conv2d as the reference)."""
    rng = np.random.default_rng(16)
    n, ci, cm, co, h, w = 2, 5, 9, 4, 6, 7
    x = _rand(rng, (n, ci, h, w))
    w1, w2 = _rand(rng, (cm, ci)), _rand(rng, (co, cm))
    b1, b2 = _rand(rng, cm), _rand(rng, co)
    case = dict(n=n, h=h, w=w, c_in=ci, c_mid=cm, c_out=co, k=1, stride=1, pad=0, dtype="f64", layout=layout,
                act=["none"] * 3)
    y = _nchw(oracle.pw_pw(case, _to_layout(x, layout), w1, b1, w2, b2), layout)
    ref = F.conv2d(torch.from_numpy(x), torch.from_numpy((w2 @ w1)[:, :, None, None]),
                   torch.from_numpy(w2 @ b1 + b2)).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("act", [("relu", "none"), ("none", "relu")])
def test_pw_pw_int8_matches_integer_reference(act):
    """int8 PW -> PW against numpy int64 matmuls and a round-half-even requantisation
    (np.round on exactly representable quotients), saturated per stage."""
    rng = np.random.default_rng(17)
    n, ci, cm, co, h, w = 2, 40, 72, 24, 5, 6
    rq = ((3, 4, -127, 127), (5, 7, -128, 127), (1, 0, -128, 127))
    # small magnitudes keep most results inside the int8 range (saturation is exercised too)
    x = rng.integers(-8, 9, (n, h, w, ci)).astype(np.int8)
    w1 = rng.integers(-8, 9, (cm, ci)).astype(np.int8)
    w2 = rng.integers(-8, 9, (co, cm)).astype(np.int8)
    b1 = rng.integers(-500, 500, cm).astype(np.int32)
    b2 = rng.integers(-500, 500, co).astype(np.int32)
    case = dict(n=n, h=h, w=w, c_in=ci, c_mid=cm, c_out=co, k=1, stride=1, pad=0, dtype="i8", layout="nhwc",
                act=list(act) + ["none"], rq=list(rq))

    def stage(t, wt, b, r, a):
        acc = t.astype(np.int64) @ wt.astype(np.int64).T + b.astype(np.int64)
        q = np.round(acc.astype(np.float64) * r[0] / 2.0 ** r[1])
        lo, hi = (max(r[2], 0), max(r[3], 0)) if a == "relu" else (r[2], r[3])
        return np.clip(q, lo, hi).astype(np.int8)

    mid = stage(x, w1, b1, rq[0], act[0])
    ref = stage(mid, w2, b2, rq[1], act[1])
    # spread results: mostly inside the int8 range, some saturated, few zeros beyond ReLU's
    assert 0.5 < np.mean(np.abs(ref.astype(int)) < 127) < 1 and np.mean(mid != 0) > 0.4 and np.mean(ref != 0) > 0.4
    y = oracle.pw_pw(case, x, w1, b1, w2, b2)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
def test_pw_dw_pw_matches_torch(layout):
    rng = np.random.default_rng(15)
    n, ci, cm, co, h, w, k, s, p = 2, 3, 8, 5, 9, 7, 3, 1, 1
    x = _rand(rng, (n, ci, h, w)) * 3
    w1, b1 = _rand(rng, (cm, ci)), _rand(rng, (cm,))
    wd, bd = _rand(rng, (cm, k, k)), _rand(rng, (cm,))
    w2, b2 = _rand(rng, (co, cm)), _rand(rng, (co,))
    case = dict(n=n, h=h, w=w, c_in=ci, c_mid=cm, c_out=co, k=k, stride=s, pad=p, dtype="f64",
                layout=layout, act=["relu6", "relu6", "none"])
    y = _nchw(oracle.pw_dw_pw(case, _to_layout(x, layout), w1, b1, wd, bd, w2, b2), layout)
    t = F.relu6(F.conv2d(torch.from_numpy(x), torch.from_numpy(w1[:, :, None, None]), torch.from_numpy(b1)))
    t = F.relu6(F.conv2d(t, torch.from_numpy(wd[:, None]), torch.from_numpy(bd), stride=s, padding=p, groups=cm))
    t = F.conv2d(t, torch.from_numpy(w2[:, :, None, None]), torch.from_numpy(b2))
    np.testing.assert_allclose(y, t.numpy(), rtol=1e-11, atol=1e-11)


# --------------------------------------------------------------------------------------
# Hand-worked examples (tests/golden/hand_dw_examples.txt)
# --------------------------------------------------------------------------------------

def _golden_dw():
    rows = []
    with open(os.path.join(GOLDEN, "hand_dw_examples.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            name, hw, ksp, xs, ws, ys = (t.strip() for t in line.split("|"))
            h, w = map(int, hw.split())
            k, s, p = map(int, ksp.split())
            rows.append((name, h, w, k, s, p, list(map(float, xs.split())),
                         list(map(float, ws.split())), list(map(float, ys.split()))))
    return rows


@pytest.mark.parametrize("row", _golden_dw(), ids=lambda r: r[0])
@pytest.mark.parametrize("dtype", ["f64", "f32", "bf16"])
def test_hand_worked_dw_examples(row, dtype):
    name, h, w, k, s, p, xs, ws, ys = row
    conv = {"f64": np.float64, "f32": np.float32}
    enc = (lambda a: _bf16_np(a)) if dtype == "bf16" else (lambda a: np.asarray(a, conv[dtype]))
    case = dict(n=1, h=h, w=w, c_in=1, c_mid=1, c_out=1, k=k, stride=s, pad=p, dtype=dtype, layout="nchw")
    x = enc(np.array(xs).reshape(1, 1, h, w))
    wd = enc(np.array(ws).reshape(1, k, k))
    y = oracle.dw(case, x, wd, None)
    yv = _bf16_to_f32(y) if dtype == "bf16" else y
    assert yv.ravel().tolist() == ys
    # followed by a 1x1 conv of weight 2: every value doubles
    y2 = oracle.dw_pw(case, x, wd, None, enc(np.array([[2.0]])), None)
    y2v = _bf16_to_f32(y2) if dtype == "bf16" else y2
    assert y2v.ravel().tolist() == [2 * v for v in ys]


# --------------------------------------------------------------------------------------
# Exact invariants
# --------------------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16", "i8"])
@pytest.mark.parametrize("s", [1, 2])
@pytest.mark.parametrize("act", ["none", "relu"])
def test_identity_kernels_are_exact(dtype, s, act):
    """Centre-delta DW and identity PW: y = act(x[:, :, ::s, ::s]) bit-exactly."""
    case = Case("dw_pw", 2, 9, 7, 6, 6, 6, 3, s, 1, dtype, "nchw", (act, act, "none"),
                ((1, 0, -128, 127),) * 3, dist_x="i8" if dtype == "i8" else "n01", seed=5)
    inp = make_inputs(case)
    x = inp["x"]
    one = {"f32": np.float32(1), "bf16": np.uint16(0x3F80), "i8": np.int8(1)}[dtype]
    wd = np.zeros((6, 3, 3), dtype=x.dtype)
    wd[:, 1, 1] = one
    wp = np.zeros((6, 6), dtype=x.dtype)
    np.fill_diagonal(wp, one)
    y = oracle.dw_pw(case, x, wd, None, wp, None)
    ref = x[:, :, ::s, ::s]
    if act == "relu":
        if dtype == "bf16":
            ref = np.where(_bf16_to_f32(ref) > 0, ref, np.uint16(0))
        else:
            ref = np.maximum(ref, 0).astype(x.dtype)
    assert np.array_equal(y, ref)
    # isolated stages: delta DW -> y = PW(x); identity PW -> y = DW(x)
    if dtype != "i8" and act == "none" and s == 1:
        y1 = oracle.dw_pw(case, x, wd, None, inp["w_pw"], None)
        y2 = oracle.pw(case.with_(op="pw", k=1, pad=0), x, inp["w_pw"], None)
        assert np.array_equal(y1, y2)
        y3 = oracle.dw_pw(case, x, inp["w_dw"], None, wp, None)
        y4 = oracle.dw(case.with_(op="dw"), x, inp["w_dw"], None)
        assert np.array_equal(y3, y4)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("op", ["dw_pw", "pw_dw", "pw_dw_pw"])
def test_power_of_two_homogeneity_is_bit_exact(dtype, op):
    """f(2^k x) = 2^k f(x) exactly (act none/relu, biases scaled alike)."""
    case = Case(op, 1, 8, 6, 4, 8 if op != "dw_pw" else 4, 5 if op == "pw_dw_pw" else (8 if op == "pw_dw" else 6),
                3, 1, 1, dtype, "nhwc", ("relu", "relu", "none"), dist_x="n01", bias=True, seed=9)
    inp = make_inputs(case)
    y = oracle.run(op, case, inp)
    scaled = dict(inp)
    if dtype == "f32":
        scaled["x"] = (inp["x"] * np.float32(8)).astype(np.float32)
        yv = y
    else:
        scaled["x"] = _bf16_np(_bf16_to_f32(inp["x"]) * 8)
        yv = _bf16_to_f32(y)
    # every stage then sees 8x inputs with unchanged weights, so every bias scales by 8
    for key in ("b_dw", "b_pw", "b_pw1", "b_pw2"):
        if scaled.get(key) is not None:
            scaled[key] = (scaled[key] * np.float32(8)).astype(np.float32)
    y8 = oracle.run(op, case, scaled)
    y8v = y8 if dtype == "f32" else _bf16_to_f32(y8)
    assert np.array_equal(y8v, (yv * 8).astype(np.float32))


def test_linearity_within_rounding():
    case = Case("dw_pw", 1, 9, 9, 5, 5, 7, 3, 2, 1, "f64", "nchw", dist_x="n01", seed=3)
    a = make_inputs(case)
    b = make_inputs(case, seed=4)
    xa, xb = a["x"], b["x"]
    ya = oracle.dw_pw(case, xa, a["w_dw"], None, a["w_pw"], None)
    yb = oracle.dw_pw(case, xb, a["w_dw"], None, a["w_pw"], None)
    yab = oracle.dw_pw(case, 0.75 * xa - 2.5 * xb, a["w_dw"], None, a["w_pw"], None)
    np.testing.assert_allclose(yab, 0.75 * ya - 2.5 * yb, rtol=1e-12, atol=1e-12)
    # bilinear in (Wd, P)
    yw = oracle.dw_pw(case, xa, 3 * a["w_dw"], None, -2 * a["w_pw"], None)
    np.testing.assert_allclose(yw, -6 * ya, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "i8"])
@pytest.mark.parametrize("op", ["dw_pw", "pw_dw", "pw_dw_pw"])
def test_layout_and_batch_independence(dtype, op):
    rq = ((1, 4, -127, 127),) * 3
    case = Case(op, 3, 7, 10, 6, 6 if op == "dw_pw" else 10, 4 if op != "pw_dw" else 10, 3, 2, 1,
                dtype, "nchw", ("relu", "none", "relu"), rq,
                dist_x="i8small" if dtype == "i8" else "n01", dist_w="i8small", bias=True, seed=21)
    inp = make_inputs(case)
    y = oracle.run(op, case, inp)
    nh = dict(inp)
    nh["x"] = np.ascontiguousarray(np.transpose(inp["x"], (0, 2, 3, 1)))
    y_nhwc = oracle.run(op, case.with_(layout="nhwc"), nh)
    assert np.array_equal(np.transpose(y_nhwc, (0, 3, 1, 2)), y)
    for b in range(case.n):
        one = dict(inp)
        one["x"] = np.ascontiguousarray(inp["x"][b:b + 1])
        assert np.array_equal(oracle.run(op, case.with_(n=1), one), y[b:b + 1])


def test_f32_path_rounds_exact_result_once_per_stage():
    """Single stage: the f32 result is the exact (f64) result rounded to float32."""
    case = Case("dw", 2, 11, 9, 5, 5, 5, 3, 1, 1, "f32", "nchw", dist_x="n01", bias=True, seed=31)
    inp = make_inputs(case)
    y32 = oracle.dw(case, inp["x"], inp["w_dw"], inp["b_dw"])
    c64 = case.with_(dtype="f64")
    y64 = oracle.dw(c64, inp["x"].astype(np.float64), inp["w_dw"].astype(np.float64),
                    inp["b_dw"].astype(np.float64))
    assert np.array_equal(y32, y64.astype(np.float32))


def test_relu6_clamps():
    case = dict(n=1, h=1, w=3, c_in=1, c_mid=1, c_out=1, k=1, stride=1, pad=0, dtype="f64",
                layout="nchw", act=["relu6"] * 3)
    y = oracle.pw(case, np.array([[[[-3.0, 2.5, 9.0]]]]), np.array([[1.0]]), None)
    assert y.ravel().tolist() == [0.0, 2.5, 6.0]


# --------------------------------------------------------------------------------------
# Integer path
# --------------------------------------------------------------------------------------

def _golden_rq():
    rows = []
    with open(os.path.join(GOLDEN, "requant_rne.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            rows.append(tuple(int(t) for t in line.split()))
    return rows


@pytest.mark.parametrize("row", _golden_rq())
def test_requant_table(row):
    acc, mult, shift, qmin, qmax, expected = row
    assert oracle.requant(acc, mult, shift, qmin, qmax) == expected


def _rq_fraction(acc, mult, shift, qmin, qmax):
    q = round(Fraction(acc * mult, 2 ** shift))  # Python rounds half to even
    return max(qmin, min(qmax, q))


def test_requant_exhaustive_against_fraction():
    for shift in (0, 1, 2, 3, 8):
        for mult in (1, 3, 7):
            for acc in range(-1200, 1201):
                assert oracle.requant(acc, mult, shift, -127, 127) == _rq_fraction(acc, mult, shift, -127, 127)
    big = [2 ** 31 - 1, -2 ** 31, 123456789, -987654321]
    for acc in big:
        for mult, shift in ((1, 8), (1073741824, 40), (12345, 20)):
            assert oracle.requant(acc, mult, shift, -128, 127) == _rq_fraction(acc, mult, shift, -128, 127)


def _int_conv_reference(x, wd, bd, wp, bp, k, s, p, rq, acts):
    """DW -> requant -> PW -> requant using float64 conv (exact for these magnitudes)
    and Fraction rounding."""
    t = F.conv2d(torch.from_numpy(x.astype(np.float64)), torch.from_numpy(wd.astype(np.float64)[:, None]),
                 stride=s, padding=p, groups=x.shape[1]).numpy()
    t = np.rint(t).astype(np.int64)
    if bd is not None:
        t = t + bd.astype(np.int64)[None, :, None, None]
    rqv = np.vectorize(lambda a: _rq_fraction(int(a), *rq[0]))
    m = rqv(t)
    if acts[0] == "relu":
        m = np.maximum(m, 0)
    u = F.conv2d(torch.from_numpy(m.astype(np.float64)), torch.from_numpy(wp.astype(np.float64)[:, :, None, None])).numpy()
    u = np.rint(u).astype(np.int64)
    if bp is not None:
        u = u + bp.astype(np.int64)[None, :, None, None]
    y = np.vectorize(lambda a: _rq_fraction(int(a), *rq[1]))(u)
    if acts[1] == "relu":
        y = np.maximum(y, 0)
    return y.astype(np.int8)


@pytest.mark.parametrize("dist,rq", [("i8", (1, 8, -127, 127)), ("i8small", (1, 4, -127, 127)), ("i8", (5, 11, -128, 127))])
@pytest.mark.parametrize("act", [("none", "none"), ("relu", "relu")])
def test_int8_dw_pw_matches_integer_reference(dist, rq, act):
    case = Case("dw_pw", 2, 9, 8, 12, 12, 5, 5, 2, 2, "i8", "nchw", act + ("none",), (rq, rq, rq),
                dist_x=dist, dist_w=dist, bias=True, seed=41)
    inp = make_inputs(case)
    y = oracle.dw_pw(case, inp["x"], inp["w_dw"], inp["b_dw"], inp["w_pw"], inp["b_pw"])
    ref = _int_conv_reference(inp["x"], inp["w_dw"], inp["b_dw"], inp["w_pw"], inp["b_pw"],
                              5, 2, 2, (rq, rq), act)
    assert np.array_equal(y, ref)


def test_int8_saturation_fraction_matches_analysis():
    """U{-127..127} inputs and weights with 5x5 DW and scale 2^-8 saturate heavily
    (analysis: sigma(acc/256) ~ 106, about 23% of DW outputs at +-127)."""
    case = Case("dw", 1, 40, 40, 16, 16, 16, 5, 1, 2, "i8", "nchw", rq=((1, 8, -127, 127),) * 3,
                dist_x="i8", dist_w="i8", seed=42)
    inp = make_inputs(case)
    y = oracle.dw(case, inp["x"], inp["w_dw"], None)
    interior = y[:, :, 2:-2, 2:-2]
    frac = np.mean(np.abs(interior.astype(np.int32)) == 127)
    assert 0.15 < frac < 0.32


def test_int32_overflow_is_reported():
    case = dict(n=1, h=1, w=1, c_in=1, c_mid=1, c_out=1, k=1, stride=1, pad=0, dtype="i8",
                layout="nchw", rq=[(1, 0, -127, 127)] * 3)
    x = np.array([[[[127]]]], dtype=np.int8)
    w = np.array([[127]], dtype=np.int8)
    b = np.array([2 ** 31 - 100], dtype=np.int32)
    with pytest.raises(oracle.OracleError):
        oracle.pw(case, x, w, b)


def test_int8_relu6_is_the_quantised_clamp():
    """int8 ReLU6: clamp to [max(qmin, 0), qmax], qmax holding 6.0 in output units. Worked
    by hand for requantisation by 2^-2 (scale 1/4, so 6.0 is 24): accumulators
    -40, 7, 50, 200 (diagonal weights -1, 1, 1, 2 on inputs 40, 7, 50, 100) give
    rne(-10) = -10, rne(1.75) = 2, rne(12.5) = 12 (ties to even), rne(50) = 50;
    saturated to [-127, 24]: -10, 2, 12, 24; clamped at 0: 0, 2, 12, 24."""
    x = np.array([40, 7, 50, 100], dtype=np.int8).reshape(1, 1, 1, 4)
    w = np.diag([-1, 1, 1, 2]).astype(np.int8)
    base = dict(n=1, h=1, w=1, c_in=4, c_mid=4, c_out=4, k=1, stride=1, pad=0, dtype="i8", layout="nhwc",
                rq=[(1, 2, -127, 24)] * 3)
    got = {a: oracle.pw(dict(base, act=[a] * 3), x, w, None).ravel().tolist() for a in ("none", "relu", "relu6")}
    assert got["none"] == [-10, 2, 12, 24]
    assert got["relu6"] == [0, 2, 12, 24]
    # the same as ReLU with the same range: 6 lives in qmax
    assert got["relu6"] == got["relu"]


# --------------------------------------------------------------------------------------
# bfloat16 rounding
# --------------------------------------------------------------------------------------

def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(51)
    vals = np.concatenate([
        rng.standard_normal(4000).astype(np.float32) * np.float32(3.0),
        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 3.4e38, -3.4e38, 1e-40, 0.0, -0.0,
                  np.inf, -np.inf, 65504.0, 1.00390625, 1.01171875], dtype=np.float32),
    ])
    ref = _bf16_np(vals)
    got = np.array([oracle.bf16_bits(v) for v in vals], dtype=np.uint16)
    assert np.array_equal(got, ref)
    assert oracle.bf16_bits(1.0 + 2 ** -8) == 0x3F80  # tie -> even (down)
    assert oracle.bf16_bits(1.0 + 3 * 2 ** -8) == 0x3F82  # tie -> even (up)
    assert oracle.bf16_bits(3.4e38) == 0x7F80  # rounds up to +inf
    nan = oracle.bf16_bits(float("nan"))
    assert (nan & 0x7F80) == 0x7F80 and (nan & 0x7F) != 0


@pytest.mark.parametrize("dtype", ["f32", "bf16", "i8"])
@pytest.mark.parametrize("op", ["dw_pw", "pw_dw", "pw_dw_pw", "pw_pw"])
def test_module_equals_chain_of_single_layers(dtype, op):
    """A module computes exactly its layer-by-layer chain: each stage's output is cast to
    the storage precision before the next stage reads it (fusion moves data only). Each
    single layer is pinned above (exact result rounded once), so this pins the
    intermediate casts."""
    rq = ((1, 6, -127, 127), (3, 9, -127, 127), (1, 7, -127, 127))
    cm = 6 if op == "dw_pw" else 9
    co = {"dw_pw": 5, "pw_dw": 9, "pw_dw_pw": 4, "pw_pw": 7}[op]
    case = Case(op, 2, 9, 8, 6, cm, co, 3, 2, 1, dtype, "nhwc", ("relu", "relu6" if dtype != "i8" else "none", "relu"),
                rq, dist_x="i8small" if dtype == "i8" else "n01", dist_w="i8small", bias=True, seed=61)
    inp = make_inputs(case)
    y = oracle.run(op, case, inp)
    base = dict(n=2, dtype=dtype, layout="nhwc")

    def stage_dw(t, h, w, c, wd, bd, i):
        return oracle.dw(dict(base, h=h, w=w, c_in=c, c_mid=c, c_out=c, k=3, stride=2, pad=1,
                              act=[case.act[i]] * 3, rq=[rq[i]] * 3), t, wd, bd)

    def stage_pw(t, h, w, ci, co_, wp, bp, i):
        return oracle.pw(dict(base, h=h, w=w, c_in=ci, c_mid=co_, c_out=co_, k=1, stride=1, pad=0,
                              act=[case.act[i]] * 3, rq=[rq[i]] * 3), t, wp, bp)

    ho, wo = oracle.out_hw(9, 8, 3, 2, 1)
    if op == "dw_pw":
        m = stage_dw(inp["x"], 9, 8, 6, inp["w_dw"], inp["b_dw"], 0)
        ref = stage_pw(m, ho, wo, 6, co, inp["w_pw"], inp["b_pw"], 1)
    elif op == "pw_dw":
        m = stage_pw(inp["x"], 9, 8, 6, cm, inp["w_pw"], inp["b_pw"], 0)
        ref = stage_dw(m, 9, 8, cm, inp["w_dw"], inp["b_dw"], 1)
    elif op == "pw_pw":  # spatial size unchanged: k, stride and pad do not apply
        m = stage_pw(inp["x"], 9, 8, 6, cm, inp["w_pw1"], inp["b_pw1"], 0)
        ref = stage_pw(m, 9, 8, cm, co, inp["w_pw2"], inp["b_pw2"], 1)
    else:
        m = stage_pw(inp["x"], 9, 8, 6, cm, inp["w_pw1"], inp["b_pw1"], 0)
        m = stage_dw(m, 9, 8, cm, inp["w_dw"], inp["b_dw"], 1)
        ref = stage_pw(m, ho, wo, cm, co, inp["w_pw2"], inp["b_pw2"], 2)
    assert np.array_equal(y, ref)


# --------------------------------------------------------------------------------------
# int8 per-channel requantisation
# --------------------------------------------------------------------------------------

def _i8_case(op, ci, cm, co, k=3, s=1, acts=("relu", "none", "relu"), layout="nhwc"):
    return dict(op=op, n=2, h=7, w=6, c_in=ci, c_mid=cm, c_out=co, k=k, stride=s, pad=k // 2, dtype="i8",
                layout=layout, act=list(acts), rq=[(1, 6, -127, 127), (3, 8, -128, 127), (1, 5, -127, 127)],
                dist_x="i8small", dist_w="i8small", bias=True, seed=77)


def _i8_inputs(c):
    from paper_2404_19331_amd.workloads import Case, make_inputs
    kw = {k: v for k, v in c.items() if k != "op"}
    return make_inputs(Case(c["op"], **{k: kw[k] for k in ("n", "h", "w", "c_in", "c_mid", "c_out", "k", "stride",
                                                              "pad", "dtype", "layout")}, act=tuple(c["act"]),
                            rq=tuple(c["rq"]), dist_x="i8small", dist_w="i8small", bias=True, seed=c["seed"]))


def _stage_channels(op, c):
    return {"dw_pw": [c["c_in"], c["c_out"]], "pw_dw": [c["c_mid"], c["c_mid"]], "pw_pw": [c["c_mid"], c["c_out"]],
            "pw_dw_pw": [c["c_mid"], c["c_mid"], c["c_out"]], "dw": [c["c_in"]], "pw": [c["c_out"]]}[op]


@pytest.mark.parametrize("op", ["dw_pw", "pw_dw", "pw_pw", "pw_dw_pw", "dw", "pw"])
def test_per_channel_requant_with_equal_channels_is_per_tensor(op):
    c = _i8_case(op, 12, 12 if op in ("dw_pw", "dw") else 20, 12 if op in ("dw", "pw_dw") else 8,
                 k=1 if op in ("pw", "pw_pw") else 3)
    if op == "pw_dw":
        c["c_out"] = c["c_mid"]
    inp = _i8_inputs(c)
    ref = oracle.run(op, c, inp)
    chans = _stage_channels(op, c)
    pc = dict(c, rq_channel=[(np.full(n, r[0]), np.full(n, r[1])) for n, r in zip(chans, c["rq"])])
    assert np.array_equal(oracle.run(op, pc, inp), ref)


def test_per_channel_requant_selects_each_channels_own_scale():
    """A PW layer requantised per output channel equals, channel by channel, the layer run
    with that channel's (mult, shift) as the per-tensor requantisation."""
    c = _i8_case("pw", 16, 16, 6, k=1, acts=("none",) * 3)
    inp = _i8_inputs(c)
    mults, shifts = np.array([1, 3, 5, 1, 7, 2]), np.array([2, 4, 6, 8, 5, 3])
    got = oracle.run("pw", dict(c, rq_channel=[(mults, shifts)]), inp)
    for ch in range(6):
        one = oracle.run("pw", dict(c, rq=[(int(mults[ch]), int(shifts[ch]), -127, 127)] * 3), inp)
        assert np.array_equal(got[..., ch], one[..., ch])
    # not vacuous: one shared scale gives a different result
    shared = oracle.run("pw", dict(c, rq=[(1, 2, -127, 127)] * 3), inp)
    assert not np.array_equal(got, shared) and np.mean(got != 0) > 0.3


def test_per_channel_requant_composes_stage_by_stage():
    """DW -> PW with per-channel requantisation of both stages equals the DW layer and the
    PW layer run one after the other with the same per-channel requantisation."""
    c = _i8_case("dw_pw", 10, 10, 7)
    inp = _i8_inputs(c)
    rng = np.random.default_rng(3)
    pc0 = (rng.integers(1, 8, 10), rng.integers(3, 9, 10))
    pc1 = (rng.integers(1, 8, 7), rng.integers(5, 11, 7))
    fused = oracle.run("dw_pw", dict(c, rq_channel=[pc0, pc1]), inp)
    mid = oracle.dw(dict(c, rq_channel=[pc0]), inp["x"], inp["w_dw"], inp["b_dw"])
    c2 = dict(c, h=mid.shape[1], w=mid.shape[2], c_in=10, c_out=7, act=[c["act"][1]] * 3, rq=[c["rq"][1]] * 3,
              rq_channel=[pc1])
    assert np.array_equal(fused, oracle.pw(c2, mid, inp["w_pw"], inp["b_pw"]))


def test_per_channel_requant_hand_values():
    # one pixel, identity weights on inputs 40 and 50: channel 0 by 3/2^2 -> rne(30) = 30,
    # channel 1 by 1/2^3 -> rne(6.25) = 6
    x = np.array([40, 50], dtype=np.int8).reshape(1, 1, 1, 2)
    w = np.eye(2, dtype=np.int8)
    c = dict(n=1, h=1, w=1, c_in=2, c_mid=2, c_out=2, k=1, stride=1, pad=0, dtype="i8", layout="nhwc",
             act=["none"] * 3, rq=[(1, 0, -127, 127)] * 3, rq_channel=[(np.array([3, 1]), np.array([2, 3]))])
    assert oracle.pw(c, x, w, None).ravel().tolist() == [30, 6]


# --------------------------------------------------------------------------------------
# Asymmetric int8: zero points (a code q stands for scale * (q - zero point))
# --------------------------------------------------------------------------------------

ZP_OPS = ["dw_pw", "pw_dw", "pw_pw", "pw_dw_pw", "dw", "pw"]


def _zp_case(op, **kw):
    c = _i8_case(op, 12, 12 if op in ("dw_pw", "dw") else 20, 12 if op in ("dw", "pw_dw") else 8,
                 k=1 if op in ("pw", "pw_pw") else 3, s=2 if op in ("dw_pw", "pw_dw_pw") else 1)
    if op == "pw_dw":
        c["c_out"] = c["c_mid"]
    c.update(kw)
    return c


@pytest.mark.parametrize("op", ZP_OPS)
def test_input_zero_point_equals_centred_input(op):
    """With input zero point z, every module equals the symmetric (z = 0) module run on the
    centred codes x - z (whenever those fit int8): zero padding means real 0 in both,
    so a padding or centring mistake in any stage shows at the borders."""
    z = 5
    c = _zp_case(op)
    inp = _i8_inputs(c)  # x in [-8, 8], so x + z fits int8
    shifted = dict(inp, x=(inp["x"].astype(np.int16) + z).astype(np.int8))
    got = oracle.run(op, dict(c, zp_in=z), shifted)
    assert np.array_equal(got, oracle.run(op, c, inp))
    # not vacuous: the same codes read as symmetric differ
    assert not np.array_equal(oracle.run(op, c, shifted), got)


@pytest.mark.parametrize("op", ["dw_pw", "pw_dw", "pw_pw", "pw_dw_pw"])
def test_intermediate_zero_point_is_invisible_without_saturation(op):
    """A zero point on an intermediate only relabels its codes: when no intermediate code
    saturates, the module's output does not depend on it (the next stage subtracts what
    the previous one added, and pads with the new code of real 0)."""
    rq = [(1, 9, -128, 127), (1, 9, -128, 127), (1, 5, -128, 127)]
    c = _zp_case(op, rq=rq, act=["relu", "relu", "none"])
    inp = _i8_inputs(c)
    ref = oracle.run(op, c, inp)
    nstages = 3 if op == "pw_dw_pw" else 2
    for zs in ((17,), (-23,), (40, -31)):
        rqz = [tuple(r) + (zs[i] if i < len(zs) and i < nstages - 1 else 0,) for i, r in enumerate(rq)]
        assert np.array_equal(oracle.run(op, dict(c, rq=rqz), inp), ref), zs
    # the intermediates really are small: a wrong centring would move the output
    assert np.abs(ref).max() > 0


@pytest.mark.parametrize("op", ZP_OPS)
@pytest.mark.parametrize("act", ["none", "relu"])
def test_output_zero_point_offsets_the_codes(op, act):
    """Without saturation the output codes move by exactly the output zero point; ReLU
    clamps at the zero point, so it is max(symmetric ReLU output + z, z)."""
    z = -9
    last = {"dw": 0, "pw": 0, "pw_dw_pw": 2}.get(op, 1)
    rq = [(1, 6, -128, 127), (3, 8, -128, 127), (1, 5, -128, 127)]
    acts = ["relu", "none", "relu"]
    acts[last] = act
    c = _zp_case(op, rq=rq, act=acts)
    inp = _i8_inputs(c)
    ref = oracle.run(op, c, inp).astype(np.int32)
    assert ref.max() + z <= 127 and ref.min() + z >= -128
    rqz = [tuple(r) + ((z,) if i == last else (0,)) for i, r in enumerate(rq)]
    got = oracle.run(op, dict(c, rq=rqz), inp).astype(np.int32)
    assert np.array_equal(got, ref + z)
    if act == "relu":
        assert (got >= z).all() and (got == z).any()


def test_zero_point_hand_values():
    """Worked by hand.
    DW 3x3, pad 1, on a 1x1 image: only the centre tap lies inside. Code 10 with input
    zero point 3 is the value 7; centre weight 2 gives 14; output zero point -5 gives code
    9. (Padding with code 0 instead of real 0 would add 8 * 5 * (0 - 3) = -120.)
    PW on one pixel, codes (10, -4) with input zero point 2, i.e. values (8, -6), bias 5,
    requantised by 2^-1 with output zero point -7:
      weights (3, -1):  24 + 6 + 5 = 35  -> rne(17.5) = 18 (tie to even)  -> 11
      weights (-3, 1): -24 - 6 + 5 = -25 -> rne(-12.5) = -12 (tie to even) -> -19,
    which ReLU clamps at the zero point: -7."""
    wd = np.full((1, 3, 3), 5, dtype=np.int8)
    wd[0, 1, 1] = 2
    c = dict(n=1, h=1, w=1, c_in=1, c_mid=1, c_out=1, k=3, stride=1, pad=1, dtype="i8", layout="nchw",
             act=["none"] * 3, rq=[(1, 0, -128, 127, -5)] * 3, zp_in=3)
    assert oracle.dw(c, np.array([[[[10]]]], dtype=np.int8), wd, None).ravel().tolist() == [9]
    x = np.array([10, -4], dtype=np.int8).reshape(1, 1, 1, 2)
    w = np.array([[3, -1], [-3, 1]], dtype=np.int8)
    b = np.array([5, 5], dtype=np.int32)
    c = dict(n=1, h=1, w=1, c_in=2, c_mid=2, c_out=2, k=1, stride=1, pad=0, dtype="i8", layout="nhwc",
             rq=[(1, 1, -128, 127, -7)] * 3, zp_in=2)
    assert oracle.pw(dict(c, act=["none"] * 3), x, w, b).ravel().tolist() == [11, -19]
    assert oracle.pw(dict(c, act=["relu"] * 3), x, w, b).ravel().tolist() == [11, -7]


def test_int8_zero_points_match_float_convolution_reference():
    """DW -> PW with zero points on input, intermediate and output against torch's float64
    convolutions of the centred values (zero padding = real 0 by torch's definition) and
    exact Fraction rounding, saturating heavily (wide inputs, U{-127..127})."""
    zin, zmid, zout = -20, 13, 31
    rq = [(5, 11, -128, 127, zmid), (3, 12, -100, 120, zout)]
    case = Case("dw_pw", 2, 9, 8, 12, 12, 5, 5, 2, 2, "i8", "nchw", ("relu", "none", "none"),
                (rq[0], rq[1], rq[1]), dist_x="i8", dist_w="i8", bias=True, seed=43)
    inp = make_inputs(case)
    y = oracle.run("dw_pw", dict(case.as_dict(), rq=rq, zp_in=zin), inp)

    def requant(t, r):
        q = np.vectorize(lambda a: _rq_fraction(int(a), r[0], r[1], -2 ** 40, 2 ** 40))(t) + r[4]
        return np.maximum(np.clip(q, r[2], r[3]), r[4])  # relu at the zero point

    x = torch.from_numpy(inp["x"].astype(np.float64) - zin)
    t = F.conv2d(x, torch.from_numpy(inp["w_dw"].astype(np.float64)[:, None]), stride=2, padding=2, groups=12)
    m = requant(np.rint(t.numpy()).astype(np.int64) + inp["b_dw"].astype(np.int64)[None, :, None, None], rq[0])
    u = F.conv2d(torch.from_numpy(m.astype(np.float64) - zmid),
                 torch.from_numpy(inp["w_pw"].astype(np.float64)[:, :, None, None]))
    t2 = np.rint(u.numpy()).astype(np.int64) + inp["b_pw"].astype(np.int64)[None, :, None, None]
    ref = np.clip(np.vectorize(lambda a: _rq_fraction(int(a), 3, 12, -2 ** 40, 2 ** 40))(t2) + zout, -100, 120)
    assert np.array_equal(y, ref.astype(np.int8))
    assert np.mean(np.abs(m) >= 127) > 0.01 or np.mean(m == zmid) > 0.05


def test_zero_point_validation():
    c = _zp_case("pw")
    inp = _i8_inputs(c)
    for bad in (dict(zp_in=128), dict(zp_in=-129), dict(rq=[(1, 6, -127, 127, 200)] * 3)):
        with pytest.raises(oracle.OracleError):
            oracle.run("pw", dict(c, **bad), inp)


def test_c4_spread_cases_leave_most_outputs_unsaturated():
    """The spread-keeping int8 C4 cases really exercise the contraction and rounding: most
    of the oracle's outputs are strictly inside (-127, 127) and take many distinct values
    (the named configuration saturates most of them)."""
    from paper_2404_19331_amd.workloads import config_c4_spread
    for case in config_c4_spread():
        small = case.with_(n=1)
        y = oracle.run(case.op, small, make_inputs(small))
        inner = np.mean(np.abs(y.astype(np.int32)) < 127)
        assert inner > 0.95, (case.name, inner)
        assert len(np.unique(y)) > 100, case.name


def _t_bf16_round(t64):
    """float64 tensor -> bfloat16 bits the way the stage cast is defined: to float32
    (nearest even), then to bfloat16 (nearest even), by torch's own conversions."""
    return t64.to(torch.float32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _t_vals(bits):
    return torch.from_numpy(_bf16_to_f32(bits).astype(np.float64))


@pytest.mark.parametrize("k,s,p", [(3, 1, 1), (3, 2, 1), (5, 1, 2), (5, 2, 0)])
def test_bf16_stage_cast_matches_torch_float64_convolutions(k, s, p):
    """bf16 oracle = float64 convolutions (torch) with each stage rounded to bf16
    nearest-even, element for element, for the single DW and PW layers and the DW->PW
    module (whose intermediate is rounded before the PW). Truncating instead of rounding
    at either stage changes many of these outputs, so the pin sees the cast's mode."""
    case = Case("dw_pw", 2, 11, 9, 24, 24, 20, k, s, p, "bf16", "nchw", ("relu", "relu6", "none"), bias=True,
                dist_x="n01", seed=424)
    inp = make_inputs(case)
    x, wd, bd, wp, bp = (inp[n] for n in ("x", "w_dw", "b_dw", "w_pw", "b_pw"))
    xt, wdt, wpt = _t_vals(x), _t_vals(wd), _t_vals(wp)
    bdt, bpt = torch.from_numpy(bd.astype(np.float64)), torch.from_numpy(bp.astype(np.float64))
    c = case.c_in
    dw64 = F.conv2d(xt, wdt.reshape(c, 1, k, k), bdt, stride=s, padding=p, groups=c).clamp(min=0)
    mid = _t_bf16_round(dw64)
    pw64 = (F.conv2d(_t_vals(mid), wpt.reshape(case.c_out, c, 1, 1), bpt)).clamp(0, 6)
    ref_dwpw = _t_bf16_round(pw64)
    assert np.array_equal(oracle.dw_pw(case, x, wd, bd, wp, bp), ref_dwpw)
    assert np.array_equal(oracle.dw(case, x, wd, bd), mid)
    pw_case = case.with_(h=mid.shape[2], w=mid.shape[3], k=1, stride=1, pad=0, act=("relu6", "none", "none"),
                         c_in=c, c_mid=c)
    assert np.array_equal(oracle.pw(pw_case, mid, wp, bp), ref_dwpw)
    # the rounding mode matters on these inputs: truncation differs
    trunc = (dw64.to(torch.float32).numpy().view(np.uint32) >> 16).astype(np.uint16)
    assert np.mean(trunc != mid) > 0.2
