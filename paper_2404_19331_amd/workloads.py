"""Seeded synthetic workloads for the fused DW/PW modules.

This module only describes layer shapes and draws seeded random tensors. It holds none
of the modules' arithmetic; both the CPU oracle and the HIP path consume what it
produces, so the same bytes reach both.

Shapes follow the layers the paper evaluates (arXiv 2404.19331, Sec. V-B: MobileNet
v1/v2-style depthwise separable and inverted-residual blocks, and convolutional ViT
token grids) plus an EfficientNet-style int8 MBConv pair. Values are synthetic: the
modules' timing does not depend on them, and no trained weights are used.

Recipe (every array drawn on the CPU with numpy's PCG64 in the order x, then the
weights in execution order):
  * x:  U[-1, 1] ("u11"), N(0, 1) ("n01"), U{-127..127} ("i8"), U{-8..8} ("i8small")
  * float weights: N(0, 1/fan_in); fan_in = K*K for depthwise, C_in for pointwise
  * int8 weights: U{-127..127} ("i8") or U{-8..8} ("i8small")
  * bf16 tensors: drawn in float32, then rounded to bfloat16 (nearest-even)
  * biases: none for the named configurations; tests that exercise bias draw
    N(0, 0.25) (float) or U{-2000..2000} (int32).
"""
from dataclasses import dataclass, field, replace
from typing import Tuple

import math

import numpy as np

BASE_SEED = 2404_19331

ACT3 = Tuple[str, str, str]
RQ = Tuple[int, int, int, int]  # (mult, shift, qmin, qmax)

RQ_C4 = (1, 8, -127, 127)  # per-tensor scale 2^-8, symmetric int8 range


@dataclass(frozen=True)
class Case:
    """One module invocation: module name, geometry, precision, layout, epilogues."""
    op: str                      # dw_pw | pw_dw | pw_dw_pw | pw_pw | dw | pw
    n: int
    h: int
    w: int
    c_in: int
    c_mid: int
    c_out: int
    k: int = 3
    stride: int = 1
    pad: int = 1
    dtype: str = "f32"           # f32 | bf16 | i8
    layout: str = "nchw"         # nchw | nhwc
    act: ACT3 = ("none", "none", "none")
    rq: Tuple[RQ, RQ, RQ] = ((1, 0, -127, 127),) * 3
    dist_x: str = "u11"
    dist_w: str = "fan_in"
    bias: bool = False
    seed: int = BASE_SEED
    name: str = ""
    zp_in: int = 0               # int8 zero point of x (rq entries may carry a 5th: output zero point)

    def with_(self, **kw):
        return replace(self, **kw)

    def as_dict(self):
        return dict(op=self.op, n=self.n, h=self.h, w=self.w, c_in=self.c_in, c_mid=self.c_mid,
                    c_out=self.c_out, k=self.k, stride=self.stride, pad=self.pad,
                    dtype=self.dtype, layout=self.layout, act=list(self.act),
                    rq=[list(r) for r in self.rq], zp_in=self.zp_in, name=self.name)


def _x_shape(case):
    if case.layout == "nchw":
        return (case.n, case.c_in, case.h, case.w)
    return (case.n, case.h, case.w, case.c_in)


def _to_bf16_bits(a):
    import torch  # conversion only (round to nearest even), CPU
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def _draw_x(rng, case):
    shape = _x_shape(case)
    d = case.dist_x
    if d == "u11":
        a = rng.uniform(-1.0, 1.0, size=shape)
    elif d == "n01":
        a = rng.standard_normal(size=shape)
    elif d == "i8":
        return rng.integers(-127, 128, size=shape, dtype=np.int64).astype(np.int8)
    elif d == "i8small":
        return rng.integers(-8, 9, size=shape, dtype=np.int64).astype(np.int8)
    else:
        raise ValueError(d)
    return _cast_float(a, case.dtype)


def _cast_float(a, dtype):
    if dtype == "f32":
        return a.astype(np.float32)
    if dtype == "bf16":
        return _to_bf16_bits(a.astype(np.float32))
    if dtype == "f64":
        return a.astype(np.float64)
    raise ValueError(dtype)


def _draw_w(rng, case, shape, fan_in):
    if case.dtype == "i8":
        lo, hi = (-8, 8) if case.dist_w == "i8small" else (-127, 127)
        return rng.integers(lo, hi + 1, size=shape, dtype=np.int64).astype(np.int8)
    a = rng.standard_normal(size=shape) * np.sqrt(1.0 / fan_in)
    return _cast_float(a, case.dtype)


def _draw_b(rng, case, cnt):
    if not case.bias:
        return None
    if case.dtype == "i8":
        return rng.integers(-2000, 2001, size=cnt, dtype=np.int64).astype(np.int32)
    b = rng.normal(0.0, 0.25, size=cnt)
    return b.astype(np.float64 if case.dtype == "f64" else np.float32)


def make_inputs(case, seed=None):
    """Seeded inputs of a case as a dict of contiguous numpy arrays in storage format
    (float32, uint16 bfloat16 bits, int8, float64). Keys depend on the module."""
    rng = np.random.default_rng(case.seed if seed is None else seed)
    out = {"x": _draw_x(rng, case)}
    k = case.k
    if case.op == "dw_pw":
        out["w_dw"] = _draw_w(rng, case, (case.c_in, k, k), k * k)
        out["w_pw"] = _draw_w(rng, case, (case.c_out, case.c_in), case.c_in)
        out["b_dw"] = _draw_b(rng, case, case.c_in)
        out["b_pw"] = _draw_b(rng, case, case.c_out)
    elif case.op == "pw_dw":
        out["w_pw"] = _draw_w(rng, case, (case.c_mid, case.c_in), case.c_in)
        out["w_dw"] = _draw_w(rng, case, (case.c_mid, k, k), k * k)
        out["b_pw"] = _draw_b(rng, case, case.c_mid)
        out["b_dw"] = _draw_b(rng, case, case.c_mid)
    elif case.op == "pw_dw_pw":
        out["w_pw1"] = _draw_w(rng, case, (case.c_mid, case.c_in), case.c_in)
        out["w_dw"] = _draw_w(rng, case, (case.c_mid, k, k), k * k)
        out["w_pw2"] = _draw_w(rng, case, (case.c_out, case.c_mid), case.c_mid)
        out["b_pw1"] = _draw_b(rng, case, case.c_mid)
        out["b_dw"] = _draw_b(rng, case, case.c_mid)
        out["b_pw2"] = _draw_b(rng, case, case.c_out)
    elif case.op == "pw_pw":
        out["w_pw1"] = _draw_w(rng, case, (case.c_mid, case.c_in), case.c_in)
        out["w_pw2"] = _draw_w(rng, case, (case.c_out, case.c_mid), case.c_mid)
        out["b_pw1"] = _draw_b(rng, case, case.c_mid)
        out["b_pw2"] = _draw_b(rng, case, case.c_out)
    elif case.op == "dw":
        out["w_dw"] = _draw_w(rng, case, (case.c_in, k, k), k * k)
        out["b_dw"] = _draw_b(rng, case, case.c_in)
    elif case.op == "pw":
        out["w_pw"] = _draw_w(rng, case, (case.c_out, case.c_in), case.c_in)
        out["b_pw"] = _draw_b(rng, case, case.c_out)
    else:
        raise ValueError(case.op)
    return out


# ---------------------------------------------------------------------------
# Named configurations
# ---------------------------------------------------------------------------

# MobileNetV1 (width 1.0, 224x224 input) depthwise-separable layers:
# (input spatial size, channels, depthwise stride, pointwise output channels)
MOBILENET_V1 = [
    (112, 32, 1, 64), (112, 64, 2, 128), (56, 128, 1, 128), (56, 128, 2, 256),
    (28, 256, 1, 256), (28, 256, 2, 512), (14, 512, 1, 512), (14, 512, 1, 512),
    (14, 512, 1, 512), (14, 512, 1, 512), (14, 512, 1, 512), (14, 512, 2, 1024),
    (7, 1024, 1, 1024),
]

VIT_GRIDS = [(56, 64, 192), (28, 192, 384), (14, 384, 768)]


def config_c1():
    """DW3x3+ReLU -> PW 32->64 +ReLU, fp32 NCHW, batch 1, 56x56."""
    return [Case("dw_pw", 1, 56, 56, 32, 32, 64, 3, 1, 1, "f32", "nchw", ("relu", "relu", "none"),
                 dist_x="u11", seed=BASE_SEED + 1, name="C1 dwpw 56x56x32->64 f32 b1")]


def config_c2():
    """Inverted residual PW 24->144 ReLU6, DW3x3 ReLU6, PW 144->24 linear, fp32, b1, 56x56."""
    return [Case("pw_dw_pw", 1, 56, 56, 24, 144, 24, 3, 1, 1, "f32", "nchw",
                 ("relu6", "relu6", "none"), dist_x="u11", seed=BASE_SEED + 2,
                 name="C2 pwdwpw 56x56 24->144->24 f32 b1")]


def config_c3(batches=(1, 32)):
    """All 13 MobileNetV1 DW3x3+PW layers, bf16 NHWC, ReLU after each conv."""
    out = []
    for b in batches:
        for li, (hw, c, s, co) in enumerate(MOBILENET_V1, start=1):
            out.append(Case("dw_pw", b, hw, hw, c, c, co, 3, s, 1, "bf16", "nhwc",
                            ("relu", "relu", "none"), dist_x="u11",
                            seed=BASE_SEED + 3 + 100 * li + b,
                            name="C3 L%d %dx%dx%d s%d ->%d bf16 b%d" % (li, hw, hw, c, s, co, b)))
    return out


def config_c4():
    """EfficientNet-B0-style int8 MBConv DW5x5+PW pairs, NHWC, batch 8, requant 2^-8 RNE."""
    rq = (RQ_C4, RQ_C4, RQ_C4)
    return [
        Case("dw_pw", 8, 112, 112, 96, 96, 24, 5, 2, 2, "i8", "nhwc", ("none",) * 3, rq,
             dist_x="i8", dist_w="i8", seed=BASE_SEED + 4 + 100,
             name="C4a dwpw5x5s2 112x112x96->24 i8 b8"),
        Case("dw_pw", 8, 14, 14, 480, 480, 112, 5, 1, 2, "i8", "nhwc", ("none",) * 3, rq,
             dist_x="i8", dist_w="i8", seed=BASE_SEED + 4 + 200,
             name="C4b dwpw5x5s1 14x14x480->112 i8 b8"),
    ]


def config_c4_spread():
    """The C4 shapes (EfficientNet-B0-style int8 DW5x5+PW, NHWC, batch 8) with
    requantisation shifts sized to each stage's accumulator spread, as config_pwpw does:
    with the named configuration's 2^-8 most results saturate at +-127, which would leave
    the bit-exact comparison mostly comparing the clamp. U{-127..127} operands have
    standard deviation 127/sqrt(3) = s; a K*K depthwise sum has s^2 * K, a C-wide
    pointwise sum over inputs of spread d has d * s * sqrt(C); each shift is the smallest
    that brings its stage to a spread of at most 48."""
    sd = 127 / math.sqrt(3)
    out = []
    for j, (n, hw, c, co, k, st) in enumerate([(8, 112, 96, 24, 5, 2), (8, 14, 480, 112, 5, 1)]):
        s1 = int(math.ceil(math.log2(sd * sd * k / 48)))
        d1 = sd * sd * k / 2 ** s1  # spread of the depthwise output
        s2 = int(math.ceil(math.log2(d1 * sd * math.sqrt(c) / 48)))
        rq = ((1, s1, -127, 127), (1, s2, -127, 127), RQ_C4)
        out.append(Case("dw_pw", n, hw, hw, c, c, co, k, st, k // 2, "i8", "nhwc", ("none",) * 3, rq,
                        dist_x="i8", dist_w="i8", seed=BASE_SEED + 4 + 1000 + 100 * j,
                        name="C4%s-spread dwpw%dx%ds%d %dx%dx%d->%d i8 b%d" % ("ab"[j], k, k, st, hw, hw, c, co, n)))
    return out


def config_c5():
    """Convolutional-ViT token-grid DW3x3+PW projections, bf16 NHWC, batch 64, linear."""
    return [Case("dw_pw", 64, hw, hw, c, c, co, 3, 1, 1, "bf16", "nhwc", ("none",) * 3,
                 dist_x="n01", seed=BASE_SEED + 5 + 100 * i,
                 name="C5 %dx%dx%d->%d bf16 b64" % (hw, hw, c, co))
            for i, (hw, c, co) in enumerate(VIT_GRIDS, start=1)]


# MobileNetV2 expansion / projection widths (spatial size, c_in, expanded, c_out) used
# as two fused pointwise layers without the depthwise layer between them.
PWPW_SHAPES = [(56, 24, 144, 24), (28, 32, 192, 32), (14, 64, 384, 64), (14, 96, 576, 96), (7, 160, 960, 160)]


def config_pwpw():
    """PW -> PW pairs (the paper's PwPw module, frequent in its int8 plans), int8 NHWC,
    batch 8, ReLU after the first layer. Each stage requantises by a power of two sized to
    its contraction: U{-127..127} operands have standard deviation 127/sqrt(3), so a
    C-wide sum has 127^2/3 * sqrt(C); the shift brings that to about 48, keeping nearly
    all results inside the int8 range. The second stage reads ReLU output, whose root mean
    square is about 48/sqrt(2)."""
    sd = 127 / math.sqrt(3)
    out = []
    for i, (hw, ci, cm, co) in enumerate(PWPW_SHAPES, start=1):
        s1 = int(round(math.log2(sd * sd * math.sqrt(ci) / 48)))
        s2 = int(round(math.log2(48 / math.sqrt(2) * sd * math.sqrt(cm) / 48)))
        rq = ((1, s1, -127, 127), (1, s2, -127, 127), RQ_C4)
        out.append(Case("pw_pw", 8, hw, hw, ci, cm, co, 1, 1, 0, "i8", "nhwc", ("relu", "none", "none"), rq,
                        dist_x="i8", dist_w="i8", seed=BASE_SEED + 6 + 100 * i,
                        name="PWPW %dx%dx%d->%d->%d i8 b8" % (hw, hw, ci, cm, co)))
    return out


# MobileNetV2 inverted-residual stages after the stem convolution (112x112x32 input):
# (expansion t, output channels c, repeats, stride of the first block).
MNV2_STAGES = [(1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2), (6, 96, 3, 1), (6, 160, 3, 2),
               (6, 320, 1, 1)]


@dataclass
class ChainSpec:
    """A sequence of DW/PW layers (no skip connections) with its input and seed."""
    n: int
    h: int
    w: int
    c: int
    dtype: str
    layout: str
    layers: list
    seed: int = BASE_SEED
    name: str = ""
    zp_in: int = 0               # int8 zero point of x (rq entries may carry a 5th: output zero point)


def mobilenetv2_chain(n=8, dtype="i8", layout="nhwc", h=112, w=112, stages=None, final_pw=True,
                      zero_points=False):
    """The DW and PW layers of MobileNetV2 after its stem (51 layers at full depth): per
    block an expansion PW (t > 1), a DW 3x3 and a linear projection PW, then the final PW
    to 1280 channels. Float types use ReLU6 after the expansion and the DW; int8 uses ReLU
    there (its requantisation by a power of two has no output scale that would place 6.0)
    and requantises every layer by 2^-s, s sized to the layer's accumulator spread
    (U{-127..127} weights, inputs of RMS about 48 or, after ReLU, 34) so outputs spread over
    the int8 range. zero_points (int8): asymmetric tensors, the input and every ReLU output
    with zero point -128 (real 0 at the bottom of the code range), linear outputs with 3."""
    stages = MNV2_STAGES if stages is None else stages
    act = "relu" if dtype == "i8" else "relu6"
    sd_w = 127 / math.sqrt(3)
    layers = []
    c = 32
    sd_in = [sd_w]  # RMS of the current int8 activations (input drawn as U{-127..127})

    def rq_for(fan_in, relu):
        s = int(round(math.log2(max(1.0, sd_in[0] * sd_w * math.sqrt(fan_in) / 48))))
        sd_in[0] = 48 / math.sqrt(2) if relu else 48.0
        if zero_points:
            return (1, s, -127, 127, -128 if relu else 3)
        return (1, s, -127, 127)

    for t, co, reps, s0 in stages:
        for r in range(reps):
            if t != 1:
                layers.append(dict(kind="pw", c_out=c * t, act=act, rq=rq_for(c, True)))
            layers.append(dict(kind="dw", k=3, stride=s0 if r == 0 else 1, pad=1, act=act, rq=rq_for(9, True)))
            cm = c * t
            layers.append(dict(kind="pw", c_out=co, act="none", rq=rq_for(cm, False)))
            c = co
    if final_pw:
        layers.append(dict(kind="pw", c_out=1280, act=act, rq=rq_for(c, True)))
    return ChainSpec(n, h, w, 32, dtype, layout, layers, seed=BASE_SEED + 7,
                     name="MobileNetV2 body %d layers %s%s %s b%d" % (len(layers), dtype,
                                                                    " zero points" if zero_points else "", layout, n),
                     zp_in=-128 if zero_points else 0)


def make_chain_inputs(spec, seed=None):
    """Seeded input and per-layer weights/biases of a chain, storage format as make_inputs:
    x, then for each layer its weights ([c][k][k] DW, [c_out][c_in] PW) and bias."""
    rng = np.random.default_rng(spec.seed if seed is None else seed)
    case = Case("pw", spec.n, spec.h, spec.w, spec.c, spec.c, spec.c, 1, 1, 0, spec.dtype, spec.layout,
                dist_x="i8" if spec.dtype == "i8" else "n01", dist_w="i8", bias=True)
    x = _draw_x(rng, case)
    ws, bs = [], []
    c = spec.c
    for L in spec.layers:
        if L["kind"] == "dw":
            k = L["k"]
            ws.append(_draw_w(rng, case, (c, k, k), k * k))
            bs.append(_draw_b(rng, case, c))
        else:
            ws.append(_draw_w(rng, case, (L["c_out"], c), c))
            bs.append(_draw_b(rng, case, L["c_out"]))
            c = L["c_out"]
    return x, ws, bs


CONFIGS = {"C1": config_c1, "C2": config_c2, "C3": config_c3, "C4": config_c4, "C5": config_c5}


def all_cases():
    out = []
    for f in CONFIGS.values():
        out.extend(f())
    return out
