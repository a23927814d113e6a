"""GPU parity of asymmetric int8 (zero points) against the CPU oracle, bit-exact.

Zero points run on the first-generation kernels, the int8 persistent kernels (their own
tests in test_gpu_v3_zero_points.py) and the PW->PW register kernel's
instances of at most 192 output channels. First generation: the window a depthwise stage reads is
padded with its input's code of real 0, the depthwise sum and each pointwise contraction
lose (input zero point) x (weight sum), the border of the PW -> DW intermediate holds the
intermediate's code of real 0, and every epilogue adds its output zero point and clamps
ReLU / ReLU6 there. Cases cover every module in both layouts, the vector and the
element staging paths (channel rows that are and are not 16-byte multiples), ragged
tiles and channel blocks, an image smaller than the filter footprint (mostly padding),
strides 1 and 2, zero points at the int8 extremes, per-channel requantisation together
with zero points, explicit tilings, the layer-by-layer path and a chain run through
fcm_chain_run. The register kernel takes the weight-row sums from the operands in its
registers; its instances run with every split of the intermediate chunks over 1, 2 and 4
waves.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import Case, make_inputs, mobilenetv2_chain, make_chain_inputs

from gpu_util import (dev_inputs, oracle_chain, oracle_ref, run_chain, run_fused, run_unfused, to_dev, to_np,
                      torch)

pytestmark = pytest.mark.gpu

OPS = {  # op: (c_in, c_mid, c_out, k, stride)
    "dw_pw": [(24, 24, 20, 3, 1), (32, 32, 48, 5, 2)],
    "pw_dw": [(24, 40, 40, 3, 1), (32, 64, 64, 5, 2)],
    "pw_dw_pw": [(24, 40, 20, 3, 1), (16, 64, 48, 3, 2)],
    "pw_pw": [(24, 40, 20, 1, 1), (32, 64, 48, 1, 1)],
    "dw": [(24, 24, 24, 3, 1), (48, 48, 48, 5, 2)],
    "pw": [(24, 24, 20, 1, 1), (64, 64, 96, 1, 1)],
}
ZPS = {0: (-128, (17, -5, 100)), 1: (37, (-90, 6, -31))}  # (zp_in, output zero point of each stage)


def _first_gen(v):
    return not any(g in fcm.variant_name(v) for g in ("2<", "3<", "4<"))


def _case(op, shape_i, layout, h=13, w=11, n=2):
    ci, cm, co, k, s = OPS[op][shape_i]
    zin, zs = ZPS[shape_i]
    rq = tuple((1, sh, -128, 127, z) for sh, z in zip((6, 5, 6), zs))
    return Case(op, n, h, w, ci, cm, co, k, s, k // 2, "i8", layout, ("relu", "relu6", "none"), rq,
                dist_x="i8", dist_w="i8small", bias=True, seed=4100 + 7 * shape_i + len(op),
                name="zp-%s-%d-%s-%dx%d" % (op, shape_i, layout, h, w), zp_in=zin)


def _check(case, got, ref):
    assert np.array_equal(got, ref), "%s: %d of %d differ" % (case.name, int(np.sum(got != ref)), ref.size)
    # not degenerate: the output takes many codes
    assert len(np.unique(ref)) > 8, case.name


CASES = [_case(op, i, lay) for op in OPS for i in range(2) for lay in ("nhwc", "nchw")]
CASES += [_case(op, 0, "nhwc", h=2, w=3, n=1) for op in ("dw_pw", "pw_dw", "pw_dw_pw", "dw")]


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_zero_point_parity(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    got = to_np(run_fused(case, d))
    assert np.array_equal(got, ref), "%s: %d of %d differ" % (case.name, int(np.sum(got != ref)), ref.size)
    if case.h > 3:
        assert len(np.unique(ref)) > 8, case.name
    p = fcm.plan(case.op, fcm.desc_from_case(case))
    v = p.variant
    assert _first_gen(v) or (case.op == "pw_pw" and fcm.variant_name(v).startswith("k_pwpw4<i8,")) or \
        fcm.variant_name(v).startswith(("k_dwpw3<i8,", "k_pw3<i8,", "k_dw3<i8,")), \
        fcm.variant_name(v)
    if case.op not in ("dw", "pw"):
        assert np.array_equal(to_np(run_unfused(case, d)), ref), case.name + " (layer-by-layer)"


@pytest.mark.parametrize("op", list(OPS))
def test_zero_point_explicit_tilings(op):
    # first-generation tilings (PW->PW on NHWC plans the register kernel: its own test below)
    case = _case(op, 1, "nchw" if op == "pw_pw" else "nhwc", h=19, w=17)
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    desc = fcm.desc_from_case(case)
    best = fcm.plan(op, desc)
    if not _first_gen(best.variant):  # (the planner chose a newer kernel: take the first-generation one)
        best = fcm.plan(op, fcm.desc_from_case(case.with_(layout="nchw")))
        assert _first_gen(best.variant)
    n = 0
    for th in (1, 2, 4, 8):
        for tw in (4, 8, 16):
            for cob in (16, 32, 48, 64):
                try:
                    p = fcm.plan_evaluate(op, desc, th, tw, best.c_block, cob, best.variant)
                except fcm.FcmError:
                    continue
                got = to_np(run_fused(case, d, plan=p))
                assert np.array_equal(got, ref), "%s tile %dx%d cob %d" % (case.name, th, tw, cob)
                n += 1
    assert n >= 2, case.name


@pytest.mark.parametrize("op", list(OPS))
def test_zero_points_with_per_channel_requant(op):
    case = _case(op, 0, "nhwc", h=9, w=10)
    ci, cm, co = case.c_in, case.c_mid, case.c_out
    chans = {"dw_pw": [ci, co], "pw_dw": [cm, cm], "pw_dw_pw": [cm, cm, co], "pw_pw": [cm, co], "dw": [ci],
             "pw": [co]}[op]
    rng = np.random.default_rng(12)
    pcs = [(rng.integers(1, 8, n), rng.integers(5, 10, n)) for n in chans]
    inp = make_inputs(case)
    ref = oracle.run(op, dict(case.as_dict(), rq_channel=pcs), inp)
    d = dev_inputs(inp, case.dtype)
    T = torch()
    rqc = [T.from_numpy(np.concatenate(pc).astype(np.int32)).cuda() for pc in pcs]
    got = to_np(run_fused(case, d, rq_channel=rqc))
    assert np.array_equal(got, ref), case.name


def test_zero_point_chain_matches_layer_by_layer_oracle():
    """A MobileNetV2-style chain with a zero point on every tensor: the planned chain
    (fused groups) and the unfused chain both equal the oracle run layer by layer."""
    spec = mobilenetv2_chain(n=2, dtype="i8", h=32, w=32, stages=[(1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 2, 2)],
                             final_pw=False)
    rng = np.random.default_rng(5)
    layers = []
    for L in spec.layers:
        L = dict(L)
        L["rq"] = tuple(L["rq"]) + (int(rng.integers(-60, 60)),)
        layers.append(L)
    spec = dataclasses.replace(spec, layers=layers, zp_in=-128)
    x, ws, bs = make_chain_inputs(spec)
    ref = oracle_chain(spec, x, ws, bs)
    xd = to_dev(x, "i8")
    wd = [to_dev(w, "i8") for w in ws]
    bd = [to_dev(b, "i8") for b in bs]
    for objective in ("bytes", "unfused"):
        y, p = run_chain(spec, objective, xd, wd, bd)
        assert np.array_equal(to_np(y), ref), objective
    assert p.fused_layers == 0
    y, p = run_chain(spec, "bytes", xd, wd, bd)
    assert p.fused_layers > 0
    assert len(np.unique(ref)) > 8


REG_SHAPES = [(40, 200, 40), (36, 100, 20), (64, 960, 4), (24, 144, 24), (128, 64, 128), (16, 64, 16),
              (160, 960, 160), (192, 100, 180)]


@pytest.mark.parametrize("ci,cm,co", REG_SHAPES, ids=lambda v: str(v))
def test_zero_points_register_kernel_every_variant_and_split(ci, cm, co):
    case = Case("pw_pw", 2, 13, 11, ci, cm, co, 1, 1, 0, "i8", "nhwc", ("relu", "none", "none"),
                ((1, 8, -128, 127, -37), (5, 9, -128, 100, 21), (1, 1, -128, 127)), dist_x="i8",
                dist_w="i8small", bias=True, seed=4300 + ci + co, name="zp-reg-%d-%d-%d" % (ci, cm, co), zp_in=-128)
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    assert len(np.unique(ref)) > 8
    d = dev_inputs(inp, case.dtype)
    desc = fcm.desc_from_case(case)
    assert fcm.variant_name(fcm.plan("pw_pw", desc).variant).startswith("k_pwpw4<i8,")
    nch = -(-cm // 64)
    n = 0
    for v in range(fcm.lib().fcm_variant_count()):
        name = fcm.variant_name(v)
        if not name.startswith("k_pwpw4<i8,"):
            continue
        pb = int(name.rstrip(">").split(",")[3])
        for s in (1, 2, 4):
            if s > nch:
                continue
            try:
                p = fcm.plan_evaluate("pw_pw", desc, 1, 16 * pb, 64, -(-co // 16) * 16, v, splits=s)
            except fcm.FcmError:
                continue
            got = to_np(run_fused(case, d, plan=p))
            assert np.array_equal(got, ref), "%s %s splits %d: %d differ" % (case.name, name, s, int(np.sum(got != ref)))
            n += 1
    assert n >= 2
