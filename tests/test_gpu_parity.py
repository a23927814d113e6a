"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Small cases span several tiles, ragged spatial tails, ragged channel chunks and blocks,
every module x element type x layout x depthwise geometry, with biases and activations.
The named configurations run at full size: the whole output is compared (every image of
MobileNetV1 batch 32 and of the 14x14 token grid at batch 64); on the two large token grids
the oracle recomputes a strided sample of images (every 8th, plus the last; images are
independent), compared against the full-batch GPU result.
"""
import re

import numpy as np
import pytest

from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import (Case, make_inputs, config_c1, config_c2, config_c3, config_c4, config_c5,
                                             config_c4_spread, config_pwpw)

import oracle
from gpu_util import (assert_close, batch_slice, dev_inputs, oracle_ref, run_fused, run_unfused, to_np, torch)

pytestmark = pytest.mark.gpu

KS = [(3, 1), (3, 2), (5, 1), (5, 2)]
RQ_SMALL = ((1, 4, -127, 127), (3, 7, -128, 127), (1, 6, -127, 127))
ACTS = {"f32": ("relu6", "relu", "none"), "bf16": ("relu", "none", "relu6"), "i8": ("relu", "none", "relu")}


def _small_cases():
    out = []
    for dt in ("f32", "bf16", "i8"):
        for lay in ("nchw", "nhwc"):
            for op in ("dw_pw", "pw_dw", "pw_dw_pw", "dw"):
                for k, s in KS:
                    cm = 40 if op == "dw_pw" or op == "dw" else 72
                    co = {"dw_pw": 24, "pw_dw": cm, "pw_dw_pw": 24, "dw": 40}[op]
                    out.append(Case(op, 2, 13, 11, 40, cm, co, k, s, k // 2, dt, lay, ACTS[dt], RQ_SMALL,
                                    dist_x="i8small" if dt == "i8" else "n01", dist_w="i8small", bias=True,
                                    seed=1000 + len(out), name="%s-%s-%s-k%ds%d" % (op, dt, lay, k, s)))
            out.append(Case("pw", 2, 13, 11, 40, 40, 24, 1, 1, 0, dt, lay, ACTS[dt], RQ_SMALL,
                            dist_x="i8small" if dt == "i8" else "n01", dist_w="i8small", bias=True,
                            seed=1000 + len(out), name="pw-%s-%s" % (dt, lay)))
            out.append(Case("pw_pw", 2, 13, 11, 40, 72, 24, 1, 1, 0, dt, lay, ACTS[dt], RQ_SMALL,
                            dist_x="i8small" if dt == "i8" else "n01", dist_w="i8small", bias=True,
                            seed=1000 + len(out), name="pw_pw-%s-%s" % (dt, lay)))
    return out


SMALL = _small_cases()


@pytest.mark.parametrize("case", SMALL, ids=lambda c: c.name)
def test_small_parity(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    got = to_np(run_fused(case, dev_inputs(inp, case.dtype)))
    assert_close(got, ref, case.dtype, case.name)


EDGE = [
    # 1x1 image, every tap but the centre in the padding
    Case("dw_pw", 3, 1, 1, 16, 16, 8, 3, 1, 1, "f32", "nhwc", ("relu", "none", "none"), bias=True, seed=1),
    Case("pw_dw", 1, 1, 1, 8, 16, 16, 3, 2, 1, "bf16", "nchw", ("relu6", "relu", "none"), bias=True, seed=2),
    # image smaller than the filter's reach, k=5 pad=2 on 2x3
    Case("pw_dw_pw", 2, 2, 3, 8, 24, 8, 5, 1, 2, "f32", "nchw", ("relu6", "relu6", "none"), bias=True, seed=3),
    Case("dw_pw", 1, 2, 3, 8, 8, 8, 5, 2, 2, "i8", "nhwc", ("relu", "relu", "none"), RQ_SMALL,
         dist_x="i8small", dist_w="i8small", bias=True, seed=4),
    # single channel in and out (every channel dimension ragged)
    Case("dw_pw", 1, 9, 9, 1, 1, 1, 3, 1, 1, "bf16", "nhwc", ("none", "none", "none"), bias=True, seed=5),
    Case("pw_dw_pw", 1, 9, 7, 1, 1, 1, 3, 2, 1, "i8", "nchw", ("relu", "none", "none"), RQ_SMALL,
         dist_x="i8small", dist_w="i8small", bias=True, seed=6),
    # channel rows that are not 16-byte multiples (scalar staging / store paths)
    Case("dw_pw", 2, 10, 12, 20, 20, 12, 3, 1, 1, "bf16", "nhwc", ("relu", "relu", "none"), bias=True, seed=7),
    Case("pw_dw", 2, 10, 12, 20, 36, 36, 3, 2, 1, "i8", "nhwc", ("relu", "relu", "none"), RQ_SMALL,
         dist_x="i8small", dist_w="i8small", bias=True, seed=8),
    Case("pw", 2, 7, 7, 24, 24, 24, 1, 1, 0, "i8", "nhwc", ("none",) * 3, RQ_SMALL,
         dist_x="i8small", dist_w="i8small", bias=True, seed=9),
    # no padding, valid convolution shrinking the image
    Case("dw_pw", 2, 9, 8, 32, 32, 48, 3, 1, 0, "f32", "nchw", ("relu", "relu", "none"), bias=True, seed=10),
    Case("dw", 2, 12, 10, 48, 48, 48, 5, 2, 0, "bf16", "nhwc", ("relu6", "none", "none"), bias=True, seed=11),
    # many channels: several contraction chunks and output blocks, odd sizes
    Case("dw_pw", 1, 6, 5, 600, 600, 300, 3, 1, 1, "bf16", "nhwc", ("relu", "none", "none"), bias=True, seed=12),
    Case("pw_dw_pw", 1, 6, 5, 100, 200, 150, 3, 1, 1, "bf16", "nhwc", ("relu6", "relu6", "none"), bias=True,
         seed=13),
    # int8 ReLU6: the quantised clamp [0, qmax] (qmax = 6.0 in output units), every module
    Case("dw_pw", 2, 10, 12, 40, 40, 24, 3, 1, 1, "i8", "nhwc", ("relu6", "relu6", "none"),
         ((1, 4, -127, 40), (1, 6, -128, 30), (1, 6, -127, 127)), dist_x="i8small", dist_w="i8small", bias=True,
         seed=20),
    Case("pw_dw_pw", 2, 10, 12, 24, 48, 16, 3, 2, 1, "i8", "nchw", ("relu6", "relu6", "relu6"),
         ((1, 4, -127, 40), (1, 6, -128, 30), (1, 5, -127, 20)), dist_x="i8small", dist_w="i8small", bias=True,
         seed=21),
    Case("pw_pw", 2, 10, 12, 32, 72, 16, 1, 1, 0, "i8", "nhwc", ("relu6", "relu6", "none"),
         ((1, 5, -127, 30), (1, 6, -128, 25), (1, 6, -127, 127)), dist_x="i8small", dist_w="i8small", bias=True,
         seed=22),
    Case("pw_dw", 2, 10, 12, 32, 48, 48, 5, 1, 2, "i8", "nhwc", ("relu6", "relu6", "none"),
         ((1, 5, -127, 30), (1, 6, -128, 25), (1, 6, -127, 127)), dist_x="i8small", dist_w="i8small", bias=True,
         seed=23),
    # PW -> PW: ragged channel rows, single channels, many chunks and output blocks
    Case("pw_pw", 2, 10, 12, 20, 36, 12, 1, 1, 0, "i8", "nhwc", ("relu", "none", "none"), RQ_SMALL,
         dist_x="i8small", dist_w="i8small", bias=True, seed=14),
    Case("pw_pw", 1, 9, 7, 1, 1, 1, 1, 1, 0, "bf16", "nchw", ("relu6", "none", "none"), bias=True, seed=15),
    Case("pw_pw", 1, 6, 5, 600, 300, 200, 1, 1, 0, "bf16", "nhwc", ("relu", "none", "none"), bias=True, seed=16),
    Case("pw_pw", 3, 1, 1, 16, 48, 8, 1, 1, 0, "f32", "nhwc", ("relu", "relu", "none"), bias=True, seed=17),
]


@pytest.mark.parametrize("case", EDGE, ids=lambda c: "%s-%s-%dx%d-c%d-%d" % (c.op, c.dtype, c.h, c.w, c.c_in, c.c_out))
def test_edge_parity(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    got = to_np(run_fused(case, dev_inputs(inp, case.dtype)))
    assert_close(got, ref, case.dtype, case.name)


# ---------------------------------------------------------------------------------
# Named configurations at full size
# ---------------------------------------------------------------------------------

FULL = config_c1() + config_c2() + config_c3(batches=(1, 32)) + config_c4() + config_c4_spread() + config_pwpw() + \
    [c for c in config_c5() if c.h == 14]
SAMPLED = [c for c in config_c5() if c.h != 14]


@pytest.mark.parametrize("case", FULL, ids=lambda c: c.name.replace(" ", "_"))
def test_config_parity_full(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    got = to_np(run_fused(case, dev_inputs(inp, case.dtype)))
    assert_close(got, ref, case.dtype, case.name)


@pytest.mark.parametrize("case", SAMPLED, ids=lambda c: c.name.replace(" ", "_"))
def test_config_parity_sampled_images(case):
    inp = make_inputs(case)
    got = to_np(run_fused(case, dev_inputs(inp, case.dtype)))
    idx = list(range(0, case.n, 8)) + [case.n - 1]
    ref = oracle_ref(case.with_(n=len(idx)), batch_slice(inp, idx))
    assert_close(got[idx], ref, case.dtype, case.name)


# ---------------------------------------------------------------------------------
# Fused vs layer-by-layer, determinism, tilings
# ---------------------------------------------------------------------------------

UNFUSED = [c for c in SMALL if c.op in ("dw_pw", "pw_dw", "pw_dw_pw", "pw_pw") and c.layout == "nhwc"] + \
    config_c1() + config_c2() + config_c4() + config_c4_spread() + config_pwpw()


@pytest.mark.parametrize("case", UNFUSED, ids=lambda c: c.name.replace(" ", "_"))
def test_layer_by_layer_chain_matches_oracle(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    lbl = to_np(run_unfused(case, d))
    assert_close(lbl, ref, case.dtype, case.name + " (layer-by-layer)")
    if case.dtype == "i8":  # unique result: fused and unfused are bit-identical
        assert np.array_equal(to_np(run_fused(case, d)), lbl)


@pytest.mark.parametrize("case", [c for c in SMALL if c.layout == "nhwc" and c.k == 3 and c.stride == 2],
                         ids=lambda c: c.name)
def test_run_to_run_bitwise_determinism(case):
    d = dev_inputs(make_inputs(case), case.dtype)
    a = to_np(run_fused(case, d))
    b = to_np(run_fused(case, d))
    assert np.array_equal(a, b)


def test_full_size_bench_plan_is_bitwise_deterministic():
    """MobileNetV1 layer 7 at batch 32 with the plan the benchmark times: two runs agree bit
    for bit (every workgroup range, split and ring position is exercised at full size)."""
    case = [c for c in config_c3(batches=(32,)) if c.name.startswith("C3 L7 ")][0]
    d = dev_inputs(make_inputs(case), case.dtype)
    p = fcm.plan(case.op, fcm.desc_from_case(case))
    a = to_np(run_fused(case, d, plan=p))
    b = to_np(run_fused(case, d, plan=p))
    assert np.array_equal(a, b)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("op", ["dw_pw", "pw_dw", "pw_dw_pw", "pw_pw"])
def test_power_of_two_homogeneity_bit_exact(dt, op):
    k, pad = (1, 0) if op == "pw_pw" else (3, 1)
    case = Case(op, 2, 12, 9, 24, 24 if op == "dw_pw" else 48, 16 if op != "pw_dw" else 48, k, 1, pad, dt, "nhwc",
                ("relu", "relu", "none"), dist_x="n01", bias=False, seed=77)
    inp = make_inputs(case)
    d = dev_inputs(inp, case.dtype)
    y = run_fused(case, d)
    d8 = dict(d)
    d8["x"] = (d["x"].float() * 8).to(d["x"].dtype)
    y8 = run_fused(case, d8)
    assert torch().equal(y8.float(), y.float() * 8)


def _tilings(case, limit=12):
    """Several explicit tilings of the case that the compiled kernels implement."""
    desc = fcm.desc_from_case(case)
    best = fcm.plan(case.op, desc)
    out = []
    for th in (1, 2, 4, 8):
        for tw in (4, 8, 16):
            for cob in (16, 32, 48, 64):
                try:
                    p = fcm.plan_evaluate(case.op, desc, th, tw, best.c_block, cob, best.variant)
                except fcm.FcmError:
                    continue
                out.append(p)
    step = max(1, len(out) // limit)
    return [best] + out[::step][:limit]


@pytest.mark.parametrize("case", [c for c in SMALL if c.layout == "nhwc" and c.k == 5 and c.stride == 1],
                         ids=lambda c: c.name)
def test_explicit_tilings_agree(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    for p in _tilings(case):
        got = to_np(run_fused(case, d, plan=p))
        assert_close(got, ref, case.dtype, "%s tile %dx%d cob %d" % (case.name, p.tile_h, p.tile_w, p.co_block))


def test_every_output_element_is_written():
    case = Case("dw_pw", 2, 21, 19, 40, 40, 36, 3, 2, 1, "f32", "nchw", ("none",) * 3, bias=True, seed=99)
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    out = torch().full(ref.shape, float("nan"), dtype=torch().float32, device="cuda")
    got = to_np(run_fused(case, d, out=out))
    assert_close(got, ref, case.dtype, "nan-poisoned output")


# ---------------------------------------------------------------------------------
# int8 per-channel requantisation (first-generation kernels)
# ---------------------------------------------------------------------------------

PC_OPS = [("dw_pw", 24, 24, 16, 3), ("pw_dw", 16, 40, 40, 3), ("pw_dw_pw", 16, 40, 12, 3), ("pw_pw", 20, 36, 12, 1),
          ("dw", 24, 24, 24, 5), ("pw", 24, 24, 20, 1)]


@pytest.mark.parametrize("layout", ["nhwc", "nchw"])
@pytest.mark.parametrize("op,ci,cm,co,k", PC_OPS)
def test_per_channel_requant_parity(op, ci, cm, co, k, layout):
    case = Case(op, 2, 11, 9, ci, cm, co, k, 1, k // 2, "i8", layout, ("relu", "relu6", "none"),
                ((1, 6, -127, 127), (1, 7, -128, 40), (1, 6, -127, 127)), dist_x="i8small", dist_w="i8small",
                bias=True, seed=3000 + len(op) + k, name="pc-%s-%s" % (op, layout))
    chans = {"dw_pw": [ci, co], "pw_dw": [cm, cm], "pw_dw_pw": [cm, cm, co], "pw_pw": [cm, co], "dw": [ci],
             "pw": [co]}[op]
    rng = np.random.default_rng(11)
    pcs = [(rng.integers(1, 8, n), rng.integers(4, 10, n)) for n in chans]
    inp = make_inputs(case)
    ref = oracle.run(op, dict(case.as_dict(), rq_channel=pcs), inp)
    d = dev_inputs(inp, case.dtype)
    T = torch()
    rqc = [T.from_numpy(np.concatenate(pc).astype(np.int32)).cuda() for pc in pcs]
    got = to_np(run_fused(case, d, rq_channel=rqc))
    assert_close(got, ref, "i8", case.name)
    # the shared scale gives another result (the per-channel scales were used)
    assert not np.array_equal(got, to_np(run_fused(case, d)))
    desc = fcm.desc_from_case(case)
    name = fcm.variant_name(fcm.plan(op, fcm.make_desc(desc.n, desc.h, desc.w, desc.c_in, desc.c_mid, desc.c_out,
                                                       desc.k, desc.stride, desc.pad, "i8", layout,
                                                       rq_channel=rqc)).variant)
    # the first-generation kernels or, where they implement the module, the int8 persistent ones
    assert re.search(r"\d<", name) is None or re.match(r"k_(dwpw|dw|pw)3<i8,", name), name
