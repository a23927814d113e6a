"""GPU parity of the PW -> PW register kernel (k_pwpw4), forced through explicit plans.

Every compiled variant that implements a case runs with each pixel group's intermediate
chunks on 1, 2 and 4 waves of a workgroup (partial sums added through LDS), against the
CPU oracle. Cases cover ragged pixel groups (workgroups whose last waves have no pixel
group but still meet the barrier), ragged output-channel tiles, channel rows that are
not 16-byte multiples (word-wise operand loads), input channels needing 1 to 4 MFMA
k-steps and every element type. Split plans of two shapes run back to back and repeat
bit-exactly.
"""
import numpy as np
import pytest

from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import Case, make_inputs

from gpu_util import assert_close, dev_inputs, oracle_ref, run_fused, to_np

pytestmark = pytest.mark.gpu

RQ = ((1, 6, -127, 127), (3, 9, -128, 127), (1, 6, -127, 127))
ELT = {"f32": 4, "bf16": 2, "i8": 1}


def _cases():
    out = []
    shapes = {
        "i8": [(40, 200, 40), (36, 100, 20), (200, 64, 160), (64, 960, 4), (24, 144, 24)],
        "bf16": [(40, 72, 24), (100, 50, 36), (8, 300, 120), (64, 64, 64)],
        "f32": [(20, 36, 12), (60, 30, 64), (4, 8, 4)],
    }
    for dt, shp in shapes.items():
        for ci, cm, co in shp:
            out.append(Case("pw_pw", 2, 13, 11, ci, cm, co, 1, 1, 0, dt, "nhwc",
                            ("relu" if dt == "i8" else "relu6", "relu", "none"), RQ,
                            dist_x="i8small" if dt == "i8" else "n01", dist_w="i8small", bias=True,
                            seed=2100 + len(out), name="pwpw4-%s-%d-%d-%d" % (dt, ci, cm, co)))
    out.append(Case("pw_pw", 1, 1, 3, 16, 64, 16, 1, 1, 0, "i8", "nhwc", ("none",) * 3, RQ,
                    dist_x="i8small", dist_w="i8small", bias=False, seed=2199, name="pwpw4-i8-3px"))
    return out


CASES = _cases()


def _v4_plans(case):
    desc = fcm.desc_from_case(case)
    e = ELT[case.dtype]
    nch = -(-case.c_mid * e // 64)
    plans = []
    for v in range(fcm.lib().fcm_variant_count()):
        name = fcm.variant_name(v)
        if not name.startswith("k_pwpw4<%s," % case.dtype):
            continue
        pb = int(name.rstrip(">").split(",")[3])
        for s in (1, 2, 4):
            if s > nch:
                continue
            try:
                plans.append(fcm.plan_evaluate("pw_pw", desc, 1, 16 * pb, 64 // e, -(-case.c_out // 16) * 16, v,
                                               splits=s))
            except fcm.FcmError:
                pass
    return plans


def test_every_case_has_register_kernel_plans():
    for c in CASES:
        assert _v4_plans(c), c.name
    # the planner picks the register kernel for NHWC int8 pairs
    p = fcm.plan("pw_pw", fcm.desc_from_case(CASES[0]))
    assert fcm.variant_name(p.variant).startswith("k_pwpw4")


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_register_kernel_every_variant_and_split(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    plans = _v4_plans(case)
    for p in plans:
        got = to_np(run_fused(case, d, plan=p))
        assert_close(got, ref, case.dtype, "%s %s splits %d" % (case.name, fcm.variant_name(p.variant), p.splits))


def test_split_plans_back_to_back_repeat():
    # alternate split plans of two shapes (different pixel-group counts) several times
    big = Case("pw_pw", 4, 9, 10, 32, 192, 48, 1, 1, 0, "i8", "nhwc", ("relu", "none", "none"), RQ,
               dist_x="i8small", dist_w="i8small", bias=True, seed=2201, name="big")
    small = big.with_(n=1, h=3, w=5, seed=2202, name="small")
    runs = []
    for c in (big, small):
        inp = make_inputs(c)
        d = dev_inputs(inp, c.dtype)
        ps = [p for p in _v4_plans(c) if p.splits > 1]
        assert ps
        runs.append((c, d, oracle_ref(c, inp), ps))
    for _ in range(3):
        for c, d, ref, ps in runs:
            for p in ps:
                got = to_np(run_fused(c, d, plan=p))
                assert np.array_equal(got, ref), "%s splits %d" % (c.name, p.splits)
