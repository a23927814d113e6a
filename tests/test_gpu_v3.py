"""GPU parity of the persistent NHWC kernels (DW->PW, PW, DW), forced through explicit plans.

Every compiled persistent variant that implements a case runs at several tile shapes
(full and ragged pixel blocks) and compared with the CPU oracle. A capped grid makes
each workgroup stream many (tile, channel chunk) items, which exercises the LDS ring
across tile boundaries, at depths from 2 (one item in flight) to 8 where the tiling
allows it, and split plans (2-4 workgroups per work tile, combined by a second kernel).
"""
import pytest

from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import Case, make_inputs

from gpu_util import assert_close, dev_inputs, oracle_ref, run_fused, to_np

pytestmark = pytest.mark.gpu

RQ = ((1, 5, -127, 127), (3, 8, -128, 127), (1, 6, -127, 127))
ELT = {"f32": 4, "bf16": 2, "i8": 1}
TILES = ((4, 16), (8, 8), (7, 9), (16, 16), (3, 5), (1, 13))


def _cases():
    out = []
    geo = [(3, 1), (3, 2), (5, 1), (5, 2)]
    for dt, (ci, co) in (("bf16", (40, 24)), ("bf16", (72, 200)), ("f32", (20, 36)), ("i8", (48, 32)),
                         ("i8", (144, 80)), ("f32", (36, 12)), ("i8", (48, 24)), ("f32", (20, 6))):
        for k, s in geo:
            act2 = "relu6" if dt != "i8" else "none"
            out.append(Case("dw_pw", 2, 13, 11, ci, ci, co, k, s, k // 2, dt, "nhwc", ("relu", act2, "none"), RQ,
                            dist_x="i8small" if dt == "i8" else "n01", dist_w="i8small", bias=True,
                            seed=1700 + len(out), name="dwpw3-%s-c%d-co%d-k%ds%d" % (dt, ci, co, k, s)))
            out.append(Case("dw", 2, 13, 11, ci, ci, ci, k, s, k // 2, dt, "nhwc",
                            ("relu6" if dt != "i8" else "relu",) * 3, RQ,
                            dist_x="i8small" if dt == "i8" else "n01", dist_w="i8small", bias=True,
                            seed=1800 + len(out), name="dw3-%s-c%d-k%ds%d" % (dt, ci, k, s)))
        out.append(Case("pw", 2, 13, 11, ci, ci, co, 1, 1, 0, dt, "nhwc", ("relu",) * 3, RQ,
                        dist_x="i8small" if dt == "i8" else "n01", dist_w="i8small", bias=True,
                        seed=1900 + len(out), name="pw3-%s-c%d-co%d" % (dt, ci, co)))
    out.append(Case("dw_pw", 3, 5, 7, 64, 64, 48, 3, 1, 1, "bf16", "nhwc", ("relu", "none", "none"), bias=True,
                    seed=1990, name="dwpw3-bf16-small-image"))
    out.append(Case("dw_pw", 2, 1, 1, 32, 32, 16, 3, 2, 1, "bf16", "nhwc", ("none", "none", "none"), bias=True,
                    seed=1991, name="dwpw3-bf16-1x1"))
    out.append(Case("dw_pw", 1, 6, 5, 600, 600, 300, 3, 1, 1, "bf16", "nhwc", ("relu", "none", "none"), bias=True,
                    seed=1992, name="dwpw3-bf16-c600-co300"))
    return out


# (workgroup cap, ring depth, splits); 0 = the planner's choice
LAUNCH = ((0, 0, 1), (3, 2, 1), (3, 0, 1), (2, 5, 1), (2, 8, 1), (0, 0, 2), (3, 0, 3), (0, 2, 4))


def _v3_plans(case, launch=((0, 0, 1),)):
    desc = fcm.desc_from_case(case)
    cb = 64 // ELT[case.dtype]
    plans = []
    for v in range(fcm.lib().fcm_variant_count()):
        name = fcm.variant_name(v)
        if not name.startswith(("k_dwpw3", "k_pw3", "k_dw3")):
            continue
        for th, tw in TILES:
            cobs = [cb] if case.op == "dw" else [16 * int(name.split(",")[4])]
            for cob in cobs:
                for cap, depth, splits in launch:
                    try:
                        p = fcm.plan_evaluate(case.op, desc, th, tw, cb, cob, v, workgroups=cap, depth=depth,
                                              splits=splits)
                    except fcm.FcmError:
                        continue
                    plans.append(p)
    return plans


CASES = _cases()


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_persistent_variants_match_oracle(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    plans = _v3_plans(case, launch=LAUNCH)
    assert plans, "no persistent variant implements %s" % case.name
    for p in plans:
        got = to_np(run_fused(case, d, plan=p))
        assert_close(got, ref, case.dtype, "%s %s tile %dx%d grid %d depth %d splits %d" % (
            case.name, fcm.variant_name(p.variant), p.tile_h, p.tile_w, p.workgroups, p.depth, p.splits))
