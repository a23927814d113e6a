"""GPU parity of the deep DW->PW kernels (bf16, 3x3), forced through explicit plans.

Every compiled instance runs at the planner's grid and at small capped grids (one
workgroup streams many tiles and chunks through its three-deep load pipeline, the
epilogue of one tile overlapping the next tile's loads), on images with ragged tiles,
chunk counts per workgroup that are and are not multiples of three, a ragged last
output-channel block, biases and activations; compared with the CPU oracle at the bf16
tolerance. Input channels not in whole 32-channel chunks (64-channel pairs for the
two-chunk instances) are not offered to these kernels (checked on the CPU with the
planner).
"""
import re

import pytest

from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import Case, make_inputs

from gpu_util import assert_close, dev_inputs, oracle_ref, run_fused, to_np

pytestmark = pytest.mark.gpu

CAPS = (0, 3, 7)


def _cases():
    out = []
    for s in (1, 2):
        for n, h, w, ci, co in ((2, 9, 11, 64, 136), (1, 14, 14, 288, 256), (3, 7, 7, 96, 520), (2, 1, 1, 32, 16),
                                (1, 15, 16, 512, 72)):
            out.append(Case("dw_pw", n, h, w, ci, ci, co, 3, s, 1, "bf16", "nhwc", ("relu6", "relu", "none"),
                            bias=True, seed=4000 + len(out), name="dwpw7-n%d-%dx%d-c%d-co%d-s%d" % (n, h, w, ci, co, s)))
    out.append(Case("dw_pw", 2, 14, 14, 96, 96, 264, 3, 1, 1, "bf16", "nhwc", ("none", "none", "none"), bias=False,
                    seed=4100, name="dwpw7-co264-nobias"))
    return out


def _v7_plans(case):
    desc = fcm.desc_from_case(case)
    plans = []
    for v in range(fcm.lib().fcm_variant_count()):
        name = fcm.variant_name(v)
        if not name.startswith("k_dwpw7<"):
            continue
        th, tw = [int(t) for t in name.split(",")[3].split("x")]
        cob = 64 * int(re.search(r"ct(\d+)", name).group(1))
        for cap in CAPS:
            try:
                p = fcm.plan_evaluate(case.op, desc, th, tw, 32, cob, v, workgroups=cap)
            except fcm.FcmError:
                continue
            plans.append(p)
    return plans


CASES = _cases()


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_deep_variants_match_oracle(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    plans = _v7_plans(case)
    assert plans, "no deep variant implements %s" % case.name
    for p in plans:
        got = to_np(run_fused(case, d, plan=p))
        assert_close(got, ref, case.dtype, "%s %s grid %d" % (case.name, fcm.variant_name(p.variant), p.workgroups))


def test_every_deep_variant_is_exercised():
    names = {fcm.variant_name(p.variant) for c in CASES for p in _v7_plans(c)}
    every = {fcm.variant_name(v) for v in range(fcm.lib().fcm_variant_count())
             if fcm.variant_name(v).startswith("k_dwpw7<")}
    assert every and names == every, sorted(every - names)
