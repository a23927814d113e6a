"""GPU parity of the streaming NHWC kernels (DW->PW, PW, DW), forced through explicit plans.

Each streaming variant has one compiled tile and output-channel block; every variant that
implements a case runs at the planner's grid and at small capped grids, so that one
workgroup streams many (tile, channel block) items and the deferred epilogue of one item
overlaps the next item's copies, across image borders, ragged tiles, ragged channel chunks
(input channels not a multiple of the 64-byte chunk) and ragged output-channel blocks.
Compared with the CPU oracle at the bf16 tolerance.
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
    for k, s in ((3, 1), (3, 2)):
        for ci, co, h, w in ((40, 24, 19, 23), (96, 200, 17, 30), (264, 72, 9, 33), (64, 136, 1, 1), (32, 26, 3, 5)):
            out.append(Case("dw_pw", 2, h, w, ci, ci, co, k, s, 1, "bf16", "nhwc", ("relu", "relu6", "none"),
                            bias=True, seed=2500 + len(out), name="dwpw5-c%d-co%d-%dx%d-k%ds%d" % (ci, co, h, w, k, s)))
        for ci, h, w in ((40, 19, 23), (136, 10, 37)):
            out.append(Case("dw", 2, h, w, ci, ci, ci, k, s, 1, "bf16", "nhwc", ("relu6",) * 3, bias=True,
                            seed=2600 + len(out), name="dw5-c%d-%dx%d-k%ds%d" % (ci, h, w, k, s)))
    for ci, co, h, w in ((40, 24, 19, 23), (96, 200, 9, 35), (264, 136, 5, 7)):
        out.append(Case("pw", 2, h, w, ci, ci, co, 1, 1, 0, "bf16", "nhwc", ("relu",) * 3, bias=True,
                        seed=2700 + len(out), name="pw5-c%d-co%d-%dx%d" % (ci, co, h, w)))
    return out


def _v5_plans(case):
    desc = fcm.desc_from_case(case)
    plans = []
    for v in range(fcm.lib().fcm_variant_count()):
        name = fcm.variant_name(v)
        if not name.startswith(("k_dwpw5<", "k_pw5<", "k_dw5<")):
            continue
        th, tw = [int(t) for t in name.split(",")[3].split("x")]
        m = re.search(r"ct(\d+),wc(\d+)", name)
        cob = 32 if name.startswith("k_dw5<") else 16 * int(m.group(1)) * int(m.group(2))
        for cap in CAPS:
            try:
                p = fcm.plan_evaluate(case.op, desc, th, tw, 32, cob, v, workgroups=cap)
            except fcm.FcmError:
                continue
            plans.append(p)
    return plans


CASES = _cases()


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_streaming_variants_match_oracle(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    plans = _v5_plans(case)
    assert plans, "no streaming variant implements %s" % case.name
    for p in plans:
        got = to_np(run_fused(case, d, plan=p))
        assert_close(got, ref, case.dtype, "%s %s grid %d" % (case.name, fcm.variant_name(p.variant), p.workgroups))


def test_every_streaming_variant_is_exercised():
    names = {fcm.variant_name(p.variant) for c in CASES for p in _v5_plans(c)}
    every = {fcm.variant_name(v) for v in range(fcm.lib().fcm_variant_count())
             if fcm.variant_name(v).startswith(("k_dwpw5<", "k_pw5<", "k_dw5<"))}
    assert every and names == every, sorted(every - names)
