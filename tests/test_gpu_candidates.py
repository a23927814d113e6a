"""GPU parity of every plan the benchmark's device timing may choose.

bench.py runs, for each layer of every named configuration, the fastest of the planner's
candidate plans (fcm_plan_candidates, at most 12, caller workspace up to 64 MiB), and for
the layer-by-layer comparison the fastest candidate of each stage. Here every one of those
candidates runs at full size and is compared with the CPU oracle: the whole output where
the oracle finishes in seconds, a strided sample of images on the two large token grids
(images are independent). Unfused stage candidates are checked through the whole
layer-by-layer chain, one stage's candidate at a time with the planner's plans elsewhere.
"""
import numpy as np
import pytest

import bench
from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import make_inputs, config_c1, config_c2, config_c3, config_c4, config_c5

from gpu_util import assert_close_dev, batch_slice, dev_inputs, oracle_ref, run_fused

pytestmark = pytest.mark.gpu

MAX_CANDIDATES = 12
WORKSPACE = 64 << 20

CASES = config_c1() + config_c2() + config_c3(batches=(1, 32)) + config_c4() + config_c5()


def _sample(case):
    """Images compared: all, or every 8th plus the last on the large token grids."""
    if case.op == "dw_pw" and case.n == 64 and case.h != 14:
        return list(range(0, case.n, 8)) + [case.n - 1]
    return None


def _ref(case, inp):
    idx = _sample(case)
    if idx is None:
        return oracle_ref(case, inp), None
    return oracle_ref(case.with_(n=len(idx)), batch_slice(inp, idx)), idx


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name.replace(" ", "_"))
def test_every_candidate_plan_matches_oracle(case):
    inp = make_inputs(case)
    ref, idx = _ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    desc = fcm.desc_from_case(case)
    ws = WORKSPACE if case.op == "dw_pw" else 0
    cands = fcm.plan_candidates(case.op, desc, MAX_CANDIDATES, ws)
    assert cands
    for p in cands:
        got = run_fused(case, d, plan=p)
        if idx is not None:
            got = got[idx]
        assert_close_dev(got, ref, case.dtype, "%s %s %dx%d splits %d" % (
            case.name, fcm.variant_name(p.variant), p.tile_h, p.tile_w, p.splits))


def _unfused(case, d, plans):
    kw = dict(stride=case.stride, pad=case.pad, layout=case.layout, plans=plans, zp_in=case.zp_in)
    rq = list(case.rq) if case.dtype == "i8" else None
    if case.op == "dw_pw":
        return fcm.dw_then_pw(d["x"], d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), act=case.act[:2], rq=rq,
                              **kw)
    return fcm.pw_then_dw_then_pw(d["x"], d["w_pw1"], d["w_dw"], d["w_pw2"], d.get("b_pw1"), d.get("b_dw"),
                                  d.get("b_pw2"), act=case.act, rq=rq, **kw)


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name.replace(" ", "_"))
def test_every_unfused_stage_candidate_matches_oracle(case):
    inp = make_inputs(case)
    ref, idx = _ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    stages = bench.stage_ops(case)
    descs = [bench.stage_desc(fcm, case, s) for s in stages]
    base = [fcm.plan(s[0], sd) for s, sd in zip(stages, descs)]
    for i, (s, sd) in enumerate(zip(stages, descs)):
        for p in fcm.plan_candidates(s[0], sd, MAX_CANDIDATES, WORKSPACE if s[0] == "pw" else 0):
            plans = list(base)
            plans[i] = p
            got = _unfused(case, d, plans)
            if idx is not None:
                got = got[idx]
            assert_close_dev(got, ref, case.dtype, "%s stage %d %s %dx%d splits %d" % (
                case.name, i, fcm.variant_name(p.variant), p.tile_h, p.tile_w, p.splits))


def test_candidate_outputs_are_bit_identical_for_int8():
    """int8 results are unique: every candidate of the int8 layers gives the same bytes."""
    for case in config_c4():
        d = dev_inputs(make_inputs(case), case.dtype)
        desc = fcm.desc_from_case(case)
        outs = [run_fused(case, d, plan=p).cpu().numpy() for p in fcm.plan_candidates(case.op, desc, 12, WORKSPACE)]
        assert all(np.array_equal(outs[0], o) for o in outs[1:])
