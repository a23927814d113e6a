"""GPU parity of the whole-module fp32 kernels for small batches, forced through explicit
plans: every compiled instance that implements a case (module, depthwise geometry) runs
on images that leave ragged tiles at the right and bottom, with channel counts that are
not multiples of the 16-channel MFMA chunk (and a few that are), both layouts, biases and
activations; compared with the CPU oracle at the fp32 tolerance. (The kernels take input
and depthwise channel counts in fours; output channels are free.) The last PW stage's
split of channel chunks over waves (fewer output tiles than waves) is covered by the small
output-channel counts.
"""
import pytest

from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import Case, make_inputs

from gpu_util import assert_close, dev_inputs, oracle_ref, run_fused, to_np

pytestmark = pytest.mark.gpu

ACTS = ("relu6", "relu", "none")


def _cases():
    out = []
    geo = [(3, 1), (3, 2), (5, 1), (5, 2)]
    for lay in ("nchw", "nhwc"):
        for k, s in geo:
            for ci, co in ((24, 64), (8, 5), (40, 24)):
                out.append(Case("dw_pw", 2, 13, 11, ci, ci, co, k, s, k // 2, "f32", lay, ACTS, bias=True,
                                seed=3000 + len(out), name="dwpw6-%s-c%d-co%d-k%ds%d" % (lay, ci, co, k, s)))
            for ci, cm in ((24, 40), (4, 20)) if k == 3 else ():
                out.append(Case("pw_dw", 2, 13, 11, ci, cm, cm, k, s, k // 2, "f32", lay, ACTS, bias=True,
                                seed=3100 + len(out), name="pwdw6-%s-c%d-cm%d-k%ds%d" % (lay, ci, cm, k, s)))
            for ci, cm, co in ((24, 144, 24), (4, 36, 3), (16, 48, 40)) if (k, s) != (5, 2) else ():
                out.append(Case("pw_dw_pw", 2, 13, 11, ci, cm, co, k, s, k // 2, "f32", lay, ACTS, bias=True,
                                seed=3200 + len(out), name="pwdwpw6-%s-c%d-cm%d-co%d-k%ds%d" % (lay, ci, cm, co, k, s)))
    out.append(Case("pw_dw_pw", 1, 3, 2, 24, 144, 24, 3, 1, 1, "f32", "nchw", ACTS, bias=False, seed=3300,
                    name="pwdwpw6-tiny-image"))
    out.append(Case("dw_pw", 1, 1, 1, 32, 32, 64, 3, 2, 1, "f32", "nchw", ACTS, bias=True, seed=3301,
                    name="dwpw6-1x1"))
    return out


def _v6_plans(case):
    desc = fcm.desc_from_case(case)
    last = case.c_mid if case.op == "pw_dw" else case.c_out
    plans = []
    for v in range(fcm.lib().fcm_variant_count()):
        name = fcm.variant_name(v)
        if not name.startswith(("k_dwpw6<", "k_pwdw6<", "k_pwdwpw6<")):
            continue
        th, tw = [int(t) for t in name.split(",")[3].rstrip(">").split("x")]
        try:
            plans.append(fcm.plan_evaluate(case.op, desc, th, tw, 16, -(-last // 16) * 16, v))
        except fcm.FcmError:
            continue
    return plans


CASES = _cases()


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_small_batch_kernels_match_oracle(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    plans = _v6_plans(case)
    assert plans, "no small-batch kernel implements %s" % case.name
    for p in plans:
        got = to_np(run_fused(case, d, plan=p))
        assert_close(got, ref, case.dtype, "%s %s" % (case.name, fcm.variant_name(p.variant)))


def test_every_small_batch_variant_is_exercised():
    names = {fcm.variant_name(p.variant) for c in CASES for p in _v6_plans(c)}
    every = {fcm.variant_name(v) for v in range(fcm.lib().fcm_variant_count())
             if fcm.variant_name(v).startswith(("k_dwpw6<", "k_pwdw6<", "k_pwdwpw6<"))}
    assert every and names == every, sorted(every - names)
