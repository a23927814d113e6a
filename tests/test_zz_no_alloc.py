"""GPU: fcm_dw_pw_noalloc (split partial sums in the library's fixed per-GPU array)
against fcm_dw_pw_ws (the same plans with a caller workspace), through the C ABI, on two
calls in a row, the second with a smaller input (symmetric int8, int8 with zero points and
per-channel requantisation, bf16); and its refusal of plans that need more than the array
holds."""
import numpy as np
import pytest

from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import Case, config_c4_spread, make_inputs

from gpu_util import assert_close, dev_inputs, to_np, torch
import oracle

pytestmark = pytest.mark.gpu
EINVAL = 1


def _split_plan(case, splits):
    desc = fcm.desc_from_case(case)
    e = {"f32": 4, "bf16": 2, "i8": 1}[case.dtype]
    for v in range(fcm.lib().fcm_variant_count()):
        name = fcm.variant_name(v)
        if name.startswith("k_dwpw3<%s,%d,%d," % (case.dtype, case.k, case.stride)):
            ct = int(name.split(",")[4])
            try:
                return fcm.plan_evaluate("dw_pw", desc, 7, 7, 64 // e, 16 * ct, v, splits=splits)
            except fcm.FcmError:
                continue
    raise AssertionError(case.name)


def _both(case, plan):
    """(noalloc result, caller-workspace result) of the case under `plan` (None = planner)."""
    T = torch()
    d = dev_inputs(make_inputs(case), case.dtype)
    kw = dict(stride=case.stride, pad=case.pad, act=case.act[:2], layout=case.layout,
              rq=list(case.rq) if case.dtype == "i8" else None)
    desc = fcm.desc_from_case(case)
    p = plan if plan is not None else fcm.plan_limited("dw_pw", desc, fcm.NOALLOC_SCRATCH_BYTES)
    ws = T.empty(max(16, fcm.workspace_bytes(desc, p)), dtype=T.uint8, device="cuda")
    ref = fcm.dw_pw(d["x"], d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), plan=p, workspace=ws, **kw)
    got = fcm.dw_pw_noalloc(d["x"], d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), plan=plan, **kw)
    T.cuda.synchronize()
    return to_np(got), to_np(ref)


@pytest.mark.parametrize("splits", [4, 2])
def test_noalloc_int8_two_calls_second_smaller(splits):
    big = config_c4_spread()[1]                      # 8 x 14x14x480 -> 112
    small = big.with_(n=2, h=9, w=11, seed=big.seed + 1)  # then a smaller input
    for case in (big, small):
        p = _split_plan(case, splits)
        assert 0 < fcm.workspace_bytes(fcm.desc_from_case(case), p) <= fcm.NOALLOC_SCRATCH_BYTES
        got, ref = _both(case, p)
        assert np.array_equal(got, ref), case.name


def test_noalloc_int8_zero_points_per_channel_two_calls():
    """Split plans of the int8 kernel instances with zero points and per-channel scales:
    each split's share of the zero-point term goes into the array with its partial sums,
    and the combine requantises per channel; bit-exact against the workspace path and the
    oracle."""
    T = torch()
    base = config_c4_spread()[1]  # 8 x 14x14x480 -> 112
    rq = tuple(tuple(r[:4]) + (z,) for r, z in zip(base.rq, (-7, 11, 0)))
    big = base.with_(rq=rq, zp_in=-20, name="noalloc-zp-pc-big")
    small = big.with_(n=2, h=9, w=11, seed=big.seed + 1, name="noalloc-zp-pc-small")
    rng = np.random.default_rng(77)
    for case in (big, small):
        pcs = [(rng.integers(1 << 14, 1 << 16, n), rng.integers(20, 26, n)) for n in (case.c_in, case.c_out)]
        rqc = [T.from_numpy(np.concatenate(pc).astype(np.int32)).cuda() for pc in pcs]
        desc = fcm.desc_from_case(case)
        for i, t in enumerate(rqc):
            desc.rq_channel[i] = t.data_ptr()
        p = _split_plan(case, 4)
        p = fcm.plan_evaluate("dw_pw", desc, p.tile_h, p.tile_w, p.c_block, p.co_block, p.variant, splits=4)
        assert p.splits == 4 and 0 < fcm.workspace_bytes(desc, p) <= fcm.NOALLOC_SCRATCH_BYTES
        inp = make_inputs(case)
        ref = oracle.run("dw_pw", dict(case.as_dict(), rq_channel=pcs), inp)
        assert len(np.unique(ref)) > 8, case.name
        d = dev_inputs(inp, case.dtype)
        kw = dict(stride=case.stride, pad=case.pad, act=case.act[:2], layout=case.layout, rq=list(case.rq),
                  rq_channel=rqc, zp_in=case.zp_in, plan=p)
        ws = T.empty(fcm.workspace_bytes(desc, p), dtype=T.uint8, device="cuda")
        via_ws = fcm.dw_pw(d["x"], d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), workspace=ws, **kw)
        got = fcm.dw_pw_noalloc(d["x"], d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), **kw)
        T.cuda.synchronize()
        assert np.array_equal(to_np(got), ref), case.name
        assert np.array_equal(to_np(via_ws), ref), case.name


def test_noalloc_bf16_planner_choice_two_calls():
    a = Case("dw_pw", 1, 14, 14, 512, 512, 512, 3, 1, 1, "bf16", "nhwc", ("relu", "relu", "none"), bias=True,
             dist_x="n01", seed=901, name="noalloc-bf16-a")
    b = a.with_(h=7, w=7, c_in=256, c_mid=256, c_out=128, seed=902, name="noalloc-bf16-b")
    for case in (a, b):
        got, ref = _both(case, None)
        assert_close(got, ref, "bf16", case.name)


def test_noalloc_refuses_plans_beyond_its_array():
    case = Case("dw_pw", 32, 14, 14, 512, 512, 512, 3, 1, 1, "bf16", "nhwc", ("relu", "relu", "none"), seed=903)
    p = _split_plan(case, 2)  # 2 x 256 work tiles x 49 pixels x 256 channels x 4 bytes = 25.7 MB
    assert fcm.workspace_bytes(fcm.desc_from_case(case), p) > fcm.NOALLOC_SCRATCH_BYTES
    d = dev_inputs(make_inputs(case.with_(n=1)), case.dtype)  # pointers only: refused before launch
    T = torch()
    x = T.zeros((32, 14, 14, 512), dtype=T.bfloat16, device="cuda")
    with pytest.raises(fcm.FcmError) as e:
        fcm.dw_pw_noalloc(x, d["w_dw"], d["w_pw"], act=("relu", "relu"), layout="nhwc", plan=p)
    assert e.value.status == EINVAL
