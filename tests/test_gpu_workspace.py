"""GPU: split plans run with a caller workspace (the library allocates nothing).

A split plan spreads each work tile's input-channel chunks over several workgroups; their
partial sums go to the caller's workspace and a second kernel adds them in split order.
int8 sums are exact, so split and unsplit plans, and two concurrent split launches on two
streams with two workspaces, give bit-identical results equal to the oracle's."""
import numpy as np
import pytest

from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import Case, config_c4_spread, make_inputs

from gpu_util import assert_close, dev_inputs, oracle_ref, run_fused, to_np, torch

pytestmark = pytest.mark.gpu


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
    raise AssertionError("no persistent kernel implements %s" % case.name)


def test_two_streams_two_workspaces_bit_identical_int8():
    case = config_c4_spread()[1]  # 14x14x480 -> 112, int8, batch 8: 8 channel chunks
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    T = torch()
    p = _split_plan(case, 4)
    need = fcm.workspace_bytes(fcm.desc_from_case(case), p)
    assert p.splits == 4 and need > 0
    ws = [T.empty(need, dtype=T.uint8, device="cuda") for _ in range(2)]
    streams = [T.cuda.Stream(), T.cuda.Stream()]
    outs = []
    T.cuda.synchronize()
    for s, w in zip(streams, ws):
        with T.cuda.stream(s):
            outs.append(fcm.dw_pw(d["x"], d["w_dw"], d["w_pw"], stride=case.stride, pad=case.pad, act=case.act[:2],
                                  rq=list(case.rq), layout=case.layout, plan=p, workspace=w, stream=s))
    T.cuda.synchronize()
    a, b = to_np(outs[0]), to_np(outs[1])
    assert np.array_equal(a, b)
    assert_close(a, ref, "i8", case.name + " split 4")
    unsplit = to_np(run_fused(case, d, plan=_split_plan(case, 1)))
    assert np.array_equal(a, unsplit)


def test_split_plan_without_workspace_is_refused_and_short_one_too():
    case = config_c4_spread()[1]
    d = dev_inputs(make_inputs(case), case.dtype)
    p = _split_plan(case, 2)
    need = fcm.workspace_bytes(fcm.desc_from_case(case), p)
    T = torch()
    with pytest.raises(ValueError):
        fcm.dw_pw(d["x"], d["w_dw"], d["w_pw"], stride=case.stride, pad=case.pad, act=case.act[:2],
                  rq=list(case.rq), layout=case.layout, plan=p, workspace=T.empty(need - 16, dtype=T.uint8,
                                                                                    device="cuda"))


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_split_plans_float_match_the_oracle(dt):
    case = Case("dw_pw", 2, 14, 14, 512, 512, 256, 3, 1, 1, dt, "nhwc", ("relu", "relu", "none"), bias=True,
                dist_x="n01", seed=4242, name="split-%s" % dt)
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    for splits in (2, 4, 8):
        got = to_np(run_fused(case, d, plan=_split_plan(case, splits)))
        assert_close(got, ref, dt, "%s splits %d" % (case.name, splits))


@pytest.mark.parametrize("dt,co", [("f32", 18), ("f32", 20), ("bf16", 18), ("bf16", 36)])
def test_split_plans_ragged_output_channels(dt, co):
    """The combine kernel stores four output channels per thread with one aligned store, and
    one by one where c_out leaves a partial group of four (c_out % 4 != 0): both match the
    oracle at every split count."""
    case = Case("dw_pw", 2, 9, 11, 256, 256, co, 3, 1, 1, dt, "nhwc", ("relu", "none", "none"), bias=True,
                dist_x="n01", seed=4300 + co, name="split-%s-co%d" % (dt, co))
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    for splits in (2, 4, 8):
        p = _split_plan(case, splits)
        assert p.splits == splits
        got = to_np(run_fused(case, d, plan=p))
        assert_close(got, ref, dt, "%s splits %d" % (case.name, splits))
