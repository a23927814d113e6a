"""GPU parity of whole chains (FusePlanner over a network, Sec. IV): the MobileNetV2 body
(51 DW/PW layers after the stem, no skip connections) planned three ways -- least
Eq. 1-4 bytes, least modelled time, every layer alone -- and run through fcm_chain_run,
against the CPU oracle applied layer by layer. int8 is bit-exact end to end. Float chains
are compared with the oracle at the parity tolerance over their first stages, and the full
bf16 body kernel by kernel, each kernel fed the device's own output of the kernel before:
rounding a layer's result to bfloat16 in a different order can flip a last bit that later
layers carry along, so end to end the full float chains are compared between the plans."""
import numpy as np
import pytest

from paper_2404_19331_amd.workloads import MNV2_STAGES, mobilenetv2_chain, make_chain_inputs

from gpu_util import assert_close, oracle_chain, run_chain, to_dev, to_np

pytestmark = pytest.mark.gpu

OBJECTIVES = ("bytes", "time", "unfused")


def _dev(spec):
    x, ws, bs = make_chain_inputs(spec)
    return (x, ws, bs), (to_dev(x, spec.dtype), [to_dev(w, spec.dtype) for w in ws],
                         [to_dev(b, spec.dtype) for b in bs])


@pytest.mark.parametrize("layout", ["nhwc", "nchw"])
def test_int8_mobilenetv2_chain_bit_exact(layout):
    spec = mobilenetv2_chain(n=2, dtype="i8", layout=layout, h=112 if layout == "nhwc" else 56,
                             w=112 if layout == "nhwc" else 56)
    host, dev = _dev(spec)
    ref = oracle_chain(spec, *host)
    assert 0.05 < np.mean(ref != 0) and np.mean(np.abs(ref.astype(int)) == 127) < 0.2  # a spread result
    for obj in OBJECTIVES:
        got, plan = run_chain(spec, obj, *dev)
        assert np.array_equal(to_np(got), ref), "%s plan (%d groups, %d fused layers)" % (
            obj, plan.num_groups, plan.fused_layers)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_float_chain_first_stages_match_oracle(dtype):
    spec = mobilenetv2_chain(n=2, dtype=dtype, stages=MNV2_STAGES[:3], final_pw=False)
    host, dev = _dev(spec)
    ref = oracle_chain(spec, *host)
    for obj in OBJECTIVES:
        got, plan = run_chain(spec, obj, *dev)
        assert_close(to_np(got), ref, dtype, "%s chain, %s plan" % (dtype, obj))


def test_bf16_full_chain_plans_agree():
    spec = mobilenetv2_chain(n=2, dtype="bf16")
    _, dev = _dev(spec)
    outs = {obj: to_np(run_chain(spec, obj, *dev)[0]) for obj in OBJECTIVES}
    for obj in ("bytes", "time"):
        assert_close(outs[obj], outs["unfused"], "bf16", "full bf16 chain, %s plan vs layer by layer" % obj)


def test_autotuned_chain_plan_runs_bit_exact():
    from paper_2404_19331_amd import fcm
    from paper_2404_19331_amd.autotune import chain_autotune
    spec = mobilenetv2_chain(n=2, dtype="i8", stages=MNV2_STAGES[:4], final_pw=False)
    host, dev = _dev(spec)
    ref = oracle_chain(spec, *host)
    d = fcm.chain_desc(spec.n, spec.h, spec.w, spec.c, spec.layers, spec.dtype, spec.layout)
    plan, timed = chain_autotune(d, reps=3)
    assert plan.num_groups >= 1 and len(timed) >= len(spec.layers)
    got = fcm.chain_run(d, plan, dev[0], dev[1], dev[2])
    assert np.array_equal(to_np(got), ref)


@pytest.mark.parametrize("objective", OBJECTIVES)
def test_bf16_full_chain_each_kernel_against_oracle(objective):
    """Every kernel of the full bf16 MobileNetV2 body at its true depth: the planned chain runs
    one group (kernel) at a time, each group fed the device's own output of the group
    before, and each group's output is compared with the oracle applied to that group's
    layers on the same input, so no rounding carries from one kernel into the next
    comparison."""
    import dataclasses
    from paper_2404_19331_amd import fcm
    spec = mobilenetv2_chain(n=2, dtype="bf16")
    host, dev = _dev(spec)
    d = fcm.chain_desc(spec.n, spec.h, spec.w, spec.c, spec.layers, spec.dtype, spec.layout)
    plan = fcm.chain_plan(d, objective)
    firsts = [plan.first[i] for i in range(plan.num_groups)] + [len(spec.layers)]
    assert firsts[0] == 0 and all(a < b for a, b in zip(firsts, firsts[1:]))
    x = dev[0]
    h, w, c = spec.h, spec.w, spec.c
    for g in range(plan.num_groups):
        a, b = firsts[g], firsts[g + 1]
        sub = dataclasses.replace(spec, h=h, w=w, c=c, layers=spec.layers[a:b])
        sd = fcm.chain_desc(sub.n, h, w, c, sub.layers, sub.dtype, sub.layout)
        sp = fcm.ChainPlan()
        sp.objective, sp.num_groups, sp.first[0], sp.op[0], sp.plan[0] = plan.objective, 1, 0, plan.op[g], plan.plan[g]
        y = fcm.chain_run(sd, sp, x, dev[1][a:b], dev[2][a:b])
        ref = oracle_chain(sub, to_np(x), host[1][a:b], host[2][a:b])
        assert_close(to_np(y), ref, "bf16", "%s plan, kernel %d (layers %d..%d)" % (objective, g, a, b - 1))
        x = y
        for L in sub.layers:
            if L["kind"] == "dw":
                h, w = fcm.out_hw(h, w, L["k"], L["stride"], L["pad"])
            else:
                c = L["c_out"]
