"""Host-side tests of the chain planner (FusePlanner over a network, Sec. IV): the
partition it returns is the least-cost one (checked against brute force over every
partition of short random chains, using the module planner's own estimates), the
pairwise rule of Sec. IV-B (fuse exactly when the module's Eq. 1-4 estimate is below its
layers'), the layer-by-layer objective, shapes and workspace, and rejected chains."""
import itertools

import numpy as np
import pytest

from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import mobilenetv2_chain

EINVAL, EUNSUPPORTED = 1, 2
KINDS = {"dw_pw": ("dw", "pw"), "pw_dw": ("pw", "dw"), "pw_pw": ("pw", "pw"), "pw_dw_pw": ("pw", "dw", "pw"),
         "dw": ("dw",), "pw": ("pw",)}


def _random_chain(rng, nl, dtype):
    layers = []
    for _ in range(nl):
        if rng.random() < 0.5:
            layers.append(dict(kind="pw", c_out=int(rng.choice([16, 24, 48, 96, 144])),
                               act="relu" if rng.random() < 0.5 else "none", rq=(1, 9, -127, 127)))
        else:
            layers.append(dict(kind="dw", k=int(rng.choice([3, 5])), stride=int(rng.choice([1, 2])), pad=1,
                               act="relu", rq=(1, 5, -127, 127)))
            layers[-1]["pad"] = layers[-1]["k"] // 2
    return layers


def _group_desc(n, h, w, c, layers, first, op, dtype):
    """fcm_desc of module `op` over layers[first:], or None if they do not form it."""
    kinds = KINDS[op]
    sub = layers[first:first + len(kinds)]
    if len(sub) != len(kinds) or tuple(L["kind"] for L in sub) != kinds:
        return None
    for L in layers[:first]:  # shape at `first`
        if L["kind"] == "pw":
            c = L["c_out"]
        else:
            h, w = fcm.out_hw(h, w, L["k"], L["stride"], L["pad"])
    k = stride = 1
    pad = 0
    chans = [c]
    for L in sub:
        if L["kind"] == "dw":
            k, stride, pad = L["k"], L["stride"], L["pad"]
            chans.append(chans[-1])
        else:
            chans.append(L["c_out"])
    c_mid = chans[1] if op != "dw_pw" else c
    return fcm.make_desc(n, h, w, c, c_mid, chans[-1], k=k, stride=stride, pad=pad, dtype=dtype, layout="nhwc",
                         act=[L["act"] for L in sub], rq=[L["rq"] for L in sub])


def _brute_force_bytes(n, h, w, c, layers, dtype):
    """Least summed bytes_paper over every partition of the chain into modules."""
    memo = {}

    def best(i):
        if i == len(layers):
            return 0
        if i in memo:
            return memo[i]
        out = None
        for op in KINDS:
            d = _group_desc(n, h, w, c, layers, i, op, dtype)
            if d is None:
                continue
            try:
                b = fcm.plan(op, d).bytes_paper
            except fcm.FcmError:
                continue
            v = b + best(i + len(KINDS[op]))
            out = v if out is None else min(out, v)
        memo[i] = out
        return out

    return best(0)


@pytest.mark.parametrize("seed", range(12))
def test_chain_plan_is_the_least_cost_partition(seed):
    rng = np.random.default_rng(seed)
    nl = int(rng.integers(1, 8))
    dtype = ["i8", "bf16", "f32"][seed % 3]
    layers = _random_chain(rng, nl, dtype)
    n, h, w, c = 2, 28, 28, 32
    d = fcm.chain_desc(n, h, w, c, layers, dtype)
    p = fcm.chain_plan(d, "bytes")
    assert p.bytes_paper == _brute_force_bytes(n, h, w, c, layers, dtype)
    # the groups tile the chain and each group's plan is the module planner's own
    nxt = 0
    for first, op, plan in p.groups():
        assert first == nxt
        desc = _group_desc(n, h, w, c, layers, first, op, dtype)
        assert plan.as_dict() == fcm.plan(op, desc).as_dict()
        nxt += len(KINDS[op])
    assert nxt == nl
    assert p.bytes_paper <= p.bytes_lbl_paper
    u = fcm.chain_plan(d, "unfused")
    assert u.num_groups == nl and u.fused_layers == 0 and u.bytes_paper == p.bytes_lbl_paper
    assert [op for _, op, _ in u.groups()] == [L["kind"] for L in layers]
    t = fcm.chain_plan(d, "time")
    assert t.time_est <= t.time_lbl_est + 1e-12


@pytest.mark.parametrize("pair", ["dw_pw", "pw_dw", "pw_pw"])
def test_two_layer_chain_follows_the_pairwise_rule(pair):
    # Sec. IV-B: fuse when the module's estimate is below the sum of its layers'
    for hw_, c in ((56, 32), (14, 512), (7, 960)):
        layers = [dict(kind=k, c_out=c if k == "pw" else 0, k=3, stride=1, pad=1, act="relu",
                       rq=(1, 8, -127, 127)) for k in KINDS[pair]]
        d = fcm.chain_desc(8, hw_, hw_, c, layers, "i8")
        p = fcm.chain_plan(d, "bytes")
        desc = _group_desc(8, hw_, hw_, c, layers, 0, pair, "i8")
        fused = fcm.plan(pair, desc).bytes_paper < p.bytes_lbl_paper
        assert (p.num_groups == 1) == fused
        assert (p.fused_layers == 2) == fused


def test_mobilenetv2_chain_shapes_and_workspace():
    sp = mobilenetv2_chain(n=8, dtype="i8")
    assert len(sp.layers) == 51
    d = fcm.chain_desc(sp.n, sp.h, sp.w, sp.c, sp.layers, sp.dtype, sp.layout)
    assert fcm.chain_output_shape(d) == (8, 7, 7, 1280)
    for obj in ("bytes", "time", "unfused"):
        p = fcm.chain_plan(d, obj)
        # the largest activation between groups, and two 256-byte aligned buffers of it
        sizes = []
        h, w, c = sp.h, sp.w, sp.c
        ends = [first + len(KINDS[op]) for first, op, _ in p.groups()][:-1]
        for i, L in enumerate(sp.layers):
            if L["kind"] == "pw":
                c = L["c_out"]
            else:
                h, w = fcm.out_hw(h, w, L["k"], L["stride"], L["pad"])
            if i + 1 in ends:
                sizes.append(8 * h * w * c)
        assert p.act_bytes_max == max(sizes)
        assert fcm.lib().fcm_chain_workspace_bytes(p) == 2 * (-(-max(sizes) // 256) * 256)
    fused = fcm.chain_plan(d, "bytes")
    assert 0 < fused.fused_layers < 51 and fused.bytes_paper < fused.bytes_lbl_paper


def test_chain_validation():
    good = [dict(kind="pw", c_out=32, act="relu"), dict(kind="dw", k=3, stride=1, pad=1)]
    bad_layers = [
        [dict(kind="pw", c_out=0)],                        # no output channels
        [dict(kind="dw", k=3, stride=0, pad=1)],           # stride 0
        [dict(kind="dw", k=5, stride=1, pad=0)] * 3,       # 4x4 image shrinks below the filter
    ]
    for layers in bad_layers:
        d = fcm.chain_desc(1, 4, 4, 8, layers, "f32")
        with pytest.raises(fcm.FcmError) as e:
            fcm.chain_plan(d, "bytes")
        assert e.value.status == EINVAL
    d = fcm.chain_desc(1, 8, 8, 8, good, "f32")
    d.num_layers = 0
    with pytest.raises(fcm.FcmError):
        fcm.chain_plan(d, "bytes")
    d = fcm.chain_desc(1, 8, 8, 8, good, "f32")
    assert fcm.lib().fcm_chain_plan(fcm.ctypes.byref(d), 7, None, fcm.ctypes.byref(fcm.ChainPlan())) == EINVAL
    # a 7x7 depthwise layer has no kernel: the chain cannot be planned
    d = fcm.chain_desc(1, 8, 8, 8, [dict(kind="dw", k=7, stride=1, pad=3)], "i8")
    with pytest.raises(fcm.FcmError) as e:
        fcm.chain_plan(d, "bytes")
    assert e.value.status == EUNSUPPORTED


def test_chain_run_rejects_a_plan_of_another_chain():
    a = fcm.chain_desc(1, 8, 8, 8, [dict(kind="pw", c_out=8), dict(kind="pw", c_out=8)], "f32")
    b = fcm.chain_desc(1, 8, 8, 8, [dict(kind="dw", k=3, stride=1, pad=1), dict(kind="pw", c_out=8)], "f32")
    pa = fcm.chain_plan(a, "unfused")
    ptrs = (fcm.ctypes.c_void_p * 2)()
    st = fcm.lib().fcm_chain_run(fcm.ctypes.byref(b), fcm.ctypes.byref(pa), None, ptrs, None, None, None, None)
    assert st == EINVAL and "does not match" in fcm.last_error()


def test_chain_groups_carry_zero_points():
    """With zero points, each group of a chain plan is the module planner's plan of the
    group's descriptor with the zero points it sees: the chain input's (or the previous
    layer's output zero point) as input, its layers' as outputs."""
    sp = mobilenetv2_chain(n=4, dtype="i8", h=56, w=56, stages=[(1, 16, 1, 1), (6, 24, 2, 2)], final_pw=False,
                           zero_points=True)
    assert sp.zp_in == -128 and all(len(L["rq"]) == 5 for L in sp.layers)
    d = fcm.chain_desc(sp.n, sp.h, sp.w, sp.c, sp.layers, sp.dtype, sp.layout, zp_in=sp.zp_in)
    for obj in ("bytes", "time", "unfused"):
        p = fcm.chain_plan(d, obj)
        for first, op, plan in p.groups():
            g = _group_desc(sp.n, sp.h, sp.w, sp.c, sp.layers, first, op, "i8")
            g.zp_in = sp.zp_in if first == 0 else sp.layers[first - 1]["rq"][4]
            assert plan.as_dict() == fcm.plan(op, g).as_dict(), (obj, first, op)
