"""GPU parity of the int8 persistent kernels (DW->PW, PW, DW) under zero points and
per-channel requantisation, bit-exact against the CPU oracle, forced through explicit
plans, unsplit and split (channel chunks over several workgroups, partial sums combined
by a second kernel).

With an input zero point the copy waves rewrite the window positions outside the image
with the input's code of real 0 once an item's copies have landed, and fold the input zero
point times each channel's weight sum into the depthwise bias; a pointwise contraction
reading codes of zero point z loses z times each weight row's sum, which every compute
lane accumulates from its A operands and completes at the epilogue; every epilogue adds
its output zero point and clamps ReLU at it. Every compiled persistent variant runs at
several tile shapes (tiles on the image border and inside, ragged pixel blocks), ring
depths and capped grids (a workgroup streams many tiles, so the rewrite follows the ring
across tiles), channel counts with a ragged last chunk, zero points at the int8
extremes, strides 1 and 2 and filters 3 and 5.

Per-channel requantisation (a multiplier and a shift per output channel of a stage, staged
beside the biases) runs on the same cases, on every stage or on one stage only, with and
without the zero points: multipliers up to 2^30 (64-bit products), shifts from 0 to 62.
"""
import pytest

from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import Case, make_inputs

from gpu_util import dev_inputs, oracle_ref, run_fused, to_np
import oracle

import numpy as np

pytestmark = pytest.mark.gpu

TILES = ((4, 16), (8, 8), (7, 9), (3, 5), (1, 13))
LAUNCH = ((0, 0), (3, 2), (2, 3), (2, 8))  # (workgroup cap, ring depth); 0 = the planner's choice
ZPS = ((-128, (17, -5)), (37, (-90, 6)), (127, (0, 100)), (0, (-128, 3)))  # (zp_in, output zero points)


def _cases():
    out = []
    for j, (k, s, ci, co) in enumerate(((3, 1, 48, 32), (3, 2, 144, 80), (5, 1, 48, 24), (5, 2, 96, 40))):
        zin, zs = ZPS[j]
        rq = ((1, 6, -128, 127, zs[0]), (1, 7, -128, 127, zs[1]), (1, 6, -128, 127, 0))
        for op, c_out, acts in (("dw_pw", co, ("relu", "relu6", "none")), ("dw", ci, ("relu", "none", "none")),
                                ("pw", co, ("relu", "none", "none"))):
            kk, ss = (1, 1) if op == "pw" else (k, s)
            out.append(Case(op, 2, 13, 11, ci, ci, c_out, kk, ss, kk // 2, "i8", "nhwc", acts, rq,
                            dist_x="i8", dist_w="i8small", bias=True, seed=5100 + len(out), zp_in=zin,
                            name="zp3-%s-c%d-co%d-k%ds%d-z%d" % (op, ci, c_out, kk, ss, zin)))
    # mostly padding: an image smaller than the filter footprint
    out.append(Case("dw_pw", 1, 2, 3, 64, 64, 48, 3, 1, 1, "i8", "nhwc", ("relu", "none", "none"),
                    ((1, 5, -128, 127, -128), (1, 7, -128, 127, 9), (1, 6, -128, 127, 0)),
                    dist_x="i8", dist_w="i8small", bias=True, seed=5190, zp_in=-128, name="zp3-dwpw-2x3"))
    return out


def _plans(case, rqc=()):
    desc = fcm.desc_from_case(case)
    for i, t in enumerate(rqc):
        if t is not None:
            desc.rq_channel[i] = t.data_ptr()  # (rqc outlives the plans' use)
    plans = []
    for v in range(fcm.lib().fcm_variant_count()):
        name = fcm.variant_name(v)
        if not name.startswith(("k_dwpw3<i8,", "k_pw3<i8,", "k_dw3<i8,")):
            continue
        cob = 64 if case.op == "dw" else 16 * int(name.split(",")[4])
        for th, tw in TILES:
            for cap, depth in LAUNCH:
                try:
                    p = fcm.plan_evaluate(case.op, desc, th, tw, 64, cob, v, workgroups=cap, depth=depth)
                except fcm.FcmError:
                    continue
                assert p.splits == 1
                plans.append(p)
            for splits in (2, 3):  # each split subtracts its own share of the zero-point term
                try:
                    p = fcm.plan_evaluate(case.op, desc, th, tw, 64, cob, v, splits=splits)
                except fcm.FcmError:
                    continue
                assert p.splits == splits
                plans.append(p)
    return plans


CASES = _cases()


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_persistent_zero_points_match_oracle(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    if case.h > 3:
        assert len(np.unique(ref)) > 8, case.name  # not degenerate
    d = dev_inputs(inp, case.dtype)
    plans = _plans(case)
    assert plans, "no persistent variant implements %s" % case.name
    if case.c_in > 64 and case.op != "dw":
        assert any(p.splits > 1 for p in plans), case.name  # not vacuous
    for p in plans:
        got = to_np(run_fused(case, d, plan=p))
        assert np.array_equal(got, ref), "%s %s tile %dx%d grid %d depth %d splits %d: %d of %d differ" % (
            case.name, fcm.variant_name(p.variant), p.tile_h, p.tile_w, p.workgroups, p.depth, p.splits,
            int(np.sum(got != ref)), ref.size)
    # the planner's own plan for the asymmetric descriptor is a persistent one too
    p = fcm.plan(case.op, fcm.desc_from_case(case))
    assert fcm.variant_name(p.variant).startswith(("k_dwpw3<i8,", "k_pw3<i8,", "k_dw3<i8,"))


def _stage_channels(case):
    return {"dw_pw": [case.c_in, case.c_out], "dw": [case.c_in], "pw": [case.c_out]}[case.op]


def _per_channel(n, seed):
    """Multipliers and shifts of n channels: scales from about 2^-8 to 2^-2 with
    multipliers up to 2^30, plus the edge channels (1, 0) (the accumulator itself,
    saturated) and a shift of 62."""
    rng = np.random.default_rng(seed)
    mult = rng.integers(1, 1 << 30, n)
    shift = np.floor(np.log2(mult)).astype(np.int64) + rng.integers(2, 9, n)
    mult[0], shift[0] = 1, 0
    if n > 5:
        mult[5], shift[5] = (1 << 30) - 1, 62
    return mult.astype(np.int64), np.clip(shift, 0, 62)


PC_CASES = [c for c in CASES if c.h > 3]


@pytest.mark.parametrize("stages", ["all", "first", "last"])
@pytest.mark.parametrize("case", PC_CASES, ids=lambda c: c.name)
def test_persistent_per_channel_requant_matches_oracle(case, stages):
    import dataclasses
    import torch
    chans = _stage_channels(case)
    if stages != "all" and len(chans) == 1:
        pytest.skip("a one-stage module: every stage is the first and the last")
    pcs = [_per_channel(n, 60 + 7 * i + len(case.name)) for i, n in enumerate(chans)]
    if stages == "first":
        pcs = [pcs[0]] + [None] * (len(pcs) - 1)
    elif stages == "last":
        pcs = [None] * (len(pcs) - 1) + [pcs[-1]]
    rqc = [None if pc is None else torch.from_numpy(np.concatenate(pc).astype(np.int32)).cuda() for pc in pcs]
    for zp in (True, False):
        c = case if zp else dataclasses.replace(case, zp_in=0, rq=tuple(tuple(r[:4]) + (0,) for r in case.rq))
        inp = make_inputs(c)
        ref = oracle.run(c.op, dict(c.as_dict(), rq_channel=pcs), inp)
        assert len(np.unique(ref)) > 8, c.name
        d = dev_inputs(inp, c.dtype)
        plans = _plans(c, rqc)
        assert plans, c.name
        if c.c_in > 64 and c.op != "dw":
            assert any(p.splits > 1 for p in plans), c.name  # not vacuous
        for p in plans:
            got = to_np(run_fused(c, d, plan=p, rq_channel=rqc))
            assert np.array_equal(got, ref), "%s zp %s pc %s %s tile %dx%d grid %d depth %d splits %d: %d of %d differ" % (
                c.name, zp, stages, fcm.variant_name(p.variant), p.tile_h, p.tile_w, p.workgroups, p.depth, p.splits,
                int(np.sum(got != ref)), ref.size)
        # not vacuous: the stage scales change the result; the planner picks this kernel
        assert not np.array_equal(to_np(run_fused(c, d)), ref)
        desc = fcm.desc_from_case(c)
        for i, t in enumerate(rqc):
            if t is not None:
                desc.rq_channel[i] = t.data_ptr()
        p = fcm.plan(c.op, desc)
        assert fcm.variant_name(p.variant).startswith(("k_dwpw3<i8,", "k_pw3<i8,", "k_dw3<i8,"))
