"""GPU parity of the NHWC LDS-DMA kernels, forced through explicit plans.

Every compiled LDS-DMA variant that implements a case is run with several output-channel
blocks and compared with the CPU oracle; shapes are ragged against the fixed tiles, the
64-byte channel chunk and the output-channel blocks.
"""
import numpy as np
import pytest

from paper_2404_19331_amd import fcm
from paper_2404_19331_amd.workloads import Case, make_inputs

from gpu_util import assert_close, dev_inputs, oracle_ref, run_fused, to_np

pytestmark = pytest.mark.gpu

RQ = ((1, 5, -127, 127), (3, 8, -128, 127), (1, 6, -127, 127))
ELT = {"f32": 4, "bf16": 2, "i8": 1}


def _cases():
    out = []
    geo = [(3, 1), (3, 2), (5, 1), (5, 2)]
    for dt, (ci, co) in (("bf16", (40, 24)), ("bf16", (72, 200)), ("f32", (20, 36)), ("i8", (48, 32)),
                         ("i8", (144, 80))):
        for k, s in geo:
            out.append(Case("dw_pw", 2, 13, 11, ci, ci, co, k, s, k // 2, dt, "nhwc",
                            ("relu", "relu6" if dt != "i8" else "none", "none"), RQ,
                            dist_x="i8small" if dt == "i8" else "n01", dist_w="i8small", bias=True,
                            seed=700 + len(out), name="dwpw-%s-c%d-co%d-k%ds%d" % (dt, ci, co, k, s)))
            out.append(Case("dw", 2, 13, 11, ci, ci, ci, k, s, k // 2, dt, "nhwc", ("relu6" if dt != "i8" else "relu",) * 3,
                            RQ, dist_x="i8small" if dt == "i8" else "n01", dist_w="i8small", bias=True,
                            seed=800 + len(out), name="dw-%s-c%d-k%ds%d" % (dt, ci, k, s)))
        out.append(Case("pw", 2, 13, 11, ci, ci, co, 1, 1, 0, dt, "nhwc", ("relu",) * 3, RQ,
                        dist_x="i8small" if dt == "i8" else "n01", dist_w="i8small", bias=True,
                        seed=900 + len(out), name="pw-%s-c%d-co%d" % (dt, ci, co)))
    # a full-image tile where the image is smaller than the tile, and a 1x1 image
    out.append(Case("dw_pw", 3, 5, 7, 64, 64, 48, 3, 1, 1, "bf16", "nhwc", ("relu", "none", "none"), bias=True,
                    seed=990, name="dwpw-bf16-small-image"))
    out.append(Case("dw_pw", 2, 1, 1, 32, 32, 16, 3, 2, 1, "bf16", "nhwc", ("none", "none", "none"), bias=True,
                    seed=991, name="dwpw-bf16-1x1"))
    return out


def _v2_plans(case):
    desc = fcm.desc_from_case(case)
    cb = 64 // ELT[case.dtype]
    last = case.c_in if case.op == "dw" else case.c_out
    plans = []
    for v in range(fcm.lib().fcm_variant_count()):
        name = fcm.variant_name(v)
        if not name.startswith(("k_dwpw2", "k_pw2", "k_dw2")):
            continue
        for th, tw in ((8, 8), (8, 16)):
            cobs = [cb] if case.op == "dw" else sorted({16, 64, -(-last // 16) * 16, 256})
            for cob in cobs:
                try:
                    p = fcm.plan_evaluate(case.op, desc, th, tw, cb, cob, v)
                except fcm.FcmError:
                    continue
                plans.append(p)
    return plans


CASES = _cases()


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_lds_dma_variants_match_oracle(case):
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    plans = _v2_plans(case)
    assert plans, "no LDS-DMA variant implements %s" % case.name
    for p in plans:
        got = to_np(run_fused(case, d, plan=p))
        assert_close(got, ref, case.dtype, "%s %s cob=%d" % (case.name, fcm.variant_name(p.variant), p.co_block))


def test_misaligned_tensors_fall_back():
    """LDS-DMA kernels need 16-byte aligned tensors; a misaligned view must still give the
    oracle's result (the planner then picks a kernel without DMA staging)."""
    import torch
    case = Case("dw_pw", 1, 9, 9, 32, 32, 16, 3, 1, 1, "bf16", "nhwc", ("relu", "none", "none"), bias=True,
                seed=992)
    inp = make_inputs(case)
    ref = oracle_ref(case, inp)
    d = dev_inputs(inp, case.dtype)
    big = torch.empty(d["x"].numel() + 8, dtype=d["x"].dtype, device="cuda")
    xv = big[1:1 + d["x"].numel()].view(d["x"].shape)   # 2-byte offset: not 16-byte aligned
    xv.copy_(d["x"])
    d2 = dict(d)
    d2["x"] = xv
    got = to_np(run_fused(case, d2))
    assert_close(got, ref, case.dtype, "misaligned x")
