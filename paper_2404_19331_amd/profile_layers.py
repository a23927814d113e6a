"""Launch sequence for per-layer hardware counters of the DW->PW layers of a workload.

    python -m paper_2404_19331_amd.profile_layers --workload C3b32 [--reps 10] > manifest.json

Run it under rocprofv3 (one run per counter group, plus one with --kernel-trace); then
`python -m paper_2404_19331_amd.rocprof_report layers --manifest manifest.json ...` turns
the dispatches into a per-layer table. For every layer, in this order and each group
synchronised: a plain device copy of 256 MiB (a float multiply by one, which calibrates
the byte counters) three times, the fused module `reps` times, then its two unfused
stages (DW, then PW) `reps` times each, all with the planner's own plans (the default
entry points). Input and output buffers rotate over sets of at least 512 MiB so that the
Infinity Cache does not serve a repeated working set. The manifest (stdout, JSON) gives
the launch roles in order and the planner's byte figures for each launch; every launch
goes through the C ABI.
"""
import argparse
import json
import sys

import numpy as np

from . import fcm
from .workloads import config_c3, config_c4, config_c5, make_inputs

ROTATE = 512 << 20
CALIB_BYTES = 256 << 20


def _cases(name):
    if name == "C3b32":
        return config_c3(batches=(32,))
    if name == "C3b1":
        return config_c3(batches=(1,))
    if name == "C5":
        return config_c5()
    if name == "C4":
        return config_c4()
    raise ValueError(name)


def _plan_info(p):
    return {"variant": fcm.variant_name(p.variant), "tile": [int(p.tile_h), int(p.tile_w)],
            "co_block": int(p.co_block), "workgroups": int(p.workgroups), "bytes_ideal": int(p.bytes_ideal),
            "bytes_tiled": int(p.bytes_tiled), "bytes_paper": int(p.bytes_paper)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="C3b32")
    ap.add_argument("--reps", type=int, default=10)
    a = ap.parse_args()
    import torch
    assert torch.cuda.is_available(), "needs a GPU"
    fcm.lib()
    src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)

    def dev(v):
        if v is None:
            return None
        if v.dtype == np.uint16:
            return torch.from_numpy(v.view(np.int16).copy()).view(torch.bfloat16).cuda()
        return torch.from_numpy(v).cuda()

    manifest = {"workload": a.workload, "reps": a.reps, "calib_bytes": CALIB_BYTES, "layers": []}
    for c in _cases(a.workload):
        if c.op != "dw_pw" or c.layout != "nhwc":
            continue
        d = {k: dev(v) for k, v in make_inputs(c).items()}
        desc = fcm.desc_from_case(c)
        plan = fcm.plan_limited("dw_pw", desc, 0)
        ho, wo = fcm.out_hw(c.h, c.w, c.k, c.stride, c.pad)
        x0 = d["x"]
        per_set = x0.numel() * x0.element_size() * (1 + c.c_out * ho * wo / (c.c_in * c.h * c.w))
        nsets = max(2, int(-(-ROTATE // per_set)))
        xs = [x0] + [x0.clone() for _ in range(nsets - 1)]
        ys = [torch.empty((c.n, ho, wo, c.c_out), dtype=x0.dtype, device="cuda") for _ in range(nsets)]
        mids = [torch.empty((c.n, ho, wo, c.c_in), dtype=x0.dtype, device="cuda") for _ in range(2)]
        rq = list(c.rq) if c.dtype == "i8" else None
        kw = dict(stride=c.stride, pad=c.pad, layout=c.layout)
        fused = [fcm.dw_pw(x, d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), act=c.act[:2], rq=rq, plan=plan,
                           out=y, prepare=True, **kw) for x, y in zip(xs, ys)]
        dws = [fcm.dw(x, d["w_dw"], d.get("b_dw"), act=c.act[0], rq=rq[0] if rq else None, out=mids[i % 2],
                      prepare=True, **kw) for i, x in enumerate(xs)]
        pws = [fcm.pw(mids[i % 2], d["w_pw"], d.get("b_pw"), act=c.act[1], rq=rq[1] if rq else None, layout=c.layout,
                      out=y, prepare=True) for i, y in enumerate(ys)]
        dw_desc = fcm.make_desc(c.n, c.h, c.w, c.c_in, c.c_in, c.c_in, c.k, c.stride, c.pad, c.dtype, c.layout,
                                (c.act[0],), [rq[0]] if rq else None)
        pw_desc = fcm.make_desc(c.n, ho, wo, c.c_in, c.c_in, c.c_out, 1, 1, 0, c.dtype, c.layout, (c.act[1],),
                                [rq[1]] if rq else None)
        torch.cuda.synchronize()
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        for group in (fused, dws, pws):
            for r in range(a.reps):
                group[r % len(group)]()
            torch.cuda.synchronize()
        manifest["layers"].append({
            "layer": c.name, "fused": _plan_info(plan),
            "dw": _plan_info(fcm.plan_limited("dw", dw_desc, 0)), "pw": _plan_info(fcm.plan_limited("pw", pw_desc, 0))})
        del xs, ys, mids, fused, dws, pws, d
        torch.cuda.empty_cache()
        print("profile_layers: %s done" % c.name, file=sys.stderr, flush=True)
    print(json.dumps(manifest), flush=True)


if __name__ == "__main__":
    main()
