"""Chain planning with the hardware in the loop: every candidate group of a chain (each
single layer, and each run of adjacent layers that forms a DW->PW, PW->DW, PW->PW or
PW->DW->PW module) is planned by the module planner, launched on the device and timed;
the partition of least measured time is chosen by the same dynamic programming as
fcm_chain_plan. The result is an fcm_chain_plan_t that fcm_chain_run accepts (it checks
that the groups tile the chain). Planning only: every launch goes through the C ABI."""
import ctypes

from . import fcm

_KINDS = {"dw_pw": ("dw", "pw"), "pw_dw": ("pw", "dw"), "pw_pw": ("pw", "pw"), "pw_dw_pw": ("pw", "dw", "pw"),
          "dw": ("dw",), "pw": ("pw",)}
_ELT = {0: 4, 1: 2, 2: 1}
MEASURED = 3  # fcm_chain_plan_t.objective of an autotuned plan


def _layers(desc):
    kinds = {v: k for k, v in fcm.LAYER_KIND.items()}
    acts = {v: k for k, v in fcm.ACT.items()}
    out = []
    for i in range(desc.num_layers):
        L = desc.layers[i]
        out.append(dict(kind=kinds[L.kind], c_out=L.c_out, k=L.k, stride=L.stride, pad=L.pad, act=acts[L.act],
                        rq=(L.rq.mult, L.rq.shift, L.rq.qmin, L.rq.qmax, L.rq.zero_point)))
    return out


def _shapes(desc, layers):
    h, w, c = desc.h, desc.w, desc.c
    out = [(h, w, c)]
    for L in layers:
        if L["kind"] == "pw":
            c = L["c_out"]
        else:
            h, w = fcm.out_hw(h, w, L["k"], L["stride"], L["pad"])
        out.append((h, w, c))
    return out


def _time_group(torch, sub, plan, op, x, weights, reps):
    """Mean microseconds of one group's launch (events on the current stream)."""
    cp = fcm.ChainPlan()
    cp.objective = MEASURED
    cp.num_groups = 1
    cp.first[0] = 0
    cp.op[0] = fcm.OP[op]
    cp.plan[0] = plan
    run = fcm.chain_run(sub, cp, x, weights, [None] * len(weights), prepare=True)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(reps):
        run()
    t1.record()
    torch.cuda.synchronize()
    return 1000.0 * t0.elapsed_time(t1) / reps


def chain_autotune(desc, reps=20, device="cuda"):
    """Plan `desc` (an fcm.ChainDesc) by timing every candidate group on `device` with
    zero-filled tensors of the chain's shapes. Returns (ChainPlan, {(first, op): us})."""
    import torch
    td = {0: torch.float32, 1: torch.bfloat16, 2: torch.int8}[desc.dtype]
    nhwc = desc.layout == fcm.LAYOUT["nhwc"]
    layers = _layers(desc)
    shapes = _shapes(desc, layers)
    n = len(layers)
    timed, plans = {}, {}
    for i in range(n):
        for op, kinds in _KINDS.items():
            sub_layers = layers[i:i + len(kinds)]
            if len(sub_layers) != len(kinds) or tuple(L["kind"] for L in sub_layers) != kinds:
                continue
            h, w, c = shapes[i]
            zp = desc.zp_in if i == 0 else layers[i - 1]["rq"][4]
            sub = fcm.chain_desc(desc.n, h, w, c, sub_layers, desc.dtype, desc.layout, zp_in=zp)
            plan = _module_plan(sub, op)
            if plan is None:
                continue
            x = torch.zeros((desc.n, h, w, c) if nhwc else (desc.n, c, h, w), dtype=td, device=device)
            ws, cc = [], c
            for L in sub_layers:
                if L["kind"] == "dw":
                    ws.append(torch.zeros((cc, L["k"], L["k"]), dtype=td, device=device))
                else:
                    ws.append(torch.zeros((L["c_out"], cc), dtype=td, device=device))
                    cc = L["c_out"]
            timed[(i, op)] = _time_group(torch, sub, plan, op, x, ws, reps)
            plans[(i, op)] = plan
    # dynamic programming over measured times (singles first; strictly smaller replaces)
    best, pick = [0.0] * (n + 1), [None] * n
    order = ["dw", "pw", "dw_pw", "pw_dw", "pw_pw", "pw_dw_pw"]
    for i in range(n - 1, -1, -1):
        b = None
        for op in order:
            if (i, op) not in timed:
                continue
            cost = timed[(i, op)] + best[i + len(_KINDS[op])]
            if b is None or cost < b:
                b, pick[i] = cost, op
        if b is None:
            raise fcm.FcmError(2, "chain_autotune: layer %d has no kernel" % i)
        best[i] = b
    cp = fcm.ChainPlan()
    cp.objective = MEASURED
    g, i, act_max = 0, 0, 0
    while i < n:
        op = pick[i]
        cp.first[g], cp.op[g], cp.plan[g] = i, fcm.OP[op], plans[(i, op)]
        cp.bytes_paper += plans[(i, op)].bytes_paper
        span = len(_KINDS[op])
        if span > 1:
            cp.fused_layers += span
        i += span
        if i < n:
            h, w, c = shapes[i]
            act_max = max(act_max, desc.n * h * w * c * _ELT[desc.dtype])
        g += 1
    cp.num_groups = g
    cp.act_bytes_max = act_max
    cp.time_est = best[0] * 1e-6
    cp.time_lbl_est = sum(timed[(i, L["kind"])] for i, L in enumerate(layers) if (i, L["kind"]) in timed) * 1e-6
    return cp, timed


def _module_plan(sub, op):
    """fcm_plan of module `op` over a chain's layers (which the chain planner kept apart)."""
    layers = _layers(sub)
    k = s = 1
    p = 0
    chans = [sub.c]
    for L in layers:
        if L["kind"] == "dw":
            k, s, p = L["k"], L["stride"], L["pad"]
            chans.append(chans[-1])
        else:
            chans.append(L["c_out"])
    c_mid = chans[1] if op in ("pw_dw", "pw_pw", "pw_dw_pw") else sub.c
    d = fcm.make_desc(sub.n, sub.h, sub.w, sub.c, c_mid, chans[-1], k=k, stride=s, pad=p, dtype=sub.dtype,
                      layout=sub.layout, act=[L["act"] for L in layers], rq=[L["rq"] for L in layers],
                      zp_in=sub.zp_in)
    try:
        return fcm.plan_limited(op, d, 0)  # chain groups run without a split workspace
    except fcm.FcmError:
        return None


# ------------------------------------------------------------------------------------
# One module or layer: the fastest of the planner's candidate plans, timed on the device
# ------------------------------------------------------------------------------------

def time_calls(torch, calls, launches, repeats=3, stream=None):
    """Median over `repeats` of the mean microseconds per launch of `launches` launches
    cycling through `calls` (prepared launches on `stream`), between two events on it."""
    stream = stream or torch.cuda.current_stream()
    for f in calls[:3]:
        f()
    torch.cuda.synchronize()
    out = []
    k = 0
    for _ in range(repeats):
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(launches):
            calls[k % len(calls)]()
            k += 1
        t1.record(stream)
        torch.cuda.synchronize()
        out.append(1000.0 * t0.elapsed_time(t1) / launches)
    return sorted(out)[len(out) // 2]


def fastest_plan(torch, plans, make_calls, agrees, launches=30, repeats=5, margin=0.05):
    """Time every plan of `plans` (the first is the planner's choice) and return
    (fastest plan, [(plan, microseconds or None), ...]). make_calls(plan) gives prepared
    launches over rotating buffers; agrees(plan) runs the plan once and says whether its
    output matches the planner's choice (bit-exact for int8, within rounding for floats):
    a plan that does not is never chosen. The plans are timed in turn, `repeats` rounds,
    each plan's median kept (drift over the rounds falls on every plan alike); another plan
    replaces the planner's choice only when it is faster by more than `margin` (relative),
    so that timing noise between near-equal plans does not change the choice from run to
    run."""
    calls = []
    for i, p in enumerate(plans):
        calls.append(None if i > 0 and not agrees(p) else make_calls(p))
    samples = [[] for _ in plans]
    for _ in range(repeats):
        for i, c in enumerate(calls):
            if c is not None:
                samples[i].append(time_calls(torch, c, launches, 1))
    timed = []
    best, best_t = None, None
    for i, p in enumerate(plans):
        if calls[i] is None:
            timed.append((p, None))
            continue
        t = sorted(samples[i])[len(samples[i]) // 2]
        timed.append((p, t))
        if best is None or t < best_t:
            best, best_t = p, t
    t0 = timed[0][1]
    if best is not plans[0] and best_t > t0 * (1.0 - margin):
        best = plans[0]
    return best, timed
