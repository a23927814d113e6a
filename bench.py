"""Benchmark of the fused DW/PW modules on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload C3b32] [--configs all]

Headline: a step is one pass of the fused path over every layer of the workload (one
fused kernel per layer, MobileNetV1's 13 DW->PW layers at batch 32 by default) on one
batch of seeded synthetic input; `value` is the algorithmic bytes of a step (input,
weights and output of every layer, once) over its time. The same layers are timed layer by
layer (one DW and one PW kernel per layer, intermediate through HBM) as the unfused
comparison.

Every configuration (C1 to C5) is then measured layer by layer with the same protocol:
10 warm-up launches, then 5 repeats of at least 50 back-to-back launches cycling through
rotating buffer sets of at least 512 MiB in total (the 256 MiB Infinity Cache cannot serve
a repeated working set), the median repeat's mean per launch; fused and unfused alike,
plus a hot-cache figure (one buffer set launched repeatedly), labelled as such.

Plans: each fused module and each unfused stage runs the fastest of the planner's
candidate plans (fcm_plan_candidates), timed here on the device, among those whose
output agrees with the planner's own choice; both sides may use split plans with a
caller workspace. Inputs are resident in HBM before any timed region.

Prints ONE JSON line: metric/value, per-layer microseconds fused and unfused, per-config
entries, the roofline of the dominant kernel (HIP events on the launch stream), and the
CPU oracle timed on a bounded sample (plus its single-thread time on C1).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

ROTATE_BYTES = 512 << 20
WORKSPACE_BYTES = 64 << 20  # caller workspace offered to split plans
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "i8": 5000.0, "f32": 157.3}
# the depthwise taps run on the vector ALU: fp32 FMA (fp32 and bf16 paths); int8 one
# multiply-accumulate per lane and cycle (256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz x 2 x 2)
VALU_PEAK_TFLOPS = {"bf16": 157.3, "f32": 157.3, "i8": 78.6}
METRIC = "fused DW+PW layer us and achieved HBM GB/s (% roofline) vs unfused DW->PW"
CONFIGS = ("C1", "C2", "C3b1", "C3b32", "C4", "C5")
WARMUP_LAUNCHES = 10
REPEATS = 5
MIN_LAUNCHES = 50


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="C3b32",
                    choices=["C1", "C2", "C3b1", "C3b32", "C4", "C5", "PWPW", "MNV2", "MNV2bf16", "MNV2zp"])
    ap.add_argument("--configs", default="all",
                    help="per-config layer measurements: 'all', 'none' or a comma-separated list of " +
                         ", ".join(CONFIGS))
    ap.add_argument("--no-tune", action="store_true", help="run the planner's own plans (no device timing)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU-baseline sample time")
    ap.add_argument("--layers", default=None, help="comma-separated layer indices of the headline (subset)")
    ap.add_argument("--calib", action="store_true",
                    help="also run a plain 256 MiB device copy (reference for profiler byte counters)")
    ap.add_argument("--energy", type=float, default=0.0, metavar="SECONDS",
                    help="also measure energy per step, fused and unfused: the GPU's power sensor sampled "
                         "while the step loop runs for this many seconds each (0 = off)")
    return ap.parse_args()


def workload_cases(name):
    from paper_2404_19331_amd import workloads as W
    if name == "C1":
        return W.config_c1(), "DW3x3+ReLU -> PW 32->64+ReLU, 56x56, fp32 NCHW, batch 1"
    if name == "C2":
        return W.config_c2(), "inverted residual PW 24->144 ReLU6, DW3x3 ReLU6, PW 144->24, 56x56, fp32 NCHW, batch 1"
    if name == "C3b1":
        return W.config_c3(batches=(1,)), "MobileNetV1 13 DW3x3+PW layers (224x224 input), bf16 NHWC, ReLU, batch 1"
    if name == "C3b32":
        return W.config_c3(batches=(32,)), "MobileNetV1 13 DW3x3+PW layers (224x224 input), bf16 NHWC, ReLU, batch 32"
    if name == "C4":
        return W.config_c4(), "EfficientNet-B0-style int8 DW5x5+PW (112x112x96 s2 ->24; 14x14x480 ->112), NHWC, batch 8"
    if name == "PWPW":
        return W.config_pwpw(), "MobileNetV2-width PW->PW pairs (expand ReLU, project), int8 NHWC, batch 8"
    return W.config_c5(), "CvT/CMT-style token grids DW3x3+PW (56x56x64->192, 28x28x192->384, 14x14x384->768), bf16 NHWC, batch 64"


def elt(dtype):
    return {"f32": 4, "bf16": 2, "i8": 1}[dtype]


def out_hw(c):
    return (c.h + 2 * c.pad - c.k) // c.stride + 1, (c.w + 2 * c.pad - c.k) // c.stride + 1


def layer_stats(c):
    """Algorithmic bytes (input + weights + output once) and flops of one fused layer
    (depthwise and pointwise flops apart), and the unfused intermediate bytes (written
    once and read once per intermediate)."""
    e = elt(c.dtype)
    ho, wo = out_hw(c)
    kk = c.k * c.k
    x = c.n * c.h * c.w * c.c_in
    if c.op == "dw_pw":
        w = c.c_in * kk + c.c_out * c.c_in
        y = c.n * ho * wo * c.c_out
        mids = [c.n * ho * wo * c.c_in]
        dw = 2 * c.n * ho * wo * c.c_in * kk
        pw = 2 * c.n * ho * wo * c.c_in * c.c_out
    elif c.op == "pw_dw_pw":
        w = c.c_mid * c.c_in + c.c_mid * kk + c.c_out * c.c_mid
        y = c.n * ho * wo * c.c_out
        mids = [c.n * c.h * c.w * c.c_mid, c.n * ho * wo * c.c_mid]
        dw = 2 * c.n * ho * wo * c.c_mid * kk
        pw = 2 * (c.n * c.h * c.w * c.c_mid * c.c_in + c.n * ho * wo * c.c_mid * c.c_out)
    elif c.op == "pw_pw":
        w = c.c_mid * c.c_in + c.c_out * c.c_mid
        y = c.n * c.h * c.w * c.c_out
        mids = [c.n * c.h * c.w * c.c_mid]
        dw = 0
        pw = 2 * c.n * c.h * c.w * c.c_mid * (c.c_in + c.c_out)
    else:  # pw_dw
        w = c.c_mid * c.c_in + c.c_mid * kk
        y = c.n * ho * wo * c.c_mid
        mids = [c.n * c.h * c.w * c.c_mid]
        dw = 2 * c.n * ho * wo * c.c_mid * kk
        pw = 2 * c.n * c.h * c.w * c.c_mid * c.c_in
    fused = (x + w + y) * e
    unfused = fused + 2 * sum(mids) * e
    return dict(bytes=fused, bytes_unfused=unfused, flops=dw + pw, flops_dw=dw, flops_pw=pw, x=x * e, y=y * e,
                mids=[m * e for m in mids])


def roof(c, stats, us):
    """The binding roof of a layer and the fraction of it reached in `us` microseconds:
    max(t_HBM, t_compute) / t_measured, t_HBM = algorithmic bytes / 8 TB/s, t_compute =
    depthwise flops on the vector ALU + pointwise flops on the matrix cores."""
    t_hbm = stats["bytes"] / (HBM_PEAK_GBS * 1e9)
    t_cmp = stats["flops_dw"] / (VALU_PEAK_TFLOPS[c.dtype] * 1e12) + stats["flops_pw"] / (
        MFMA_PEAK_TFLOPS[c.dtype] * 1e12)
    bound = "hbm" if t_hbm >= t_cmp else ("mfma" if stats["flops_pw"] / MFMA_PEAK_TFLOPS[c.dtype] >=
                                          stats["flops_dw"] / VALU_PEAK_TFLOPS[c.dtype] else "valu")
    return bound, max(t_hbm, t_cmp) / (us * 1e-6)


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2404_19331_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def stage_ops(c):
    """The unfused stages of a module: (op, n, h, w, c_in, c_out, k, stride, pad, stage)."""
    ho, wo = out_hw(c)
    if c.op == "dw_pw":
        return [("dw", c.h, c.w, c.c_in, c.c_in, c.k, c.stride, c.pad, 0), ("pw", ho, wo, c.c_in, c.c_out, 1, 1, 0, 1)]
    if c.op == "pw_dw":
        return [("pw", c.h, c.w, c.c_in, c.c_mid, 1, 1, 0, 0), ("dw", c.h, c.w, c.c_mid, c.c_mid, c.k, c.stride, c.pad, 1)]
    if c.op == "pw_pw":
        return [("pw", c.h, c.w, c.c_in, c.c_mid, 1, 1, 0, 0), ("pw", c.h, c.w, c.c_mid, c.c_out, 1, 1, 0, 1)]
    return [("pw", c.h, c.w, c.c_in, c.c_mid, 1, 1, 0, 0), ("dw", c.h, c.w, c.c_mid, c.c_mid, c.k, c.stride, c.pad, 1),
            ("pw", ho, wo, c.c_mid, c.c_out, 1, 1, 0, 2)]


def stage_desc(fcm, c, s):
    """Descriptor of one unfused stage (an entry of stage_ops) as fcm.dw / fcm.pw build it."""
    op, h, w, ci, co, k, st, pad, i = s
    rq = [c.rq[i]] if c.dtype == "i8" else None
    zp = c.zp_in if i == 0 else (int(c.rq[i - 1][4]) if c.dtype == "i8" and len(c.rq[i - 1]) > 4 else 0)
    return fcm.make_desc(c.n, h, w, ci, ci, co, k, st, pad, c.dtype, c.layout, (c.act[i],), rq, zp_in=zp)


def plan_info(fcm, p):
    return {"variant": fcm.variant_name(p.variant), "tile": [int(p.tile_h), int(p.tile_w)],
            "c_block": int(p.c_block), "co_block": int(p.co_block), "workgroups": int(p.workgroups),
            "splits": int(p.splits)}


class Layer:
    """One layer of a workload on the device: rotating buffer sets, the fused module's and
    the unfused stages' plans (tuned on the device unless told not to), prepared
    launches."""

    def __init__(self, case, torch, fcm, make_inputs, to_dev, tune=True, log=None):
        from paper_2404_19331_amd.autotune import fastest_plan
        self.case = c = case
        self.torch, self.fcm = torch, fcm
        self.stats = layer_stats(case)
        d = {k: to_dev(v) for k, v in make_inputs(case).items()}
        self.d = d
        ho, wo = out_hw(c)
        self.nsets = max(2, -(-ROTATE_BYTES // (self.stats["x"] + self.stats["y"])))
        x0 = d["x"]

        def shaped(ch, h, w):
            return (c.n, ch, h, w) if c.layout == "nchw" else (c.n, h, w, ch)

        self.stages = stage_ops(c)
        ych = c.c_mid if c.op == "pw_dw" else c.c_out
        self.xs = [x0] + [x0.clone() for _ in range(self.nsets - 1)]
        self.ys = [torch.empty(shaped(ych, ho, wo), dtype=x0.dtype, device=x0.device) for _ in range(self.nsets)]
        self.mids = [[torch.empty(shaped(s[4], *fcm.out_hw(s[1], s[2], s[5], s[6], s[7])), dtype=x0.dtype,
                                  device=x0.device) for s in self.stages[:-1]] for _ in range(self.nsets)]
        self.ws = torch.empty(WORKSPACE_BYTES, dtype=torch.uint8, device=x0.device)
        self.rq = list(c.rq) if c.dtype == "i8" else None
        self.desc = fcm.desc_from_case(c)
        self.static = fcm.plan(c.op, self.desc)
        self.stage_descs = [self._stage_desc(s) for s in self.stages]
        self.static_stages = [fcm.plan(s[0], sd) for s, sd in zip(self.stages, self.stage_descs)]
        self.plan, self.stage_plans = self.static, list(self.static_stages)
        self.tuning = None
        if tune:
            ntune = min(self.nsets, 32)
            # fused module
            ref = self.fused_call(0, self.static)()
            ref = ref.clone()
            ws_max = WORKSPACE_BYTES if c.op == "dw_pw" else 0
            cands = fcm.plan_candidates(c.op, self.desc, 12, ws_max)
            self.plan, timed = fastest_plan(
                torch, cands, lambda p: [self.fused_call(j, p) for j in range(ntune)],
                lambda p: self._agrees(self.fused_call(0, p)(), ref))
            self.tuning = {"fused": [(plan_info(fcm, p), None if t is None else round(t, 3)) for p, t in timed]}
            # unfused stages, each on the planner's own output of the stage before
            self.unfused_call(0, self.static_stages)()
            st_timed = []
            for i, (s, sd) in enumerate(zip(self.stages, self.stage_descs)):
                sref = self.stage_call(i, 0, self.static_stages[i])().clone()
                cands = fcm.plan_candidates(s[0], sd, 12, WORKSPACE_BYTES if s[0] == "pw" else 0)
                best, timed = fastest_plan(
                    torch, cands, lambda p, i=i: [self.stage_call(i, j, p) for j in range(ntune)],
                    lambda p, i=i, sref=sref: self._agrees(self.stage_call(i, 0, p)(), sref))
                self.stage_plans[i] = best
                st_timed.append([(plan_info(fcm, p), None if t is None else round(t, 3)) for p, t in timed])
            self.tuning["unfused"] = st_timed
            torch.cuda.synchronize()
            if log:
                log("  %s: fused %s (planner %s), unfused %s" % (
                    c.name, fcm.variant_name(self.plan.variant), fcm.variant_name(self.static.variant),
                    " + ".join(fcm.variant_name(p.variant) for p in self.stage_plans)))
        self.fused_calls = [self.fused_call(j, self.plan) for j in range(self.nsets)]
        self.unfused_calls = [self.unfused_call(j, self.stage_plans) for j in range(self.nsets)]

    def _stage_desc(self, s):
        return stage_desc(self.fcm, self.case, s)

    def _agrees(self, got, ref):
        torch = self.torch
        if self.case.dtype == "i8":
            return bool(torch.equal(got, ref))
        g, r = got.float(), ref.float()
        if not bool(torch.isfinite(g).all()):
            return False
        if self.case.dtype == "f32":
            tol = 1e-4 + 1e-5 * r.abs()
        else:
            rms = torch.sqrt(torch.mean(r * r))
            tol = 2e-2 * torch.maximum(r.abs(), rms)
        return bool(((g - r).abs() <= tol).all())

    def fused_call(self, j, plan):
        c, d, fcm = self.case, self.d, self.fcm
        x, y, rq = self.xs[j], self.ys[j], self.rq
        kw = dict(stride=c.stride, pad=c.pad, layout=c.layout, out=y, prepare=True, plan=plan)
        if c.op == "dw_pw":
            ws = self.ws if fcm.workspace_bytes(self.desc, plan) else None
            return fcm.dw_pw(x, d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), act=c.act[:2], rq=rq,
                             workspace=ws, zp_in=c.zp_in, **kw)
        if c.op == "pw_dw_pw":
            return fcm.pw_dw_pw(x, d["w_pw1"], d["w_dw"], d["w_pw2"], d.get("b_pw1"), d.get("b_dw"), d.get("b_pw2"),
                                act=c.act, rq=rq, zp_in=c.zp_in, **kw)
        if c.op == "pw_pw":
            kw.pop("stride"), kw.pop("pad")
            return fcm.pw_pw(x, d["w_pw1"], d["w_pw2"], d.get("b_pw1"), d.get("b_pw2"), act=c.act[:2], rq=rq,
                             zp_in=c.zp_in, **kw)
        return fcm.pw_dw(x, d["w_pw"], d["w_dw"], d.get("b_pw"), d.get("b_dw"), act=c.act[:2], rq=rq,
                         zp_in=c.zp_in, **kw)

    def _stage_weights(self, i):
        c, d = self.case, self.d
        if c.op == "dw_pw":
            return [(d["w_dw"], d.get("b_dw")), (d["w_pw"], d.get("b_pw"))][i]
        if c.op == "pw_dw":
            return [(d["w_pw"], d.get("b_pw")), (d["w_dw"], d.get("b_dw"))][i]
        if c.op == "pw_pw":
            return [(d["w_pw1"], d.get("b_pw1")), (d["w_pw2"], d.get("b_pw2"))][i]
        return [(d["w_pw1"], d.get("b_pw1")), (d["w_dw"], d.get("b_dw")), (d["w_pw2"], d.get("b_pw2"))][i]

    def stage_call(self, i, j, plan):
        """Prepared launch of unfused stage i on buffer set j."""
        c, fcm = self.case, self.fcm
        s = self.stages[i]
        x = self.xs[j] if i == 0 else self.mids[j][i - 1]
        y = self.ys[j] if i == len(self.stages) - 1 else self.mids[j][i]
        w, b = self._stage_weights(i)
        sd = self.stage_descs[i]
        rq = self.rq[s[8]] if self.rq else None
        if s[0] == "dw":
            return fcm.dw(x, w, b, stride=s[6], pad=s[7], act=c.act[s[8]], rq=rq, layout=c.layout, plan=plan,
                          out=y, prepare=True, zp_in=int(sd.zp_in))
        ws = self.ws if fcm.workspace_bytes(sd, plan) else None
        return fcm.pw(x, w, b, act=c.act[s[8]], rq=rq, layout=c.layout, plan=plan, out=y, prepare=True,
                      zp_in=int(sd.zp_in), workspace=ws)

    def unfused_call(self, j, plans):
        from paper_2404_19331_amd.fcm import _Chain
        return _Chain([self.stage_call(i, j, p) for i, p in enumerate(plans)])

    def calls(self, which):
        return self.fused_calls if which == "fused" else self.unfused_calls


def _preroll(torch):
    """Keep the GPU busy briefly so the host enqueues the timed launches ahead of it."""
    try:
        torch.cuda._sleep(20_000_000)
    except Exception:
        pass


def time_steps(torch, layers, which, steps, warmup, stream):
    """Warm up, then time `steps` steps (each launches every layer once) between two
    events on the launch stream. Returns ms per step."""
    calls = [L.calls(which) for L in layers]
    k = 0
    for _ in range(warmup):
        for cl in calls:
            cl[k % len(cl)]()
        k += 1
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    _preroll(torch)
    t0.record(stream)
    for _ in range(steps):
        for cl in calls:
            cl[k % len(cl)]()
        k += 1
    t1.record(stream)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / steps


def time_layer(torch, cl, stream, hot=False):
    """The measurement protocol for one layer's launches `cl` (one per rotating buffer
    set): WARMUP_LAUNCHES launches, then REPEATS repeats of max(MIN_LAUNCHES, sets)
    back-to-back launches between two events on the launch stream; the median repeat's
    microseconds per launch. hot: buffer set 0 only, MIN_LAUNCHES per repeat (a
    hot-cache figure)."""
    seq = [cl[0]] if hot else cl
    launches = MIN_LAUNCHES if hot else max(MIN_LAUNCHES, len(seq))
    k = 0
    for _ in range(WARMUP_LAUNCHES):
        seq[k % len(seq)]()
        k += 1
    torch.cuda.synchronize()
    reps = []
    for _ in range(REPEATS):
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        _preroll(torch)
        t0.record(stream)
        for _ in range(launches):
            seq[k % len(seq)]()
            k += 1
        t1.record(stream)
        torch.cuda.synchronize()
        reps.append(1000.0 * t0.elapsed_time(t1) / launches)
    return sorted(reps)[REPEATS // 2]


def layer_entry(fcm, L, fu, uu, hot):
    st = L.stats
    bound, frac = roof(L.case, st, fu)
    e = {"layer": L.case.name, "fused_us": round(fu, 3), "unfused_us": round(uu, 3), "speedup": round(uu / fu, 3),
         "hot_cache_fused_us": round(hot, 3), "bytes": int(st["bytes"]), "bytes_unfused": int(st["bytes_unfused"]),
         "flops": int(st["flops"]), "gbs": round(st["bytes"] / (fu * 1e-6) / 1e9, 1),
         "hbm_frac": round(st["bytes"] / (fu * 1e-6) / 1e9 / HBM_PEAK_GBS, 4), "bound": bound,
         "roof_frac": round(frac, 4), "plan": plan_info(fcm, L.plan),
         "planner_plan": fcm.variant_name(L.static.variant),
         "unfused_plans": [fcm.variant_name(p.variant) for p in L.stage_plans]}
    return e


def power_sensor():
    """Path of the GPU's socket-power sensor (hwmon, microwatts), or None."""
    import glob
    for pat in ("/sys/class/drm/card*/device/hwmon/hwmon*/power1_input",
                "/sys/class/drm/card*/device/hwmon/hwmon*/power1_average"):
        for path in sorted(glob.glob(pat)):
            try:
                with open(path) as f:
                    int(f.read().strip())
                return path
            except (OSError, ValueError):
                continue
    return None


class PowerSampler:
    """Reads the power sensor every `period` seconds on a thread: [(time, watts)]."""

    def __init__(self, path, period=0.005):
        import threading
        self.path, self.period, self.samples = path, period, []
        self._stop = threading.Event()
        self._t = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        while not self._stop.is_set():
            try:
                with open(self.path) as f:
                    self.samples.append((time.perf_counter(), int(f.read().strip()) * 1e-6))
            except (OSError, ValueError):
                pass
            time.sleep(self.period)

    def __enter__(self):
        self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._t.join()


def measure_energy(torch, step, seconds, images, path):
    """Energy per step of `step` (enqueues one step): the step loop runs for about
    `seconds` (batches of steps between synchronisations) while the power sensor is
    sampled; energy = mean sampled power x wall time, over the steps completed. Also the
    idle power over one second before, and the energy above idle."""
    with PowerSampler(path) as idle:
        time.sleep(1.0)
    p_idle = sum(w for _, w in idle.samples) / max(1, len(idle.samples))
    for _ in range(3):
        step()
    torch.cuda.synchronize()
    steps = 0
    with PowerSampler(path) as ps:
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < seconds:
            for _ in range(10):
                step()
            steps += 10
            torch.cuda.synchronize()
        t1 = time.perf_counter()
    inside = [w for t, w in ps.samples if t0 <= t <= t1]
    p = sum(inside) / max(1, len(inside))
    j_step = p * (t1 - t0) / steps
    return {"watts_mean": round(p, 1), "watts_idle": round(p_idle, 1), "samples": len(inside),
            "seconds": round(t1 - t0, 3), "steps": steps, "ms_per_step_wall": round(1e3 * (t1 - t0) / steps, 4),
            "joules_per_step": round(j_step, 5), "mj_per_image": round(1e3 * j_step / images, 4),
            "mj_per_image_above_idle": round(1e3 * (p - p_idle) * (t1 - t0) / steps / images, 4)}


def energy_block(torch, steps_by_name, seconds, images):
    path = power_sensor()
    if path is None:
        return {"error": "no readable GPU power sensor"}
    out = {"sensor": path, "method": "hwmon socket power sampled every 5 ms during a %.1f s step loop" % seconds}
    for name, step in steps_by_name.items():
        print("bench: energy of the %s step" % name, file=sys.stderr, flush=True)
        out[name] = measure_energy(torch, step, seconds, images, path)
    if "fused" in out and "unfused" in out:
        out["ratio_unfused_over_fused"] = round(out["unfused"]["joules_per_step"] / out["fused"]["joules_per_step"], 3)
    return out


def bench_chain(a, torch, fcm):
    """End-to-end MobileNetV2 body (51 DW/PW layers after the stem, batch 32, NHWC): the
    chain planned by timing every candidate group on the device (value), by least modelled
    time, by least Eq. 1-4 bytes and layer by layer, each run through fcm_chain_run; a step
    is one pass of the whole chain over one batch."""
    import numpy as np
    from paper_2404_19331_amd.workloads import mobilenetv2_chain, make_chain_inputs
    dtype = "bf16" if a.workload == "MNV2bf16" else "i8"
    spec = mobilenetv2_chain(n=32, dtype=dtype, zero_points=a.workload == "MNV2zp")
    x, ws, bs = make_chain_inputs(spec)

    def dev(v):
        if v is None:
            return None
        if v.dtype == np.uint16:
            return torch.from_numpy(v.view(np.int16).copy()).view(torch.bfloat16).cuda()
        return torch.from_numpy(v).cuda()

    xd, wd, bd = dev(x), [dev(w) for w in ws], [dev(b) for b in bs]
    nsets = max(2, -(-ROTATE_BYTES // (xd.numel() * xd.element_size())))
    xs = [xd] + [xd.clone() for _ in range(nsets - 1)]
    d = fcm.chain_desc(spec.n, spec.h, spec.w, spec.c, spec.layers, spec.dtype, spec.layout, zp_in=spec.zp_in)
    stream = torch.cuda.current_stream()
    res = {}
    from paper_2404_19331_amd.autotune import chain_autotune
    tuned, _ = chain_autotune(d)
    print("bench: autotuned chain plan ready (%d groups)" % tuned.num_groups, file=sys.stderr, flush=True)
    for obj in ("measured", "time", "bytes", "unfused"):
        p = tuned if obj == "measured" else fcm.chain_plan(d, obj)
        calls = [fcm.chain_run(d, p, xv, wd, bd, prepare=True) for xv in xs]
        for k in range(a.warmup):
            calls[k % nsets]()
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        _preroll(torch)
        t0.record(stream)
        for k in range(a.steps):
            calls[k % nsets]()
        t1.record(stream)
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / a.steps
        ideal = sum(int(p.plan[g].bytes_ideal) for g in range(p.num_groups))
        res[obj] = {"ms_per_step": round(ms, 4), "images_per_s": round(spec.n / (ms * 1e-3), 1),
                    "groups": int(p.num_groups), "fused_layers": int(p.fused_layers),
                    "bytes_paper": int(p.bytes_paper), "bytes_ideal": ideal,
                    "gbs": round(ideal / (ms * 1e-3) / 1e9, 1), "time_est_ms": round(p.time_est * 1e3, 4),
                    "ops": [op for _, op, _ in p.groups()]}
        print("bench: chain %s plan %.3f ms (%d groups)" % (obj, ms, p.num_groups), file=sys.stderr, flush=True)
    best = res["measured"]
    out = {
        "metric": "MobileNetV2 body end-to-end images/s (chain FusePlanner, groups timed on the device) vs "
                  "layer-by-layer",
        "value": best["images_per_s"],
        "unit": "images/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": best["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dtype, "data": "synthetic (seeded, random-init weights)",
        "config": {"workload": spec.name, "name": a.workload, "layers": len(spec.layers), "batch": spec.n,
                   "layout": spec.layout, "parallelism": "none (1 GPU)"},
        "chains": res,
        "speedup_vs_unfused": round(res["unfused"]["ms_per_step"] / best["ms_per_step"], 3),
        "roofline": {"bound": "hbm", "achieved": best["gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(best["gbs"] / HBM_PEAK_GBS, 4), "kernel": "whole chain", "traffic": None},
        "cpu_baseline": None,
    }
    if a.energy > 0:
        steps = {}
        for obj, name in (("measured", "fused"), ("unfused", "unfused")):
            p = tuned if obj == "measured" else fcm.chain_plan(d, obj)
            cl = [fcm.chain_run(d, p, xv, wd, bd, prepare=True) for xv in xs]
            it = iter(range(1 << 62))
            steps[name] = (lambda cl=cl, it=it: cl[next(it) % len(cl)]())
        out["energy"] = energy_block(torch, steps, a.energy, spec.n)
    print(json.dumps(out), flush=True)
    return 0




def cpu_baseline(cases, target_s):
    """The oracle (as it stands) on a bounded sample of the workload: every layer on a
    subset of the batch's images (images are independent); and its single-thread time on
    C1 (one image, fp32)."""
    import oracle
    from paper_2404_19331_amd.workloads import make_inputs, config_c1
    oracle.build()
    threads = oracle.num_threads()

    def run(cs, nimg):
        t = 0.0
        moved = 0
        for c in cs:
            cc = c.with_(n=min(nimg, c.n))
            inp = make_inputs(cc)
            t0 = time.perf_counter()
            oracle.run(cc.op, cc, inp)
            t += time.perf_counter() - t0
            moved += layer_stats(cc)["bytes"]
        return t, moved

    t1, _ = run(cases, 1)
    nimg = max(1, min(max(c.n for c in cases), int(target_s / max(t1, 1e-3))))
    t, moved = run(cases, nimg) if nimg > 1 else run(cases, 1)
    oracle.set_num_threads(1)
    c1 = config_c1()
    t_c1 = min(run(c1, 1)[0] for _ in range(3))
    oracle.set_num_threads(threads)
    return {"value": round(moved / t / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": "all %d layers, %d of %d images each (images are independent); %.1f s of oracle time" % (
                len(cases), min(nimg, max(c.n for c in cases)), max(c.n for c in cases), t),
            "c1_single_thread_ms": round(1e3 * t_c1, 3)}


def layer_shape(c):
    """Geometry of a layer (what a kernel's traffic per launch depends on), as text."""
    return "n%d %dx%d %d->%d k%d s%d" % (c.n, c.h, c.w, c.c_in, c.c_out, c.k, c.stride)


def load_traffic(workload, kernel_name, shape):
    """HBM bytes per launch of a kernel on layers of one shape, from the rocprofv3 FETCH_SIZE /
    WRITE_SIZE runs (profiles/traffic.json), only if they were taken on the current kernel
    sources and on that shape."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    ent = rec.get("%s|%s" % (workload, kernel_name))
    if not ent or ent.get("source_hash") != kernel_source_hash() or ent.get("shape") != shape:
        return None
    return ent.get("bytes_per_launch")


def log(msg):
    print("bench: " + msg, file=sys.stderr, flush=True)


def build_layers(torch, fcm, cases, tune):
    import numpy as np
    from paper_2404_19331_amd.workloads import make_inputs

    def to_dev(v):
        if v is None:
            return None
        if v.dtype == np.uint16:
            return torch.from_numpy(v.view(np.int16).copy()).view(torch.bfloat16).cuda()
        return torch.from_numpy(v).cuda()

    layers = [Layer(c, torch, fcm, make_inputs, to_dev, tune=tune, log=log) for c in cases]
    torch.cuda.synchronize()
    return layers


def measure_config(torch, fcm, name, tune, stream):
    cases, desc = workload_cases(name)
    log("config %s: %d layers" % (name, len(cases)))
    layers = build_layers(torch, fcm, cases, tune)
    ent = []
    for L in layers:
        fu = time_layer(torch, L.fused_calls, stream)
        uu = time_layer(torch, L.unfused_calls, stream)
        hot = time_layer(torch, L.fused_calls, stream, hot=True)
        ent.append(layer_entry(fcm, L, fu, uu, hot))
    del layers
    torch.cuda.empty_cache()
    fu = sum(e["fused_us"] for e in ent)
    uu = sum(e["unfused_us"] for e in ent)
    c0 = cases[0]
    return {"workload": desc, "dtype": c0.dtype, "layout": c0.layout, "batch": c0.n,
            "fused_us": round(fu, 3), "unfused_us": round(uu, 3), "speedup": round(uu / fu, 3),
            "gbs": round(sum(e["bytes"] for e in ent) / (fu * 1e-6) / 1e9, 1), "layers": ent}


def main():
    a = parse()
    if a.gpus != 1:
        print("bench.py measures one GPU: the fused modules run on a single device and this build has no "
              "multi-GPU path (requested --gpus %d)." % a.gpus, file=sys.stderr)
        return 2
    import torch
    from paper_2404_19331_amd import fcm

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    fcm.lib()
    if a.workload.startswith("MNV2"):
        return bench_chain(a, torch, fcm)
    tune = not a.no_tune
    cases, desc = workload_cases(a.workload)
    if a.layers:
        keep = [int(i) for i in a.layers.split(",")]
        cases = [cases[i] for i in keep]
    stream = torch.cuda.current_stream()
    log("%s: %d layers, planning%s" % (a.workload, len(cases), " and tuning on the device" if tune else ""))
    layers = build_layers(torch, fcm, cases, tune)
    log("plans ready")

    fused_ms = time_steps(torch, layers, "fused", a.steps, a.warmup, stream)
    unf_ms = time_steps(torch, layers, "unfused", a.steps, a.warmup, stream)
    log("timed %d steps fused (%.3f ms/step) and unfused (%.3f ms/step)" % (a.steps, fused_ms, unf_ms))
    fused_us = [time_layer(torch, L.fused_calls, stream) for L in layers]
    unf_us = [time_layer(torch, L.unfused_calls, stream) for L in layers]
    hot_us = [time_layer(torch, L.fused_calls, stream, hot=True) for L in layers]

    tot_bytes = sum(L.stats["bytes"] for L in layers)
    value = tot_bytes / (fused_ms * 1e-3) / 1e9
    # dominant kernel: the compiled kernel (variant) on one layer shape taking the largest
    # share of the fused step; its achieved rate = its algorithmic bytes (flops) per launch
    # / its mean launch duration over those layers (each layer is launched equally often).
    groups = {}
    for i, L in enumerate(layers):
        groups.setdefault((int(L.plan.variant), layer_shape(L.case)), []).append(i)
    dkey = max(groups, key=lambda k: sum(fused_us[i] for i in groups[k]))
    dv, dshape = dkey
    idx = groups[dkey]
    t_us = sum(fused_us[i] for i in idx)
    g_bytes = sum(layers[i].stats["bytes"] for i in idx)
    g_flops = sum(layers[i].stats["flops"] for i in idx)
    dt = layers[idx[0]].case.dtype
    balance = MFMA_PEAK_TFLOPS[dt] * 1e12 / (HBM_PEAK_GBS * 1e9)
    if g_flops / g_bytes < balance:
        rf = {"bound": "hbm", "achieved": round(g_bytes / (t_us * 1e-6) / 1e9, 1), "peak": HBM_PEAK_GBS,
              "unit": "GB/s"}
    else:
        rf = {"bound": "mfma", "achieved": round(g_flops / (t_us * 1e-6) / 1e12, 2),
              "peak": MFMA_PEAK_TFLOPS[dt], "unit": "TFLOP/s"}
    rf["frac"] = round(rf["achieved"] / rf["peak"], 4)
    kname = fcm.variant_name(dv)
    rf["kernel"] = kname
    rf["layers"] = [layers[i].case.name for i in idx]
    rf["bytes_per_launch"] = int(g_bytes / len(idx))
    rf["us_per_launch"] = round(t_us / len(idx), 3)
    rf["shape"] = dshape
    rf["traffic"] = load_traffic(a.workload, kname, dshape)

    per_layer = [layer_entry(fcm, L, fu, uu, ho) for L, fu, uu, ho in zip(layers, fused_us, unf_us, hot_us)]
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(fused_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cases[0].dtype,
        "data": "synthetic (seeded, random-init weights)",
        "config": {"workload": desc, "name": a.workload, "layers": len(layers), "batch": cases[0].n,
                   "layout": cases[0].layout, "parallelism": "none (1 GPU)",
                   "rotating_buffers_bytes_min": ROTATE_BYTES,
                   "plans": "fastest of the planner's candidates timed on the device" if tune else "planner"},
        "protocol": "per layer: %d warm-up launches, median of %d repeats of >= %d launches over rotating buffers "
                    ">= %d MiB; hot_cache_fused_us: one buffer set repeated" % (
                        WARMUP_LAUNCHES, REPEATS, MIN_LAUNCHES, ROTATE_BYTES >> 20),
        "unfused": {"ms_per_step": round(unf_ms, 5),
                    "value": round(tot_bytes / (unf_ms * 1e-3) / 1e9, 2),
                    "speedup_fused": round(unf_ms / fused_ms, 3)},
        "roofline": rf,
        "layers": per_layer,
    }
    if a.energy > 0:
        def step_of(which):
            calls = [L.calls(which) for L in layers]
            it = iter(range(1 << 62))

            def step():
                k = next(it)
                for cl in calls:
                    cl[k % len(cl)]()
            return step
        out["energy"] = energy_block(torch, {"fused": step_of("fused"), "unfused": step_of("unfused")}, a.energy,
                                     cases[0].n)
    if a.calib:
        # plain device copy of known size for the profiler's byte counters: a float
        # multiply by one reads 256 MiB and writes 256 MiB
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        out["calib_copy_bytes"] = 256 << 20
    del layers
    torch.cuda.empty_cache()

    names = CONFIGS if a.configs == "all" else ([] if a.configs == "none" else a.configs.split(","))
    out["configs"] = {}
    for name in names:
        if name == a.workload and not a.layers:
            ent = per_layer
            fu = sum(e["fused_us"] for e in ent)
            uu = sum(e["unfused_us"] for e in ent)
            out["configs"][name] = {"workload": desc, "dtype": cases[0].dtype, "layout": cases[0].layout,
                                    "batch": cases[0].n, "fused_us": round(fu, 3), "unfused_us": round(uu, 3),
                                    "speedup": round(uu / fu, 3),
                                    "gbs": round(sum(e["bytes"] for e in ent) / (fu * 1e-6) / 1e9, 1),
                                    "layers": "as the headline's"}
            continue
        out["configs"][name] = measure_config(torch, fcm, name, tune, stream)
    if not a.no_cpu_baseline:
        log("timing the CPU oracle sample")
        out["cpu_baseline"] = cpu_baseline(cases, a.cpu_seconds)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
