"""Benchmark of the fused DW/PW modules on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload C3b32]

A step is one pass of the fused path over every layer of the workload (plan lookup +
one fused kernel per layer) on one batch of seeded synthetic input. The same layers are
then timed layer-by-layer (one DW and one PW kernel per layer, intermediate through HBM)
as the unfused comparison. Inputs are resident in HBM before the timed region. Each
layer cycles through rotating buffer sets totalling >= 512 MiB so that the 256 MiB
Infinity Cache cannot serve a repeated working set.

Prints ONE JSON line: metric/value (achieved HBM GB/s = algorithmic bytes / time),
per-layer microseconds fused and unfused, the roofline of the dominant kernel (measured
with HIP events on the launch stream), and the CPU oracle timed on a bounded sample.
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
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "i8": 5000.0, "f32": 157.3}
METRIC = "fused DW+PW layer us and achieved HBM GB/s (% roofline) vs unfused DW->PW"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="C3b32",
                    choices=["C1", "C2", "C3b1", "C3b32", "C4", "C5", "PWPW", "MNV2", "MNV2bf16", "MNV2zp"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target CPU-baseline sample time")
    ap.add_argument("--layers", default=None, help="comma-separated layer indices (subset)")
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
    """Algorithmic bytes (input + weights + output once) and flops of one fused layer,
    and the unfused intermediate bytes (written once and read once per intermediate)."""
    e = elt(c.dtype)
    ho, wo = out_hw(c)
    kk = c.k * c.k
    x = c.n * c.h * c.w * c.c_in
    if c.op == "dw_pw":
        w = c.c_in * kk + c.c_out * c.c_in
        y = c.n * ho * wo * c.c_out
        mids = [c.n * ho * wo * c.c_in]
        flops = 2 * c.n * ho * wo * c.c_in * (kk + c.c_out)
    elif c.op == "pw_dw_pw":
        w = c.c_mid * c.c_in + c.c_mid * kk + c.c_out * c.c_mid
        y = c.n * ho * wo * c.c_out
        mids = [c.n * c.h * c.w * c.c_mid, c.n * ho * wo * c.c_mid]
        flops = 2 * (c.n * c.h * c.w * c.c_mid * c.c_in + c.n * ho * wo * c.c_mid * (kk + c.c_out))
    elif c.op == "pw_pw":
        w = c.c_mid * c.c_in + c.c_out * c.c_mid
        y = c.n * c.h * c.w * c.c_out
        mids = [c.n * c.h * c.w * c.c_mid]
        flops = 2 * c.n * c.h * c.w * c.c_mid * (c.c_in + c.c_out)
    else:  # pw_dw
        w = c.c_mid * c.c_in + c.c_mid * kk
        y = c.n * ho * wo * c.c_mid
        mids = [c.n * c.h * c.w * c.c_mid]
        flops = 2 * (c.n * c.h * c.w * c.c_mid * c.c_in + c.n * ho * wo * c.c_mid * kk)
    fused = (x + w + y) * e
    unfused = fused + 2 * sum(mids) * e
    return dict(bytes=fused, bytes_unfused=unfused, flops=flops, x=x * e, y=y * e, mids=[m * e for m in mids])


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2404_19331_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


class Layer:
    """Device buffers (rotating sets) and pre-marshalled launches for one layer."""

    def __init__(self, case, torch, fcm, make_inputs, to_dev):
        self.case = c = case
        self.stats = layer_stats(case)
        d = {k: to_dev(v) for k, v in make_inputs(case).items()}
        ho, wo = out_hw(c)
        self.nsets = max(2, -(-ROTATE_BYTES // (self.stats["x"] + self.stats["y"])))
        x0 = d["x"]

        def shaped(ch, h, w):
            shp = (c.n, ch, h, w)
            return shp if c.layout == "nchw" else (c.n, h, w, ch)

        ych = c.c_mid if c.op == "pw_dw" else c.c_out
        if c.op == "dw_pw":
            mid_shapes = [shaped(c.c_in, ho, wo)]
        elif c.op == "pw_dw_pw":
            mid_shapes = [shaped(c.c_mid, c.h, c.w), shaped(c.c_mid, ho, wo)]
        else:  # pw_dw, pw_pw
            mid_shapes = [shaped(c.c_mid, c.h, c.w)]
        self.desc = fcm.desc_from_case(c)
        self.plan = fcm.plan(c.op, self.desc)
        rq = list(c.rq) if c.dtype == "i8" else None
        self.fused_calls, self.unfused_calls = [], []
        for j in range(self.nsets):
            x = x0 if j == 0 else x0.clone()
            y = torch.empty(shaped(ych, ho, wo), dtype=x0.dtype, device=x0.device)
            mids = [torch.empty(s, dtype=x0.dtype, device=x0.device) for s in mid_shapes]
            kw = dict(stride=c.stride, pad=c.pad, layout=c.layout, out=y, prepare=True)
            if c.op == "dw_pw":
                f = fcm.dw_pw(x, d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), act=c.act[:2], rq=rq,
                              plan=self.plan, **kw)
                u = fcm.dw_then_pw(x, d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), act=c.act[:2], rq=rq,
                                   mid=mids[0], **kw)
            elif c.op == "pw_dw_pw":
                f = fcm.pw_dw_pw(x, d["w_pw1"], d["w_dw"], d["w_pw2"], d.get("b_pw1"), d.get("b_dw"),
                                 d.get("b_pw2"), act=c.act, rq=rq, plan=self.plan, **kw)
                u = fcm.pw_then_dw_then_pw(x, d["w_pw1"], d["w_dw"], d["w_pw2"], d.get("b_pw1"), d.get("b_dw"),
                                           d.get("b_pw2"), act=c.act, rq=rq, mids=(mids[0], mids[1]), **kw)
            elif c.op == "pw_pw":
                kp = dict(layout=c.layout, out=y, prepare=True)
                f = fcm.pw_pw(x, d["w_pw1"], d["w_pw2"], d.get("b_pw1"), d.get("b_pw2"), act=c.act[:2], rq=rq,
                              plan=self.plan, **kp)
                u = fcm.pw_then_pw(x, d["w_pw1"], d["w_pw2"], d.get("b_pw1"), d.get("b_pw2"), act=c.act[:2], rq=rq,
                                   mid=mids[0], **kp)
            else:
                f = fcm.pw_dw(x, d["w_pw"], d["w_dw"], d.get("b_pw"), d.get("b_dw"), act=c.act[:2], rq=rq,
                              plan=self.plan, **kw)
                u = fcm.pw_then_dw(x, d["w_pw"], d["w_dw"], d.get("b_pw"), d.get("b_dw"), act=c.act[:2], rq=rq,
                                   mid=mids[0], **kw)
            self.fused_calls.append(f)
            self.unfused_calls.append(u)
        self.i = 0

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


def time_layer(torch, layer, which, launches, stream):
    """Average microseconds per launch of one layer: `launches` back-to-back launches
    over its rotating buffer sets between two events on the launch stream."""
    cl = layer.calls(which)
    for j in range(min(len(cl), 3)):
        cl[j]()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    _preroll(torch)
    t0.record(stream)
    for j in range(launches):
        cl[j % len(cl)]()
    t1.record(stream)
    torch.cuda.synchronize()
    return 1000.0 * t0.elapsed_time(t1) / launches


def cpu_baseline(cases, target_s):
    """The oracle (as it stands) on a bounded sample of the workload: every layer on a
    subset of the batch's images (images are independent)."""
    import oracle
    from paper_2404_19331_amd.workloads import make_inputs
    oracle.build()
    threads = oracle.num_threads()

    def run(nimg):
        t = 0.0
        moved = 0
        for c in cases:
            cc = c.with_(n=min(nimg, c.n))
            inp = make_inputs(cc)
            t0 = time.perf_counter()
            oracle.run(cc.op, cc, inp)
            t += time.perf_counter() - t0
            moved += layer_stats(cc)["bytes"]
        return t, moved

    t1, _ = run(1)
    nimg = max(1, min(max(c.n for c in cases), int(target_s / max(t1, 1e-3))))
    t, moved = run(nimg) if nimg > 1 else run(1)
    return {"value": round(moved / t / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": "all %d layers, %d of %d images each (images are independent); %.1f s of oracle time" % (
                len(cases), min(nimg, max(c.n for c in cases)), max(c.n for c in cases), t)}


def load_traffic(workload, kernel_name):
    """HBM bytes per launch of a kernel from the rocprofv3 FETCH_SIZE / WRITE_SIZE runs
    (profiles/traffic.json), only if they were taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    ent = rec.get("%s|%s" % (workload, kernel_name))
    if not ent or ent.get("source_hash") != kernel_source_hash():
        return None
    return ent.get("bytes_per_launch")


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


def main():
    a = parse()
    if a.gpus != 1:
        print("bench.py measures one GPU: the fused modules run on a single device and this build has no "
              "multi-GPU path (requested --gpus %d)." % a.gpus, file=sys.stderr)
        return 2
    import numpy as np
    import torch
    from paper_2404_19331_amd import fcm
    from paper_2404_19331_amd.workloads import make_inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    fcm.lib()
    if a.workload.startswith("MNV2"):
        return bench_chain(a, torch, fcm)
    cases, desc = workload_cases(a.workload)
    if a.layers:
        keep = [int(i) for i in a.layers.split(",")]
        cases = [cases[i] for i in keep]

    def to_dev(v):
        if v is None:
            return None
        if v.dtype == np.uint16:
            return torch.from_numpy(v.view(np.int16).copy()).view(torch.bfloat16).cuda()
        return torch.from_numpy(v).cuda()

    stream = torch.cuda.current_stream()
    layers = [Layer(c, torch, fcm, make_inputs, to_dev) for c in cases]
    torch.cuda.synchronize()
    print("bench: %s, %d layers, plans ready" % (a.workload, len(layers)), file=sys.stderr, flush=True)

    fused_ms = time_steps(torch, layers, "fused", a.steps, a.warmup, stream)
    unf_ms = time_steps(torch, layers, "unfused", a.steps, a.warmup, stream)
    print("bench: timed %d steps fused (%.3f ms/step) and unfused (%.3f ms/step)" % (a.steps, fused_ms, unf_ms),
          file=sys.stderr, flush=True)
    launches = max(a.steps, 100)
    fused_us = [time_layer(torch, L, "fused", launches, stream) for L in layers]
    unf_us = [time_layer(torch, L, "unfused", launches, stream) for L in layers]

    tot_bytes = sum(L.stats["bytes"] for L in layers)
    value = tot_bytes / (fused_ms * 1e-3) / 1e9
    # dominant kernel: the compiled kernel (variant) taking the largest share of the fused
    # step; its achieved rate = its algorithmic bytes (flops) per launch / its mean launch
    # duration, over every layer it runs (each layer is launched equally often).
    groups = {}
    for i, L in enumerate(layers):
        groups.setdefault(int(L.plan.variant), []).append(i)
    dv = max(groups, key=lambda v: sum(fused_us[i] for i in groups[v]))
    idx = groups[dv]
    t_us = sum(fused_us[i] for i in idx)
    g_bytes = sum(layers[i].stats["bytes"] for i in idx)
    g_flops = sum(layers[i].stats["flops"] for i in idx)
    dt = layers[idx[0]].case.dtype
    balance = MFMA_PEAK_TFLOPS[dt] * 1e12 / (HBM_PEAK_GBS * 1e9)
    if g_flops / g_bytes < balance:
        roof = {"bound": "hbm", "achieved": round(g_bytes / (t_us * 1e-6) / 1e9, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": round(g_flops / (t_us * 1e-6) / 1e12, 2),
                "peak": MFMA_PEAK_TFLOPS[dt], "unit": "TFLOP/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    kname = fcm.variant_name(dv)
    roof["kernel"] = kname
    roof["layers"] = [layers[i].case.name for i in idx]
    roof["bytes_per_launch"] = int(g_bytes / len(idx))
    roof["us_per_launch"] = round(t_us / len(idx), 3)
    roof["traffic"] = load_traffic(a.workload, kname)

    per_layer = []
    for L, fu, uu in zip(layers, fused_us, unf_us):
        st = L.stats
        per_layer.append({
            "layer": L.case.name, "fused_us": round(fu, 3), "unfused_us": round(uu, 3),
            "speedup": round(uu / fu, 3), "bytes": int(st["bytes"]), "bytes_unfused": int(st["bytes_unfused"]),
            "gbs": round(st["bytes"] / (fu * 1e-6) / 1e9, 1),
            "hbm_frac": round(st["bytes"] / (fu * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "tile": [int(L.plan.tile_h), int(L.plan.tile_w), int(L.plan.c_block), int(L.plan.co_block)],
            "wgs": int(L.plan.workgroups)})

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
                   "rotating_buffers_bytes_min": ROTATE_BYTES},
        "unfused": {"ms_per_step": round(unf_ms, 5),
                    "value": round(sum(L.stats["bytes"] for L in layers) / (unf_ms * 1e-3) / 1e9, 2),
                    "speedup_fused": round(unf_ms / fused_ms, 3)},
        "roofline": roof,
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
    if not a.no_cpu_baseline:
        print("bench: timing CPU oracle sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(cases, a.cpu_seconds)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
