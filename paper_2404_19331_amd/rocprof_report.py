"""Summaries of rocprofv3 output for the fused-module kernels.

  python -m paper_2404_19331_amd.rocprof_report stats KERNEL_STATS_CSV [--title T] [--command C]
      per-kernel launch statistics (from `rocprofv3 --kernel-trace --stats`) as a text table

  python -m paper_2404_19331_amd.rocprof_report traffic --workload W --variant NAME [--kernel SYMBOL]
          --fetch COUNTER_CSV --write COUNTER_CSV [--calib-bytes B] [--out profiles/traffic.json]
      HBM bytes per launch of one compiled variant from two `rocprofv3 --pmc` runs of
      `bench.py --calib` (FETCH_SIZE, then WRITE_SIZE). Each counter is scaled by what it
      reads for the bench's plain device copy of known size (a float multiply by one over
      B bytes that reads B and writes B bytes), so the unit and the coverage of the counter
      cancel out. The entry is keyed by workload and variant and stamped with the hash of
      the kernel sources; bench.py reports it only while the sources are unchanged.
      --kernel gives the demangled kernel name (as the stats table prints it) for variants
      whose name kernel_symbol does not map.

  python -m paper_2404_19331_amd.rocprof_report counters CSV [CSV ...] --kernel SUBSTRING [--title T]
          [--command C]
      mean per dispatch of every counter of `rocprofv3 --pmc` runs, for the kernels whose
      demangled name contains SUBSTRING, one row per kernel and counter
  python -m paper_2404_19331_amd.rocprof_report layers --manifest MANIFEST_JSON --fetch CSV
          --write CSV --mfma CSV --trace KERNEL_TRACE_CSV [--title T] [--command C]
      per-layer table of a `profile_layers` run: for the fused module and for its two
      unfused stages, the mean launch time, the HBM bytes per launch (FETCH_SIZE and
      WRITE_SIZE scaled by the calibration copy that precedes each layer) against the
      planner's figures (bytes_ideal: input + weights + output once; bytes_tiled: per-tile
      staging; bytes_paper: Eq. 1-4), and the matrix-core busy fraction
      (SQ_VALU_MFMA_BUSY_CYCLES over 1024 SIMDs x 2.4 GHz x the launch time).
"""
import argparse
import csv
import json
import os
import re
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

_MODE = {"k_dwpw3": 0, "k_pw3": 1, "k_dw3": 2}
_DT = {"f32": "TF32", "bf16": "TBF16", "i8": "TI8"}


def kernel_symbol(variant, split=False, qx=0):
    """Demangled kernel name of a variant: persistent, e.g. k_dwpw3<bf16,3,1,1,16,p16> ->
    void fcm::k_fused3<fcm::TBF16, 3, 1, 1, 16, 0, 16, 1, false, 0>(fcm::KArgs) (the instance
    of unsplit symmetric plans; split=True names the one of split plans, qx = 1 / 2 the int8
    instances with zero points / with per-channel requantisation); streaming (k_dwpw5<...>),
    whole-module (k_dwpw6<...>) and deep (k_dwpw7<...>) variants map to their single instance."""
    m5 = re.match(r"(k_\w+5)<(\w+),(\d+),(\d+),(\d+)x(\d+),ct(\d+),wc(\d+)>$", variant)
    if m5:  # streaming kernels: k_fused5<DT, K, S, MODE, TH, TW, CTW, WC>
        fam, dt, k, s, th, tw, ct, wc = m5.groups()
        mode = {"k_dwpw5": 0, "k_pw5": 1, "k_dw5": 2}[fam]
        return "void fcm::k_fused5<fcm::%s, %s, %s, %d, %s, %s, %s, %s>(fcm::KArgs)" % (_DT[dt], k, s, mode, th, tw, ct, wc)
    m7 = re.match(r"k_dwpw7<bf16,3,(\d+),(\d+)x(\d+),ct(\d+)(?:,k(\d+))?>$", variant)
    if m7:  # deep kernels: k_deep7<S, TH, TW, CTW, KC>
        s7, th, tw, ct, kc = m7.groups()
        return "void fcm::k_deep7<%s, %s, %s, %s, %s>(fcm::KArgs)" % (s7, th, tw, ct, kc or "1")
    m6 = re.match(r"(k_\w+6)<f32,(\d+),(\d+),(\d+)x(\d+)>$", variant)
    if m6:  # whole-module fp32 kernels: k_small6<MODE, K, S, TH, TW>
        fam, k, s, th, tw = m6.groups()
        mode = {"k_dwpw6": 0, "k_pwdw6": 1, "k_pwdwpw6": 2}[fam]
        return "void fcm::k_small6<%d, %s, %s, %s, %s>(fcm::KArgs)" % (mode, k, s, th, tw)
    m = re.match(r"(k_\w+3)<(\w+),(\d+),(\d+),(\d+),(\d+),p(\d+)(?:,k(\d+))?>$", variant)
    if not m:
        raise ValueError("not a persistent, streaming or whole-module kernel variant name: %s" % variant)
    fam, dt, k, s, bpw, ct, pitch, ks = m.groups()
    if fam == "k_pw3":
        k = s = "1"
    return "void fcm::k_fused3<fcm::%s, %s, %s, %s, %s, %d, %s, %s, %s, %d>(fcm::KArgs)" % (
        _DT[dt], k, s, bpw, ct, _MODE[fam], pitch, ks or "1", "true" if split else "false", qx)


def read_counters(path):
    """{(kernel name, counter): [value per dispatch]} and {kernel name: [grid sizes]}."""
    vals, grids = defaultdict(list), defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            vals[(r["Kernel_Name"], r["Counter_Name"])].append(float(r["Counter_Value"]))
            grids[r["Kernel_Name"]].append(int(r["Grid_Size"]))
    return vals, grids


def _calib(vals, grids, counter):
    """Counter value of the calibration copy: the multiply kernel with the largest grid."""
    best = None
    for name, gs in grids.items():
        if "MulFunctor" not in name or (name, counter) not in vals:
            continue
        if best is None or max(gs) > best[0]:
            best = (max(gs), [v for v, g in zip(vals[(name, counter)], gs) if g == max(gs)])
    if not best:
        raise SystemExit("no calibration copy (MulFunctor kernel) with counter %s: run bench.py --calib" % counter)
    return sum(best[1]) / len(best[1])


def _mean(vals, name, counter):
    v = vals.get((name, counter))
    if not v:
        raise SystemExit("kernel %s has no %s samples" % (name, counter))
    return sum(v) / len(v)


def traffic(args):
    sym = args.kernel or kernel_symbol(args.variant, args.split)
    fv, fg = read_counters(args.fetch)
    wv, wg = read_counters(args.write)
    f_k, w_k = _mean(fv, sym, "FETCH_SIZE"), _mean(wv, sym, "WRITE_SIZE")
    f_c, w_c = _calib(fv, fg, "FETCH_SIZE"), _calib(wv, wg, "WRITE_SIZE")
    rb = f_k / f_c * args.calib_bytes
    wb = w_k / w_c * args.calib_bytes
    sys.path.insert(0, ROOT)
    import bench  # the hash of the kernel sources that bench.py checks
    ent = {"variant": args.variant, "kernel": sym, "read_bytes_per_launch": int(rb), "write_bytes_per_launch": int(wb),
           "bytes_per_launch": int(rb + wb), "launches": len(fv[(sym, "FETCH_SIZE")]),
           "fetch_kib_per_launch": round(f_k, 1), "write_kib_per_launch": round(w_k, 1),
           "calib_fetch_kib": round(f_c, 1), "calib_write_kib": round(w_c, 1), "calib_bytes": args.calib_bytes,
           "source_hash": bench.kernel_source_hash()}
    if args.shape:
        ent["shape"] = args.shape
    rec = {}
    if os.path.exists(args.out):
        with open(args.out) as f:
            rec = json.load(f)
    rec["%s|%s" % (args.workload, args.variant)] = ent
    with open(args.out, "w") as f:
        json.dump(rec, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps(ent))


def _dispatches(path, field="counter"):
    """[(dispatch id, kernel name, {counter: value} or duration ns)] in dispatch order."""
    with open(path) as f:
        rows = list(csv.DictReader(f))
    if field == "trace":
        out = [(int(r["Dispatch_Id"]), r["Kernel_Name"], int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
               for r in rows]
        return sorted(out)
    by = {}
    for r in rows:
        d = by.setdefault(int(r["Dispatch_Id"]), [r["Kernel_Name"], {}])
        d[1][r["Counter_Name"]] = d[1].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return sorted((k, v[0], v[1]) for k, v in by.items())


def _segments(disp, nlayers, reps):
    """Per layer: (calibration dispatches, fused, dw, pw) of a profile_layers run: each
    layer starts with three calibration copies (MulFunctor) followed by 3 x reps launches."""
    out, i = [], 0
    for _ in range(nlayers):
        while i < len(disp) and "MulFunctor" not in disp[i][1]:
            i += 1
        cal = disp[i:i + 3]
        body = disp[i + 3:i + 3 + 3 * reps]
        if len(cal) < 3 or len(body) < 3 * reps:
            raise SystemExit("dispatch sequence shorter than the manifest says")
        out.append((cal, body[:reps], body[reps:2 * reps], body[2 * reps:]))
        i += 3 + 3 * reps
    return out


def layers(args):
    with open(args.manifest) as f:
        man = json.load(f)
    reps, nl, cb = man["reps"], len(man["layers"]), man["calib_bytes"]
    fetch = _segments(_dispatches(args.fetch), nl, reps)
    write = _segments(_dispatches(args.write), nl, reps)
    mfma = _segments(_dispatches(args.mfma), nl, reps)
    trace = _segments(_dispatches(args.trace, "trace"), nl, reps)

    def mean(xs):
        xs = xs[1:] if len(xs) > 2 else xs  # the first launch of a group warms the instruction cache
        return sum(xs) / len(xs)

    out = []
    if args.title:
        out.append(args.title)
    if args.command:
        out.append("commands:\n" + args.command)
    out.append("")
    out.append("HBM MB = (FETCH_SIZE + WRITE_SIZE) per launch, scaled by the calibration copy of %d MiB "
               "(read and written) preceding each layer; ideal = input + weights + output once; tiled = the "
               "planner's per-tile staging bytes; paper = Eq. 1-4; MFMA = matrix-core busy fraction." % (cb >> 20))
    out.append("%-34s %-34s %7s %7s %7s %7s %7s %6s %5s | %7s %7s %7s %5s" % (
        "layer", "fused kernel", "us", "HBM_MB", "ideal", "tiled", "paper", "HBM/id", "MFMA",
        "unf_us", "unf_HBM", "unf_id", "HBM/id"))
    rows = []
    for li, L in enumerate(man["layers"]):
        res = {}
        for role, k in (("fused", 1), ("dw", 2), ("pw", 3)):
            fcal = mean([d[2]["FETCH_SIZE"] for d in fetch[li][0]])
            wcal = mean([d[2]["WRITE_SIZE"] for d in write[li][0]])
            rb = mean([d[2]["FETCH_SIZE"] for d in fetch[li][k]]) / fcal * cb
            wb = mean([d[2]["WRITE_SIZE"] for d in write[li][k]]) / wcal * cb
            us = mean([d[2] for d in trace[li][k]]) / 1e3
            busy = mean([d[2].get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) for d in mfma[li][k]])
            res[role] = {"us": us, "hbm": rb + wb, "read": rb, "write": wb,
                         "mfma": busy / (1024 * us * 1e3 * 2.4), "kernel": fetch[li][k][0][1]}
        f, dwr, pwr = res["fused"], res["dw"], res["pw"]
        fi, ui = L["fused"]["bytes_ideal"], L["dw"]["bytes_ideal"] + L["pw"]["bytes_ideal"]
        uhbm = dwr["hbm"] + pwr["hbm"]
        out.append("%-34s %-34s %7.2f %7.2f %7.2f %7.2f %7.2f %6.2f %5.2f | %7.2f %7.2f %7.2f %5.2f" % (
            L["layer"][:34], L["fused"]["variant"][:34], f["us"], f["hbm"] / 1e6, fi / 1e6,
            L["fused"]["bytes_tiled"] / 1e6, L["fused"]["bytes_paper"] / 1e6, f["hbm"] / fi, f["mfma"],
            dwr["us"] + pwr["us"], uhbm / 1e6, ui / 1e6, uhbm / ui))
        rows.append({"layer": L["layer"], "fused": dict(f, plan=L["fused"]), "dw": dict(dwr, plan=L["dw"]),
                     "pw": dict(pwr, plan=L["pw"])})
    print("\n".join(out))
    if args.json:
        with open(args.json, "w") as fh:
            json.dump(rows, fh, indent=1)


def stats(args):
    with open(args.csv) as f:
        rows = list(csv.DictReader(f))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    out = []
    if args.title:
        out.append(args.title)
    if args.command:
        out.append("command: " + args.command)
    out.append("")
    out.append("%-72s %6s %12s %10s %10s %10s" % ("kernel", "calls", "total_us", "avg_us", "min_us", "max_us"))
    for r in rows[:args.top]:
        out.append("%-72s %6d %12.1f %10.3f %10.3f %10.3f" % (
            r["Name"][:72], int(r["Calls"]), float(r["TotalDurationNs"]) / 1e3, float(r["AverageNs"]) / 1e3,
            float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3))
    print("\n".join(out))


def counters(a):
    rows = defaultdict(list)
    for path in a.csv:
        vals, _ = read_counters(path)
        for (kernel, counter), v in vals.items():
            if a.kernel in kernel:
                rows[(kernel, counter)] += v
    out = []
    if a.title:
        out.append(a.title)
    if a.command:
        out.append("command: " + a.command)
    if out:
        out.append("")
    out.append("%-60s %-34s %10s %16s" % ("kernel", "counter", "dispatches", "mean per dispatch"))
    for (kernel, counter) in sorted(rows):
        v = rows[(kernel, counter)]
        out.append("%-60s %-34s %10d %16.1f" % (kernel[:60], counter, len(v), sum(v) / len(v)))
    print("\n".join(out))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--title", default="")
    s.add_argument("--command", default="")
    s.add_argument("--top", type=int, default=16)
    t = sub.add_parser("traffic")
    t.add_argument("--workload", required=True)
    t.add_argument("--variant", required=True)
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--split", action="store_true", help="the split-plan instance of the variant")
    t.add_argument("--calib-bytes", type=int, default=256 << 20)
    t.add_argument("--out", default=os.path.join(ROOT, "profiles", "traffic.json"))
    t.add_argument("--kernel", default="", help="demangled kernel name (default: from the variant name)")
    t.add_argument("--shape", default="", help="layer shape the run launched the kernel on (bench.py --layers)")
    c = sub.add_parser("counters")
    c.add_argument("csv", nargs="+")
    c.add_argument("--kernel", required=True)
    c.add_argument("--title", default="")
    c.add_argument("--command", default="")
    l = sub.add_parser("layers")
    l.add_argument("--manifest", required=True)
    l.add_argument("--fetch", required=True)
    l.add_argument("--write", required=True)
    l.add_argument("--mfma", required=True)
    l.add_argument("--trace", required=True)
    l.add_argument("--title", default="")
    l.add_argument("--command", default="")
    l.add_argument("--json", default="")
    a = ap.parse_args()
    {"stats": stats, "traffic": traffic, "counters": counters, "layers": layers}[a.cmd](a)


if __name__ == "__main__":
    main()
