"""Summaries of rocprofv3 output for the fused-module kernels.

  python -m paper_2404_19331_amd.rocprof_report stats KERNEL_STATS_CSV [--title T] [--command C]
      per-kernel launch statistics (from `rocprofv3 --kernel-trace --stats`) as a text table

  python -m paper_2404_19331_amd.rocprof_report traffic --workload W --variant NAME
          --fetch COUNTER_CSV --write COUNTER_CSV [--calib-bytes B] [--out profiles/traffic.json]
      HBM bytes per launch of one compiled variant from two `rocprofv3 --pmc` runs of
      `bench.py --calib` (FETCH_SIZE, then WRITE_SIZE). Each counter is scaled by what it
      reads for the bench's plain device copy of known size (a float multiply by one over
      B bytes that reads B and writes B bytes), so the unit and the coverage of the counter
      cancel out. The entry is keyed by workload and variant and stamped with the hash of
      the kernel sources; bench.py reports it only while the sources are unchanged.
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


def kernel_symbol(variant, split=False):
    """Demangled kernel name of a persistent variant, e.g. k_dwpw3<bf16,3,1,1,16,p16> ->
    void fcm::k_fused3<fcm::TBF16, 3, 1, 1, 16, 0, 16, 1, false>(fcm::KArgs) (the instance
    of unsplit plans; split=True names the one of split plans)."""
    m = re.match(r"(k_\w+3)<(\w+),(\d+),(\d+),(\d+),(\d+),p(\d+)(?:,k(\d+))?>$", variant)
    if not m:
        raise ValueError("not a persistent-kernel variant name: %s" % variant)
    fam, dt, k, s, bpw, ct, pitch, ks = m.groups()
    if fam == "k_pw3":
        k = s = "1"
    return "void fcm::k_fused3<fcm::%s, %s, %s, %s, %s, %d, %s, %s, %s>(fcm::KArgs)" % (
        _DT[dt], k, s, bpw, ct, _MODE[fam], pitch, ks or "1", "true" if split else "false")


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
    sym = kernel_symbol(args.variant, args.split)
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
    rec = {}
    if os.path.exists(args.out):
        with open(args.out) as f:
            rec = json.load(f)
    rec["%s|%s" % (args.workload, args.variant)] = ent
    with open(args.out, "w") as f:
        json.dump(rec, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps(ent))


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
    a = ap.parse_args()
    (stats if a.cmd == "stats" else traffic)(a)


if __name__ == "__main__":
    main()
