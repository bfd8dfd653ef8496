"""Summaries of rocprofv3 CSV output for profiles/ (measurement helper; not
used by the library).

  python -m paper_2607_24981_amd.profsum kernels DIR --title T --command C
      per-kernel call count, total / average / min duration and launch shape
      from DIR/*_kernel_stats.csv and DIR/*_kernel_trace.csv
  python -m paper_2607_24981_amd.profsum traffic FETCH_DIR WRITE_DIR --workload W
      --stage S --kernel K --source F [--source F ...] --copy-mib N --command C
      HBM bytes per launch of the kernels whose name starts with K: FETCH_SIZE
      and WRITE_SIZE (KiB per dispatch) scaled by what the same counters read
      for the plain device copy of N MiB that the profiled command made first
      (the __amd_rocclr_copyBuffer dispatch with the largest FETCH_SIZE);
      updates profiles/traffic.json and prints a text summary.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
import statistics
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def short(name: str) -> str:
    name = name.replace("ilw::(anonymous namespace)::", "").replace("void ", "")
    return re.sub(r"\(.*$", "", name)


def source_digest(paths) -> str:
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def kernels(args):
    stats = glob.glob(os.path.join(args.dir, "**", "*kernel_stats.csv"), recursive=True)
    trace = glob.glob(os.path.join(args.dir, "**", "*kernel_trace.csv"), recursive=True)
    if not stats:
        sys.exit(f"no *kernel_stats.csv under {args.dir}")
    shapes = {}
    if trace:
        for r in csv.DictReader(open(trace[0])):
            k = short(r["Kernel_Name"])
            if k not in shapes:
                shapes[k] = (r["Grid_Size_X"], r["Grid_Size_Y"], r["Grid_Size_Z"],
                             r["Workgroup_Size_X"], r["LDS_Block_Size"], r["VGPR_Count"],
                             r["Accum_VGPR_Count"], r["Scratch_Size"])
    print(f"# {args.title}")
    print(f"# command: {args.command}")
    print("# source: rocprofv3 --kernel-trace --stats --output-format csv (kernel_stats.csv)")
    print(f"{'calls':>7} {'total_us':>11} {'avg_us':>8} {'min_us':>8} {'pct':>6}  kernel")
    for r in csv.DictReader(open(stats[0])):
        print(f"{int(r['Calls']):7d} {float(r['TotalDurationNs']) / 1e3:11.1f} "
              f"{float(r['AverageNs']) / 1e3:8.2f} {float(r['MinNs']) / 1e3:8.2f} "
              f"{float(r['Percentage']):6.2f}  {short(r['Name'])}")
    if shapes:
        print("# launch shape of the first dispatch: grid (threads), workgroup, LDS bytes, "
              "VGPR, AGPR, scratch")
        for k, (gx, gy, gz, wx, lds, v, a, sc) in shapes.items():
            print(f"#   {k}: grid {gx}x{gy}x{gz} wg {wx} lds {lds} vgpr {v} agpr {a} "
                  f"scratch {sc}")


def _pmc(dirname, counter):
    rows = []
    for f in glob.glob(os.path.join(dirname, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] == counter:
                rows.append((int(r["Dispatch_Id"]), short(r["Kernel_Name"]),
                             float(r["Counter_Value"])))
    if not rows:
        sys.exit(f"no {counter} rows under {dirname}")
    return rows


def traffic(args):
    fetch = _pmc(args.fetch_dir, "FETCH_SIZE")
    write = _pmc(args.write_dir, "WRITE_SIZE")
    copies_f = [v for _, k, v in fetch if k.startswith("__amd_rocclr_copyBuffer")]
    copies_w = [v for _, k, v in write if k.startswith("__amd_rocclr_copyBuffer")]
    known_kib = args.copy_mib * 1024.0
    f_scale = known_kib / max(copies_f)
    w_scale = known_kib / max(copies_w)
    kf = [v for _, k, v in fetch if k.startswith(args.kernel)]
    kw = [v for _, k, v in write if k.startswith(args.kernel)]
    if not kf or not kw:
        sys.exit(f"no dispatch of {args.kernel}")
    names = sorted({k for _, k, _ in fetch if k.startswith(args.kernel)})
    fetch_b = statistics.mean(kf) * f_scale * 1024
    write_b = statistics.mean(kw) * w_scale * 1024
    rec = {"kernel": args.kernel, "variants": names, "dispatches": len(kf),
           "fetch_bytes_per_launch": round(fetch_b), "write_bytes_per_launch": round(write_b),
           "hbm_bytes_per_launch": round(fetch_b + write_b),
           "copy_scale_fetch": round(f_scale, 4), "copy_scale_write": round(w_scale, 4),
           "source_sha256_16": source_digest(args.source), "sources": args.source,
           "command": args.command}
    path = os.path.join(ROOT, "profiles", "traffic.json")
    table = json.load(open(path)) if os.path.exists(path) else {}
    table.setdefault(args.workload, {})[args.stage] = rec
    with open(path, "w") as f:
        json.dump(table, f, indent=1, sort_keys=True)
        f.write("\n")
    print(f"# HBM traffic of {args.kernel}* in {args.workload} (stage {args.stage})")
    print(f"# command: {args.command}")
    print("# source: rocprofv3 --pmc FETCH_SIZE, then --pmc WRITE_SIZE (KiB per dispatch)")
    print(f"# calibration: plain device copy of {args.copy_mib} MiB reads FETCH_SIZE "
          f"{max(copies_f):.0f} KiB, WRITE_SIZE {max(copies_w):.0f} KiB -> scale "
          f"{f_scale:.4f} / {w_scale:.4f}")
    print(f"dispatches {len(kf)}  variants {', '.join(names)}")
    print(f"FETCH_SIZE mean {statistics.mean(kf):.1f} KiB -> {fetch_b / 1e6:.3f} MB per launch")
    print(f"WRITE_SIZE mean {statistics.mean(kw):.1f} KiB -> {write_b / 1e6:.3f} MB per launch")
    print(f"HBM bytes per launch {(fetch_b + write_b) / 1e6:.3f} MB")


def main():
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    k = sub.add_parser("kernels")
    k.add_argument("dir")
    k.add_argument("--title", required=True)
    k.add_argument("--command", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("fetch_dir")
    t.add_argument("write_dir")
    t.add_argument("--workload", required=True)
    t.add_argument("--stage", required=True)
    t.add_argument("--kernel", required=True)
    t.add_argument("--source", action="append", required=True)
    t.add_argument("--copy-mib", type=float, required=True)
    t.add_argument("--command", required=True)
    args = ap.parse_args()
    kernels(args) if args.cmd == "kernels" else traffic(args)


if __name__ == "__main__":
    main()
