"""Summaries of rocprofv3 CSV output for profiles/ (measurement helper; not
used by the library).

  python -m paper_2607_24981_amd.profsum kernels DIR --title T --command C
      per-kernel call count, total / average / min duration and launch shape
      from DIR/*_kernel_stats.csv and DIR/*_kernel_trace.csv, and per launch
      grid for kernels launched with several grids
  python -m paper_2607_24981_amd.profsum traffic FETCH_DIR WRITE_DIR --workload W
      --stage S --kernel K --source F [--source F ...] --copy-mib N --command C
      HBM bytes per launch of the kernels whose name starts with K (per
      variant, the dispatches with its largest grid): FETCH_SIZE and
      WRITE_SIZE (KiB per dispatch) scaled by what the same counters read
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
    by_grid = {}  # (kernel, grid) -> durations in ns
    if trace:
        for r in csv.DictReader(open(trace[0])):
            k = short(r["Kernel_Name"])
            grid = f"{r['Grid_Size_X']}x{r['Grid_Size_Y']}x{r['Grid_Size_Z']}"
            by_grid.setdefault((k, grid), []).append(
                int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
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
    multi = {k for k, _ in by_grid if sum(1 for k2, _ in by_grid if k2 == k) > 1}
    if multi:
        print("# kernels launched with several grids (e.g. a batch split over streams and "
              "a whole-batch pass), from the trace:")
        print(f"#{'calls':>6} {'avg_us':>8} {'min_us':>8}  kernel  grid (threads)")
        for (k, grid), d in sorted(by_grid.items()):
            if k in multi:
                print(f"#{len(d):6d} {statistics.mean(d) / 1e3:8.2f} {min(d) / 1e3:8.2f}  "
                      f"{k}  {grid}")
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
                             float(r["Counter_Value"]), int(r["Grid_Size"])))
    if not rows:
        sys.exit(f"no {counter} rows under {dirname}")
    return rows


def traffic(args):
    fetch = _pmc(args.fetch_dir, "FETCH_SIZE")
    write = _pmc(args.write_dir, "WRITE_SIZE")
    copies_f = [v for _, k, v, _ in fetch if k.startswith("__amd_rocclr_copyBuffer")]
    copies_w = [v for _, k, v, _ in write if k.startswith("__amd_rocclr_copyBuffer")]
    known_kib = args.copy_mib * 1024.0
    f_scale = known_kib / max(copies_f)
    w_scale = known_kib / max(copies_w)
    # Per variant, only the dispatches with its largest grid count: the
    # whole-batch launches that the per-launch timing measures (a batch split
    # over streams launches the same kernels on parts of the batch too).
    names = sorted({k for _, k, _, _ in fetch if k.startswith(args.kernel)})
    top = {n: max(g for _, k, _, g in fetch if k == n) for n in names}
    grids = {}
    for _, k, v, g in fetch:
        if k in top:
            grids.setdefault((k, g), []).append(v)
    kf = [v for _, k, v, g in fetch if k in top and g == top[k]]
    kw = [v for _, k, v, g in write if k in top and g == top[k]]
    if not kf or not kw:
        sys.exit(f"no dispatch of {args.kernel}")
    fetch_b = statistics.mean(kf) * f_scale * 1024
    write_b = statistics.mean(kw) * w_scale * 1024
    rec = {"kernel": args.kernel, "variants": names, "dispatches": len(kf),
           "grids": {n: top[n] for n in names},
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
    print("# FETCH_SIZE per (variant, grid in threads); the largest grid of each variant "
          "(whole-batch launches) is used")
    for (k, g), v in sorted(grids.items()):
        print(f"#   {k}  grid {g}: {len(v)} dispatches, mean {statistics.mean(v):.1f} KiB")
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
