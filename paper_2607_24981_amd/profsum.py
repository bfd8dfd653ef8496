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
  python -m paper_2607_24981_amd.profsum counters DIR [DIR ...] --title T --command C
      --label NAME=PATTERN[@PREV][#GRID] [--label ...] [--ops NAME=OPS] [--units NAME=N:WHAT]
      per labelled kernel, the mean of every counter over its dispatches from
      DIR/**/*counter_collection.csv (one directory per --pmc pass), and the
      derived figures: int8 MFMA ops (MOPS_I8 x 512) against the algorithmic
      ops given with --ops, MFMA busy and VALU busy as fractions of the
      SIMD-cycles of the dispatch (GRBM_GUI_ACTIVE is summed over the 8
      XCDs), VALU instructions per wave and per unit (--units, e.g. scores or
      outputs per dispatch), LDS busy and bank-conflict share, and the share
      of wave time spent waiting.  A dispatch takes the first label whose
      PATTERN is in its kernel name and, with @PREV, whose preceding dispatch
      has PREV in its name (with #GRID: whose grid has GRID threads).
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


MI355X_CUS, MI355X_SIMDS, MI355X_XCDS = 256, 1024, 8


def counters(args):
    import collections
    per = collections.defaultdict(dict)  # (dir, dispatch) -> {counter: value}
    meta = {}
    for d in args.dirs:
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                key = (d, int(r["Dispatch_Id"]))
                per[key][r["Counter_Name"]] = float(r["Counter_Value"])
                meta[key] = (short(r["Kernel_Name"]), int(r["Grid_Size"]),
                             int(r["Workgroup_Size"]), int(r["LDS_Block_Size"]),
                             int(r["VGPR_Count"]), int(r["Accum_VGPR_Count"]),
                             int(r["Scratch_Size"]))
    rules = []
    for spec in args.label:
        name, pat = spec.split("=", 1)
        pat, _, grid = pat.partition("#")
        pat, _, prev = pat.partition("@")
        rules.append((name, pat, prev, int(grid) if grid else 0))
    ops = dict((k, float(v)) for k, v in (o.split("=", 1) for o in args.ops or []))
    units = {}
    for u in args.units or []:
        k, v = u.split("=", 1)
        n, _, what = v.partition(":")
        units[k] = (float(n), what or "unit")
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    shape = {}
    ndisp = collections.defaultdict(lambda: collections.Counter())
    for d in args.dirs:
        ids = sorted(i for (dd, i) in meta if dd == d)
        prev = ""
        for i in ids:
            k = meta[(d, i)][0]
            for name, pat, pv, gr in rules:
                if pat in k and (not pv or pv in prev) and (not gr or gr == meta[(d, i)][1]):
                    for c, v in per[(d, i)].items():
                        agg[name][c].append(v)
                    ndisp[name][d] += 1
                    shape[name] = (k,) + meta[(d, i)][1:]
                    break
            prev = k
    print(f"# {args.title}")
    print(f"# command: {args.command}")
    print("# source: rocprofv3 --pmc (one pass per counter group), counter_collection.csv; "
          "per label the mean over its dispatches")
    print(f"# MI355X: {MI355X_CUS} CUs, {MI355X_SIMDS} SIMDs, {MI355X_XCDS} XCDs; one "
          "v_mfma_i32_16x16x64_i8 = 32768 int8 ops = 64 MOPS_I8 units = 16 MFMA-busy cycles")
    for name, _, _, _ in rules:
        if name not in agg:
            continue
        m = {c: statistics.mean(v) for c, v in agg[name].items()}
        n = max(ndisp[name].values())  # dispatches per pass
        k, grid, wg, lds, vgpr, agpr, scr = shape[name]
        print(f"\n[{name}] {k}")
        print(f"  dispatches {n}; grid {grid} threads, workgroup {wg}, LDS {lds} B, "
              f"VGPR {vgpr}, AGPR {agpr}, scratch {scr}")
        gui = m.get("GRBM_GUI_ACTIVE")
        cyc = gui / MI355X_XCDS if gui else None
        waves = m.get("SQ_WAVES")
        if cyc:
            print(f"  GRBM_GUI_ACTIVE {gui:.0f} (summed over XCDs) -> {cyc:.0f} cycles, "
                  f"{cyc / 2.4e3:.2f} us at 2.4 GHz (counter run: dispatches serialized)")
        if "SQ_INSTS_VALU_MFMA_MOPS_I8" in m:
            mops = m["SQ_INSTS_VALU_MFMA_MOPS_I8"] * 512
            line = f"  int8 MFMA ops {mops / 1e9:.4f} G"
            if name in ops:
                line += f" (algorithmic {ops[name] / 1e9:.4f} G, ratio {mops / ops[name]:.3f})"
            print(line)
        if "SQ_VALU_MFMA_BUSY_CYCLES" in m and cyc:
            print(f"  MFMA busy {m['SQ_VALU_MFMA_BUSY_CYCLES'] / (cyc * MI355X_SIMDS):.4f} of "
                  f"SIMD-cycles")
        if "SQ_ACTIVE_INST_VALU" in m and cyc:
            print(f"  VALU busy {m['SQ_ACTIVE_INST_VALU'] / (cyc * MI355X_CUS):.4f} "
                  f"(SQ_ACTIVE_INST_VALU / (CUs x cycles))")
        if waves:
            for c in ("SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_INSTS_LDS", "SQ_INSTS_SALU",
                      "SQ_INSTS_VALU_INT32", "SQ_INSTS_VALU_INT64", "SQ_INSTS_VMEM_RD",
                      "SQ_INSTS_VMEM_WR"):
                if c in m:
                    extra = ""
                    if c == "SQ_INSTS_VALU" and name in units:
                        cnt, what = units[name]
                        extra = f", {m[c] * 64 / cnt:.2f} lane-instructions per {what}"
                    print(f"  {c} {m[c]:.0f} ({m[c] / waves:.1f} per wave{extra})")
        if "SQ_LDS_IDX_ACTIVE" in m and cyc:
            la = m["SQ_LDS_IDX_ACTIVE"]
            print(f"  LDS busy {la / (cyc * MI355X_CUS):.4f}; bank-conflict cycles "
                  f"{m.get('SQ_LDS_BANK_CONFLICT', 0) / la if la else 0:.4f} of LDS-active cycles")
        if "SQ_WAIT_INST_ANY" in m and "SQ_WAVE_CYCLES" in m:
            print(f"  waves waiting on instruction dependencies "
                  f"{m['SQ_WAIT_INST_ANY'] / m['SQ_WAVE_CYCLES']:.4f} of wave-cycles"
                  + (f" (LDS {m['SQ_WAIT_INST_LDS'] / m['SQ_WAVE_CYCLES']:.4f})"
                     if "SQ_WAIT_INST_LDS" in m else ""))
        rest = sorted(c for c in m if not c.startswith(("SQ_INSTS", "GRBM")))
        print("  raw: " + ", ".join(f"{c} {m[c]:.4g}" for c in rest))


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
    c = sub.add_parser("counters")
    c.add_argument("dirs", nargs="+")
    c.add_argument("--title", required=True)
    c.add_argument("--command", required=True)
    c.add_argument("--label", action="append", required=True)
    c.add_argument("--ops", action="append")
    c.add_argument("--units", action="append")
    args = ap.parse_args()
    {"kernels": kernels, "traffic": traffic, "counters": counters}[args.cmd](args)


if __name__ == "__main__":
    main()
