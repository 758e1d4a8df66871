"""Summaries of rocprofv3 output for the profiles/ folder.

  stats   KERNEL_STATS_CSV TITLE COMMAND        -> markdown table (stdout)
  traffic FETCH_CSV WRITE_CSV OUT_JSON ...     -> calibrated HBM bytes per dispatch

`traffic` reads two `rocprofv3 --pmc FETCH_SIZE` / `--pmc WRITE_SIZE` runs of
the same program (counter_collection.csv, values in KiB per dispatch),
scales each counter by what it reads for a plain copy kernel of known size in
the same run, and records the per-dispatch averages of the named kernels
together with a hash of the kernel sources (a summary whose hash no longer
matches the sources is stale).
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import sys

PKG = os.path.dirname(os.path.abspath(__file__))


def sources_hash(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def short_name(n: str) -> str:
    n = re.sub(r"\(.*", "", n).replace("void ", "")
    return n[:80]


def cmd_stats(args):
    rows = list(csv.DictReader(open(args.csv)))
    print(f"# {args.title}\n")
    print("Command (from the repository root on one MI355X, after `cd /tmp && export "
          "TMPDIR=/tmp`):\n")
    print("```\n" + args.command + "\n```\n")
    print("| kernel | calls | avg us | min us | max us | % time |")
    print("|---|---:|---:|---:|---:|---:|")
    for r in rows[:args.top]:
        print(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
              f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
              f"{float(r['Percentage']):.2f} |")


def per_dispatch(path, counter, name_re, grid=None):
    vals = []
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter or not re.search(name_re, r["Kernel_Name"]):
            continue
        if grid is not None and int(r["Grid_Size"]) != grid:
            continue
        vals.append(float(r["Counter_Value"]))
    if not vals:
        raise SystemExit(f"no {counter} rows for {name_re} in {path}")
    return sum(vals) / len(vals), len(vals)


def cmd_traffic(args):
    cal_f, _ = per_dispatch(args.fetch, "FETCH_SIZE", args.cal_kernel, args.cal_grid)
    cal_w, _ = per_dispatch(args.write, "WRITE_SIZE", args.cal_kernel, args.cal_grid)
    f_factor = args.cal_bytes / (cal_f * 1024.0)
    w_factor = args.cal_bytes / (cal_w * 1024.0)
    out = {"workload": args.workload, "command_fetch": args.command_fetch,
           "command_write": args.command_write,
           "calibration": {"kernel": args.cal_kernel, "grid": args.cal_grid,
                           "bytes_each_way": args.cal_bytes,
                           "fetch_kib": cal_f, "write_kib": cal_w,
                           "fetch_factor": round(f_factor, 4), "write_factor": round(w_factor, 4)},
           "sources": args.sources, "sources_hash": sources_hash(
               [os.path.join(os.path.dirname(PKG), s) for s in args.sources]),
           "kernels": {}}
    for k in args.kernel:
        fk, n = per_dispatch(args.fetch, "FETCH_SIZE", k)
        wk, _ = per_dispatch(args.write, "WRITE_SIZE", k)
        out["kernels"][k] = {"dispatches": n, "fetch_kib": fk, "write_kib": wk,
                             "hbm_bytes": fk * 1024.0 * f_factor + wk * 1024.0 * w_factor}
    with open(args.out, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out, indent=1))


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("title")
    s.add_argument("command")
    s.add_argument("--top", type=int, default=14)
    t = sub.add_parser("traffic")
    t.add_argument("fetch")
    t.add_argument("write")
    t.add_argument("out")
    t.add_argument("--workload", required=True)
    t.add_argument("--kernel", action="append", required=True)
    t.add_argument("--cal-kernel", required=True)
    t.add_argument("--cal-grid", type=int, default=None)
    t.add_argument("--cal-bytes", type=float, required=True)
    t.add_argument("--sources", nargs="+", required=True)
    t.add_argument("--command-fetch", required=True)
    t.add_argument("--command-write", required=True)
    a = ap.parse_args(argv)
    {"stats": cmd_stats, "traffic": cmd_traffic}[a.cmd](a)


if __name__ == "__main__":
    main(sys.argv[1:])
