"""Summaries of rocprofv3 output for the profiles/ folder.

  stats   KERNEL_STATS_CSV TITLE COMMAND        -> markdown table (stdout)
  traffic FETCH_CSV WRITE_CSV OUT_JSON ...     -> calibrated HBM bytes per dispatch
  pmc     OUT_MD TITLE --csv ... --kernel ...  -> MFMA busy share, executed MFMA flops,
                                                 instruction mix per dispatch

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


def per_dispatch_all(path, name_re):
    """{counter: (mean value per dispatch, dispatches)} and the mean dispatch
    duration in ns, over the dispatches of kernels matching name_re."""
    vals, dur = {}, {}
    for r in csv.DictReader(open(path)):
        if not re.search(name_re, r["Kernel_Name"]):
            continue
        vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
        dur[r["Dispatch_Id"]] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    if not vals:
        raise SystemExit(f"no rows for {name_re} in {path}")
    return ({k: (sum(v) / len(v), len(v)) for k, v in vals.items()},
            sum(dur.values()) / len(dur))


def cmd_pmc(args):
    """Counter summary per kernel.  SQ_* counters are summed over the whole
    GPU; GRBM_GUI_ACTIVE is summed over the XCDs, so one XCD's busy clocks
    are GRBM_GUI_ACTIVE / xcds.  SQ_VALU_MFMA_BUSY_CYCLES counts SIMD clocks
    with the matrix core busy, so dividing it by (SIMDs x busy clocks) gives
    the share of the matrix cores' time spent on MFMA work; one unit of
    SQ_INSTS_VALU_MFMA_MOPS_* is 512 flops."""
    simds = args.cus * 4
    lines = [f"# rocprofv3 counters: {args.title}", "",
             "Commands (repository root, after `cd /tmp && export TMPDIR=/tmp`; one counter set per run):",
             "", "```"] + args.command + ["```", ""]
    out = {}
    for k in args.kernel:
        # each counter keeps the dispatch duration of the run it was read in
        c, dur_of = {}, {}
        for path in args.csv:
            v, dur = per_dispatch_all(path, k)
            for n, (x, _) in v.items():
                c[n], dur_of[n] = x, dur
            n_disp = next(iter(v.values()))[1]
        dur_ns = sum(dur_of.values()) / len(dur_of)
        gui = c.get("GRBM_GUI_ACTIVE", 0.0) / args.xcds
        row = {"dispatches": n_disp, "duration_us": dur_ns / 1e3}
        if gui:
            row["clock_ghz"] = gui / dur_of["GRBM_GUI_ACTIVE"]
        if "SQ_VALU_MFMA_BUSY_CYCLES" in c and gui:
            row["mfma_busy"] = c["SQ_VALU_MFMA_BUSY_CYCLES"] / (simds * gui)
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in c:
            fl = 512.0 * c["SQ_INSTS_VALU_MFMA_MOPS_BF16"]
            row["mfma_bf16_gflop"] = fl / 1e9
            row["mfma_bf16_tflops"] = fl / dur_of["SQ_INSTS_VALU_MFMA_MOPS_BF16"] / 1e3
            row["mfma_bf16_frac_of_peak"] = row["mfma_bf16_tflops"] / args.bf16_peak
            if "clock_ghz" in row:
                row["frac_of_peak_at_clock"] = (row["mfma_bf16_tflops"] / args.bf16_peak
                                                * args.peak_clock / row["clock_ghz"])
        if "SQ_INSTS_MFMA" in c and "SQ_VALU_MFMA_BUSY_CYCLES" in c and c["SQ_INSTS_MFMA"]:
            row["mfma_busy_clk_per_inst"] = c["SQ_VALU_MFMA_BUSY_CYCLES"] / c["SQ_INSTS_MFMA"]
        if c.get("SQ_WAVES"):
            row["insts_per_wave"] = {n[9:]: c[n] / c["SQ_WAVES"] for n in sorted(c)
                                     if n.startswith("SQ_INSTS_")}
        if c.get("SQ_WAVE_CYCLES"):
            row["share_of_wave_cycles"] = {n[3:]: c[n] / c["SQ_WAVE_CYCLES"] for n in sorted(c)
                                           if n.startswith(("SQ_WAIT_", "SQ_ACTIVE_INST_"))}
        row["counters"] = c
        out[k] = row
    lines += ["| kernel | dispatches | avg us (counters on) | busy clock GHz | MFMA busy "
              "| MFMA bf16 TFLOP/s executed | of 2.5 PF/s | of peak at the busy clock |",
              "|---|---:|---:|---:|---:|---:|---:|---:|"]
    fmt = lambda r, n, f: (f % r[n]) if n in r else "-"
    for k, r in out.items():
        lines.append(f"| `{k}` | {r['dispatches']} | {r['duration_us']:.1f} | "
                     f"{fmt(r, 'clock_ghz', '%.2f')} | {fmt(r, 'mfma_busy', '%.3f')} | "
                     f"{fmt(r, 'mfma_bf16_tflops', '%.1f')} | "
                     f"{fmt(r, 'mfma_bf16_frac_of_peak', '%.3f')} | "
                     f"{fmt(r, 'frac_of_peak_at_clock', '%.3f')} |")
    for k, r in out.items():
        lines += ["", f"## `{k}`", ""]
        if "mfma_busy_clk_per_inst" in r:
            lines.append(f"MFMA busy clocks per MFMA instruction: {r['mfma_busy_clk_per_inst']:.2f}")
            lines.append("")
        if "insts_per_wave" in r:
            lines.append("Instructions per wave: " + ", ".join(
                f"{n} {v:,.0f}" for n, v in r["insts_per_wave"].items()))
            lines.append("")
        if "share_of_wave_cycles" in r:
            lines.append("Share of wave-cycles: " + ", ".join(
                f"{n} {v:.3f}" for n, v in r["share_of_wave_cycles"].items()))
            lines.append("")
        lines.append("Raw counters per dispatch: " + ", ".join(
            f"{n} {v:,.0f}" for n, v in sorted(r["counters"].items())))
    for note in args.note or []:
        lines += ["", note]
    if args.json:
        d = {"workload": args.workload, "commands": args.command, "sources": args.sources,
             "sources_hash": sources_hash([os.path.join(os.path.dirname(PKG), x)
                                           for x in args.sources]),
             "kernels": {k: {n: v for n, v in r.items() if n != "counters"}
                         for k, r in out.items()}}
        with open(args.json, "w") as f:
            json.dump(d, f, indent=1)
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


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
    m = sub.add_parser("pmc")
    m.add_argument("out")
    m.add_argument("title")
    m.add_argument("--csv", action="append", required=True)
    m.add_argument("--command", action="append", required=True)
    m.add_argument("--kernel", action="append", required=True)
    m.add_argument("--cus", type=int, default=256)
    m.add_argument("--xcds", type=int, default=8)
    m.add_argument("--bf16-peak", type=float, default=2500.0, help="TFLOP/s")
    m.add_argument("--peak-clock", type=float, default=2.4, help="GHz the peak is quoted at")
    m.add_argument("--note", action="append", help="paragraph appended to the summary")
    m.add_argument("--json", help="also write the derived figures here, with a hash of --sources")
    m.add_argument("--workload", default=None)
    m.add_argument("--sources", nargs="+", default=[])
    a = ap.parse_args(argv)
    {"stats": cmd_stats, "traffic": cmd_traffic, "pmc": cmd_pmc}[a.cmd](a)


if __name__ == "__main__":
    main(sys.argv[1:])
