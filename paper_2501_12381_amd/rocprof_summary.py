"""Summarise rocprofv3 CSV output (kernel stats, kernel trace, PMC counters).

    python -m paper_2501_12381_amd.rocprof_summary stats DIR
    python -m paper_2501_12381_amd.rocprof_summary traffic FETCH_DIR WRITE_DIR --copy-bytes N \
        --workload NAME --kernel-map gspn_scan_bwd=resident_bwd_kernel [...] [--calls K] [--json OUT]

`counters DIR --kernel PATTERN` prints the mean per-dispatch value of every
counter collected for the kernels whose name contains PATTERN.

`stats` prints per-kernel call count and average/min/max duration from a
`rocprofv3 --kernel-trace --stats --output-format csv` run.

`traffic` turns two counter runs (`--pmc FETCH_SIZE`, `--pmc WRITE_SIZE`, each
reported in KiB per dispatch) into HBM bytes per launch.  Each counter is
scaled by the factor that makes it read the known byte count of the plain copy
kernel the benchmark runs for calibration (`--copy-bytes` read and written),
so the result is in the same units as the algorithmic bytes.  With `--calls K`
the bytes of all dispatches matching a pattern are summed and divided by K:
the traffic of one API call that launches several kernels (the two-pass
forward), when the profiled run made K such calls.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import sys
from collections import defaultdict


def _find(d: str, suffix: str) -> list[str]:
    return sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True))


def _col(row: dict, *names):
    low = {k.lower(): v for k, v in row.items()}
    for n in names:
        if n.lower() in low:
            return low[n.lower()]
    raise KeyError(f"none of {names} in {list(row)}")


def kernel_stats(d: str) -> dict:
    """name -> dict(calls, avg_ns, min_ns, max_ns) from the kernel trace (or stats) CSV."""
    out = {}
    traces = _find(d, "kernel_trace.csv")
    if traces:
        durs = defaultdict(list)
        for path in traces:
            for row in csv.DictReader(open(path)):
                name = _col(row, "Kernel_Name", "KernelName", "Name")
                start = int(_col(row, "Start_Timestamp", "BeginNs", "Start"))
                end = int(_col(row, "End_Timestamp", "EndNs", "End"))
                durs[name].append(end - start)
        for name, v in durs.items():
            out[name] = dict(calls=len(v), avg_ns=sum(v) / len(v), min_ns=min(v), max_ns=max(v))
        return out
    for path in _find(d, "kernel_stats.csv"):
        for row in csv.DictReader(open(path)):
            name = _col(row, "Name", "Kernel_Name")
            out[name] = dict(calls=int(_col(row, "Calls")), avg_ns=float(_col(row, "AverageNs")),
                             min_ns=float(_col(row, "MinNs")), max_ns=float(_col(row, "MaxNs")))
    return out


def counter_values(d: str, counter: str) -> dict:
    """kernel name -> list of per-dispatch values of one counter."""
    vals = defaultdict(lambda: defaultdict(float))
    for path in _find(d, "counter_collection.csv"):
        for row in csv.DictReader(open(path)):
            if _col(row, "Counter_Name", "CounterName") != counter:
                continue
            name = _col(row, "Kernel_Name", "KernelName")
            disp = _col(row, "Dispatch_Id", "DispatchId", "Correlation_Id")
            vals[name][disp] += float(_col(row, "Counter_Value", "CounterValue", "Value"))
    return {k: list(v.values()) for k, v in vals.items()}


def all_counters(d: str, pattern: str) -> dict:
    """counter name -> mean per-dispatch value over the kernels whose name contains pattern."""
    vals = defaultdict(lambda: defaultdict(float))
    for path in _find(d, "counter_collection.csv"):
        for row in csv.DictReader(open(path)):
            if pattern not in _col(row, "Kernel_Name", "KernelName"):
                continue
            disp = _col(row, "Dispatch_Id", "DispatchId", "Correlation_Id")
            vals[_col(row, "Counter_Name", "CounterName")][disp] += float(
                _col(row, "Counter_Value", "CounterValue", "Value"))
    return {k: sum(v.values()) / len(v) for k, v in vals.items()}


def short(name: str, width: int = 90) -> str:
    return name if len(name) <= width else name[: width - 3] + "..."


def cmd_stats(args) -> int:
    st = kernel_stats(args.dir)
    if not st:
        print(f"no kernel trace or stats CSV under {args.dir}", file=sys.stderr)
        return 1
    total = sum(v["avg_ns"] * v["calls"] for v in st.values())
    print(f"{'calls':>6} {'avg_us':>10} {'min_us':>10} {'max_us':>10} {'share':>6}  kernel")
    for name, v in sorted(st.items(), key=lambda kv: -kv[1]["avg_ns"] * kv[1]["calls"]):
        share = v["avg_ns"] * v["calls"] / total
        print(f"{v['calls']:>6} {v['avg_ns'] / 1e3:>10.2f} {v['min_ns'] / 1e3:>10.2f} "
              f"{v['max_ns'] / 1e3:>10.2f} {share:>6.1%}  {short(name)}")
    return 0


def _match(name: str, pattern: str) -> bool:
    """pattern: substrings separated by '|'; the name matches if it contains any."""
    return any(p in name for p in pattern.split("|"))


def cmd_traffic(args) -> int:
    fetch = counter_values(args.fetch_dir, "FETCH_SIZE")
    write = counter_values(args.write_dir, "WRITE_SIZE")
    copy_f = [v for k, vs in fetch.items() if _match(k, args.copy_kernel) for v in vs]
    copy_w = [v for k, vs in write.items() if _match(k, args.copy_kernel) for v in vs]
    if not copy_f or not copy_w:
        print("copy-calibration kernel not found in the counter runs", file=sys.stderr)
        return 1
    # both counters read KiB per dispatch; the copy moves copy_bytes each way
    sf = args.copy_bytes / (max(copy_f) * 1024.0)
    sw = args.copy_bytes / (max(copy_w) * 1024.0)
    result = {"workload": args.workload, "copy_bytes": args.copy_bytes,
              "fetch_scale": sf, "write_scale": sw, "kernels": {}}
    print(f"copy calibration: FETCH_SIZE x {sf:.4f}, WRITE_SIZE x {sw:.4f}")
    for item in args.kernel_map:
        call, pattern = item.split("=", 1)
        f = [v for k, vs in fetch.items() if _match(k, pattern) for v in vs]
        w = [v for k, vs in write.items() if _match(k, pattern) for v in vs]
        if not f or not w:
            print(f"{call}: kernel matching {pattern!r} not found", file=sys.stderr)
            return 1
        div_f, div_w = (args.calls, args.calls) if args.calls else (len(f), len(w))
        fb = sum(f) / div_f * 1024.0 * sf
        wb = sum(w) / div_w * 1024.0 * sw
        result["kernels"][call] = {"kernel": pattern, "fetch_bytes_per_launch": fb,
                                   "write_bytes_per_launch": wb,
                                   "hbm_bytes_per_launch": fb + wb,
                                   "dispatches": len(f), "calls": args.calls or len(f)}
        print(f"{call} ({pattern}): fetch {fb / 1e6:.1f} MB + write {wb / 1e6:.1f} MB "
              f"= {(fb + wb) / 1e6:.1f} MB per launch")
    if args.json:
        if args.source_hash:
            result["kernel_source_hash"] = args.source_hash
        with open(args.json, "w") as fh:
            json.dump(result, fh, indent=1)
    return 0


def cmd_counters(args) -> int:
    vals = all_counters(args.dir, args.kernel)
    if not vals:
        print(f"no counters for kernels matching {args.kernel!r} under {args.dir}", file=sys.stderr)
        return 1
    for k in sorted(vals):
        print(f"{k:32s} {vals[k]:20.1f}")
    return 0


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    t = sub.add_parser("traffic")
    t.add_argument("fetch_dir")
    t.add_argument("write_dir")
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--copy-kernel", default="copy_calibration")
    t.add_argument("--workload", required=True)
    t.add_argument("--kernel-map", nargs="+", required=True)
    t.add_argument("--calls", type=int, default=0,
                   help="API calls in the profiled run (sum the matching dispatches over them)")
    t.add_argument("--json")
    t.add_argument("--source-hash")
    c = sub.add_parser("counters")
    c.add_argument("dir")
    c.add_argument("--kernel", required=True, help="substring of the kernel name")
    args = ap.parse_args(argv)
    return {"stats": cmd_stats, "traffic": cmd_traffic, "counters": cmd_counters}[args.cmd](args)


if __name__ == "__main__":
    sys.exit(main())
