"""Summaries of rocprofv3 output for the library's kernels.

    python -m paper_2608_04048_amd.profiling counters <dir> [--match NAME ...]
    python -m paper_2608_04048_amd.profiling stats <kernel_stats.csv> [--match NAME ...]

``counters`` reads every *_counter_collection.csv under <dir> (from
``rocprofv3 --pmc ... --output-format csv``) and prints, per kernel and
counter, the mean value per dispatch, the number of dispatches and the mean
dispatch duration. ``stats`` filters a *_kernel_stats.csv (from
``rocprofv3 --kernel-trace --stats``). Kernels are selected by substring
(default: the RRQ kernels and the runtime's copy kernel used to calibrate
byte counters).
"""

from __future__ import annotations

import argparse
import csv
import glob
import os
import sys
from collections import defaultdict

DEFAULT_MATCH = ["construct_kernel", "reconstruct_kernel", "copyBuffer"]


def _short(name: str) -> str:
    name = name.replace("rrq_detail::(anonymous namespace)::", "")
    return name.split("(")[0] if "(" in name else name


def counters(directory: str, match):
    sums = defaultdict(float)
    dispatches = defaultdict(set)
    durations = {}
    for path in glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True):
        with open(path, newline="") as fh:
            for row in csv.DictReader(fh):
                kname = row.get("Kernel_Name", "")
                if not any(m in kname for m in match):
                    continue
                key = (_short(kname), row["Counter_Name"])
                did = row.get("Dispatch_Id") or row.get("Correlation_Id")
                sums[key] += float(row["Counter_Value"])
                dispatches[key].add(did)
                try:
                    durations[(_short(kname), did)] = (int(row["End_Timestamp"]) -
                                                       int(row["Start_Timestamp"]))
                except (KeyError, ValueError):
                    pass
    out = []
    for (k, c), total in sorted(sums.items()):
        n = len(dispatches[(k, c)])
        ds = [v for (kk, _), v in durations.items() if kk == k]
        out.append((k, c, total / n, n, (sum(ds) / len(ds) / 1e3) if ds else float("nan")))
    return out


def stats(path: str, match):
    rows = []
    with open(path, newline="") as fh:
        for row in csv.DictReader(fh):
            if any(m in row["Name"] for m in match):
                rows.append((_short(row["Name"]), int(row["Calls"]), float(row["AverageNs"]) / 1e3,
                             float(row["MinNs"]) / 1e3, float(row["MaxNs"]) / 1e3))
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("counters")
    a.add_argument("directory")
    a.add_argument("--match", nargs="*", default=DEFAULT_MATCH)
    b = sub.add_parser("stats")
    b.add_argument("path")
    b.add_argument("--match", nargs="*", default=DEFAULT_MATCH)
    args = ap.parse_args(argv)
    if args.cmd == "counters":
        print("| kernel | counter | mean per dispatch | dispatches | mean duration (us) |")
        print("|---|---|---:|---:|---:|")
        for k, c, v, n, d in counters(args.directory, args.match):
            print(f"| {k} | {c} | {v:.6g} | {n} | {d:.1f} |")
    else:
        print("| kernel | calls | average (us) | min (us) | max (us) |")
        print("|---|---:|---:|---:|---:|")
        for k, n, avg, mn, mx in stats(args.path, args.match):
            print(f"| {k} | {n} | {avg:.1f} | {mn:.1f} | {mx:.1f} |")


if __name__ == "__main__":
    sys.exit(main())
