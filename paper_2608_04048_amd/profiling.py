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

DEFAULT_MATCH = ["construct_kernel", "reconstruct_kernel", "linear_kernel", "decode_kernel",
                 "batch_kernel", "prefill_kernel",
                 "stream_probe_kernel", "read_probe_kernel", "write_probe_kernel",
                 "construct_probe_kernel", "reconstruct_probe_kernel",
                 "copyBuffer"]


def _short(name: str) -> str:
    name = name.replace("rrq_detail::", "").replace("(anonymous namespace)::", "")
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


KERNEL_SOURCE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "rrq_kernels.hip")


def kernel_source_sha256(path: str = KERNEL_SOURCE) -> str:
    import hashlib
    with open(path, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()


def _mean_counter(directory, kernel, counter):
    for k, c, v, n, d in counters(directory, [kernel]):
        if c == counter and kernel in k:
            return v, n, d
    raise KeyError(f"{counter} for {kernel} not found under {directory}")


def traffic(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, kernel, copy_bytes):
    """HBM bytes per dispatch of `kernel`: FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch) each scaled by bytes / counter of a plain device copy of
    copy_bytes bytes."""
    fetch_kib, n_f, d_f = _mean_counter(fetch_dir, kernel, "FETCH_SIZE")
    write_kib, n_w, d_w = _mean_counter(write_dir, kernel, "WRITE_SIZE")
    copy_fetch_kib = _mean_counter(copy_fetch_dir, "copyBuffer", "FETCH_SIZE")[0]
    copy_write_kib = _mean_counter(copy_write_dir, "copyBuffer", "WRITE_SIZE")[0]
    f_scale = copy_bytes / (copy_fetch_kib * 1024)
    w_scale = copy_bytes / (copy_write_kib * 1024)
    read = fetch_kib * 1024 * f_scale
    written = write_kib * 1024 * w_scale
    return {"fetch_kib": fetch_kib, "write_kib": write_kib, "copy_fetch_kib": copy_fetch_kib,
            "copy_write_kib": copy_write_kib, "fetch_scale": f_scale, "write_scale": w_scale,
            "read_bytes": read, "written_bytes": written, "traffic_bytes": read + written,
            "dispatches": (n_f, n_w), "mean_us": (d_f, d_w)}


def read_traffic_profile(path):
    """(kernel_source_sha256, traffic_bytes_per_launch) recorded in a traffic
    profile, or None."""
    try:
        text = open(path).read()
    except OSError:
        return None
    vals = {}
    for line in text.splitlines():
        for key in ("kernel_source_sha256", "traffic_bytes_per_launch"):
            if line.strip().startswith(key + ":"):
                vals[key] = line.split(":", 1)[1].strip().strip("`")
    if len(vals) != 2:
        return None
    return vals["kernel_source_sha256"], float(vals["traffic_bytes_per_launch"])


def stats(path: str, match):
    rows = []
    with open(path, newline="") as fh:
        for row in csv.DictReader(fh):
            if any(m in row["Name"] for m in match):
                rows.append((_short(row["Name"]), int(row["Calls"]), float(row["AverageNs"]) / 1e3,
                             float(row["MinNs"]) / 1e3, float(row["MaxNs"]) / 1e3))
    return rows


def trace(path: str, match, first: int = 0):
    """Per-kernel durations from a rocprofv3 kernel-trace csv, in dispatch
    order: (kernel, calls, average, min, max, average of the first `first`
    dispatches) in microseconds. The first dispatches of a kernel are the
    ones of the leg that runs first in the profiled program."""
    per = defaultdict(list)
    with open(path, newline="") as fh:
        for row in csv.DictReader(fh):
            name = row.get("Kernel_Name", "")
            if not any(m in name for m in match):
                continue
            per[_short(name)].append((int(row["Start_Timestamp"]),
                                      (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) / 1e3))
    out = []
    for k, v in per.items():
        v.sort()
        d = [x for _, x in v]
        head = d[:first] if first > 0 else []
        out.append((k, len(d), sum(d) / len(d), min(d), max(d),
                    sum(head) / len(head) if head else float("nan")))
    out.sort(key=lambda r: -r[1] * r[2])
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("counters")
    a.add_argument("directory")
    a.add_argument("--match", nargs="*", default=DEFAULT_MATCH)
    b = sub.add_parser("stats")
    b.add_argument("path")
    b.add_argument("--match", nargs="*", default=DEFAULT_MATCH)
    tr = sub.add_parser("trace")
    tr.add_argument("path")
    tr.add_argument("--match", nargs="*", default=DEFAULT_MATCH)
    tr.add_argument("--first", type=int, default=0)
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-fetch", required=True)
    t.add_argument("--copy-write", required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--kernel", required=True)
    t.add_argument("--source", default=KERNEL_SOURCE,
                   help="the kernel's source file, whose hash the summary records")
    args = ap.parse_args(argv)
    if args.cmd == "traffic":
        r = traffic(args.fetch, args.write, args.copy_fetch, args.copy_write, args.kernel,
                    args.copy_bytes)
        print(f"kernel: `{args.kernel}`")
        print(f"kernel_source: `{os.path.relpath(args.source, os.path.dirname(os.path.dirname(KERNEL_SOURCE)))}`")
        print(f"kernel_source_sha256: `{kernel_source_sha256(args.source)}`")
        print(f"traffic_bytes_per_launch: `{r['traffic_bytes']:.6e}`")
        print()
        print("| quantity | value |")
        print("|---|---:|")
        print(f"| FETCH_SIZE per dispatch (KiB) | {r['fetch_kib']:.6g} |")
        print(f"| WRITE_SIZE per dispatch (KiB) | {r['write_kib']:.6g} |")
        print(f"| copy probe: bytes copied | {args.copy_bytes} |")
        print(f"| copy probe FETCH_SIZE (KiB) | {r['copy_fetch_kib']:.6g} |")
        print(f"| copy probe WRITE_SIZE (KiB) | {r['copy_write_kib']:.6g} |")
        print(f"| fetch scale (bytes per counted byte) | {r['fetch_scale']:.4f} |")
        print(f"| write scale | {r['write_scale']:.4f} |")
        print(f"| HBM bytes read per launch | {r['read_bytes']:.6e} |")
        print(f"| HBM bytes written per launch | {r['written_bytes']:.6e} |")
        print(f"| dispatches profiled (fetch, write) | {r['dispatches']} |")
        return 0
    if args.cmd == "trace":
        print(f"| kernel | calls | average (us) | min (us) | max (us) | average of the first {args.first} (us) |")
        print("|---|---:|---:|---:|---:|---:|")
        for k, n, avg, mn, mx, hd in trace(args.path, args.match, args.first):
            print(f"| {k} | {n} | {avg:.1f} | {mn:.1f} | {mx:.1f} | {hd:.1f} |")
        return 0
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
