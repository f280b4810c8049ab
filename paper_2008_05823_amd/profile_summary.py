"""Summaries of rocprofv3 output for the SAEF kernels (measurement tooling).

Reads the CSV files that ``rocprofv3 --kernel-trace --stats --output-format
csv`` and ``rocprofv3 --pmc FETCH_SIZE`` / ``--pmc WRITE_SIZE`` write, and
prints a short text summary:

* per kernel: calls and average duration (kernel trace statistics);
* per kernel: HBM bytes per dispatch from FETCH_SIZE and WRITE_SIZE, each
  scaled by the factor that makes the same counter read exactly the size of
  a plain device-to-device copy of known size found in the same run;
* or, from a kernel trace alone (``--trace``), per (kernel, workgroup count):
  the dispatches after the first ``--skip`` ones, their average duration,
  and the duration of the first one.

Usage:
  python -m paper_2008_05823_amd.profile_summary --stats DIR/x_kernel_stats.csv
      --fetch DIR/y_counter_collection.csv --write DIR/z_counter_collection.csv
      --copy-bytes 2147483648 [--source-hash HASH]
  python -m paper_2008_05823_amd.profile_summary --trace DIR/x_kernel_trace.csv [--skip N]
"""
from __future__ import annotations

import argparse
import collections
import csv
import re


def short_name(name: str) -> str:
    m = re.search(r"saef::\(anonymous namespace\)::(\w+)(<[^>]*>)?", name)
    if m:
        return m.group(1) + (m.group(2) or "")
    return name.split("(")[0][:60]


def kernel_stats(path: str):
    rows = list(csv.DictReader(open(path)))
    return [(short_name(r["Name"]), int(r["Calls"]), float(r["AverageNs"]) / 1e3,
             float(r["Percentage"])) for r in rows]


def counter_per_kernel(path: str):
    """{kernel: [(grid_size, value_kib), ...]} of one counter."""
    out = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        out[short_name(r["Kernel_Name"])].append((int(r["Grid_Size"]), float(r["Counter_Value"])))
    return out


def copy_factor(per_kernel, copy_bytes: int, expect_kib: float) -> float:
    """Scale that turns the counter of the known-size copy into its true size."""
    vals = [v for g, v in per_kernel.get("__amd_rocclr_copyBuffer", []) if v > 0.25 * expect_kib]
    if not vals:
        raise SystemExit("no copy dispatch of the expected size in the counter file")
    return (copy_bytes / 1024.0) / (sum(vals) / len(vals)) if expect_kib else 1.0


def trace_table(path: str, skip: int) -> None:
    """Per (kernel, workgroup count): dispatches after the first `skip`, their
    average duration and the first dispatch's duration."""
    runs = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        wg = int(r["Grid_Size_X"]) // max(1, int(r["Workgroup_Size_X"]))
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        runs[(short_name(r["Kernel_Name"]), wg)].append(us)
    rows = []
    for (name, wg), v in runs.items():
        tail = v[skip:] or v
        rows.append((sum(tail) / len(tail), name, wg, len(tail), v[0]))
    print(f"  {'kernel':40s} {'workgroups':>10s} {'calls':>6s} {'avg_us':>10s} {'first_us':>10s}")
    for avg, name, wg, n, first in sorted(rows, reverse=True):
        if name.startswith("__amd") or name.startswith("void at::") or name.startswith("at::"):
            continue
        print(f"  {name:40s} {wg:10d} {n:6d} {avg:10.1f} {first:10.1f}")


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", default=None, help="kernel trace CSV (per launch shape table)")
    ap.add_argument("--skip", type=int, default=0, help="first dispatches of each shape left out")
    ap.add_argument("--stats")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-bytes", type=int,
                    help="bytes read (and written) by the reference device copy")
    ap.add_argument("--source-hash", default=None)
    args = ap.parse_args()
    if args.trace:
        trace_table(args.trace, args.skip)
        return 0
    if not (args.stats and args.fetch and args.write and args.copy_bytes):
        ap.error("--stats, --fetch, --write and --copy-bytes are required without --trace")

    print("kernel durations (rocprofv3 --kernel-trace --stats)")
    print(f"  {'kernel':44s} {'calls':>6s} {'avg_us':>10s} {'pct':>7s}")
    for name, calls, avg_us, pct in kernel_stats(args.stats):
        print(f"  {name:44s} {calls:6d} {avg_us:10.1f} {pct:7.2f}")

    fetch = counter_per_kernel(args.fetch)
    write = counter_per_kernel(args.write)
    ff = copy_factor(fetch, args.copy_bytes, args.copy_bytes / 1024.0)
    wf = copy_factor(write, args.copy_bytes, args.copy_bytes / 1024.0)
    print()
    print(f"HBM bytes per dispatch (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE; KiB scaled by the "
          f"copy calibration: fetch x{ff:.4f}, write x{wf:.4f}, from a {args.copy_bytes}-byte "
          f"device-to-device copy in the same run)")
    print(f"  {'kernel':44s} {'n':>4s} {'read_MB':>10s} {'write_MB':>10s} {'total_MB':>10s}")
    for name in fetch:
        if name.startswith("__amd") or name.startswith("void at::") or name.startswith("at::"):
            continue
        fv = [v for _, v in fetch[name]]
        wv = [v for _, v in write.get(name, [])]
        r = sum(fv) / len(fv) * 1024 * ff / 1e6
        w = (sum(wv) / len(wv) * 1024 * wf / 1e6) if wv else float("nan")
        print(f"  {name:44s} {len(fv):4d} {r:10.1f} {w:10.1f} {r + w:10.1f}")
    if args.source_hash:
        print()
        print(f"kernel_source_sha256_16: {args.source_hash}")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
