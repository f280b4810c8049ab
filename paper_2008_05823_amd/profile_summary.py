"""Summaries of rocprofv3 output for the SAEF kernels (measurement tooling).

Reads the CSV files that ``rocprofv3 --kernel-trace --stats --output-format
csv`` and ``rocprofv3 --pmc FETCH_SIZE`` / ``--pmc WRITE_SIZE`` write, and
prints a short text summary:

* per kernel: calls and average duration (kernel trace statistics);
* per kernel: HBM bytes per dispatch from FETCH_SIZE and WRITE_SIZE, each
  scaled by the factor that makes the same counter read exactly the bytes of
  the library's stream probe found in the same run (k_stream_probe<true>: reads
  8 N and writes 4 N bytes for N elements per launch);
* or, from a kernel trace alone (``--trace``), per (kernel, workgroup count):
  the dispatches after the first ``--skip`` ones, their average duration,
  and the duration of the first one.

Usage:
  python -m paper_2008_05823_amd.profile_summary --stats DIR/x_kernel_stats.csv
      --fetch DIR/y_counter_collection.csv --write DIR/z_counter_collection.csv
      --probe-elems N [--kernel NAME --algorithmic BYTES --counters-out FILE]
  python -m paper_2008_05823_amd.profile_summary --trace DIR/x_kernel_trace.csv [--skip N]
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
# the sources the sign-path kernels are built from (the counters in a
# summary apply to this hash only)
KERNEL_SOURCES = [os.path.join(HERE, "csrc", f)
                  for f in ("saef_kernels.hip", "saef_internal.h", "saef_device.h")]

_COMMENT = re.compile(r"//[^\n]*|/\*.*?\*/", re.S)


def code_tokens(text: str) -> str:
    """The source without its comments, whitespace runs collapsed: what the
    compiler sees, so that editing a comment keeps the hash.  (No string
    literal in these sources holds a comment opener.)"""
    return " ".join(_COMMENT.sub(" ", text).split())


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, encoding="utf-8") as fh:
            h.update(code_tokens(fh.read()).encode())
            h.update(b"\0")
    return h.hexdigest()[:16]


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


def counters_by_name(path: str):
    """{kernel: {counter: average over the kernel's dispatches}} of a
    counter-collection CSV that may hold several counters per dispatch."""
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in csv.DictReader(open(path)):
        vals[short_name(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
    return {k: {c: (sum(v) / len(v), len(v)) for c, v in cs.items()} for k, cs in vals.items()}


# Bytes of an L2-to-memory request by its counted size (gfx950 TCC counters).
READ_REQS = (("TCC_EA0_RDREQ_128B_sum", 128), ("TCC_EA0_RDREQ_64B_sum", 64),
             ("TCC_EA0_RDREQ_32B_sum", 32))


def request_bytes(reads, writes, name: str):
    """(read bytes, write bytes, dispatches) per dispatch of `name` from the
    request counts: reads 128/64/32-byte requests, writes 64-byte requests
    and the remaining (32-byte) ones.  No calibration is involved."""
    rc = reads.get(name, {})
    if not all(c in rc for c, _ in READ_REQS):
        return None
    rb = sum(rc[c][0] * size for c, size in READ_REQS)
    wc = writes.get(name, {})
    wb = float("nan")
    if "TCC_EA0_WRREQ_sum" in wc and "TCC_EA0_WRREQ_64B_sum" in wc:
        w64 = wc["TCC_EA0_WRREQ_64B_sum"][0]
        wb = w64 * 64 + (wc["TCC_EA0_WRREQ_sum"][0] - w64) * 32
    return rb, wb, rc[READ_REQS[0][0]][1]


# the 2-read/1-write stream probe (c = a + b) the counters are calibrated on
PROBE_KERNEL = "k_stream_probe<true>"


def probe_factor(per_kernel, true_kib: float) -> float:
    """Scale that turns the counter of the stream probe into its true size."""
    vals = [v for _, v in per_kernel.get(PROBE_KERNEL, []) if v > 0]
    if not vals:
        raise SystemExit("no stream-probe dispatch in the counter file")
    return true_kib / (sum(vals) / len(vals))


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


def timeline(path: str, marker: str, index: int) -> None:
    """The dispatches between the index-th and the next dispatch whose kernel
    name starts with `marker` (one iteration), in start order: queue (HIP
    stream), workgroups, start and end in microseconds from the first."""
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Start_Timestamp"]))
    marks = [i for i, r in enumerate(rows) if short_name(r["Kernel_Name"]).startswith(marker)]
    if len(marks) < index + 2:
        raise SystemExit(f"fewer than {index + 2} dispatches of {marker!r}")
    i0, i1 = marks[index], marks[index + 1]
    t0 = int(rows[i0]["Start_Timestamp"])
    print(f"  {'kernel':36s} {'queue':>5s} {'workgroups':>10s} {'start_us':>9s} {'end_us':>9s} "
          f"{'dur_us':>8s}")
    for r in rows[i0:i1 + 1]:
        s, e = int(r["Start_Timestamp"]) - t0, int(r["End_Timestamp"]) - t0
        wg = int(r["Grid_Size_X"]) // max(1, int(r["Workgroup_Size_X"]))
        print(f"  {short_name(r['Kernel_Name']):36s} {r['Queue_Id']:>5s} {wg:10d} {s / 1e3:9.1f} "
              f"{e / 1e3:9.1f} {(e - s) / 1e3:8.1f}")


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", default=None, help="kernel trace CSV (per launch shape table)")
    ap.add_argument("--skip", type=int, default=0, help="first dispatches of each shape left out")
    ap.add_argument("--timeline", default=None, metavar="MARKER:INDEX",
                    help="with --trace: the dispatches of one iteration, from the INDEX-th "
                         "dispatch of a kernel whose name starts with MARKER to the next")
    ap.add_argument("--stats")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--probe-elems", type=int,
                    help="elements per stream-probe launch (reads 8 N, writes 4 N bytes)")
    ap.add_argument("--kernel", default=None, help="kernel whose bytes go to --counters-out")
    ap.add_argument("--algorithmic", type=float, default=None,
                    help="algorithmic bytes per launch of --kernel")
    ap.add_argument("--counters-out", default=None,
                    help="write the kernel's HBM bytes per launch and the source hash here")
    ap.add_argument("--header", default=None,
                    help="comment lines (a file) put at the top of --counters-out")
    ap.add_argument("--read-reqs", default=None,
                    help="counter CSV of TCC_EA0_RDREQ_128B_sum, _64B_sum and _32B_sum")
    ap.add_argument("--write-reqs", default=None,
                    help="counter CSV of TCC_EA0_WRREQ_sum and TCC_EA0_WRREQ_64B_sum")
    ap.add_argument("--algo", action="append", default=[], metavar="KERNEL=BYTES",
                    help="algorithmic bytes per launch of a kernel, for the ratio column")
    args = ap.parse_args()
    if args.trace:
        if args.timeline:
            marker, _, index = args.timeline.rpartition(":")
            timeline(args.trace, marker, int(index))
        else:
            trace_table(args.trace, args.skip)
        return 0
    if not (args.stats and args.fetch and args.write and args.probe_elems):
        ap.error("--stats, --fetch, --write and --probe-elems are required without --trace")

    stats = kernel_stats(args.stats)
    print("kernel durations (rocprofv3 --kernel-trace --stats)")
    print(f"  {'kernel':44s} {'calls':>6s} {'avg_us':>10s} {'pct':>7s}")
    for name, calls, avg_us, pct in stats:
        print(f"  {name:44s} {calls:6d} {avg_us:10.1f} {pct:7.2f}")

    fetch = counter_per_kernel(args.fetch)
    write = counter_per_kernel(args.write)
    n = args.probe_elems
    ff = probe_factor(fetch, 8 * n / 1024.0)
    wf = probe_factor(write, 4 * n / 1024.0)
    print()
    print(f"HBM bytes per dispatch (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE; KiB scaled so that "
          f"the stream probe of the same run reads {8 * n} and writes {4 * n} bytes: fetch "
          f"x{ff:.4f}, write x{wf:.4f})")
    print(f"  {'kernel':44s} {'n':>4s} {'read_MB':>10s} {'write_MB':>10s} {'total_MB':>10s}")
    per = {}
    for name in fetch:
        if name.startswith("__amd") or name.startswith("void at::") or name.startswith("at::"):
            continue
        fv = [v for _, v in fetch[name]]
        wv = [v for _, v in write.get(name, [])]
        r = sum(fv) / len(fv) * 1024 * ff / 1e6
        w = (sum(wv) / len(wv) * 1024 * wf / 1e6) if wv else float("nan")
        per[name] = (r, w, len(fv))
        print(f"  {name:44s} {len(fv):4d} {r:10.1f} {w:10.1f} {r + w:10.1f}")
    algo = {}
    for item in args.algo:
        name, _, val = item.rpartition("=")
        algo[name] = float(val)
    if args.read_reqs:
        reads = counters_by_name(args.read_reqs)
        writes = counters_by_name(args.write_reqs) if args.write_reqs else {}
        print()
        print("HBM bytes per dispatch from request counts (rocprofv3 --pmc TCC_EA0_RDREQ_128B_sum "
              "TCC_EA0_RDREQ_64B_sum TCC_EA0_RDREQ_32B_sum, then TCC_EA0_WRREQ_sum "
              "TCC_EA0_WRREQ_64B_sum; each request at its counted size, no calibration)")
        print(f"  {'kernel':44s} {'n':>4s} {'read_MB':>10s} {'write_MB':>10s} {'total_MB':>10s} "
              f"{'algo_MB':>10s} {'ratio':>7s}")
        for name in reads:
            if name.startswith("__amd") or name.startswith("void at::") or name.startswith("at::"):
                continue
            got = request_bytes(reads, writes, name)
            if got is None:
                continue
            rb, wb, cnt = got
            a_mb = algo.get(name, float("nan")) / 1e6
            ratio = (rb + wb) / 1e6 / a_mb if name in algo else float("nan")
            print(f"  {name:44s} {cnt:4d} {rb / 1e6:10.1f} {wb / 1e6:10.1f} "
                  f"{(rb + wb) / 1e6:10.1f} {a_mb:10.1f} {ratio:7.4f}")
    src = kernel_source_hash()
    print()
    print(f"kernel_source_sha256_16: {src}")
    if args.counters_out:
        if args.kernel not in per:
            raise SystemExit(f"kernel {args.kernel!r} not in the counter files")
        r, w, cnt = per[args.kernel]
        avg = {name: us for name, _, us, _ in stats}.get(args.kernel)
        with open(args.counters_out, "w") as f:
            if args.header:
                f.write(open(args.header).read())
            f.write(f"# {args.kernel}: FETCH_SIZE x {ff:.4f} + WRITE_SIZE x {wf:.4f} (stream-probe "
                    f"calibration), average of {cnt} dispatches: read {r:.1f} MB, write "
                    f"{w:.1f} MB\n")
            if args.algorithmic:
                f.write(f"# algorithmic bytes per launch {args.algorithmic:.0f}: traffic / "
                        f"algorithmic = {(r + w) * 1e6 / args.algorithmic:.4f}\n")
            if avg is not None:
                f.write(f"# rocprofv3 average duration: {avg:.1f} us\n")
            f.write(f"kernel: {args.kernel}\n")
            f.write(f"hbm_bytes_per_launch: {(r + w) * 1e6:.0f}\n")
            f.write(f"kernel_source_sha256_16: {src}\n")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
