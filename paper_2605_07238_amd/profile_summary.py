"""Summarise rocprofv3 outputs of a benchmark run into short text reports.

Used to produce the reports committed under profiles/: per-kernel dispatch
statistics from a kernel-trace database, and per-dispatch counter averages
from --pmc CSV files (FETCH_SIZE / WRITE_SIZE scaled by a plain copy of known
size in the same run).
"""

from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import os
import re
import sqlite3
import sys


def kernel_stats(db_path: str):
    con = sqlite3.connect(db_path)
    rows = con.execute("select name, count(*), avg(end - start), min(end - start), max(end - start), "
                       "sum(end - start) from kernels group by name order by sum(end - start) desc").fetchall()
    return [(r[0], r[1], r[2] / 1e3, r[3] / 1e3, r[4] / 1e3, r[5] / 1e3) for r in rows]


def counters(csv_path: str):
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    grid = {}
    for r in csv.DictReader(open(csv_path)):
        key = (r["Kernel_Name"], r["Dispatch_Id"])
        vals[r["Kernel_Name"]][r["Counter_Name"]].append(float(r["Counter_Value"]))
        grid[key] = int(r["Grid_Size"])
    return vals


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace-db")
    ap.add_argument("--pmc", nargs="*", default=[])
    ap.add_argument("--kernel", default="k_rows|k_score",
                    help="regular expression naming the kernel whose counters are summarised")
    ap.add_argument("--copy-bytes", type=int, default=512 << 20)
    ap.add_argument("--kernel-source", nargs="*",
                    help="source files whose joint SHA-256 identifies the profiled kernel and its launch geometry")
    ap.add_argument("--cus", type=int, default=256)
    ap.add_argument("--xcds", type=int, default=8)
    args = ap.parse_args()
    out = []
    if args.trace_db:
        out.append("kernel trace (durations in us)")
        out.append("%-70s %7s %10s %10s %10s %12s" % ("kernel", "calls", "avg", "min", "max", "total"))
        for name, n, avg, mn, mx, tot in kernel_stats(args.trace_db):
            out.append("%-70s %7d %10.2f %10.2f %10.2f %12.1f" % (name[:70], n, avg, mn, mx, tot))
    fetch = write = None
    copy_fetch = copy_write = None
    kavg = {}
    for path in args.pmc:
        for kname, cs in counters(path).items():
            for cname, v in cs.items():
                if re.search(args.kernel, kname):
                    avg = sum(v) / len(v)
                    kavg[cname] = avg
                    out.append("counter %-20s %-60s avg over %d dispatches: %.1f" % (cname, kname[:60], len(v), avg))
                    if cname == "FETCH_SIZE":
                        fetch = avg
                    if cname == "WRITE_SIZE":
                        write = avg
                elif "copyBuffer" in kname and cname in ("FETCH_SIZE", "WRITE_SIZE"):
                    m = max(v)  # the calibration copy is the largest copy of the run
                    if cname == "FETCH_SIZE":
                        copy_fetch = m
                    else:
                        copy_write = m
    if fetch is not None and write is not None and copy_fetch and copy_write:
        kib = args.copy_bytes / 1024.0
        fs, ws = kib / copy_fetch, kib / copy_write
        hbm = (fetch * fs + write * ws) * 1024.0
        out.append("copy calibration: %d bytes copied read back as FETCH_SIZE %.1f KiB, WRITE_SIZE %.1f KiB"
                   % (args.copy_bytes, copy_fetch, copy_write))
        out.append("fetch_scale: %.4f" % fs)
        out.append("write_scale: %.4f" % ws)
        out.append("fetch_kib_per_dispatch: %.1f" % fetch)
        out.append("write_kib_per_dispatch: %.1f" % write)
        out.append("hbm_bytes_per_launch: %.0f" % hbm)
    if "SQ_INSTS_VALU" in kavg and "GRBM_GUI_ACTIVE" in kavg:
        # GRBM_GUI_ACTIVE is summed over the XCDs; a wave64 VALU instruction
        # occupies a 16-lane SIMD for 4 cycles
        cycles = kavg["GRBM_GUI_ACTIVE"] / args.xcds
        busy = kavg["SQ_INSTS_VALU"] * 4.0 / (args.cus * 4 * cycles)
        out.append("gpu_cycles_per_dispatch: %.0f" % cycles)
        out.append("valu_issue_busy_frac: %.3f  (SQ_INSTS_VALU x 4 / (%d CUs x 4 SIMDs x cycles))" % (busy, args.cus))
    if "GRBM_GUI_ACTIVE" in kavg:
        # memory-pipeline readings (present when those counters were taken)
        cycles = kavg["GRBM_GUI_ACTIVE"] / args.xcds
        if "TCC_HIT_sum" in kavg and "TCC_MISS_sum" in kavg:
            h, m = kavg["TCC_HIT_sum"], kavg["TCC_MISS_sum"]
            out.append("l2_hit_frac: %.3f  (TCC_HIT / (TCC_HIT + TCC_MISS))" % (h / max(1.0, h + m)))
        if "TCP_TCC_READ_REQ_LATENCY_sum" in kavg and "TCP_TCC_READ_REQ_sum" in kavg:
            lat, req = kavg["TCP_TCC_READ_REQ_LATENCY_sum"], kavg["TCP_TCC_READ_REQ_sum"]
            out.append("l1_to_l2_read_latency_cycles: %.0f  (TCP_TCC_READ_REQ_LATENCY / TCP_TCC_READ_REQ)"
                       % (lat / max(1.0, req)))
            out.append("l2_reads_in_flight_per_cu: %.1f  (TCP_TCC_READ_REQ_LATENCY / (CUs x cycles))"
                       % (lat / (args.cus * cycles)))
        if "TCP_PENDING_STALL_CYCLES_sum" in kavg:
            out.append("l1_pending_stall_frac: %.3f  (TCP_PENDING_STALL_CYCLES / (CUs x cycles))"
                       % (kavg["TCP_PENDING_STALL_CYCLES_sum"] / (args.cus * cycles)))
        if "TA_BUSY_avr" in kavg:
            out.append("ta_busy_frac: %.3f  (TA_BUSY_avr / cycles)" % (kavg["TA_BUSY_avr"] / cycles))
        if "SQ_WAIT_ANY" in kavg and "SQ_WAVE_CYCLES" in kavg:
            out.append("wave_wait_frac: %.3f  (SQ_WAIT_ANY / SQ_WAVE_CYCLES)" % (kavg["SQ_WAIT_ANY"] / kavg["SQ_WAVE_CYCLES"]))
    if args.kernel_source:
        h = hashlib.sha256()
        for path in args.kernel_source:
            h.update(open(path, "rb").read())
        out.append("kernel_source_sha256: %s" % h.hexdigest())
    print("\n".join(out))


if __name__ == "__main__":
    sys.exit(main())
