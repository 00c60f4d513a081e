"""Host-tier stores and their overlap with compute, from a rocprofv3 kernel trace.

Device-to-host copies into pinned memory run as the HIP runtime's shader copy
kernel (`__amd_rocclr_copyBuffer`), so a plain `--kernel-trace` holds every
store of the host tier with its start and end.  This script takes the last
`--stores` such copies longer than `--min-us` (the stores of the timed pass)
on the queue that carries most long copies (the library's copy stream; the
compute queue also carries input uploads and gradient read-backs) and
reports their median rate for `--state-bytes` per state, the share of
their time during which one of the library's kernels runs, and how busy the
compute stream is between the first and the last of them.

    rocprofv3 --kernel-trace --stats -f csv -d OUT -o kt -- python -u bench.py ...
    python -m paper_1806_01117_amd.trace_overlap OUT/kt_kernel_trace.csv --stores 3333 --state-bytes 16777216
"""
from __future__ import annotations

import argparse
import bisect
import csv
import json
import statistics


def _merge(intervals):
    out = []
    for s, e in sorted(intervals):
        if out and s <= out[-1][1]:
            out[-1][1] = max(out[-1][1], e)
        else:
            out.append([s, e])
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("trace", help="kt_kernel_trace.csv of a rocprofv3 --kernel-trace run")
    ap.add_argument("--stores", type=int, required=True, help="stores of the timed pass (the last ones in the trace)")
    ap.add_argument("--state-bytes", type=int, required=True, help="bytes of one stored state")
    ap.add_argument("--min-us", type=float, default=100.0, help="shorter copies are not host-tier stores")
    args = ap.parse_args()
    copies, comp = [], []
    with open(args.trace) as f:
        for r in csv.DictReader(f):
            s, e = int(r["Start_Timestamp"]), int(r["End_Timestamp"])
            if "copyBuffer" in r["Kernel_Name"]:
                if e - s > args.min_us * 1e3:
                    copies.append((s, e, r["Queue_Id"]))
            elif "ambptt" in r["Kernel_Name"]:
                comp.append((s, e))
    queues = {}
    for c in copies:
        queues[c[2]] = queues.get(c[2], 0) + 1
    q = max(queues, key=queues.get)
    stores = sorted((s, e) for s, e, qq in copies if qq == q)[-args.stores:]
    if len(stores) < args.stores:
        raise SystemExit(f"only {len(stores)} copies longer than {args.min_us} us in the trace")
    merged = _merge(comp)
    starts = [m[0] for m in merged]

    def covered(s, e):
        i, tot = max(0, bisect.bisect_right(starts, s) - 1), 0
        while i < len(merged) and merged[i][0] < e:
            tot += max(0, min(e, merged[i][1]) - max(s, merged[i][0]))
            i += 1
        return tot

    t0, t1 = stores[0][0], stores[-1][1]
    busy = sum(min(e, t1) - max(s, t0) for s, e in merged if e > t0 and s < t1)
    gaps = sorted(merged[i + 1][0] - merged[i][1] for i in range(len(merged) - 1)
                  if merged[i][1] >= t0 and merged[i + 1][0] <= t1)
    med = statistics.median(e - s for s, e in stores)
    print(json.dumps({
        "stores": len(stores),
        "median_store_us": round(med / 1e3, 2),
        "store_GBps": round(args.state_bytes / med, 2),
        "store_time_overlapped_by_compute": round(sum(covered(s, e) for s, e in stores) / sum(e - s for s, e in stores), 5),
        "span_s": round((t1 - t0) / 1e9, 3),
        "compute_busy_in_span": round(busy / (t1 - t0), 4),
        "compute_gaps": len(gaps),
        "median_gap_us": round(statistics.median(gaps) / 1e3, 2) if gaps else None,
        "p99_gap_us": round(gaps[int(0.99 * (len(gaps) - 1))] / 1e3, 2) if gaps else None,
    }))
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
