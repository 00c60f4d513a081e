"""Host-link throughput and compute/transfer overlap from a rocprofv3 run
with --kernel-trace --memory-copy-trace (CSV output).

Considers the host-to-device and device-to-host copies of exactly
--state-bytes (one checkpointed state).  For each direction: the number of
copies, the bytes, the busy time (union of the copies' intervals) and the
achieved GB/s over it.  Overlap is the fraction of the copies' busy time
(both directions together) during which at least one kernel was executing:
1.0 means no transfer ran on an idle device.

    python -m paper_1806_01117_amd.copy_overlap --dir gpurun_out/prof/c3copy --state-bytes 1572864
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os


def _csv(d: str, suffix: str) -> list[dict]:
    files = glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True)
    if not files:
        raise SystemExit(f"no *{suffix} under {d}")
    rows = []
    for f in files:
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    return rows


def _union(iv: list[tuple[int, int]]) -> list[tuple[int, int]]:
    out: list[tuple[int, int]] = []
    for a, b in sorted(iv):
        if out and a <= out[-1][1]:
            out[-1] = (out[-1][0], max(out[-1][1], b))
        else:
            out.append((a, b))
    return out


def _length(iv: list[tuple[int, int]]) -> int:
    return sum(b - a for a, b in iv)


def _intersect(x: list[tuple[int, int]], y: list[tuple[int, int]]) -> int:
    i = j = tot = 0
    while i < len(x) and j < len(y):
        a, b = max(x[i][0], y[j][0]), min(x[i][1], y[j][1])
        if a < b:
            tot += b - a
        if x[i][1] < y[j][1]:
            i += 1
        else:
            j += 1
    return tot


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--dir", required=True, help="rocprofv3 output directory")
    ap.add_argument("--state-bytes", type=int, required=True)
    args = ap.parse_args()
    kern = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in _csv(args.dir, "kernel_trace.csv")
            if "rocclr" not in r["Kernel_Name"]]
    copies = _csv(args.dir, "memory_copy_trace.csv")
    busy_k = _union(kern)
    out = {"state_bytes": args.state_bytes}
    all_iv = []
    for direction in ("HOST_TO_DEVICE", "DEVICE_TO_HOST"):
        iv = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in copies
              if direction in r.get("Direction", "") and int(r.get("Size", 0)) == args.state_bytes]
        all_iv += iv
        u = _union(iv)
        t = _length(u)
        n = len(iv)
        out[direction.lower()] = {"copies": n, "bytes": n * args.state_bytes, "busy_us": round(t / 1e3, 1),
                                  "gb_per_s": round(n * args.state_bytes / t, 2) if t else None,
                                  "mean_copy_us": round(sum(b - a for a, b in iv) / n / 1e3, 2) if n else None}
    u = _union(all_iv)
    t = _length(u)
    out["copy_busy_us"] = round(t / 1e3, 1)
    out["overlap"] = round(_intersect(u, busy_k) / t, 4) if t else None
    out["kernel_busy_us"] = round(_length(busy_k) / 1e3, 1)
    print(json.dumps(out, indent=1))
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
