"""HBM traffic per kernel launch from two rocprofv3 counter runs.

rocprofv3 reports FETCH_SIZE and WRITE_SIZE in KiB per dispatch.  Each counter
is scaled by what it reads for the 256 MiB copy that bench.py makes before
anything else (256 MiB read and 256 MiB written), so the figures are bytes
that reached HBM.  The result is merged into profiles/<workload>_pmc.json,
keyed by kernel, with the sha256 of the kernel's source so that bench.py can
drop the figure once the kernel changes.

    rocprofv3 --pmc FETCH_SIZE -f csv -d OUT/fetch -o pmc -- python -u bench.py ...
    rocprofv3 --pmc WRITE_SIZE -f csv -d OUT/write -o pmc -- python -u bench.py ...
    python -m paper_1806_01117_amd.pmc_summary --workload NAME --fetch OUT/fetch --write OUT/write \
        --kernel resident_pass=resident_pass:paper_1806_01117_amd/csrc/resident.hip
"""
from __future__ import annotations

import argparse
import csv
import glob
import gzip
import hashlib
import json
import os
import statistics

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
COPY_BYTES = 256 << 20


def _rows(d: str) -> list[dict]:
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True) + \
        glob.glob(os.path.join(d, "**", "*counter_collection.csv.gz"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    opener = gzip.open if files[0].endswith(".gz") else open
    with opener(files[0], "rt") as f:
        return sorted(csv.DictReader(f), key=lambda r: int(r["Dispatch_Id"]))


def _per_dispatch(rows: list[dict], counter: str) -> list[tuple[str, float]]:
    out = []
    for r in rows:
        if r["Counter_Name"] == counter:
            out.append((r["Kernel_Name"], float(r["Counter_Value"]) * 1024.0))
    return out


def _scale(disp: list[tuple[str, float]]) -> float:
    """bytes the reference copy moved divided by what the counter read for it:
    the first copy-named dispatch whose counter is within a factor 4 of 256 MiB"""
    for name, v in disp:
        if "copy" in name.lower() and COPY_BYTES / 4 <= v <= COPY_BYTES * 4:
            return COPY_BYTES / v
    raise SystemExit("the 256 MiB reference copy was not found in the counter run")


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", required=True)
    ap.add_argument("--fetch", required=True, help="rocprofv3 output directory of the FETCH_SIZE run")
    ap.add_argument("--write", required=True, help="rocprofv3 output directory of the WRITE_SIZE run")
    ap.add_argument("--kernel", action="append", required=True,
                    help="label=name-substring:source-file")
    ap.add_argument("--pick", choices=["median", "max"], default="median",
                    help="which of a kernel's dispatches to keep: the median, or the largest (one timed pass "
                         "among shorter calibration launches)")
    args = ap.parse_args()
    fetch = _per_dispatch(_rows(args.fetch), "FETCH_SIZE")
    write = _per_dispatch(_rows(args.write), "WRITE_SIZE")
    fs, ws = _scale(fetch), _scale(write)
    path = os.path.join(ROOT, "profiles", f"{args.workload}_pmc.json")
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        rec = {"kernels": {}}
    rec.update({"workload": args.workload, "fetch_scale": fs, "write_scale": ws,
                "note": "HBM bytes per launch: FETCH_SIZE and WRITE_SIZE (KiB per dispatch) scaled by the same "
                        "counters on a 256 MiB copy"})
    for spec in args.kernel:
        label, rest = spec.split("=", 1)
        sub, src = rest.split(":", 1)
        f = [v for n, v in fetch if sub in n]
        w = [v for n, v in write if sub in n]
        if not f or not w:
            raise SystemExit(f"kernel {sub} not found in the counter runs")
        digest = hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest()
        pick = statistics.median if args.pick == "median" else max
        rec["kernels"][label] = {"source": src, "sha256": digest, "dispatches": len(f), "pick": args.pick,
                                 "fetch_bytes": pick(f) * fs, "write_bytes": pick(w) * ws}
    with open(path, "w") as fo:
        json.dump(rec, fo, indent=1)
    print(json.dumps({k: round((v["fetch_bytes"] + v["write_bytes"]) / 1e6, 2) for k, v in rec["kernels"].items()}),
          "MB per launch")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
