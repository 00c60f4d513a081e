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

With --table (and --sq, a run of SQ_VALU_MFMA_BUSY_CYCLES,
SQ_INSTS_VALU_MFMA_MOPS_F32 and GRBM_GUI_ACTIVE) it writes nothing and prints,
per kernel instance and grid size whose name holds one of --match, the
median dispatch's duration, HBM bytes and MFMA utilisation, for kernels
launched at several shapes:

    python -m paper_1806_01117_amd.pmc_summary --table --fetch OUT/fetch --write OUT/write --sq OUT/sq \
        --match mlpv_gemm --match mlpv_dw
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
    the first copy-named dispatch whose counter is within a factor 4 of 256 MiB
    (bench.py makes the reference copy before any other copy)"""
    for name, v in disp:
        if "copy" in name.lower() and COPY_BYTES / 4 <= v <= COPY_BYTES * 4:
            return COPY_BYTES / v
    raise SystemExit("the 256 MiB reference copy was not found in the counter run")


def _instance(name: str) -> str:
    """the kernel's name with its template arguments, without the return type,
    the namespaces and the parameter list"""
    name = name.strip()
    end = len(name)
    if name.endswith(")"):  # the parameter list: the parenthesis that closes at the end
        depth = 0
        for i in range(len(name) - 1, -1, -1):
            depth += {")": 1, "(": -1}.get(name[i], 0)
            if depth == 0:
                end = i
                break
    head = name[:end]
    depth, cut = 0, 0
    for i, ch in enumerate(head):  # the last "::" outside template brackets
        depth += {"<": 1, ">": -1}.get(ch, 0)
        if depth == 0 and head.startswith("::", i):
            cut = i + 2
    return head[cut:]


def _table(args) -> int:
    groups: dict[tuple[str, str], dict[str, list]] = {}
    dur: dict[tuple[str, str], list] = {}
    counters = {"FETCH_SIZE": args.fetch, "WRITE_SIZE": args.write}
    for counter, d in counters.items():
        rows = _rows(d)
        scale = _scale(_per_dispatch(rows, counter))
        for r in rows:
            if r["Counter_Name"] == counter and any(m in r["Kernel_Name"] for m in args.match):
                key = (_instance(r["Kernel_Name"]), r["Grid_Size"])
                groups.setdefault(key, {}).setdefault(counter, []).append(float(r["Counter_Value"]) * 1024.0 * scale)
    sq: dict[tuple[str, str], dict[int, dict[str, float]]] = {}
    for r in _rows(args.sq):
        if any(m in r["Kernel_Name"] for m in args.match):
            key = (_instance(r["Kernel_Name"]), r["Grid_Size"])
            disp = sq.setdefault(key, {}).setdefault(int(r["Dispatch_Id"]), {})
            disp[r["Counter_Name"]] = disp.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
            dur.setdefault(key, {})[int(r["Dispatch_Id"])] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    print("| kernel | grid (threads) | dispatches | median us | HBM fetch MB | HBM write MB | MFMA busy | MOPS x 512 (MFLOP) |")
    print("|---|---|---|---|---|---|---|---|")
    for key in sorted(set(groups) | set(sq)):
        g = groups.get(key, {})
        fmb = statistics.median(g["FETCH_SIZE"]) / 1e6 if "FETCH_SIZE" in g else float("nan")
        wmb = statistics.median(g["WRITE_SIZE"]) / 1e6 if "WRITE_SIZE" in g else float("nan")
        line = f"| {key[0]} | {key[1]} | {len(sq.get(key, {}))} "
        if key in sq:
            d = sq[key]
            ids = sorted(d, key=lambda i: dur[key][i])
            mid = ids[len(ids) // 2]
            c = d[mid]
            act = c.get("GRBM_GUI_ACTIVE", 0.0) / 8  # per XCD
            busy = 100 * c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (act * 1024) if act else float("nan")
            line += f"| {dur[key][mid]:.1f} | {fmb:.2f} | {wmb:.2f} | {busy:.1f} % | {c.get('SQ_INSTS_VALU_MFMA_MOPS_F32', 0.0) * 512 / 1e6:.0f} |"
        else:
            line += f"| | {fmb:.2f} | {wmb:.2f} | | |"
        print(line)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--table", action="store_true", help="print per-instance medians instead of merging a record")
    ap.add_argument("--sq", help="rocprofv3 output directory of the SQ / GRBM counter run (--table)")
    ap.add_argument("--match", action="append", default=[], help="kernel-name substring (--table)")
    ap.add_argument("--workload")
    ap.add_argument("--fetch", required=True, help="rocprofv3 output directory of the FETCH_SIZE run")
    ap.add_argument("--write", required=True, help="rocprofv3 output directory of the WRITE_SIZE run")
    ap.add_argument("--kernel", action="append", default=[],
                    help="label=name-substring:source-file")
    ap.add_argument("--pick", choices=["median", "max"], default="median",
                    help="which of a kernel's dispatches to keep: the median, or the largest (one timed pass "
                         "among shorter calibration launches)")
    args = ap.parse_args()
    if args.table:
        if not args.sq or not args.match:
            raise SystemExit("--table needs --sq and at least one --match")
        return _table(args)
    if not args.workload or not args.kernel:
        raise SystemExit("--workload and at least one --kernel are required")
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
