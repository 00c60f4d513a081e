#!/usr/bin/env python3
"""Throughput of checkpointed BPTT on one MI355X.

A step is one whole forward + reverse pass (ambptt_run) over the 1000-step
LSTM workload (hidden 512, input 256, batch 64, fp32) with 10 HBM checkpoint
slots and a pinned host tier, under the asynchronous two-level schedule whose
interval comes from measured T_A and T_T.  Inputs are seeded, synthetic and
resident in HBM before the timed region starts.  By default the library runs
the pass as one resident kernel launch (weights held in registers for the
whole pass); --path steps selects one kernel launch per step.

Prints one JSON line: timesteps/s over the timed steps, the recompute factor,
the same pass under plain Revolve at the same 10 slots, the other execution
path on the same schedule, the roofline of the dominant kernel (HIP-event
durations on the compute stream) and the CPU oracle's rate on a bounded
sample.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--path auto|steps|resident]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "BPTT timesteps/sec at fixed HBM slot budget; recompute factor; MFMA % of peak"
WORKLOAD = "lstm_h512_t1000"
FP32_MFMA_PEAK_TFLOPS = 157.3


def step_flops(spec, window: int) -> dict:
    """Algorithmic flops of one launch of each per-step kernel, and of the
    three products of one step (gate GEMM, h-adjoint, weight gradient)."""
    B, D, H, G = spec.batch, spec.input, spec.hidden, spec.gates
    gate = 2.0 * B * G * H * (D + H)            # z = [x|h] W^T
    hbar = 2.0 * B * H * G * H                  # hbar = zbar W_h
    dw1 = 2.0 * G * H * (D + H + 1) * B         # dW (+ db) of one step
    return {"fwd": gate, "adj": gate + hbar, "dw": dw1 * window, "gate": gate, "hbar": hbar, "dw1": dw1}


def measured_traffic(kernel: str):
    """HBM bytes per launch of a kernel from the committed FETCH_SIZE /
    WRITE_SIZE counter runs (each scaled by a plain copy of known size), or
    None if the kernel's source has changed since those counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "lstm_h512_t1000_pmc.json")
    try:
        rec = json.load(open(path))["kernels"][kernel]
        src = open(os.path.join(ROOT, rec["source"]), "rb").read()
    except (OSError, ValueError, KeyError):
        return None
    if hashlib.sha256(src).hexdigest() != rec["sha256"]:
        return None
    return round(rec["fetch_bytes"] + rec["write_bytes"])


def cpu_baseline(wl, budget_s: float = 12.0) -> dict:
    import numpy as np
    import synth
    from oracle import bptt
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    W, b = synth.params(wl)
    cell = bptt.cell_for(wl, (W.astype(np.float64), b.astype(np.float64)))
    x0 = synth.initial_state(wl)
    st = (x0["h"].astype(np.float64), x0["c"].astype(np.float64))

    def one(n):
        w = wl.with_(n_steps=n)
        xs = synth.x_slice(w, 0, n).astype(np.float64)
        t = time.perf_counter()
        bptt.store_all(cell, n, lambda i: xs[i], st)
        return time.perf_counter() - t

    probe = 16
    dt = one(probe)
    n = int(max(probe, min(wl.n_steps, budget_s * probe / max(dt, 1e-6))))
    dt = one(n)
    return {"value": n / dt, "unit": "timesteps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"float64 store-all BPTT (numpy) over the first {n} of {wl.n_steps} steps "
                      f"at the full shapes, {dt:.1f} s"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--timing-sample", type=int, default=8)
    ap.add_argument("--path", choices=["auto", "steps", "resident"], default="auto")
    ap.add_argument("--cooperative", type=int, default=0)
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(--gpus must be 1)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_1806_01117_amd as amb
    import synth

    wl = synth.get(WORKLOAD)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    x = synth.x_slice(wl, 0, wl.n_steps)
    W, b = synth.params(wl)
    x0 = synth.initial_state(wl)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    dx, dW, db, dh, dc = t(x), t(W), t(b), t(x0["h"]), t(x0["c"])

    # a plain copy of known size (256 MiB read + 256 MiB written): the reference
    # that scales the FETCH_SIZE / WRITE_SIZE counters of a profiling run
    ref_src = torch.ones(64 << 20, device=dev)
    ref_dst = torch.empty_like(ref_src)
    ref_dst.copy_(ref_src)
    torch.cuda.synchronize()
    del ref_src, ref_dst

    spec = amb.ProblemSpec.from_workload(wl)
    r = amb.Runner(spec, device=dev)
    if args.path != "auto":
        r.set("path", 1 if args.path == "steps" else 2)
    r.set("resident_cooperative", args.cooperative)
    I_min, t_a, t_t = r.calibrate(dx, dW, db, dh, dc)
    r.set("timing_sample", args.timing_sample)
    for _ in range(args.warmup):
        r.run(dx, dW, db, dh, dc)
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        out = r.run(dx, dW, db, dh, dc)
        stats.append(out["stats"])
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    value = wl.n_steps * args.steps / el
    st = stats[-1]
    resident = st["path"] == 1

    def other_run(runner, reps):
        runner.run(dx, dW, db, dh, dc)
        torch.cuda.synchronize()
        tr = time.perf_counter()
        for _ in range(reps):
            o = runner.run(dx, dW, db, dh, dc)
        torch.cuda.synchronize()
        return wl.n_steps * reps / (time.perf_counter() - tr), o["stats"]

    reps = max(1, min(3, args.steps))
    # plain Revolve at the same HBM slot budget (no host tier), same path
    rv = amb.Runner(amb.ProblemSpec.from_workload(wl, slow_slots=0), device=dev)
    rv.set("path", 2 if resident else 1)
    rv.set("resident_cooperative", args.cooperative)
    rv_value, rv_st = other_run(rv, reps)
    rv.close()
    # the same schedule with one kernel launch per step (the other execution path)
    alt = None
    if resident:
        ps = amb.Runner(amb.ProblemSpec.from_workload(wl, interval_min=max(1, st["interval"])), device=dev)
        ps.set("path", 1)
        ps_value, ps_st = other_run(ps, reps)
        ps.close()
        alt = {"value": round(ps_value, 2), "unit": "timesteps/s", "interval": ps_st["interval"],
               "recompute_factor": round(ps_st["recompute_factor"], 4)}

    # roofline of the dominant kernel (largest device time in one pass)
    from paper_1806_01117_amd._lib import KERNEL_CLASSES
    fl = step_flops(spec, st["window"])
    kern = {}
    for i, name in enumerate(KERNEL_CLASSES):
        us = [s_["kernel_us"][i] for s_ in stats if s_["kernel_samples"][i] > 0]
        if us:
            kern[name] = (float(np.mean(us)), st["kernel_calls"][i])
    tot = {k: us * cnt for k, (us, cnt) in kern.items()}
    if resident:
        dom = "pass"
        fwd_ops = st["forward_evals"] - 1          # the first turn's forward step runs inside an adjoint
        flops = {"pass": fwd_ops * fl["gate"] + st["adjoints"] * (fl["gate"] + fl["hbar"] + fl["dw1"])}
        names = {"pass": "resident_pass: whole forward + reverse pass in one launch"}
        traffic = measured_traffic("resident_pass")
    else:
        flops = {"fwd": fl["fwd"], "adj": fl["adj"], "dw": fl["dw"]}
        cand = [k for k in tot if k in flops]
        dom = max(cand, key=tot.get) if cand else "adj"
        names = {"fwd": "step_small forward: gate GEMM + LSTM update",
                 "adj": "step_small adjoint: gate recompute + h-adjoint GEMM",
                 "dw": "dw_lds_f32 weight-gradient window"}
        traffic = measured_traffic({"fwd": "step_small_fwd", "adj": "step_small_adj"}.get(dom, dom))
    dom_us = kern[dom][0] if dom in kern else 0.0
    achieved = flops[dom] / (dom_us * 1e-6) / 1e12 if dom_us > 0 else 0.0
    r.close()

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "timesteps/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(1000 * el / args.steps, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded normal inputs, uniform weights)",
        "config": {"workload": WORKLOAD, "cell": "lstm", "batch": wl.batch, "input": wl.input,
                   "hidden": wl.hidden, "n_steps": wl.n_steps, "fast_slots": wl.fast_slots,
                   "slow_slots": spec.slow_slots, "mode": "async" if st["mode"] else "revolve",
                   "interval": st["interval"], "interval_min": I_min, "t_a_us": round(t_a, 3),
                   "t_t_us": round(t_t, 3), "window": st["window"]},
        "recompute_factor": round(st["recompute_factor"], 4),
        "plain_revolve": {"value": round(rv_value, 2), "unit": "timesteps/s",
                          "recompute_factor": round(rv_st["recompute_factor"], 4)},
        "path": "resident" if resident else "steps",
        "per_step_launches": alt,
        "kernel_us": {k: round(v[0], 3) for k, v in kern.items()},
        "kernel_calls_per_pass": {k: int(v[1]) for k, v in kern.items()},
        "device_ms_per_pass": round(sum(tot.values()) / 1000.0, 3),
        "host_enqueue_ms_per_pass": round(st["enqueue_us"] / 1000.0, 3),
        "host_run_ms_per_pass": round(st["run_us"] / 1000.0, 3),
        "host_link": {"bytes_d2h": st["bytes_d2h"], "bytes_h2d": st["bytes_h2d"],
                      "stores": st["stores"], "prefetches": st["prefetches"],
                      "prefetches_elided": st["prefetches_elided"], "compute_waits": st["compute_waits"]},
        "roofline": {"bound": "mfma", "kernel": names[dom], "achieved": round(achieved, 3),
                     "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / FP32_MFMA_PEAK_TFLOPS, 4), "traffic": traffic,
                     "avg_launch_us": round(dom_us, 3), "flops_per_launch": flops[dom]},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(line), flush=True)
    # release device memory before interpreter teardown
    del dx, dW, db, dh, dc, r, rv
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return 0


if __name__ == "__main__":
    sys.exit(main())
