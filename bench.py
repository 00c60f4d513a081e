#!/usr/bin/env python3
"""Throughput of checkpointed BPTT on one MI355X.

A step is one whole forward + reverse pass (ambptt_run) over a workload's n
recurrent steps.  The default workload is the largest one that fits one GPU:
the 20000-step LSTM (hidden 4096, input 1024, batch 512, fp32; 16 MiB of
state per step, 320 GB of states in all) with 64 HBM checkpoint slots and a
pinned host tier, under the asynchronous two-level schedule whose interval
comes from measured T_A and T_T.  Pinned host memory is limited per process,
so the host tier gets the slots that fit --pinned-gib (the schedule raises the
interval to ceil(n / (H + 1)) accordingly).  Inputs are seeded, synthetic and
resident in HBM before the timed region starts.

Passes are whole: a pass is never shortened.  When the requested warm-up and
timed passes would take longer than --max-timed-s (estimated from the
calibrated forward step), fewer passes run, and the line reports the numbers
actually run ("steps", "warmup") beside the requested ones.

Prints one JSON line: timesteps/s over the timed passes, the recompute factor,
the same pass under plain Revolve at the same HBM slots (gradients compared
element by element), store-all in HBM where its slots fit, the roofline of the
dominant kernel (HIP-event durations on the compute stream) and the CPU
oracle's rate on a bounded sample.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--path auto|steps|resident]
    python bench.py --workload lstm_h512_t1000 --sweep-n 100,1000,10000,100000
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
WORKLOAD = "lstm_h4096_t20000"
FP32_MFMA_PEAK_TFLOPS = 157.3
BF16_MFMA_PEAK_TFLOPS = 2500.0  # dense
HBM_PEAK_GBS = 8000.0


def step_costs(spec: str, n: int):
    """Relative step costs from "every:K:F" (step t costs F when t % K == 0, else 1); None for ""."""
    if not spec:
        return None
    kind, k, f = spec.split(":")
    if kind != "every" or int(k) < 1 or float(f) <= 0:
        raise SystemExit("--step-costs: expected every:K:F with K >= 1, F > 0")
    return [float(f) if t % int(k) == 0 else 1.0 for t in range(n)]


def weighted_cost(text: str, costs) -> float:
    """Cost of the forward evaluations of a canonical schedule text for the given step costs."""
    import numpy as np
    pre = np.concatenate([[0.0], np.cumsum(costs)])
    tot = costs[-1]  # the first turn's forward step
    for ln in text.splitlines()[1:]:
        p = ln.split()
        if p[0] == "A":
            tot += pre[int(p[2])] - pre[int(p[1])]
    return float(tot)


def copy_overlap(spec, st, stats, dev, wall_ms: float) -> dict:
    """Host-link rate of one state's copy (hipMemcpyAsync between HBM and
    pinned host memory, timed alone) and a lower bound on the overlap of the
    pass's copies with compute: the compute stream can be idle while a copy
    is pending for at most the wall time not covered by kernel execution, so
    overlap >= 1 - (wall - kernel time) / (copy count x copy time)."""
    import numpy as np
    import torch
    nbytes = (st["bytes_d2h"] // st["stores"]) if st["stores"] else (st["bytes_h2d"] // max(1, st["prefetches"]))
    d = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    h = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    rates = {}
    for name, (dst, src) in (("d2h", (h, d)), ("h2d", (d, h))):
        best = None
        for _ in range(6):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            dst.copy_(src, non_blocking=True)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            best = ms if best is None else min(best, ms)
        rates[name] = best
    del d, h
    release_pinned()
    n_st, n_pf = st["stores"], st["prefetches"] - st["prefetches_elided"]
    copy_ms = n_st * rates["d2h"] + n_pf * rates["h2d"]
    kernel_ms = float(np.mean([sum(s_["kernel_us"][i] * s_["kernel_calls"][i] for i in range(6)) for s_ in stats])) / 1e3
    idle_ms = max(0.0, wall_ms - kernel_ms)
    return {"state_bytes": nbytes, "d2h_us": round(1000 * rates["d2h"], 2), "h2d_us": round(1000 * rates["h2d"], 2),
            "d2h_gb_s": round(nbytes / rates["d2h"] / 1e6, 2), "h2d_gb_s": round(nbytes / rates["h2d"] / 1e6, 2),
            "copies": n_st + n_pf, "copy_ms_per_pass": round(copy_ms, 2),
            "kernel_ms_per_pass": round(kernel_ms, 2), "wall_ms_per_pass": round(wall_ms, 2),
            "overlap_lower_bound": round(1.0 - idle_ms / copy_ms, 4) if copy_ms > 0 else None}


def release_pinned() -> None:
    """Frees the pinned blocks torch's host allocator caches, so that no pinned
    memory is left for static destructors to release at process exit."""
    import torch
    torch.cuda.synchronize()
    fn = getattr(torch._C, "_host_emptyCache", None)
    if fn is not None:
        fn()


def mlp_layer_work(ws, B: int) -> tuple[dict, dict]:
    """Algorithmic flops and HBM bytes of one launch of each kernel class of
    the MLP of layers of different widths, averaged over its layers (fp32):
    forward y_{l+1} = relu(y_l W_l^T + b_l); adjoint z-bar_l from the
    recomputed z_l, the seed and u = z-bar_{l+1} W_{l+1}, formed in the same
    launch (no u for the last layer), with the copy of y_l kept for the
    weight gradient; the weight gradient of one layer."""
    n = len(ws) - 1
    f = {"fwd": 0.0, "adj": 0.0, "dw": 0.0}
    b = dict(f)
    for l in range(n):
        a, c = ws[l], ws[l + 1]
        f["fwd"] += 2.0 * B * a * c
        b["fwd"] += 4.0 * (c * a + c + B * a + B * c)             # W_l, b_l, y_l in; y_{l+1} out
        f["adj"] += 2.0 * B * a * c
        b["adj"] += 4.0 * (c * a + c + B * a + B * c + B * a)     # W_l, b_l, y_l in; z-bar_l and the copy of y_l out
        if l + 1 < n:
            d = ws[l + 2]
            f["adj"] += 2.0 * B * c * d
            b["adj"] += 4.0 * (B * d + d * c)                      # z-bar_{l+1}, W_{l+1} in
        f["dw"] += 2.0 * B * c * (a + 1)
        b["dw"] += 4.0 * (B * c + B * a + c * a + c)              # z-bar_l, y_l in; dW_l, db_l written once
    return {k: v / n for k, v in f.items()}, {k: v / n for k, v in b.items()}


_HASH_CHUNK = 64 << 20  # 4-byte elements per hashed chunk (256 MiB)


def _digest(t) -> tuple:
    """64-bit hashes of a tensor's bit patterns, one per 256 MiB chunk: the sum
    of each 32-bit word times a fixed odd multiplier of its position, mod 2^64.
    One differing element changes its chunk's hash with certainty (an odd
    multiplier times a nonzero difference is nonzero mod 2^64); several
    collide with probability about 2^-64."""
    import torch
    v = t.reshape(-1).view(torch.int32)
    g = torch.Generator(device=v.device)
    g.manual_seed(1806)
    m = torch.randint(-(2 ** 62), 2 ** 62, (min(_HASH_CHUNK, v.numel()),), generator=g, device=v.device,
                      dtype=torch.int64) * 2 + 1
    out = []
    for i in range(0, v.numel(), _HASH_CHUNK):
        c = v[i:i + _HASH_CHUNK].to(torch.int64)
        out.append(int((c * m[:c.numel()]).sum().item()))
    return ("hash64", int(v.numel()), tuple(out))


def same_gradients(a: dict, b: dict) -> bool:
    """Equality of two passes' gradients and losses, bit for bit (NaNs compare by
    their bit patterns): element by element, or by per-chunk hashes where a
    snapshot could not hold a copy."""
    import torch
    for k in ("dW", "db", "dh0", "dc0"):
        x, y = a.get(k), b.get(k)
        if (x is None) != (y is None):
            return False
        if x is None:
            continue
        if isinstance(x, tuple) or isinstance(y, tuple):
            if (x if isinstance(x, tuple) else _digest(x)) != (y if isinstance(y, tuple) else _digest(y)):
                return False
        elif not torch.equal(x.view(torch.int32), y.view(torch.int32)):
            return False
    return a["loss"] == b["loss"]


def snapshot(out: dict) -> dict:
    """A pass's gradients and loss for a later comparison: a device copy of each
    tensor, or its per-chunk hashes when a copy would take more than half of
    the free device memory (the residual MLP's fp32 dW is 134 GB)."""
    import torch
    free = torch.cuda.mem_get_info()[0]
    res = {}
    for k, v in out.items():
        if k not in ("dW", "db", "dh0", "dc0", "loss"):
            continue
        if hasattr(v, "clone"):
            nbytes = v.numel() * v.element_size()
            if nbytes > free // 2:
                res[k] = _digest(v)
            else:
                res[k] = v.clone()
                free -= nbytes
        else:
            res[k] = v
    return res


def comparison_kind(snap: dict) -> str:
    return ("64-bit hash per 256 MiB chunk for " + ", ".join(k for k, v in snap.items() if isinstance(v, tuple))
            + "; the rest element by element") if any(isinstance(v, tuple) for v in snap.values()) else \
        "element by element"


def estimate_pass_s(wl, spec, t_a_us: float, I_min: int) -> float:
    """Rough seconds per pass from the calibrated forward step: R forward steps
    and about 2.7 forward steps' worth of adjoint work per timestep."""
    import paper_1806_01117_amd as amb
    evals = amb.schedule_evals(wl.n_steps, spec.fast_slots, spec.slow_slots, max(1, I_min))[0]
    return wl.n_steps * t_a_us * 1e-6 * (evals / wl.n_steps + 2.7)


def lds_kernels(spec, knobs) -> tuple[bool, bool]:
    """Whether the fp32 large-batch path runs its gate products and its
    h-adjoint products on the LDS-tiled kernels (the library's "lds_gemm"
    rule: shapes that fit their tiles and, by default, give every CU two
    workgroups: 256 tiles of 128 x 128, or of 64 x 64)."""
    G, B, D, H = spec.gates, spec.batch, spec.input, spec.hidden
    k = dict(knobs)
    mode = k.get("lds_gemm", 1)
    cell_fit = D % 4 == 0 and H % 4 == 0 and (G * H) % 128 == 0
    prod_fit = (G * H) % 4 == 0 and H % 64 == 0 and k.get("hadj_launch", 1) != 0
    cell = mode > 0 and cell_fit and (mode == 2 or -(-B // 128) * (G * H // 128) >= 256)
    prod = mode > 0 and prod_fit and (mode == 2 or -(-B // 64) * (H // 64) >= 256)
    return cell, prod


def prod_split_parts(spec, knobs) -> int:
    """Parts of the fp32 h-adjoint product's split reduction (the library's
    "prod_split" rule: both LDS-tiled kernels in use, 128 x 128 tiles, parts
    doubled up to 4 while the grid has fewer than 512 workgroups and every
    part keeps at least 16 stages of 64); 1 where it is not split."""
    cell, prod = lds_kernels(spec, knobs)
    if not (cell and prod and dict(knobs).get("prod_split", 1) != 0):
        return 1
    M, N, K = spec.batch, spec.hidden, spec.gates * spec.hidden
    if N % 128 or K % 4:
        return 1
    tiles, parts = -(-M // 128) * (N // 128), 1
    while parts < 4 and tiles * parts < 512 and (K // 64) // (2 * parts) >= 16:
        parts *= 2
    return parts


def step_flops(spec, window: int, wide: bool = False) -> dict:
    """Algorithmic flops of one launch of each per-step kernel, and of the
    three products of one step (gate GEMM, h-adjoint, weight gradient).  On
    the wide-batch bf16 path the h-adjoint product is a launch of its own
    ("hadj"); otherwise the adjoint launch holds it."""
    B, D, H, G = spec.batch, spec.input, spec.hidden, spec.gates
    gate = 2.0 * B * G * H * (D + H)            # z = [x|h] W^T (the MLP: y W_l^T)
    hbar = 2.0 * B * H * G * H                  # hbar = zbar W_h (the MLP: zbar W_{l+1})
    dw1 = 2.0 * G * H * (D + H + 1) * B         # dW (+ db) of one step
    return {"fwd": gate, "adj": gate if wide else gate + hbar, "hadj": hbar, "dw": dw1 * window,
            "gate": gate, "hbar": hbar, "dw1": dw1}


def step_bytes(wl, spec, window: int, wide: bool) -> dict:
    """Algorithmic HBM bytes of one launch of each per-step kernel: every
    operand read once and every result written once, weights included (one
    step's weights, 50 MB and more on the wide path, are streamed again by each
    launch).  e is the operand size; c, the adjoints h-bar, c-bar and the MLP's
    y-bar are fp32."""
    B, D, H, G = spec.batch, spec.input, spec.hidden, spec.gates
    e = 2 if wl.dtype == "bf16" else 4
    K1, GH = D + H, G * H
    W, b = GH * K1 * e, GH * 4
    h, f = B * H * e, B * H * 4               # a state row block in the operand type / in fp32
    c = f if G == 4 else 0
    zbar = B * GH * e
    if wl.cell == "resmlp":                  # K1 = H, G = 1, no c
        fwd = W + b + 2 * h
        adj = W + b + h + f + zbar + f + h          # y, the N-N product's sum in, zbar, ybar, y window out
        if not wide:
            adj += zbar + W + f                     # the next layer's zbar, W_{l+1} and ybar feed the product
        hadj = zbar + W + 2 * f
        dw = 2 * B * H * e + W // e * 4 + b         # zbar and y of one layer in, dW_l and db_l written once
    else:
        fwd = W + b + B * K1 * e + c + h + c
        adj = W + b + B * K1 * e + c + f + c + zbar + c + h   # ... hbar in, cbar in, zbar, cbar, h window out
        if not wide:
            adj += zbar + GH * H * e - f            # zbar_{t+1} and W_h^T instead of the h-adjoint product
        hadj = zbar + GH * H * e + f
        R = window * B
        dw = R * GH * e + R * K1 * e + 2 * (GH * K1 * 4 + b)   # the window's operands, dW and db read and written
    return {"fwd": fwd, "adj": adj, "hadj": hadj, "dw": dw}


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch of a kernel on a workload from the committed
    FETCH_SIZE / WRITE_SIZE counter runs (each scaled by a plain copy of known
    size), or None if there are none or the kernel's source has changed since
    those counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{workload}_pmc.json")
    try:
        rec = json.load(open(path))["kernels"][kernel]
        src = open(os.path.join(ROOT, rec["source"]), "rb").read()
    except (OSError, ValueError, KeyError):
        return None
    if hashlib.sha256(src).hexdigest() != rec["sha256"]:
        return None
    return round(rec["fetch_bytes"] + rec["write_bytes"])


def cpu_baseline(wl, budget_s: float = 12.0) -> dict:
    """The float64 oracle's store-all BPTT on the host cores, on the first
    steps (layers) of the workload at its full shapes, as many as fit the
    budget after a probe."""
    import numpy as np
    import synth
    from oracle import bptt
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = len(os.sched_getaffinity(0))
    x0 = synth.initial_state(wl)
    st = tuple(x0[k].astype(np.float64) for k in ("h", "c") if k in x0)
    if wl.cell in ("resmlp", "mlp"):
        cache = {}

        def layer(l):
            if l not in cache:
                Wl, bl = synth.layer_params(wl, l)
                cache[l] = (Wl.astype(np.float64), bl.astype(np.float64))
            return cache[l]
        cell = bptt.cell_for(wl, layer=layer)
    else:
        W, b = synth.params(wl)
        cell = bptt.cell_for(wl, (W.astype(np.float64), b.astype(np.float64)))

    def one(n):
        w = wl.with_(n_steps=n)
        xs = synth.x_slice(w, 0, n).astype(np.float64)
        t = time.perf_counter()
        bptt.store_all(cell, n, lambda i: xs[i], st)
        return time.perf_counter() - t

    probe = 2 if wl.batch * wl.hidden >= (1 << 19) else 16
    dt = one(probe)
    n = int(max(probe, min(wl.n_steps, budget_s * probe / max(dt, 1e-6))))
    if n > probe:
        dt = one(n)
    return {"value": n / dt, "unit": "timesteps/s", "cores": int(threads), "kind": "oracle",
            "sample": f"float64 store-all BPTT (numpy) over the first {n} of {wl.n_steps} "
                      f"{'layers' if wl.cell in ('resmlp', 'mlp') else 'steps'} at the full shapes, {dt:.1f} s"}


def device_inputs(wl, dev):
    """Seeded inputs, generated on the host in slices (synth) and moved to HBM
    in the operand dtype; the residual MLP's layers are drawn in parallel."""
    import numpy as np
    import torch
    from concurrent.futures import ThreadPoolExecutor
    import synth
    op = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    n, B, D, H = wl.n_steps, wl.batch, wl.input, wl.hidden
    x0 = synth.initial_state(wl)
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)
    dh = t(x0["h"], op)
    dc = t(x0["c"], torch.float32) if "c" in x0 else None
    if wl.cell == "mlp":  # layers of different widths: weights and biases one after the other
        ws = wl.layer_widths()
        dW = torch.empty(sum(ws[l + 1] * ws[l] for l in range(n)), dtype=torch.float32, device=dev)
        db = torch.zeros(sum(ws[1:]), dtype=torch.float32, device=dev)
        offs = [0]
        for l in range(n):
            offs.append(offs[-1] + ws[l + 1] * ws[l])
        with ThreadPoolExecutor(min(16, len(os.sched_getaffinity(0)))) as ex:
            for l, Wl in ex.map(lambda l: (l, synth.layer_params(wl, l)[0]), range(n)):
                dW[offs[l]:offs[l + 1]].copy_(torch.from_numpy(Wl.ravel()).to(dev))
        return None, dW, db, dh, None
    if wl.cell == "resmlp":
        dx = None
        dW = torch.empty((n, H, H), dtype=op, device=dev)
        db = torch.zeros((n, H), dtype=torch.float32, device=dev)
        workers = min(16, len(os.sched_getaffinity(0)))

        def put(l):
            Wl, bl = synth.layer_params(wl, l)
            return l, torch.from_numpy(Wl).to(op)
        with ThreadPoolExecutor(workers) as ex:
            for l0 in range(0, n, 64):
                for l, Wl in ex.map(put, range(l0, min(n, l0 + 64))):
                    dW[l].copy_(Wl.to(dev))
        return dx, dW, db, dh, dc
    dx = torch.empty((n, B, D), dtype=op, device=dev)
    chunk = max(1, (256 << 20) // max(1, B * D * 4))
    for t0 in range(0, n, chunk):
        t1 = min(n, t0 + chunk)
        dx[t0:t1].copy_(torch.from_numpy(synth.x_slice(wl, t0, t1)).to(op).to(dev))
    W, b = synth.params(wl)
    return dx, t(W, op), t(b, torch.float32), dh, dc


def gemm_reference(wl, dev, reps: int = 200) -> dict:
    """The vendor GEMM (torch.matmul, hipBLASLt on ROCm) on the step products
    of a workload, back to back on the same operands: a reference for the
    library's fused step kernels, which add the cell or layer epilogue."""
    import torch
    e = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    B, D, H = wl.batch, wl.input, wl.hidden
    G = 4 if wl.cell == "lstm" else 1
    if wl.cell == "resmlp":
        shapes = {"layer product y W^T": (B, H, H, True), "adjoint product zbar W": (B, H, H, False)}
    else:
        shapes = {"gate product [x|h] W^T": (B, G * H, D + H, True), "h-adjoint product zbar W_h": (B, H, G * H, True)}
    out = {}
    for name, (M, N, K, nt) in shapes.items():
        a = torch.randn(M, K, device=dev).to(e)
        w = torch.randn(N, K, device=dev).to(e) if nt else torch.randn(K, N, device=dev).to(e)
        o = torch.empty(M, N, device=dev, dtype=e)
        f = (lambda: torch.matmul(a, w.t(), out=o)) if nt else (lambda: torch.matmul(a, w, out=o))
        for _ in range(10):
            f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            f()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1000.0 / reps
        out[name] = {"shape": [M, N, K], "us": round(us, 2), "tflops": round(2.0 * M * N * K / us / 1e6, 1)}
    return out


def sweep_n(args, knobs) -> int:
    """R(n) and timesteps/s(n) at a fixed HBM slot budget: the two-level
    schedule against plain Revolve on the same slots, one JSON line per n
    (the measured counterpart of the constant-overhead claim, Section 3 and
    Fig. 3).  Each n runs its own whole passes on the workload's shapes."""
    import torch
    import paper_1806_01117_amd as amb
    import synth
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    base = synth.get(args.workload)
    for n in [int(v) for v in args.sweep_n.split(",")]:
        wl = base.with_(n_steps=n)
        dx, dW, db, dh, dc = device_inputs(wl, dev)
        torch.cuda.synchronize()
        res = {"workload": wl.name, "n_steps": n, "fast_slots": wl.fast_slots}
        outs = {}
        for name, kw in (("async", dict(slow_slots=min(wl.host_slots, n))), ("revolve", dict(slow_slots=0))):
            spec = amb.ProblemSpec.from_workload(wl, **kw)
            r = amb.Runner(spec, device=dev)
            try:
                if args.path != "auto":
                    r.set("path", 1 if args.path == "steps" else 2)
                for k, v in knobs:
                    r.set(k, v)
                I_min = 0
                if name == "async":
                    I_min, t_a, t_t = r.calibrate(dx, dW, db, dh, dc)
                r.run(dx, dW, db, dh, dc)  # warm-up
                torch.cuda.synchronize()
                reps = max(1, min(args.steps, int(2e6 // n)))
                t0 = time.perf_counter()
                for _ in range(reps):
                    o = r.run(dx, dW, db, dh, dc)
                torch.cuda.synchronize()
                el = (time.perf_counter() - t0) / reps
                outs[name] = snapshot(o)
                st = o["stats"]
                res[name] = {"value": round(n / el, 2), "unit": "timesteps/s", "ms_per_pass": round(1000 * el, 3),
                             "recompute_factor": round(st["recompute_factor"], 4), "interval": st["interval"],
                             "mode": ["revolve", "async", "dynamic", "online"][st["mode"]], "passes": reps,
                             "path": "resident" if st["path"] == 1 else "steps"}
                if name == "async":
                    res[name].update({"interval_min": I_min, "t_a_us": round(t_a, 3), "t_t_us": round(t_t, 3)})
            finally:
                r.close()
        res["bit_identical_gradients"] = same_gradients(outs["async"], outs["revolve"])
        res["paper_model"] = {"revolve_R": round((amb.revolve_advances(n, wl.fast_slots) + 1) / n, 4)}
        print(json.dumps(res), flush=True)
        del dx, dW, db, dh, dc, outs
        torch.cuda.empty_cache()
    release_pinned()
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--max-timed-s", type=float, default=120.0,
                    help="seconds the warm-up and timed passes may take together (estimated from the calibrated "
                         "forward step); fewer whole passes run beyond it, at least one timed")
    ap.add_argument("--pinned-gib", type=float, default=56.0,
                    help="pinned host memory for the host tier (the process limit is 64 GiB); caps its slots")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--timing-sample", type=int, default=32)
    ap.add_argument("--path", choices=["auto", "steps", "resident"], default="auto")
    ap.add_argument("--cooperative", type=int, default=1, help="resident kernel: 1 cooperative launch (default), 0 plain")
    ap.add_argument("--workload", default=WORKLOAD, help="a synth workload name (default: the 4096-LSTM)")
    ap.add_argument("--n-steps", type=int, default=0, help="override the workload's step count (profiling runs)")
    ap.add_argument("--host-slots", type=int, default=-1, help="host-tier slots (default: the workload's, "
                    "capped by --pinned-gib)")
    ap.add_argument("--no-compare", dest="compare", action="store_false",
                    help="skip the plain-Revolve and other-path passes")
    ap.add_argument("--file-tier", default="", metavar="DIR",
                    help="a file in DIR below the pinned host tier, as many slots as steps; --host-slots then sizes "
                         "the pinned ring in front of it")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="only time the vendor GEMM on the workload's step products and print them")
    ap.add_argument("--sweep-n", default="", metavar="N1,N2,...",
                    help="only measure the two-level schedule against plain Revolve at each step count")
    ap.add_argument("--step-costs", default="", metavar="every:K:F",
                    help="relative step costs for the schedule (step t costs F when t % K == 0, else 1): "
                         "reversals split for unequal costs (ambptt_set_step_costs)")
    ap.add_argument("--set", action="append", default=[], metavar="KEY=VALUE",
                    help="an ambptt_set_int knob for the measured passes and the plain-Revolve comparison")
    args = ap.parse_args()
    knobs = [(k, int(v)) for k, v in (kv.split("=", 1) for kv in args.set)]
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(--gpus must be 1)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_1806_01117_amd as amb
    import synth

    if args.sweep_n:
        return sweep_n(args, knobs)
    wl = synth.get(args.workload)
    if args.n_steps > 0:
        wl = wl.with_(n_steps=args.n_steps)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.gemm_reference:
        print(json.dumps({"workload": wl.name, "vendor_gemm": gemm_reference(wl, dev)}), flush=True)
        return 0
    # a plain copy of known size (256 MiB read + 256 MiB written): the reference
    # that scales the FETCH_SIZE / WRITE_SIZE counters of a profiling run.  It
    # is the run's first copy: the inputs' upload below runs as copies of up to
    # 256 MiB too, which the counter summary must not take for it.
    ref_src = torch.ones(64 << 20, device=dev)
    ref_dst = torch.empty_like(ref_src)
    ref_dst.copy_(ref_src)
    torch.cuda.synchronize()
    del ref_src, ref_dst

    dx, dW, db, dh, dc = device_inputs(wl, dev)
    torch.cuda.synchronize()
    print(f"inputs of {wl.name} in HBM", file=sys.stderr, flush=True)

    stride = amb.query(amb.ProblemSpec.from_workload(wl))[0]
    pinned_cap = int(args.pinned_gib * 2 ** 30) // stride
    if args.host_slots >= 0:
        host_slots = args.host_slots
    else:
        host_slots = min(wl.host_slots, pinned_cap) if not args.file_tier else min(wl.host_slots, 256)
    spec = amb.ProblemSpec.from_workload(wl, slow_slots=host_slots)
    f32 = dict(dtype=torch.float32, device=dev)
    outb = {"dW": torch.empty(dW.shape, **f32), "db": torch.empty(db.shape, **f32),
            "dh0": torch.empty(dh.shape, **f32), "dc0": torch.empty(dh.shape, **f32) if dc is not None else None}
    runners = []

    def runner(sp):
        rr = amb.Runner(sp, device=dev)
        runners.append(rr)
        return rr

    try:
        return _measure(args, knobs, wl, spec, host_slots, pinned_cap, dev, dx, dW, db, dh, dc, outb, runner)
    finally:
        # every context is closed and every pinned block released before the
        # interpreter's teardown, which then makes no HIP call of ours
        for rr in runners:
            rr.close()
        del dx, dW, db, dh, dc, outb
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        release_pinned()


def _measure(args, knobs, wl, spec, host_slots, pinned_cap, dev, dx, dW, db, dh, dc, outb, runner) -> int:
    import numpy as np
    import torch

    import paper_1806_01117_amd as amb

    r = runner(spec)
    if args.path != "auto":
        r.set("path", 1 if args.path == "steps" else 2)
    r.set("resident_cooperative", args.cooperative)
    for k, v in knobs:
        r.set(k, v)
    if args.file_tier:
        r.set_file_tier(args.file_tier, wl.n_steps)
    costs = step_costs(args.step_costs, wl.n_steps)
    if costs is not None:
        r.set_step_costs(costs)
    I_min, t_a, t_t = r.calibrate(dx, dW, db, dh, dc)
    print(f"calibrated: I_min {I_min}, T_A {t_a:.2f} us, T_T {t_t:.2f} us", file=sys.stderr, flush=True)
    for k, v in knobs:  # an interval_min given here replaces the calibrated one
        if k == "interval_min":
            r.set(k, v)
            I_min = v
    r.set("timing_sample", args.timing_sample)
    # the pinned host tier and the slot events are allocated now, as a context
    # that runs pass after pass holds them, so that a timed pass without a
    # warm-up pass before it does not include pinning tens of GB
    try:
        r.set("reserve", 1)
        reserved = True
    except amb.AmbpttError as e:  # a schedule the library plans only inside the pass
        print(f"host tier not reserved ahead: {e}", file=sys.stderr, flush=True)
        reserved = False
    # whole passes only: as many of the requested ones as fit the budget
    est = estimate_pass_s(wl, spec, t_a, I_min)
    steps, warmup = args.steps, args.warmup
    if est * (steps + warmup) > args.max_timed_s:
        fit = int(args.max_timed_s // max(est, 1e-9))
        steps = max(1, min(steps, fit))
        warmup = max(0, min(warmup, fit - steps))
    print(f"estimated {est:.2f} s per pass: {warmup} warm-up and {steps} timed passes", file=sys.stderr, flush=True)
    for _ in range(warmup):
        r.run(dx, dW, db, dh, dc, out=outb)
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for i in range(steps):
        out = r.run(dx, dW, db, dh, dc, out=outb)
        stats.append(out["stats"])
        print(f"pass {i + 1}/{steps} done", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    value = wl.n_steps * steps / el
    st = stats[-1]
    resident = st["path"] == 1
    ref = snapshot(out) if args.compare else None

    def other_run(rn, reps, warm=True):
        if warm:
            rn.run(dx, dW, db, dh, dc, out=outb)
        torch.cuda.synchronize()
        tr = time.perf_counter()
        for _ in range(reps):
            o = rn.run(dx, dW, db, dh, dc, out=outb)
        torch.cuda.synchronize()
        return wl.n_steps * reps / (time.perf_counter() - tr), o

    reps = max(1, min(3, steps))
    # plain Revolve at the same HBM slot budget (no host tier), same path
    rv_value, rv_st, bitwise, rv_refused = None, None, None, None
    if args.compare:
        rv = runner(amb.ProblemSpec.from_workload(wl, slow_slots=0))
        rv.set("path", 2 if resident else 1)
        rv.set("resident_cooperative", args.cooperative)
        for k, v in knobs:
            if k != "online":  # plain Revolve knows n up front
                rv.set(k, v)
        try:
            rv_value, rvo = other_run(rv, reps, warm=steps > 1)
            rv_st = rvo["stats"]
            bitwise = same_gradients(rvo, ref)
            print(f"plain Revolve done, bit-identical gradients: {bitwise}", file=sys.stderr, flush=True)
        except amb.AmbpttError as e:
            if e.status != amb._lib.EUNSUPPORTED:
                raise
            rv_refused = str(e)  # e.g. one sized reversal of all n steps needs a table past the limit
            print(f"plain Revolve refused: {e}", file=sys.stderr, flush=True)
        rv.close()
    # states of different sizes: the same pass planned with slots of the
    # largest size in the same byte budget
    uni = None
    if args.compare and wl.cell == "mlp":
        r.set("uniform_sizes", 1)
        u_value, uo = other_run(r, reps, warm=steps > 1)
        r.set("uniform_sizes", 0)
        uni = {"value": round(u_value, 2), "unit": "timesteps/s",
               "recompute_factor": round(uo["stats"]["recompute_factor"], 4),
               "bit_identical_gradients": same_gradients(uo, ref)}
        print(f"slots of the largest size done, bit-identical gradients: {uni['bit_identical_gradients']}",
              file=sys.stderr, flush=True)
        del uo
    # store-all in HBM (a slot for every state: no recomputation, no host tier),
    # same path, where the slot pool fits in a quarter of the HBM
    sa = None
    n_state = amb.query(spec)[0]
    if args.compare and wl.n_steps * n_state <= 72 * 2 ** 30:
        sr = runner(amb.ProblemSpec.from_workload(wl, fast_slots=wl.n_steps, slow_slots=0))
        sr.set("path", 2 if resident else 1)
        sr.set("resident_cooperative", args.cooperative)
        sa_value, sao = other_run(sr, reps, warm=steps > 1)
        sa = {"value": round(sa_value, 2), "unit": "timesteps/s",
              "recompute_factor": round(sao["stats"]["recompute_factor"], 4),
              "bit_identical_gradients": same_gradients(sao, ref),
              "slot_pool_gb": round(wl.n_steps * n_state / 2 ** 30, 2)}
        print(f"store-all done, bit-identical gradients: {sa['bit_identical_gradients']}", file=sys.stderr, flush=True)
        sr.close()
        del sao
        torch.cuda.empty_cache()
    # the same schedule with one kernel launch per step (the other execution path)
    alt = None
    if resident and args.compare:
        ps = runner(amb.ProblemSpec.from_workload(wl, interval_min=max(1, st["interval"]), slow_slots=host_slots))
        ps.set("path", 1)
        for k, v in knobs:
            if k == "online":  # the same schedule
                ps.set(k, v)
        if costs is not None:
            ps.set_step_costs(costs)
        ps_value, pso = other_run(ps, reps)
        ps_st = pso["stats"]
        ps.close()
        alt = {"value": round(ps_value, 2), "unit": "timesteps/s", "interval": ps_st["interval"],
               "recompute_factor": round(ps_st["recompute_factor"], 4)}

    # roofline of the dominant kernel (largest device time in one pass)
    from paper_1806_01117_amd._lib import KERNEL_CLASSES
    peak = FP32_MFMA_PEAK_TFLOPS if wl.dtype == "f32" else BF16_MFMA_PEAK_TFLOPS
    wide = st["kernel_calls"][3] > 0
    if wl.cell == "mlp":
        fl, byts = mlp_layer_work(wl.layer_widths(), wl.batch)
    else:
        fl = step_flops(spec, st["window"], wide)
        byts = step_bytes(wl, spec, st["window"], wide)
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
        e = 2 if wl.dtype == "bf16" else 4
        GH, K1 = spec.gates * spec.hidden, spec.input + spec.hidden
        # x_t of every forward step and adjoint, W in and dW out once, each host-tier transfer through HBM once
        byts = {"pass": (st["forward_evals"] + st["adjoints"]) * spec.batch * spec.input * e
                + GH * K1 * (e + 4) + 2 * GH * 4 + st["bytes_d2h"] + st["bytes_h2d"]}
        names = {"pass": "resident_pass: whole forward + reverse pass in one launch"}
        traffic = measured_traffic(wl.name, "resident_pass")
    else:
        flops = {k: fl[k] for k in ("fwd", "adj", "hadj", "dw") if k in fl}
        cand = [k for k in tot if k in flops]
        dom = max(cand, key=tot.get) if cand else "adj"
        small = spec.batch * spec.hidden < 1024 * 256 or wl.dtype == "bf16"
        lds_cell, lds_prod = lds_kernels(spec, knobs)
        if wl.cell == "mlp":
            names = {"fwd": "mlpv_gemm forward: layer product + relu (mean over layers)",
                     "adj": "mlpv_gemm adjoint: zbar_{l+1} W_{l+1}, recompute, mask, seed (mean over layers)",
                     "dw": "mlpv_dw weight gradient of one layer (mean over layers)"}
        elif wide and wl.dtype == "f32":
            parts = prod_split_parts(spec, knobs)
            hadj_kernel = (f"prod_split_f32 ({parts} parts)" if parts > 1 else
                           "prod_gemm_f32" if lds_prod else "prod_f32")
            names = {"fwd": ("cell_gemm_f32" if lds_cell else "step_f32") + " forward: gate GEMM + cell update",
                     "adj": ("cell_gemm_f32" if lds_cell else "step_f32") + " adjoint: gate recompute + cell adjoint",
                     "hadj": hadj_kernel + " h-adjoint product zbar W_h",
                     "dw": "dw_f32_big weight-gradient window"}
        elif wide and wl.cell == "resmlp":
            names = {"fwd": "mlp_wide forward", "adj": "mlp_wide adjoint (recompute + mask)",
                     "hadj": "prod_wide NN product ybar + zbar W_{l+1}", "dw": "dw_bf16 weight gradient of one layer"}
        elif wide:
            names = {"fwd": "cell_wide forward: gate GEMM + cell update",
                     "adj": "cell_wide adjoint: gate recompute + cell adjoint",
                     "hadj": "prod_wide h-adjoint product zbar W_h", "dw": "dw_bf16 weight-gradient window"}
        elif wl.cell == "resmlp":
            names = {"fwd": "resmlp_step forward", "adj": "resmlp_step adjoint (recompute + NN product)",
                     "dw": "weight gradient of one layer"}
        else:
            k = "step_small" if small else "step_f32"
            names = {"fwd": f"{k} forward: gate GEMM + cell update", "adj": f"{k} adjoint: gate recompute + h-adjoint GEMM",
                     "dw": ("dw_bf16" if wl.dtype == "bf16" else "dw_lds_f32") + " weight-gradient window"}
        if wl.cell == "mlp":
            key = "mlpv_" + dom
        elif wide and wl.dtype == "f32":
            key = {"fwd": "cell_gemm_f32_fwd" if lds_cell else "step_f32_fwd",
                   "adj": "cell_gemm_f32_adj" if lds_cell else "step_f32_adj",
                   "hadj": "prod_split_f32" if prod_split_parts(spec, knobs) > 1 else
                   "prod_gemm_f32" if lds_prod else "prod_f32"}.get(dom, "dw_f32_big")
        elif wide:
            fam = {"fwd": "mlp_wide_fwd", "adj": "mlp_wide_adj", "hadj": "prod_wide_nn"} if wl.cell == "resmlp" else \
                {"fwd": "cell_wide_fwd", "adj": "cell_wide_adj", "hadj": "prod_wide_nt"}
            key = fam.get(dom, "dw_bf16")
        elif small:
            key = {"fwd": "step_small_fwd", "adj": "step_small_adj"}.get(dom, "dw_lds_f32")
        else:
            key = {"fwd": "step_f32_fwd", "adj": "step_f32_adj"}.get(dom, "dw_f32_big")
        traffic = measured_traffic(wl.name, key)
    dom_us = kern[dom][0] if dom in kern else 0.0
    # the roofline that bounds the kernel: HBM if its algorithmic bytes take
    # longer at 8 TB/s than its flops at the MFMA peak of its operand type
    hbm = byts[dom] / (HBM_PEAK_GBS * 1e9) > flops[dom] / (peak * 1e12)
    if hbm:
        achieved = byts[dom] / (dom_us * 1e-6) / 1e9 if dom_us > 0 else 0.0
        roof_peak, roof_unit = HBM_PEAK_GBS, "GB/s"
    else:
        achieved = flops[dom] / (dom_us * 1e-6) / 1e12 if dom_us > 0 else 0.0
        roof_peak, roof_unit = peak, "TFLOP/s"
    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "timesteps/s", "n_gpus": 1,
        "steps": steps, "warmup": warmup, "ms_per_step": round(1000 * el / steps, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic (seeded normal inputs, " + ("normal" if wl.cell in ("resmlp", "mlp") else "uniform")
                + " weights)",
        "config": {"workload": wl.name, "cell": wl.cell, "batch": wl.batch, "input": wl.input,
                   "hidden": wl.hidden, "n_steps": wl.n_steps, "fast_slots": wl.fast_slots,
                   "slow_slots": spec.slow_slots,
                   "mode": ["revolve", "async", "dynamic", "online"][st["mode"]],
                   "interval": st["interval"], "interval_min": I_min, "t_a_us": round(t_a, 3),
                   "t_t_us": round(t_t, 3), "window": st["window"],
                   "pinned_host_gib": round(host_slots * n_state / 2 ** 30, 2), "host_tier_reserved": reserved,
                   **({"host_slots_capped_by_pinned_gib": args.pinned_gib}
                      if host_slots == pinned_cap and pinned_cap < wl.host_slots and not args.file_tier else {}),
                   **({"knobs": dict(knobs)} if knobs else {}),
                   **({"file_tier": {"file_slots": wl.n_steps, "pinned_ring": host_slots,
                                     "bytes_written": st["bytes_file_w"], "bytes_read": st["bytes_file_r"]}}
                      if args.file_tier else {})},
        "recompute_factor": round(st["recompute_factor"], 4),
        # Section 3's model: R(n, s) for Revolve, R(I, s) for the two-level
        # policy (the model leaves out the sweep that the count above includes)
        "paper_model": {"revolve_R": round((amb.revolve_advances(wl.n_steps, spec.fast_slots) + 1) / wl.n_steps, 4),
                        "async_R": round((amb.revolve_advances(st["interval"], spec.fast_slots) + 1) / st["interval"], 4)
                        if st["interval"] > 0 else None},
        "plain_revolve": ({"refused": rv_refused} if rv_refused else None) if rv_st is None else {
            "value": round(rv_value, 2), "unit": "timesteps/s",
            "recompute_factor": round(rv_st["recompute_factor"], 4), "bit_identical_gradients": bitwise,
            "compared": comparison_kind(ref)},
        "store_all": sa,
        **({"slots_of_the_largest_size": uni} if uni is not None else {}),
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
        "roofline": {"bound": "hbm" if hbm else "mfma", "kernel": names[dom], "achieved": round(achieved, 3),
                     "peak": roof_peak, "unit": roof_unit,
                     "frac": round(achieved / roof_peak, 4), "traffic": traffic,
                     "avg_launch_us": round(dom_us, 3), "flops_per_launch": flops[dom],
                     "bytes_per_launch": int(byts[dom]),
                     "flop_per_byte": round(flops[dom] / max(byts[dom], 1), 1)},
    }
    if not resident and (st["stores"] or st["prefetches"]):
        line["transfer_overlap"] = copy_overlap(spec, st, stats, dev, 1000.0 * el / steps)
    if costs is not None:
        # the same pass with Revolve's own splits, weighed with the same costs
        plain = amb.schedule_text(wl.n_steps, spec.fast_slots, host_slots, max(I_min, 1))
        total = float(sum(costs))
        line["step_costs"] = {"spec": args.step_costs, "forward_cost": st["forward_cost"],
                              "weighted_recompute_factor": round(st["forward_cost"] / total, 4),
                              "revolve_splits_weighted_recompute_factor":
                                  round(weighted_cost(plain, costs) / total, 4)}
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl)
    if (steps, warmup) != (args.steps, args.warmup):
        line["requested"] = {"steps": args.steps, "warmup": args.warmup, "max_timed_s": args.max_timed_s,
                             "estimated_s_per_pass": round(est, 2)}
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
