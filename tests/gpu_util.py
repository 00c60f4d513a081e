"""Helpers shared by the GPU tests: seeded inputs from ``synth``, the HIP path
through the C ABI, the oracle on the same inputs, and the error metric."""
from __future__ import annotations

import sys

import numpy as np

import synth
from oracle import bptt

# fp32 and bf16 bars: max |g - g*| / max |g*| per gradient tensor (and the loss)
TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def inputs(wl):
    """Seeded float32 numpy inputs of a workload (bf16 values for bf16 workloads)."""
    x = synth.x_slice(wl, 0, wl.n_steps)
    W, b = synth.params(wl)
    x0 = synth.initial_state(wl)
    return x, W, b, x0


def device_inputs(wl, x, W, b, x0):
    import torch
    op = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    dev = torch.device("cuda")
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt).contiguous()
    return (t(x, op), t(W, op), t(b, torch.float32), t(x0["h"], op),
            t(x0["c"], torch.float32) if "c" in x0 else None)


def run_gpu(wl, dev_in, window: int | None = None, timing_sample: int = 0, elide: bool = True, **spec_kw):
    """One forward + reverse pass on the GPU; returns numpy results and stats."""
    import paper_1806_01117_amd as amb
    spec = amb.ProblemSpec.from_workload(wl, **spec_kw)
    say(wl.name, spec)
    r = amb.Runner(spec)
    try:
        if window is not None:
            r.set("window", window)
        if timing_sample:
            r.set("timing_sample", timing_sample)
        r.set("elide_prefetch", 1 if elide else 0)
        out = r.run(*dev_in)
    finally:
        r.close()
    res = {k: (v.float().cpu().numpy() if hasattr(v, "cpu") else v) for k, v in out.items() if v is not None}
    return res


def run_oracle(wl, x, W, b, x0):
    cell = bptt.cell_for(wl, (W.astype(np.float64), b.astype(np.float64)))
    xs = x.astype(np.float64)
    st = (x0["h"].astype(np.float64),) + ((x0["c"].astype(np.float64),) if "c" in x0 else ())
    out = bptt.store_all(cell, wl.n_steps, lambda t: xs[t], st)
    res = {"loss": out["loss"], "dW": out["dW"], "db": out["db"], "dh0": out["dx0"][0]}
    if len(out["dx0"]) > 1:
        res["dc0"] = out["dx0"][1]
    return res


def rel_err(got, want) -> float:
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    scale = np.max(np.abs(want))
    if scale == 0:
        return float(np.max(np.abs(got)))
    return float(np.max(np.abs(got - want)) / scale)


def assert_close(got: dict, want: dict, tol: float, keys=("loss", "dW", "db", "dh0", "dc0")):
    errs = {k: rel_err(got[k], want[k]) for k in keys if k in want}
    say("errors", {k: f"{v:.2e}" for k, v in errs.items()})
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"relative error above {tol}: {bad}"
    return errs


def assert_bitwise(a: dict, b: dict, keys=("loss", "dW", "db", "dh0", "dc0")):
    for k in keys:
        if k in a:
            assert np.array_equal(np.asarray(a[k]), np.asarray(b[k])), f"{k} differs between schedules"
