"""ambptt_run_noalloc against ambptt_run through the C ABI: the same pass with
the library's static scratch as workspace.  Two calls of the allocation-free
entry point in a row, the second on a smaller problem, each compared bit for
bit with ambptt_run on its own context (same kernels, same schedule) and
within tolerance of the oracle; then the refusals that keep it
allocation-free."""
import numpy as np
import pytest

import synth

from gpu_util import TOL_F32, assert_close, device_inputs, inputs, run_oracle, say

pytestmark = pytest.mark.gpu

KEYS = ("dW", "db", "dh0", "dc0")


def _runner(wl, path, **kw):
    import paper_1806_01117_amd as amb
    spec = amb.ProblemSpec.from_workload(wl, **kw)
    say("no-alloc case", wl.name, spec, "path", path)
    r = amb.Runner(spec)
    r.set("path", path)
    return r


def _out(wl, dev_in):
    import torch
    x, W, b, h0, c0 = dev_in
    f = dict(dtype=torch.float32, device=W.device)
    return {"dW": torch.full(W.shape, float("nan"), **f), "db": torch.full(b.shape, float("nan"), **f),
            "dh0": torch.full(h0.shape, float("nan"), **f),
            "dc0": torch.full(h0.shape, float("nan"), **f) if c0 is not None else None}


def _same(got, want):
    import torch
    for k in KEYS:
        if want.get(k) is not None:
            assert torch.equal(got[k], want[k]), f"{k} differs from ambptt_run"
    assert got["loss"] == want["loss"]
    for k in ("forward_evals", "stores", "prefetches", "mode", "interval", "path"):
        assert got["stats"][k] == want["stats"][k], k


@pytest.mark.parametrize("path", [pytest.param(1, id="steps"), pytest.param(2, id="resident")])
def test_noalloc_matches_run_on_two_calls_second_smaller(path):
    big = synth.get("lstm_h512_t1000").with_(batch=24, input=32, hidden=64, n_steps=40, name="noalloc_big")
    small = synth.get("lstm_h512_t1000").with_(batch=8, input=16, hidden=32, n_steps=17, name="noalloc_small",
                                               seed_index=7)
    cases = []
    for wl, kw in ((big, dict(fast_slots=3, slow_slots=40, interval_min=2)),
                   (small, dict(fast_slots=2, slow_slots=17, interval_min=1))):
        host = inputs(wl)
        dev = device_inputs(wl, *host)
        r = _runner(wl, path, **kw)
        r.set("reserve", 1)
        want = r.run(*dev)  # the existing entry point, on the bound workspace
        cases.append((wl, host, dev, r, want))
    try:
        for wl, host, dev, r, want in cases:  # two allocation-free calls in a row, big then small
            got = r.run_noalloc(*dev, out=_out(wl, dev))
            assert got["stats"]["path"] == path - 1
            assert got["stats"]["mode"] == 1, "expected the two-level schedule"
            _same(got, want)
            res = {k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in got.items() if v is not None}
            assert_close(res, run_oracle(wl, *host), TOL_F32)
        # and again on the big problem after the small one left its contents in the scratch
        wl, host, dev, r, want = cases[0]
        _same(r.run_noalloc(*dev, out=_out(wl, dev)), want)
    finally:
        for c in cases:
            c[3].close()


def test_noalloc_refuses_what_would_allocate():
    import paper_1806_01117_amd as amb
    from paper_1806_01117_amd._lib import EINVAL, AmbpttError
    wl = synth.get("lstm_h512_t1000").with_(batch=8, input=16, hidden=32, n_steps=12, name="noalloc_refuse")
    host = inputs(wl)
    dev = device_inputs(wl, *host)
    # a host tier that is not reserved yet
    r = _runner(wl, 1, fast_slots=2, slow_slots=12, interval_min=1)
    try:
        with pytest.raises(AmbpttError) as e:
            r.run_noalloc(*dev, out=_out(wl, dev))
        assert e.value.status == EINVAL and "reserve" in str(e.value)
        r.set("reserve", 1)
        got = r.run_noalloc(*dev, out=_out(wl, dev))
        assert_close({k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in got.items() if v is not None},
                     run_oracle(wl, *host), TOL_F32)
    finally:
        r.close()
    # no workspace bound at all: ambptt_run refuses, the allocation-free pass runs
    import ctypes as C
    from paper_1806_01117_amd._lib import check
    r = _runner(wl, 1, fast_slots=2, slow_slots=12, interval_min=1)
    try:
        check(r.L.ambptt_bind(r.ctx, C.c_void_p(r.pool.data_ptr()), r.pool.numel(), None, 0))
        r.set("reserve", 1)
        with pytest.raises(AmbpttError) as e:
            r.run(*dev, out=_out(wl, dev))
        assert e.value.status == EINVAL and "workspace" in str(e.value)
        got = r.run_noalloc(*dev, out=_out(wl, dev))
        assert_close({k: (v.cpu().numpy() if hasattr(v, "cpu") else v) for k, v in got.items() if v is not None},
                     run_oracle(wl, *host), TOL_F32)
    finally:
        r.close()
    # an interval not yet known
    r = _runner(wl, 1, fast_slots=2, slow_slots=12, interval_min=0)
    try:
        with pytest.raises(AmbpttError) as e:
            r.run_noalloc(*dev, out=_out(wl, dev))
        assert e.value.status == EINVAL
    finally:
        r.close()
    # a workspace beyond the 64 MiB scratch (the 2048-wide bf16 LSTM's dW window ring)
    big = synth.get("lstm_h2048_bf16_t10000").with_(n_steps=3, name="noalloc_too_big")
    spec = amb.ProblemSpec.from_workload(big, fast_slots=2, slow_slots=0)
    assert amb.query(spec)[2] > 64 << 20
    hb = inputs(big)
    db_ = device_inputs(big, *hb)
    r = amb.Runner(spec)
    try:
        with pytest.raises(AmbpttError) as e:
            r.run_noalloc(*db_, out=_out(big, db_))
        assert e.value.status == EINVAL and "scratch" in str(e.value)
    finally:
        r.close()
