"""GPU parity: the HIP path through the C ABI against the float64 oracle on
the same seeded inputs, and checkpointed runs against store-all runs bit for
bit (recomputation is deterministic, so the schedule must not change a bit)."""
import numpy as np
import pytest

import synth
from oracle import schedule as S

from gpu_util import (TOL_BF16, TOL_F32, assert_bitwise, assert_close, assert_close_relu, device_inputs,
                      inputs, run_gpu, run_oracle, say)

pytestmark = pytest.mark.gpu

# 1: one launch per step; 2: the resident whole-pass kernel
PATHS = [pytest.param(1, id="steps"), pytest.param(2, id="resident")]


def _case(wl):
    x, W, b, x0 = inputs(wl)
    return (x, W, b, x0), device_inputs(wl, x, W, b, x0)


@pytest.mark.parametrize("path", PATHS)
def test_rnn_workload_full(path):
    """64-wide tanh RNN, 128 steps, 4 slots, no host tier: Revolve, R = 517/128."""
    wl = synth.get("rnn_h64_t128")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    got = run_gpu(wl, dev, path=path)
    st = got["stats"]
    assert st["mode"] == 0 and st["forward_evals"] == 517 == S.revolve_evals(128, 4)
    assert st["recompute_factor"] == pytest.approx(517 / 128)
    assert_close(got, want, TOL_F32)
    allst = run_gpu(wl, dev, fast_slots=128, path=path)  # store-all: memory ratio 1
    assert allst["stats"]["forward_evals"] == 128
    assert_bitwise(got, allst)


@pytest.mark.parametrize("path", PATHS)
def test_lstm_small_schedules_bitwise(path):
    """A reduced 512-LSTM: Revolve, async I=1, async I=3 and store-all agree bit for bit."""
    wl = synth.get("lstm_h512_t1000").with_(n_steps=48)
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    ref = run_gpu(wl, dev, fast_slots=48, slow_slots=0, path=path)
    assert ref["stats"]["forward_evals"] == 48
    assert_close(ref, want, TOL_F32)
    for kw in (dict(fast_slots=3, slow_slots=0), dict(fast_slots=3, slow_slots=48, interval_min=1),
               dict(fast_slots=4, slow_slots=48, interval_min=3), dict(fast_slots=2, slow_slots=5, interval_min=1)):
        got = run_gpu(wl, dev, path=path, **kw)
        ev = S.schedule(48, kw["fast_slots"], kw["slow_slots"], kw.get("interval_min", 0))[0]["evals"]
        assert got["stats"]["forward_evals"] == ev
        assert_bitwise(got, ref)


@pytest.mark.parametrize("path", PATHS)
def test_lstm_ragged_shapes_and_window(path):
    """Batch not a multiple of 16, a dW window that does not divide n, no prefetch elision."""
    wl = synth.get("lstm_h512_t1000").with_(batch=5, input=16, hidden=32, n_steps=37, name="lstm_ragged")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=37, slow_slots=0, path=path)
    assert_close(a, want, TOL_F32)
    b = run_gpu(wl, dev, fast_slots=3, slow_slots=37, interval_min=2, window=3, elide=False, path=path)
    assert b["stats"]["mode"] == 1 and b["stats"]["window"] == (3 if path == 1 else 0)
    assert b["stats"]["prefetches_elided"] == 0
    assert_close(b, want, TOL_F32)
    c = run_gpu(wl, dev, fast_slots=3, slow_slots=37, interval_min=2, path=path)
    assert_bitwise(b, c, keys=("loss", "dh0", "dc0") if path == 1 else ("loss", "dW", "db", "dh0", "dc0"))


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("loss", ["half_sq_last", "mean_last", "mean_sq_all"])
def test_rnn_losses(loss, path):
    wl = synth.get("rnn_h64_t128").with_(loss=loss, n_steps=40, batch=20)
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    got = run_gpu(wl, dev, fast_slots=3, slow_slots=40, interval_min=2, path=path)
    assert_close(got, want, TOL_F32)


@pytest.mark.parametrize("path", PATHS)
def test_lstm512_workload_full(path):
    """512-LSTM, 1000 steps, 10 slots + host tier: async at I=1 and I=2, plain
    Revolve at the same 10 slots, all against the oracle and bit-exact."""
    wl = synth.get("lstm_h512_t1000")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a1 = run_gpu(wl, dev, interval_min=1, path=path)
    assert a1["stats"]["mode"] == 1 and a1["stats"]["forward_evals"] == 1000   # R = 1
    assert_close(a1, want, TOL_F32)
    a2 = run_gpu(wl, dev, interval_min=2, path=path)
    assert a2["stats"]["forward_evals"] == 1499
    assert_bitwise(a1, a2)
    rv = run_gpu(wl, dev, slow_slots=0, path=path)
    assert rv["stats"]["forward_evals"] == 3637
    assert_bitwise(a1, rv)
    say("R async I=1/2, revolve:", a1["stats"]["recompute_factor"], a2["stats"]["recompute_factor"],
        rv["stats"]["recompute_factor"])


def test_resident_abort_path():
    """A resident pass whose first wait can never be satisfied ends in the
    kernel's own timeout: the call fails with EINTERNAL, every workgroup
    exits, and the next pass on the same context is correct."""
    import paper_1806_01117_amd as amb
    wl = synth.get("lstm_h512_t1000").with_(n_steps=24)
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    spec = amb.ProblemSpec.from_workload(wl, fast_slots=3, slow_slots=24, interval_min=2)
    r = amb.Runner(spec)
    try:
        r.set("path", 2)
        r.set("resident_timeout_ms", 50)
        r.set("resident_test_stall", 1)
        with pytest.raises(amb.AmbpttError, match="timeout"):
            r.run(*dev)
        r.set("resident_test_stall", 0)
        out = r.run(*dev)
    finally:
        r.close()
    got = {k: (v.float().cpu().numpy() if hasattr(v, "cpu") else v) for k, v in out.items() if v is not None}
    assert got["stats"]["path"] == 1
    assert_close(got, want, TOL_F32)


def test_lstm_wide_ragged_weight_gradient():
    """Gradient rows 4H = 320 and columns D + H = 288 (the 128 x 128-tile weight-gradient
    kernel with partial tiles on both edges), windows that do not divide n."""
    wl = synth.get("lstm_h512_t1000").with_(batch=5, input=208, hidden=80, n_steps=23, name="lstm_wide_ragged")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=23, slow_slots=0, path=1)
    assert_close(a, want, TOL_F32)
    b = run_gpu(wl, dev, fast_slots=3, slow_slots=23, interval_min=2, window=5, path=1)
    assert b["stats"]["window"] == 5
    assert_close(b, want, TOL_F32)
    c = run_gpu(wl, dev, fast_slots=3, slow_slots=23, interval_min=2, window=7, path=1)
    assert_bitwise(b, c, keys=("loss", "dh0", "dc0"))


def test_lstm4096_shapes_short():
    """The offload-stress LSTM at its full per-step shapes (B=512, H=4096, D=1024), 4 steps."""
    wl = synth.get("lstm_h4096_t20000").with_(n_steps=4)
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=2, slow_slots=4, interval_min=1)
    assert a["stats"]["mode"] == 1
    assert_close(a, want, TOL_F32)
    b = run_gpu(wl, dev, fast_slots=1, slow_slots=0)
    assert_bitwise(a, b)


def test_lstm_f32_large_batch_hadj_launch():
    """fp32 step kernels for large batches (B = 256, H = 1024: 1024 tiles of
    16 x 16) with the h-adjoint product as its own launch and fused into the
    adjoint step: each against the oracle, each bit for bit across schedules."""
    wl = synth.get("lstm_h4096_t20000").with_(batch=256, input=64, hidden=1024, n_steps=6, name="lstm_f32_big")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=2, slow_slots=6, interval_min=1)
    assert a["stats"]["kernel_calls"][3] == 5  # one product launch per adjoint but the first turn's
    assert_close(a, want, TOL_F32)
    assert_bitwise(a, run_gpu(wl, dev, fast_slots=3, slow_slots=0))
    f = run_gpu(wl, dev, fast_slots=2, slow_slots=6, interval_min=1, opts={"hadj_launch": 0})
    assert f["stats"]["kernel_calls"][3] == 0
    assert_close(f, want, TOL_F32)
    assert_bitwise(f, run_gpu(wl, dev, fast_slots=3, slow_slots=0, opts={"hadj_launch": 0}))


def test_lstm_f32_large_batch_ragged_product():
    """The product's fallback tiles (H = 1040 is no multiple of 128: 16 x 16
    blocks), a batch that is no multiple of 32 (B = 250) and the RNN cell."""
    for cell in ("lstm", "rnn"):
        wl = synth.get("lstm_h4096_t20000").with_(cell=cell, batch=250, input=48, hidden=1040, n_steps=4,
                                                  w_scale=1.0 / 32, name=f"{cell}_f32_big_ragged")
        host, dev = _case(wl)
        want = run_oracle(wl, *host)
        a = run_gpu(wl, dev, fast_slots=2, slow_slots=4, interval_min=1)
        assert a["stats"]["kernel_calls"][3] == 3
        assert_close(a, want, TOL_F32)
        assert_bitwise(a, run_gpu(wl, dev, fast_slots=4, slow_slots=0))


def test_lstm_bf16_small_schedules():
    """bf16 operands and stored h, fp32 cell state: oracle within 2e-2, schedules bit for bit."""
    wl = synth.get("lstm_h2048_bf16_t10000").with_(batch=20, input=64, hidden=96, n_steps=30,
                                                   name="lstm_bf16_small")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    ref = run_gpu(wl, dev, fast_slots=30, slow_slots=0)
    assert ref["stats"]["forward_evals"] == 30
    assert_close(ref, want, TOL_BF16)
    for kw in (dict(fast_slots=3, slow_slots=0), dict(fast_slots=3, slow_slots=30, interval_min=2),
               dict(fast_slots=2, slow_slots=30, interval_min=1)):
        got = run_gpu(wl, dev, **kw)
        assert_bitwise(got, ref)


def test_lstm2048_bf16_shapes_short():
    """The 2048-wide bf16 LSTM at its full per-step shapes (B=128, D=1024, H=2048), 6 steps."""
    wl = synth.get("lstm_h2048_bf16_t10000").with_(n_steps=6)
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=2, slow_slots=6, interval_min=2)   # async: 8 evaluations vs Revolve's 9
    assert a["stats"]["mode"] == 1 and a["stats"]["forward_evals"] == 8
    assert_close(a, want, TOL_BF16)
    b = run_gpu(wl, dev, fast_slots=6, slow_slots=0)
    assert_bitwise(a, b)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_resmlp_small_schedules(dtype):
    """Residual MLP, depth as the sequence: oracle parity and bit-exact schedules."""
    wl = synth.get("resmlp_w4096_l2000_bf16").with_(dtype=dtype, batch=20, hidden=64, n_steps=13,
                                                    w_scale=0.1, name="resmlp_small")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    tol = TOL_F32 if dtype == "f32" else TOL_BF16
    ref = run_gpu(wl, dev, fast_slots=13, slow_slots=0)
    assert ref["stats"]["forward_evals"] == 13
    assert_close(ref, want, tol)
    for kw in (dict(fast_slots=3, slow_slots=0), dict(fast_slots=3, slow_slots=13, interval_min=2),
               dict(fast_slots=2, slow_slots=13, interval_min=1)):
        got = run_gpu(wl, dev, **kw)
        assert_bitwise(got, ref)


def test_resmlp4096_shapes_short():
    """The 4096-wide bf16 residual MLP at its full layer shape (B=256), 5 layers."""
    wl = synth.get("resmlp_w4096_l2000_bf16").with_(n_steps=5)
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=2, slow_slots=5, interval_min=1)
    assert a["stats"]["mode"] == 1
    assert_close_relu(a, want, TOL_BF16)
    b = run_gpu(wl, dev, fast_slots=5, slow_slots=0)
    assert_bitwise(a, b)
