"""Oracle parity on the paths the full-size workloads take, at their full
per-step shapes and over enough steps to reach the structures that only long
runs have:

  * the 2048-wide bf16 LSTM (B 128, D 1024, H 2048) over 130 steps: two whole
    64-step (8192-row) weight-gradient windows, the wrap of the two-window
    z-bar ring, 43 intervals of I = 3, under the fixed-interval and the
    dynamic store policy, and with Revolve recomputing inside each interval;
  * the 4096-wide fp32 LSTM (B 512, D 1024, H 4096) over 200 steps at the
    interval its pinned host tier gives it (I = 6), on 8 HBM slots, and with
    Revolve inside the intervals;
  * the 4096-wide residual MLP (B 256) over 32 layers at I = 2 on 4 HBM
    slots, in fp32 against the oracle and in bf16 bit for bit across
    schedules.

The slot counts keep the memory ratio low enough that the two-level
schedule recomputes strictly less than plain Revolve at these lengths (else
the library rightly runs plain Revolve).

Each schedule is compared with the float64 oracle (fp32 1e-4, bf16 2e-2) and,
bit for bit, with plain Revolve at the same HBM slots."""
import pytest

import synth

from gpu_util import (TOL_BF16, TOL_F32, assert_bitwise, assert_close, assert_close_relu, device_inputs, inputs,
                      run_gpu, run_oracle, say)

pytestmark = pytest.mark.gpu


def _case(wl):
    host = inputs(wl)
    return host, device_inputs(wl, *host)


def test_lstm2048_bf16_full_shapes_130_steps():
    wl = synth.get("lstm_h2048_bf16_t10000").with_(n_steps=130)
    host, dev = _case(wl)
    fixed = run_gpu(wl, dev, slow_slots=130, interval_min=3)  # s = 32
    st = fixed["stats"]
    assert st["mode"] == 1 and st["interval"] == 3 and st["window"] == 64
    say("oracle: 130 steps at B 128, D 1024, H 2048")
    want = run_oracle(wl, *host)
    assert_close(fixed, want, TOL_BF16)
    assert_bitwise(fixed, run_gpu(wl, dev, slow_slots=0))                     # plain Revolve, 32 slots
    dyn = run_gpu(wl, dev, slow_slots=130, interval_min=3, opts={"store_policy": 1})
    assert dyn["stats"]["mode"] == 2
    assert_bitwise(fixed, dyn)
    few = run_gpu(wl, dev, fast_slots=3, slow_slots=130, interval_min=8)      # Revolve on 2 slots per interval
    assert few["stats"]["mode"] == 1 and few["stats"]["forward_evals"] > 130 + 129
    assert_bitwise(fixed, few)


def test_lstm4096_full_shapes_200_steps():
    # loss over every step: with the workload's mean(h_n) alone, dL/dx_0 passes
    # 200 forget gates of about 1/2 and is ~1e-60, below fp32's range
    wl = synth.get("lstm_h4096_t20000").with_(n_steps=200, loss="mean_sq_all")
    host, dev = _case(wl)
    # 8 HBM slots for 200 steps (with 64, plain Revolve already recomputes less at this length)
    a = run_gpu(wl, dev, fast_slots=8, slow_slots=200, interval_min=6)
    assert a["stats"]["mode"] == 1 and a["stats"]["interval"] == 6 and a["stats"]["window"] == 16
    say("oracle: 200 steps at B 512, D 1024, H 4096")
    want = run_oracle(wl, *host)
    assert_close(a, want, TOL_F32)
    rv = run_gpu(wl, dev, fast_slots=8, slow_slots=0)                          # plain Revolve, 8 slots
    assert rv["stats"]["forward_evals"] > a["stats"]["forward_evals"]
    assert_bitwise(a, rv)
    few = run_gpu(wl, dev, fast_slots=3, slow_slots=200, interval_min=6)       # Revolve on 2 slots per interval
    assert_bitwise(a, few)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_resmlp4096_32_layers_interval_2(dtype):
    """fp32: against the oracle (mask-aware).  bf16: the oracle rounds only the
    stored states, the kernels also round z-bar to bf16 in every product, and
    over 32 layers their relu masks part beyond the flip band; the loss and
    dL/dy_0 are compared with the oracle, every gradient bit for bit with
    plain Revolve and store-all."""
    wl = synth.get("resmlp_w4096_l2000_bf16").with_(n_steps=32, dtype=dtype)
    host, dev = _case(wl)
    # 4 HBM slots for 32 layers (with 16, plain Revolve recomputes as little)
    a = run_gpu(wl, dev, fast_slots=4, slow_slots=32, interval_min=2)
    assert a["stats"]["mode"] == 1 and a["stats"]["interval"] == 2
    say("oracle: 32 layers at B 256, width 4096", dtype)
    want = run_oracle(wl, *host)
    if dtype == "f32":
        assert_close_relu(a, want, TOL_F32)
    else:
        assert_close(a, want, TOL_BF16, keys=("loss", "dh0"))
    assert_bitwise(a, run_gpu(wl, dev, fast_slots=4, slow_slots=0))            # plain Revolve, 4 slots
    assert_bitwise(a, run_gpu(wl, dev, fast_slots=32, slow_slots=0))           # store-all
