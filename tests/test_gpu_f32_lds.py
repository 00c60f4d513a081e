"""The LDS-tiled fp32 kernels of the large-batch path (gate product with the
cell epilogue on 128 x 128 tiles; h-adjoint product on 128 x 128 tiles with
the reduction split in parts, or on 64 x 64 tiles), forced onto shapes that
are ragged against their tiles: batches that leave a partial row tile, for
the LSTM and the tanh RNN, every loss.  Each run is compared with the oracle
and, bit for bit, across schedules; the direct-load kernels on the same
inputs meet the same tolerance."""
import pytest

import synth

from gpu_util import TOL_F32, assert_bitwise, assert_close, device_inputs, inputs, run_gpu, run_oracle, say

pytestmark = pytest.mark.gpu

LDS = {"lds_gemm": 2}


def _case(wl):
    host = inputs(wl)
    return host, device_inputs(wl, *host)


def test_lds_lstm_ragged_batch_schedules():
    # B = 300: two full row tiles and one of 44 rows; 4H = 4096 gate columns (16 column tiles)
    wl = synth.get("lstm_h4096_t20000").with_(batch=300, input=96, hidden=1024, n_steps=9, w_scale=1.0 / 32,
                                              name="lstm_f32_lds_ragged")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=3, slow_slots=9, interval_min=2, opts=LDS)
    st = a["stats"]
    assert st["mode"] == 1 and st["kernel_calls"][3] == 8  # a product launch per adjoint but the first turn's
    assert_close(a, want, TOL_F32)
    assert_bitwise(a, run_gpu(wl, dev, fast_slots=9, slow_slots=0, opts=LDS))   # store-all
    assert_bitwise(a, run_gpu(wl, dev, fast_slots=3, slow_slots=0, opts=LDS))   # plain Revolve
    old = run_gpu(wl, dev, fast_slots=3, slow_slots=9, interval_min=2, opts={"lds_gemm": 0})
    assert_close(old, want, TOL_F32)
    # the product on 64 x 64 tiles, unsplit (K = 4096 splits in 4 parts of 16 stages by default)
    whole = run_gpu(wl, dev, fast_slots=3, slow_slots=9, interval_min=2, opts=dict(LDS, prod_split=0))
    assert_close(whole, want, TOL_F32)
    assert_bitwise(whole, run_gpu(wl, dev, fast_slots=9, slow_slots=0, opts=dict(LDS, prod_split=0)))
    # the h-adjoint product fused into the direct-load adjoint beside the LDS-tiled forward
    f = run_gpu(wl, dev, fast_slots=3, slow_slots=9, interval_min=2, opts={"lds_gemm": 2, "hadj_launch": 0})
    assert f["stats"]["kernel_calls"][3] == 0
    assert_close(f, want, TOL_F32)


@pytest.mark.parametrize("loss", ["half_sq_last", "mean_sq_all", "mean_last"])
def test_lds_rnn_losses(loss):
    # tanh RNN: 256 units per column tile, B = 300 ragged against 128-row tiles
    wl = synth.get("lstm_h4096_t20000").with_(cell="rnn", loss=loss, batch=300, input=64, hidden=1024, n_steps=6,
                                              w_scale=1.0 / 32, name="rnn_f32_lds")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=2, slow_slots=6, interval_min=1, opts=LDS)
    say("rnn lds", loss, a["stats"]["kernel_calls"])
    assert_close(a, want, TOL_F32)
    assert_bitwise(a, run_gpu(wl, dev, fast_slots=6, slow_slots=0, opts=LDS))
