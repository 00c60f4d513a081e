"""GPU parity of the wide-batch bf16 kernels (batches of 48 rows and more):
the cell kernel over 64- or 128-row tiles, the adjoint's separate products
(hbar = zbar W_h; the MLP's ybar + zbar W_{l+1}), against the float64 oracle,
bit for bit across schedules, and against the small-batch kernels on the same
inputs.  Batches and widths are ragged with respect to every tile."""
import pytest

import synth

from gpu_util import (TOL_BF16, assert_bitwise, assert_close, assert_close_relu, device_inputs, inputs, run_gpu,
                      run_oracle, say)

pytestmark = pytest.mark.gpu

HADJ = 3  # kernel class of the adjoint's product launches


def _case(wl):
    x, W, b, x0 = inputs(wl)
    return (x, W, b, x0), device_inputs(wl, x, W, b, x0)


def test_wide_lstm_bf16_ragged():
    """B = 100 (two 64-row tiles, the second ragged; the product's 32-row tiles end
    ragged), H = 1536 (192 cell tiles of 64 x 64, 192 product tiles of 32 x 32), D = 64."""
    wl = synth.get("lstm_h2048_bf16_t10000").with_(batch=100, input=64, hidden=1536, n_steps=5,
                                                   name="lstm_bf16_wide")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=2, slow_slots=5, interval_min=1)
    assert a["stats"]["mode"] == 1 and a["stats"]["kernel_calls"][HADJ] == 4
    assert_close(a, want, TOL_BF16)
    b = run_gpu(wl, dev, fast_slots=2, slow_slots=0)
    assert b["stats"]["forward_evals"] > a["stats"]["forward_evals"]
    assert_bitwise(a, b)
    c = run_gpu(wl, dev, fast_slots=5, slow_slots=0, wide=False)  # the small-batch kernels
    assert c["stats"]["kernel_calls"][HADJ] == 0
    assert_close(c, want, TOL_BF16)


def test_wide_lstm_bf16_windows():
    """Weight-gradient windows of 2 steps over 7 (the last one ragged) on the
    compute stream and on a stream of their own: the same sums in the same
    order, so the same bits; against the oracle within the bf16 tolerance."""
    wl = synth.get("lstm_h2048_bf16_t10000").with_(batch=64, input=128, hidden=192, n_steps=7,
                                                   name="lstm_bf16_wide_windows")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=2, slow_slots=7, interval_min=2, window=2)
    assert a["stats"]["mode"] == 1 and a["stats"]["window"] == 2 and a["stats"]["kernel_calls"][4] == 4
    assert_close(a, want, TOL_BF16)
    b = run_gpu(wl, dev, fast_slots=2, slow_slots=0, window=2, opts={"dw_stream": 1})
    assert_bitwise(a, b)
    c = run_gpu(wl, dev, fast_slots=2, slow_slots=7, interval_min=2, window=2, opts={"host_waits": 0})
    assert c["stats"]["stores"] == a["stats"]["stores"] > 0
    assert_bitwise(a, c)  # host-tier dependencies as stream waits instead of host waits


def test_wide_lstm_bf16_long_window_ragged_columns():
    """Weight-gradient windows longer than 512 rows (the 256 x 192 tiles): B = 64 over
    20 steps in one window of 1280 rows, N = D + H = 448 columns (two full 192-column
    tiles and one of 64), against the oracle and, with 4-step windows of 256 rows
    (the 128 x 128 tiles), within rounding of the same sums."""
    wl = synth.get("lstm_h2048_bf16_t10000").with_(batch=64, input=128, hidden=320, n_steps=20,
                                                   name="lstm_bf16_wide_long_window")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=3, slow_slots=20, interval_min=2, window=20)
    assert a["stats"]["mode"] == 1 and a["stats"]["window"] == 20 and a["stats"]["kernel_calls"][4] == 1
    assert_close(a, want, TOL_BF16)
    b = run_gpu(wl, dev, fast_slots=3, slow_slots=20, interval_min=2, window=4)
    assert b["stats"]["window"] == 4 and b["stats"]["kernel_calls"][4] == 5
    assert_close(b, want, TOL_BF16)
    for k in ("loss", "dh0", "dc0"):  # the windows change only the weight-gradient sums
        assert (a[k] == b[k]).all() if k != "loss" else a[k] == b[k], k


@pytest.mark.parametrize("loss", ["half_sq_last", "mean_sq_all", "mean_last"])
def test_wide_rnn_bf16_losses(loss):
    """tanh RNN (G = 1, 64 units per tile), B = 50 on a 64-row tile, every loss."""
    wl = synth.get("lstm_h2048_bf16_t10000").with_(cell="rnn", batch=50, input=64, hidden=128, n_steps=9,
                                                   loss=loss, w_scale=0.125, h0_std=0.3, name="rnn_bf16_wide")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=9, slow_slots=0)
    assert a["stats"]["kernel_calls"][HADJ] == 8
    assert_close(a, want, TOL_BF16)
    for kw in (dict(fast_slots=2, slow_slots=0), dict(fast_slots=3, slow_slots=9, interval_min=2)):
        assert_bitwise(run_gpu(wl, dev, **kw), a)


@pytest.mark.parametrize("loss", ["half_sq_last", "mean_sq_all"])
def test_wide_resmlp_bf16_ragged(loss):
    """Residual MLP, B = 70 (two 64-row tiles, the second ragged), width 192."""
    wl = synth.get("resmlp_w4096_l2000_bf16").with_(batch=70, hidden=192, n_steps=9, loss=loss, w_scale=0.08,
                                                    name="resmlp_bf16_wide")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=9, slow_slots=0)
    assert a["stats"]["kernel_calls"][HADJ] == 8
    assert_close_relu(a, want, TOL_BF16)
    for kw in (dict(fast_slots=2, slow_slots=0), dict(fast_slots=2, slow_slots=9, interval_min=1)):
        assert_bitwise(run_gpu(wl, dev, **kw), a)
    c = run_gpu(wl, dev, fast_slots=9, slow_slots=0, wide=False)
    assert c["stats"]["kernel_calls"][HADJ] == 0
    say("small-batch kernels on the same inputs")
    assert_close_relu(c, want, TOL_BF16)
