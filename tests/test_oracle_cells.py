"""Pins for the float64 oracle cells and the store-all BPTT (CPU only).

  * central finite differences of the loss, for every parameter and every
    initial-state entry, on tiny shapes of each cell and each loss;
  * closed forms: an LSTM with all-zero weights and biases has i = f = o = 1/2,
    g = 0, so c_t = c_0 / 2^t and h_t = tanh(c_t) / 2; a residual MLP with
    zero weights is the identity and relu'(0) = 0 leaves dW = 0;
  * bfloat16 rounding against hand-worked ties and against an independent
    bit-level conversion;
  * any valid schedule replayed on the CPU equals store-all bit for bit
    (checkpointing changes which states are recomputed, not the result).
"""
import math

import numpy as np
import pytest

import synth
from oracle import bptt, schedule as S
from oracle.cells import Cell, round_bf16


def _tiny(kind, loss, B=2, D=3, H=4, seed=0, scale=0.7):
    rng = np.random.default_rng(seed)
    G = 4 if kind == "lstm" else 1
    if kind == "resmlp":
        Ws = {l: (rng.standard_normal((H, H)) * scale, rng.standard_normal(H) * 0.3) for l in range(32)}
        return Cell(kind, loss, B, 0, H, layer=lambda l: Ws[l]), Ws
    W = rng.standard_normal((G * H, D + H)) * scale
    b = rng.standard_normal(G * H) * 0.3
    return Cell(kind, loss, B, D, H, W=W, b=b), None


def _loss(cell, n, us, x0):
    return bptt.store_all(cell, n, lambda t: us[t], x0)["loss"]


def _fd_check(kind, loss, n, B=2, D=3, H=4):
    cell, Ws = _tiny(kind, loss, B, D, H)
    rng = np.random.default_rng(7)
    us = rng.standard_normal((n, B, D if kind != "resmlp" else 0))
    if kind == "lstm":
        x0 = (rng.standard_normal((B, H)) * 0.5, rng.standard_normal((B, H)) * 0.5)
    else:
        x0 = (rng.standard_normal((B, H)) * 0.5,)
    out = bptt.store_all(cell, n, lambda t: us[t], x0)
    eps = 1e-6

    def fd(get, set_):
        g = np.zeros_like(get())
        base = get().copy()
        for idx in np.ndindex(base.shape):
            p = base.copy(); p[idx] += eps; set_(p); lp = _loss(cell, n, us, x0)
            m = base.copy(); m[idx] -= eps; set_(m); lm = _loss(cell, n, us, x0)
            g[idx] = (lp - lm) / (2 * eps)
        set_(base)
        return g

    def close(a, b):
        scale = max(np.max(np.abs(b)), 1e-3)
        assert np.max(np.abs(a - b)) / scale < 1e-6, (np.max(np.abs(a - b)), scale)

    if kind == "resmlp":
        for l in range(n):
            def set_w(v, l=l):
                Ws[l] = (v, Ws[l][1]); cell._cache.pop(l, None)
            def set_b(v, l=l):
                Ws[l] = (Ws[l][0], v); cell._cache.pop(l, None)
            close(out["dW"][l], fd(lambda l=l: Ws[l][0], set_w))
            close(out["db"][l], fd(lambda l=l: Ws[l][1], set_b))
    else:
        close(out["dW"], fd(lambda: cell.W, lambda v: setattr(cell, "W", v)))
        close(out["db"], fd(lambda: cell.b, lambda v: setattr(cell, "b", v)))
    for i in range(len(x0)):
        def set_x(v, i=i):
            nonlocal x0
            x0 = tuple(v if j == i else x0[j] for j in range(len(x0)))
        close(out["dx0"][i], fd(lambda i=i: x0[i], set_x))


@pytest.mark.parametrize("loss", ["half_sq_last", "mean_sq_all", "mean_last"])
def test_fd_rnn(loss):
    _fd_check("rnn", loss, n=6)


@pytest.mark.parametrize("loss", ["half_sq_last", "mean_sq_all", "mean_last"])
def test_fd_lstm(loss):
    _fd_check("lstm", loss, n=5, B=2, D=2, H=3)


@pytest.mark.parametrize("loss", ["half_sq_last", "mean_sq_all", "mean_last"])
def test_fd_resmlp(loss):
    _fd_check("resmlp", loss, n=5, B=2, H=4)


def test_lstm_zero_weights_closed_form():
    B, D, H, n = 3, 2, 5, 6
    cell = Cell("lstm", "mean_last", B, D, H, W=np.zeros((4 * H, D + H)), b=np.zeros(4 * H))
    rng = np.random.default_rng(3)
    us = rng.standard_normal((n, B, D))
    c0 = rng.standard_normal((B, H))
    out = bptt.store_all(cell, n, lambda t: us[t], (np.zeros((B, H)), c0))
    cn = c0 / 2.0 ** n
    hn = 0.5 * np.tanh(cn)
    assert np.array_equal(out["states"][n][1], cn)
    np.testing.assert_allclose(out["states"][n][0], hn, rtol=1e-15, atol=0)
    assert out["loss"] == pytest.approx(float(np.mean(hn)), rel=1e-14)
    # L = mean(tanh(c0 / 2^n) / 2): dL/dc0 = sech^2(c_n) / 2^(n+1) / (B H); dL/dh0 = 0
    want = (1.0 - np.tanh(cn) ** 2) / 2.0 ** (n + 1) / (B * H)
    np.testing.assert_allclose(out["dx0"][1], want, rtol=1e-12)
    assert np.all(out["dx0"][0] == 0.0)


def test_resmlp_zero_weights_is_identity():
    B, w, n = 2, 6, 4
    cell = Cell("resmlp", "half_sq_last", B, 0, w, layer=lambda l: (np.zeros((w, w)), np.zeros(w)))
    y0 = np.random.default_rng(1).standard_normal((B, w))
    out = bptt.store_all(cell, n, lambda t: np.zeros((B, 0)), (y0,))
    assert out["loss"] == pytest.approx(0.5 * float(np.sum(y0 * y0)), rel=1e-15)
    assert np.array_equal(out["dx0"][0], y0)
    assert all(np.all(out["dW"][l] == 0) for l in range(n))   # relu'(0) = 0


def test_rnn_single_step_small_weight_limit():
    # with W -> 0: h1 = tanh(b), L = 1/2 |h1|^2, dL/db = sum_batch h1 (1 - h1^2)
    B, D, H = 3, 2, 4
    b = np.array([0.1, -0.4, 0.7, 0.0])
    cell = Cell("rnn", "half_sq_last", B, D, H, W=np.zeros((H, D + H)), b=b)
    out = bptt.store_all(cell, 1, lambda t: np.ones((B, D)), (np.zeros((B, H)),))
    h1 = np.tanh(b)
    np.testing.assert_allclose(out["db"], B * h1 * (1 - h1 ** 2), rtol=1e-14)
    assert out["loss"] == pytest.approx(0.5 * B * float(np.sum(h1 ** 2)), rel=1e-14)


def test_round_bf16_ties_and_bits():
    one = 1.0
    assert round_bf16(np.array(one + 2.0 ** -8)) == 1.0                      # tie -> even
    assert round_bf16(np.array(one + 3 * 2.0 ** -8)) == one + 2.0 ** -6      # tie -> even (up)
    assert round_bf16(np.array(one + 2.0 ** -8 + 2.0 ** -20)) == one + 2.0 ** -7
    assert round_bf16(np.array(-3.0)) == -3.0
    x = np.random.default_rng(5).standard_normal(100000).astype(np.float32)
    ref = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(x)).astype(np.float64)
    assert np.array_equal(round_bf16(x.astype(np.float64)), ref)


def _replay_cases():
    return [("rnn", "half_sq_last", 13, 3, 0, 0), ("rnn", "mean_sq_all", 10, 3, 5, 2),
            ("lstm", "mean_sq_all", 12, 3, 100, 3), ("lstm", "mean_last", 17, 2, 16, 1),
            ("lstm", "half_sq_last", 9, 1, 0, 0), ("resmlp", "half_sq_last", 11, 3, 4, 2),
            ("lstm", "mean_sq_all", 23, 4, 7, 2)]


@pytest.mark.parametrize("case", _replay_cases(), ids=lambda c: "-".join(map(str, c)))
def test_replay_equals_store_all_bitwise(case):
    kind, loss, n, s, H, I = case
    cell, _ = _tiny(kind, loss, B=3, D=2, H=5, seed=11)
    rng = np.random.default_rng(2)
    us = rng.standard_normal((n, 3, 2 if kind != "resmlp" else 0))
    x0 = tuple(rng.standard_normal((3, 5)) * 0.3 for _ in range(2 if kind == "lstm" else 1))
    ref = bptt.store_all(cell, n, lambda t: us[t], x0)
    head, acts = S.schedule(n, s, H, I)
    got = S.replay(cell, n, lambda t: us[t], x0, acts)
    assert got["loss"] == ref["loss"]
    if kind == "resmlp":
        assert all(np.array_equal(got["dW"][l], ref["dW"][l]) for l in range(n))
    else:
        assert np.array_equal(got["dW"], ref["dW"]) and np.array_equal(got["db"], ref["db"])
    assert all(np.array_equal(a, b) for a, b in zip(got["dx0"], ref["dx0"]))


@pytest.mark.parametrize("kind,starts", [("lstm", [0, 1, 4, 5, 9, 13]), ("rnn", [0, 6]), ("resmlp", [0, 2, 3, 10])])
def test_replay_over_chosen_starts_equals_store_all_bitwise(kind, starts):
    """Intervals of unequal length, as stores decided during the sweep make them."""
    n, s = 15, 3
    cell, _ = _tiny(kind, "mean_sq_all", B=3, D=2, H=5, seed=5)
    rng = np.random.default_rng(8)
    us = rng.standard_normal((n, 3, 2 if kind != "resmlp" else 0))
    x0 = tuple(rng.standard_normal((3, 5)) * 0.3 for _ in range(2 if kind == "lstm" else 1))
    ref = bptt.store_all(cell, n, lambda t: us[t], x0)
    head, acts = S.schedule_from_starts(n, s, 10, starts)
    got = S.replay(cell, n, lambda t: us[t], x0, acts)
    assert got["loss"] == ref["loss"]
    if kind == "resmlp":
        assert all(np.array_equal(got["dW"][l], ref["dW"][l]) for l in range(n))
    else:
        assert np.array_equal(got["dW"], ref["dW"]) and np.array_equal(got["db"], ref["db"])
    assert all(np.array_equal(a, b) for a, b in zip(got["dx0"], ref["dx0"]))


def test_replay_detects_a_wrong_restore():
    # restoring from the wrong slot must change the result (and fail the checker)
    cell, _ = _tiny("lstm", "mean_sq_all", B=2, D=2, H=3, seed=4)
    n = 10
    us = np.random.default_rng(9).standard_normal((n, 2, 2))
    x0 = (np.zeros((2, 3)), np.zeros((2, 3)))
    ref = bptt.store_all(cell, n, lambda t: us[t], x0)
    head, acts = S.schedule(n, 3)
    i = acts.index(("R", 2, 7))
    bad = acts[:i] + [("R", 1, 7)] + acts[i + 1:]      # slot 1 holds x_4, not x_7
    with pytest.raises(AssertionError):
        S.check(n, 3, 0, bad)
    got = S.replay(cell, n, lambda t: us[t], x0, bad)
    assert not np.array_equal(got["dW"], ref["dW"])


def test_workload_loss_scale_small_rnn():
    # the 64-wide RNN workload at its real shape: forward stays bounded, loss finite
    wl = synth.get("rnn_h64_t128")
    W, b = synth.params(wl)
    cell = bptt.cell_for(wl, (W, b))
    xs = synth.x_slice(wl, 0, wl.n_steps)
    h0 = synth.initial_state(wl)["h"]
    out = bptt.store_all(cell, wl.n_steps, lambda t: xs[t], (h0,))
    assert math.isfinite(out["loss"]) and 0 < out["loss"] < 0.5 * wl.batch * wl.hidden
    assert np.all(np.abs(out["states"][-1][0]) < 1)


@pytest.mark.parametrize("loss", ["half_sq_last", "mean_sq_all", "mean_last"])
def test_fd_mlp_of_different_widths(loss):
    """Central finite differences for the MLP whose layers change width (states
    of different sizes): every weight, bias and initial-state entry."""
    widths = [4, 6, 3, 5, 2, 6]
    n, B = len(widths) - 1, 2
    rng = np.random.default_rng(11)
    Ws = {l: [rng.standard_normal((widths[l + 1], widths[l])) * 0.8, rng.standard_normal(widths[l + 1]) * 0.3]
          for l in range(n)}
    cell = Cell("mlp", loss, B, 0, max(widths), layer=lambda l: tuple(Ws[l]))
    y0 = rng.standard_normal((B, widths[0]))
    zero = np.zeros((B, 0))
    run = lambda: bptt.store_all(cell, n, lambda t: zero, (y0,))
    out = run()
    eps = 1e-6

    def fd(arr):
        g = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            keep = arr[idx]
            arr[idx] = keep + eps; cell._cache.clear(); lp = run()["loss"]
            arr[idx] = keep - eps; cell._cache.clear(); lm = run()["loss"]
            arr[idx] = keep
            g[idx] = (lp - lm) / (2 * eps)
        cell._cache.clear()
        return g

    def close(a, b):
        scale = max(np.max(np.abs(b)), 1e-3)
        assert np.max(np.abs(a - b)) / scale < 1e-6, (np.max(np.abs(a - b)), scale)

    for l in range(n):
        close(out["dW"][l], fd(Ws[l][0]))
        close(out["db"][l], fd(Ws[l][1]))
    close(out["dx0"][0], fd(y0))
    assert out["dW"][2].shape == (widths[3], widths[2])
