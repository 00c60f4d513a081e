"""Float64 recurrent cells: forward step, adjoint step, loss and its seeds.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's test network is a "simple vanilla LSTM" (Section 5); the cells
and losses here are the three workload cells.  Each step maps the state x_t
and the step input u_t to x_{t+1}; the adjoint step maps (x_t, u_t, xbar_{t+1})
to xbar_t and the step's parameter-gradient contribution, by the chain rule:

    xbar_t = (d f / d x_t)^T xbar_{t+1}   (+ dL/dx_t, added by the caller)
    dtheta += (d f / d theta)^T xbar_{t+1}

Layouts (batch rows, row-major):
  state h[B][H] (and c[B][H] for the LSTM), u[B][D],
  W[G*H][D+H] acting on [u | h] (input columns first), b[G*H];
  LSTM gate blocks of W in the order i, f, g, o;
  residual MLP: layer l has W_l[w][w] (output x input), b_l[w];
  MLP of layers of different widths (states of different sizes, the case the
  paper's Sections 1.1 and 6 set beside Revolve's uniform states): layer l
  maps y_l[B][w_l] to y_{l+1} = relu(y_l W_l^T + b_l), W_l[w_{l+1}][w_l].

Precision: everything is float64.  For bf16 workloads the stored forward
state h (or y) is rounded to bfloat16 after every step, as the GPU stores it;
the cell state c and every adjoint quantity stay float64.
"""
from __future__ import annotations

import numpy as np


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 value (8 significant bits, ties to even)."""
    m, e = np.frexp(np.asarray(x, dtype=np.float64))
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


class Cell:
    """One recurrent cell with its parameters (float64)."""

    def __init__(self, kind: str, loss: str, batch: int, input: int, hidden: int,
                 bf16: bool = False, W=None, b=None, layer=None):
        self.kind, self.loss, self.bf16 = kind, loss, bf16
        self.B, self.D, self.H = batch, input, hidden
        self.G = 4 if kind == "lstm" else 1
        if kind in ("resmlp", "mlp"):
            self._layer = layer          # callable l -> (W_l, b_l)
            self._cache = {}
        else:
            self.W = np.asarray(W, np.float64)
            self.b = np.asarray(b, np.float64)
            assert self.W.shape == (self.G * hidden, input + hidden)

    # -- parameters -----------------------------------------------------
    def layer(self, l: int):
        if l not in self._cache:
            W, b = self._layer(l)
            self._cache[l] = (np.asarray(W, np.float64), np.asarray(b, np.float64))
        return self._cache[l]

    def _store(self, h):
        return round_bf16(h) if self.bf16 else h

    # -- forward step x_t -> x_{t+1} ---------------------------------------
    def step(self, t: int, state: tuple, u: np.ndarray) -> tuple:
        if self.kind == "rnn":
            (h,) = state
            z = np.concatenate([u, h], axis=1) @ self.W.T + self.b
            return (self._store(np.tanh(z)),)
        if self.kind == "lstm":
            h, c = state
            H = self.H
            z = np.concatenate([u, h], axis=1) @ self.W.T + self.b
            i, f = _sigmoid(z[:, :H]), _sigmoid(z[:, H:2 * H])
            g, o = np.tanh(z[:, 2 * H:3 * H]), _sigmoid(z[:, 3 * H:])
            c1 = f * c + i * g
            return (self._store(o * np.tanh(c1)), c1)
        (y,) = state
        W, b = self.layer(t)
        z = y @ W.T + b
        if self.kind == "mlp":
            return (self._store(np.maximum(z, 0.0)),)
        return (self._store(y + np.maximum(z, 0.0)),)

    # -- adjoint step (x_t, u_t, xbar_{t+1}) -> (xbar_t, dW_t, db_t) --------
    def adjoint(self, t: int, state: tuple, u: np.ndarray, bar_next: tuple):
        if self.kind == "rnn":
            (h,) = state
            (hb1,) = bar_next
            a_in = np.concatenate([u, h], axis=1)
            h1 = np.tanh(a_in @ self.W.T + self.b)
            a = hb1 * (1.0 - h1 * h1)                 # d tanh
            hb = a @ self.W[:, self.D:]
            return (hb,), a.T @ a_in, a.sum(axis=0)
        if self.kind == "lstm":
            h, c = state
            hb1, cb1 = bar_next
            H = self.H
            a_in = np.concatenate([u, h], axis=1)
            z = a_in @ self.W.T + self.b
            i, f = _sigmoid(z[:, :H]), _sigmoid(z[:, H:2 * H])
            g, o = np.tanh(z[:, 2 * H:3 * H]), _sigmoid(z[:, 3 * H:])
            c1 = f * c + i * g
            tc = np.tanh(c1)
            ob = hb1 * tc                                  # dL/do
            ch = cb1 + hb1 * o * (1.0 - tc * tc)           # total dL/dc_{t+1}
            zb = np.concatenate([ch * g * i * (1.0 - i),   # through sigma'(z_i)
                                 ch * c * f * (1.0 - f),   # through sigma'(z_f)
                                 ch * i * (1.0 - g * g),   # through tanh'(z_g)
                                 ob * o * (1.0 - o)], axis=1)
            hb = zb @ self.W[:, self.D:]
            return (hb, ch * f), zb.T @ a_in, zb.sum(axis=0)
        (y,) = state
        (yb1,) = bar_next
        W, b = self.layer(t)
        z = y @ W.T + b
        zb = yb1 * (z > 0.0)                               # relu'(0) = 0
        if self.kind == "mlp":                             # no identity path
            return (zb @ W,), zb.T @ y, zb.sum(axis=0)
        return (yb1 + zb @ W,), zb.T @ y, zb.sum(axis=0)

    # -- loss ------------------------------------------------------------
    # half_sq_last: L = 1/2 sum(h_n^2); mean_last: L = mean(h_n);
    # mean_sq_all: L = sum_{t=1..n} mean(h_t^2)  (the given h_0 excluded).
    def loss_term(self, t: int, n: int, state: tuple) -> float:
        h = state[0]
        if self.loss == "mean_sq_all":
            return float(np.mean(h * h)) if t >= 1 else 0.0
        if t != n:
            return 0.0
        if self.loss == "half_sq_last":
            return float(0.5 * np.sum(h * h))
        if self.loss == "mean_last":
            return float(np.mean(h))
        raise ValueError(self.loss)

    def seed(self, t: int, n: int, state: tuple):
        """dL/dh_t, or None when the loss does not read h_t."""
        h = state[0]
        if self.loss == "mean_sq_all":
            return 2.0 * h / h.size if t >= 1 else None
        if t != n:
            return None
        if self.loss == "half_sq_last":
            return h.copy()
        if self.loss == "mean_last":
            return np.full_like(h, 1.0 / h.size)
        raise ValueError(self.loss)

    def zero_bar(self, state: tuple) -> tuple:
        return tuple(np.zeros_like(s) for s in state)
