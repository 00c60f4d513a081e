"""Conventional backpropagation through time, storing every state (float64).

TEST INFRASTRUCTURE ONLY (see the package docstring).

This is the plain definition that every checkpointing schedule must
reproduce (Section 1.1; Fig. 1: all states stored, memory peak at the end of
the forward pass; Section 3: T_inf = n T_A + n T_B):

    x_{t+1} = f(x_t, u_t)                       t = 0 .. n-1
    L = sum_t loss_t(x_t)
    xbar_n = dL/dx_n
    xbar_t = (df/dx_t)^T xbar_{t+1} + dL/dx_t   t = n-1 .. 0
    dtheta = sum_t (df/dtheta_t)^T xbar_{t+1}

Gradient contributions are added in descending t and the loss terms are
summed in ascending t, in both the store-all driver and the schedule
replayer, so the two agree bit for bit when they feed the same states.
"""
from __future__ import annotations

import numpy as np

from .cells import Cell


class Reverse:
    """Accumulates the reverse sweep: one adjoint step per t, in order n-1 .. 0."""

    def __init__(self, cell: Cell, n: int, u_of):
        self.cell, self.n, self.u_of = cell, n, u_of
        self.terms = np.zeros(n + 1)
        self.next_t = n - 1
        self.bar = None
        if cell.kind in ("resmlp", "mlp"):
            self.dW, self.db = {}, {}
        else:
            self.dW = np.zeros_like(cell.W)
            self.db = np.zeros_like(cell.b)

    def adjoint(self, t: int, x_t: tuple, x_next: tuple | None = None) -> None:
        if t != self.next_t:
            raise RuntimeError(f"adjoint of step {t} out of order (expected {self.next_t})")
        cell, n = self.cell, self.n
        u = self.u_of(t)
        if x_next is None:
            x_next = cell.step(t, x_t, u)
        self.terms[t + 1] = cell.loss_term(t + 1, n, x_next)
        bar = [b.copy() for b in (self.bar if self.bar is not None else cell.zero_bar(x_next))]
        s = cell.seed(t + 1, n, x_next)
        if s is not None:
            bar[0] = bar[0] + s
        bar_t, dW_t, db_t = cell.adjoint(t, x_t, u, tuple(bar))
        if cell.kind in ("resmlp", "mlp"):
            self.dW[t], self.db[t] = dW_t, db_t
        else:
            self.dW += dW_t
            self.db += db_t
        self.bar = bar_t
        self.next_t -= 1

    def result(self) -> dict:
        if self.next_t != -1:
            raise RuntimeError("reverse sweep incomplete")
        loss = 0.0
        for v in self.terms:          # ascending t
            loss += v
        out = {"loss": loss, "dW": self.dW, "db": self.db, "dx0": self.bar}
        return out


def store_all(cell: Cell, n: int, u_of, x0: tuple) -> dict:
    """Forward sweep storing x_0 .. x_n, then the reverse sweep.

    u_of(t) returns the step input u_t as an array [B][D]; x0 is the initial
    state tuple.  Returns loss, dW, db (dicts per layer for the residual MLP)
    and dx0 (a tuple like x0).
    """
    states = [tuple(np.asarray(s, np.float64) for s in x0)]
    for t in range(n):
        states.append(cell.step(t, states[t], u_of(t)))
    rev = Reverse(cell, n, u_of)
    for t in range(n - 1, -1, -1):
        rev.adjoint(t, states[t], states[t + 1])
    out = rev.result()
    out["states"] = states
    return out


def cell_for(wl, params=None, layer=None) -> Cell:
    """Build an oracle cell for a ``synth`` workload (parameters as float32 arrays)."""
    bf16 = wl.dtype == "bf16"
    if wl.cell in ("resmlp", "mlp"):
        return Cell(wl.cell, wl.loss, wl.batch, 0, wl.hidden, bf16, layer=layer)
    W, b = params
    return Cell(wl.cell, wl.loss, wl.batch, wl.input, wl.hidden, bf16, W=W, b=b)
