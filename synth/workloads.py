"""Workload shapes and seeded input generators (no method arithmetic here).

Five recurrent workloads of the long-sequence shape the paper studies
(Section 5 uses an LSTM whose depth in time is varied).  Each names its cell,
operand precision, sizes, step count n, fast (HBM) checkpoint slots s and
slow-tier budget, the loss, and the distributions its inputs are drawn from.

Conventions (readings written down once, here):
  * N(0, v) names a variance v, so an initial hidden state drawn from
    N(0, 0.1) has standard deviation sqrt(0.1).
  * Weights are one matrix W[G*H][D+H] acting on the concatenation [x | h]
    (input columns first).  For the LSTM, G = 4 gate blocks in the order
    i, f, g, o; for the tanh RNN, G = 1.  Biases b[G*H].
  * The residual MLP treats depth as the sequence: layer l has W_l[w][w]
    (output x input) and b_l[w]; there is no per-step input.
  * Initial states and biases that are not stated are zero, except the
    forget-gate bias of the 512-wide LSTM (1.0).
  * bf16 workloads draw float32 values and round them to bfloat16 (round to
    nearest even); the arrays returned here hold those bf16 values in
    float32 so both sides see the same numbers.
  * The residual MLP's stated N(0, 0.02^2) weights make activations grow by
    a factor ~1.8 per layer at width 4096, so 2000 layers overflow to inf in
    any float format with an 8-bit exponent.  The workload therefore scales
    the standard deviation by 1/sqrt(L) (``w_std = 0.02 / sqrt(2000)``);
    kernel timing does not depend on the values.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

BASE_SEED = 1806_01117

# stream ids inside one workload's SeedSequence
_S_X, _S_W, _S_X0, _S_LAYER = 1, 2, 3, 4


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    cell: str            # "rnn" | "lstm" | "resmlp"
    dtype: str           # operand dtype: "f32" | "bf16"; accumulation, cell state and grads fp32
    batch: int
    input: int           # D (0 for resmlp)
    hidden: int          # H (or MLP width w)
    n_steps: int         # n
    fast_slots: int      # s, HBM checkpoint slots
    slow_slots: int      # host slots; 0 = no slow tier, -1 = as many as the schedule can use (n)
    loss: str            # "half_sq_last" | "mean_sq_all" | "mean_last"
    x_std: float = 1.0
    w_dist: str = "uniform"   # "uniform" (+-w_scale) | "normal" (std w_scale)
    w_scale: float = 0.0
    forget_bias: float = 0.0
    h0_std: float = 0.0       # rnn h0 / resmlp y0 standard deviation
    seed_index: int = 0
    widths: tuple = ()        # "mlp": layer widths cycled from w_0 (empty: all = hidden)

    @property
    def gates(self) -> int:
        return 4 if self.cell == "lstm" else 1

    @property
    def seed(self) -> int:
        return BASE_SEED + self.seed_index

    @property
    def host_slots(self) -> int:
        return self.n_steps if self.slow_slots < 0 else self.slow_slots

    def layer_widths(self) -> list[int] | None:
        """w_0 .. w_n of the MLP of layers of different widths (the pattern
        repeated), or None for the other cells."""
        if self.cell != "mlp":
            return None
        pat = self.widths or (self.hidden,)
        return [int(pat[t % len(pat)]) for t in range(self.n_steps + 1)]

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: dict[str, Workload] = {w.name: w for w in [
    # vanilla tanh RNN h' = tanh(W h + U x + b)
    Workload("rnn_h64_t128", "rnn", "f32", batch=4, input=32, hidden=64, n_steps=128,
             fast_slots=4, slow_slots=0, loss="half_sq_last",
             w_dist="uniform", w_scale=1.0 / math.sqrt(64), h0_std=math.sqrt(0.1), seed_index=1),
    # LSTM, fused [x;h] gate GEMM, fp32, 10 HBM slots + unlimited pinned host tier
    Workload("lstm_h512_t1000", "lstm", "f32", batch=64, input=256, hidden=512, n_steps=1000,
             fast_slots=10, slow_slots=-1, loss="mean_sq_all",
             w_dist="uniform", w_scale=1.0 / math.sqrt(512), forget_bias=1.0, seed_index=2),
    # LSTM, bf16 operands and stored h, fp32 accumulation and cell state
    Workload("lstm_h2048_bf16_t10000", "lstm", "bf16", batch=128, input=1024, hidden=2048,
             n_steps=10000, fast_slots=32, slow_slots=-1, loss="mean_last",
             w_dist="uniform", w_scale=1.0 / math.sqrt(2048), seed_index=3),
    # residual MLP, depth as the sequence, bf16 with fp32 accumulation
    Workload("resmlp_w4096_l2000_bf16", "resmlp", "bf16", batch=256, input=0, hidden=4096,
             n_steps=2000, fast_slots=16, slow_slots=-1, loss="half_sq_last",
             w_dist="normal", w_scale=0.02 / math.sqrt(2000), h0_std=1.0, seed_index=4),
    # MLP of layers of different widths (as before and after a pooling layer):
    # states of 1, 1/2 and 1/4 of the largest size, fp32, He-scaled weights
    Workload("mlp_widths_l2000", "mlp", "f32", batch=256, input=0, hidden=1024, n_steps=2000,
             fast_slots=16, slow_slots=-1, loss="half_sq_last",
             w_dist="he", w_scale=1.0, h0_std=1.0, seed_index=6, widths=(1024, 512, 256, 512)),
    # offload-stress LSTM: 16 MiB of fp32 state per step, 20000 steps
    Workload("lstm_h4096_t20000", "lstm", "f32", batch=512, input=1024, hidden=4096,
             n_steps=20000, fast_slots=64, slow_slots=-1, loss="mean_last",
             w_dist="uniform", w_scale=1.0 / 64.0, seed_index=5),
]}


def get(name: str) -> Workload:
    return WORKLOADS[name]


# ---------------------------------------------------------------------------
# bf16 input preparation (round to nearest even); not used by the method.

def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _as_operand(wl: Workload, a: np.ndarray) -> np.ndarray:
    a = np.asarray(a, dtype=np.float32)
    if wl.dtype == "bf16":
        return bf16_bits_to_f32(f32_to_bf16_bits(a))
    return a


def _rng(wl: Workload, *key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([wl.seed, *key]))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


# ---------------------------------------------------------------------------
# generators

def x_slice(wl: Workload, t0: int, t1: int) -> np.ndarray:
    """Per-step inputs x[t0:t1] as float32 [t1-t0][B][D]; x_t is seeded by t."""
    if wl.cell == "resmlp" or wl.input == 0:
        return np.zeros((t1 - t0, wl.batch, 0), np.float32)
    out = np.empty((t1 - t0, wl.batch, wl.input), np.float32)

    def fill(t: int) -> None:
        out[t - t0] = _rng(wl, _S_X, t).standard_normal((wl.batch, wl.input), dtype=np.float32) * np.float32(wl.x_std)

    steps = range(t0, t1)
    if (t1 - t0) * wl.batch * wl.input > (1 << 22):
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, steps))
    else:
        for t in steps:
            fill(t)
    return _as_operand(wl, out)


def _draw_w(wl: Workload, rng: np.random.Generator, shape) -> np.ndarray:
    if wl.w_dist == "he":  # N(0, 2 / fan_in) times w_scale
        return (rng.standard_normal(shape) * (wl.w_scale * math.sqrt(2.0 / shape[1]))).astype(np.float32)
    if wl.w_dist == "uniform":
        return (rng.random(shape) * (2.0 * wl.w_scale) - wl.w_scale).astype(np.float32)
    return (rng.standard_normal(shape) * wl.w_scale).astype(np.float32)


def params(wl: Workload) -> tuple[np.ndarray, np.ndarray]:
    """(W[G*H][D+H], b[G*H]) as float32 for the rnn and lstm cells."""
    assert wl.cell in ("rnn", "lstm")
    G, H, D = wl.gates, wl.hidden, wl.input
    W = _as_operand(wl, _draw_w(wl, _rng(wl, _S_W), (G * H, D + H)))
    b = np.zeros(G * H, np.float32)
    if wl.cell == "lstm":
        b[H:2 * H] = wl.forget_bias
    return W, b


def layer_params(wl: Workload, layer: int) -> tuple[np.ndarray, np.ndarray]:
    """(W_l, b_l) as float32 for one layer, seeded by l: [w][w] and [w] for
    the residual MLP, [w_{l+1}][w_l] and [w_{l+1}] for the MLP of layers of
    different widths."""
    assert wl.cell in ("resmlp", "mlp")
    if wl.cell == "mlp":
        ws = wl.layer_widths()
        shape = (ws[layer + 1], ws[layer])
    else:
        shape = (wl.hidden, wl.hidden)
    W = _as_operand(wl, _draw_w(wl, _rng(wl, _S_LAYER, layer), shape))
    return W, np.zeros(shape[0], np.float32)


def initial_state(wl: Workload) -> dict[str, np.ndarray]:
    B, H = wl.batch, wl.hidden
    if wl.cell == "rnn":
        h0 = _rng(wl, _S_X0).standard_normal((B, H)) * wl.h0_std
        return {"h": _as_operand(wl, h0)}
    if wl.cell == "lstm":
        return {"h": np.zeros((B, H), np.float32), "c": np.zeros((B, H), np.float32)}
    w0 = wl.layer_widths()[0] if wl.cell == "mlp" else H
    y0 = _rng(wl, _S_X0).standard_normal((B, w0)) * wl.h0_std
    return {"h": _as_operand(wl, y0)}
