"""Python face of the C ABI: torch tensors in, gradients out.

Only argument marshalling lives here.  Every step of the forward and reverse
pass, the schedule and the checkpoint tiers run in libambptt.so; if that
library is missing this module raises instead of computing anything.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import sys

from . import _lib
from ._lib import check, load


def version() -> str:
    return load().ambptt_version().decode()


def revolve_advances(n: int, s: int) -> int:
    v = load().ambptt_revolve_advances(n, s)
    if v < 0:
        raise ValueError("need n >= 1 and s >= 1")
    return int(v)


def schedule_evals(n: int, s: int, H: int = 0, interval_min: int = 0) -> tuple[int, int, str]:
    """(forward evaluations, interval, mode) of the schedule the library runs."""
    I, mode = C.c_int32(), C.c_int32()
    v = load().ambptt_schedule_evals(n, s, H, interval_min, C.byref(I), C.byref(mode))
    if v < 0:
        raise ValueError("bad schedule arguments")
    return int(v), int(I.value), ("async" if mode.value else "revolve")


def schedule_text(n: int, s: int, H: int = 0, interval_min: int = 0) -> str:
    L = load()
    need = C.c_size_t(0)
    L.ambptt_schedule_text(n, s, H, interval_min, None, 0, C.byref(need))
    if need.value == 0:
        check(L.ambptt_schedule_text(n, s, H, interval_min, None, 0, C.byref(need)))
    buf = C.create_string_buffer(need.value)
    check(L.ambptt_schedule_text(n, s, H, interval_min, buf, need.value, C.byref(need)))
    return buf.value.decode()


def _text(call) -> str:
    """A canonical-text call: size query, then the text."""
    need = C.c_size_t(0)
    call(None, 0, C.byref(need))
    if need.value == 0:
        check(call(None, 0, C.byref(need)))
    buf = C.create_string_buffer(need.value)
    check(call(buf, need.value, C.byref(need)))
    return buf.value.decode()


def schedule_text_starts(n: int, s: int, H: int, starts, costs=None) -> str:
    """Canonical text of the two-level schedule over interval starts chosen
    during the sweep (ambptt_schedule_text_starts), with every reversal split
    for the step costs when they are given (ambptt_schedule_text_starts_costs)."""
    L = load()
    arr = (C.c_int64 * len(starts))(*[int(t) for t in starts])
    if costs is None:
        return _text(lambda buf, cap, need: L.ambptt_schedule_text_starts(n, s, H, arr, len(starts), buf, cap, need))
    if len(costs) != n:
        raise ValueError("need one cost per step")
    cv = (C.c_double * n)(*[float(c) for c in costs])
    return _text(lambda buf, cap, need: L.ambptt_schedule_text_starts_costs(n, s, H, arr, len(starts), cv, buf, cap,
                                                                           need))


def interval_from_timings(t_a_us: float, t_t_us: float, s: int, rule: int = 1) -> int:
    """I_min for measured T_A and T_T (ambptt_interval_from_timings)."""
    v = load().ambptt_interval_from_timings(float(t_a_us), float(t_t_us), s, rule)
    if v < 0:
        raise ValueError("bad interval arguments")
    return int(v)


def schedule_text_costs(n: int, s: int, costs, H: int = 0, interval_min: int = 0) -> str:
    """Canonical text of the schedule split for unequal step costs
    (ambptt_schedule_text_costs)."""
    L = load()
    arr = (C.c_double * len(costs))(*[float(c) for c in costs])
    return _text(lambda buf, cap, need: L.ambptt_schedule_text_costs(n, s, H, interval_min, arr, buf, cap, need))


def schedule_text_sized(n: int, s: int, sizes, H: int = 0, interval_min: int = 0, costs=None) -> str:
    """Canonical text of the schedule for states of different sizes
    (ambptt_schedule_text_sized): sizes[0..n] in units of a common granule."""
    L = load()
    za = (C.c_int64 * len(sizes))(*[int(v) for v in sizes])
    ca = (C.c_double * len(costs))(*[float(c) for c in costs]) if costs is not None else None
    return _text(lambda buf, cap, need: L.ambptt_schedule_text_sized(n, s, H, interval_min, za, ca, buf, cap, need))


def schedule_text_online(n: int, s: int, H: int = 0, interval_min: int = 0) -> str:
    """Canonical text of the online checkpointing schedule for n steps
    (ambptt_schedule_text_online)."""
    L = load()
    return _text(lambda buf, cap, need: L.ambptt_schedule_text_online(n, s, H, interval_min, buf, cap, need))


def resident_program(n: int, s: int, H: int = 0, interval_min: int = 0, elide_prefetch: bool = True,
                     online: bool = False):
    """The resident whole-pass kernel's program for a schedule (the online one
    when `online`), as a list of (op, y, z, w) tuples (see
    ambptt_resident_program in include/ambptt.h)."""
    L = load()
    flags = int(elide_prefetch) | (2 if online else 0)
    need = C.c_size_t(0)
    L.ambptt_resident_program(n, s, H, interval_min, flags, None, 0, C.byref(need))
    if need.value == 0:
        check(L.ambptt_resident_program(n, s, H, interval_min, flags, None, 0, C.byref(need)))
    buf = (C.c_int32 * (4 * need.value))()
    check(L.ambptt_resident_program(n, s, H, interval_min, flags, buf, need.value, C.byref(need)))
    return [tuple(buf[4 * i:4 * i + 4]) for i in range(need.value)]


@dataclasses.dataclass
class ProblemSpec:
    cell: str             # "rnn" | "lstm" | "resmlp" | "mlp"
    dtype: str            # "f32" | "bf16"
    loss: str             # "half_sq_last" | "mean_sq_all" | "mean_last"
    batch: int
    input: int
    hidden: int
    n_steps: int
    fast_slots: int
    slow_slots: int = 0
    interval_min: int = 0
    widths: tuple | None = None  # "mlp": layer widths w_0 .. w_n (None: all = hidden)

    @classmethod
    def from_workload(cls, wl, **kw) -> "ProblemSpec":
        d = dict(cell=wl.cell, dtype=wl.dtype, loss=wl.loss, batch=wl.batch, input=wl.input,
                 hidden=wl.hidden, n_steps=wl.n_steps, fast_slots=wl.fast_slots,
                 slow_slots=wl.host_slots, interval_min=0,
                 widths=tuple(getattr(wl, "layer_widths", lambda: None)() or ()) or None)
        d.update(kw)
        return cls(**d)

    def c(self) -> _lib.Problem:
        return _lib.Problem(_lib.CELL[self.cell], _lib.DTYPE[self.dtype], _lib.LOSS[self.loss],
                            self.batch, self.input, self.hidden, self.n_steps, self.fast_slots,
                            self.interval_min, self.slow_slots)

    @property
    def gates(self) -> int:
        return 4 if self.cell == "lstm" else 1


def query(spec: ProblemSpec) -> tuple[int, int, int]:
    """(state stride, slot pool bytes, workspace bytes)."""
    a, b, c = C.c_size_t(), C.c_size_t(), C.c_size_t()
    p = spec.c()
    check(load().ambptt_query(C.byref(p), C.byref(a), C.byref(b), C.byref(c)))
    return a.value, b.value, c.value


def _ptr(t) -> C.c_void_p:
    return C.c_void_p(t.data_ptr()) if t is not None else C.c_void_p(0)


class Runner:
    """One context: an HBM slot pool and workspace (torch-allocated), the host tier and copy stream."""

    def __init__(self, spec: ProblemSpec, device=None, stream=None):
        import torch

        self.torch = torch
        self.spec = spec
        self.L = load()
        self.state_bytes, pool, ws = query(spec)
        self.device = torch.device(device if device is not None else "cuda")
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.pool = torch.empty(max(pool, 256), dtype=torch.uint8, device=self.device)
        self.ws = torch.empty(max(ws, 256), dtype=torch.uint8, device=self.device)
        self._p = spec.c()
        ctx = C.c_void_p()
        check(self.L.ambptt_create(C.byref(self._p), C.c_void_p(self.stream.cuda_stream), C.byref(ctx)))
        self.ctx = ctx
        check(self.L.ambptt_bind(ctx, _ptr(self.pool), self.pool.numel(), _ptr(self.ws), self.ws.numel()))
        if spec.cell == "mlp" and spec.widths:
            w = (C.c_int32 * len(spec.widths))(*[int(v) for v in spec.widths])
            check(self.L.ambptt_set_widths(ctx, w, len(spec.widths)))

    # -- checks (shapes, dtypes, device, contiguity) -------------------------
    def _check(self, name, t, shape, dtype):
        torch = self.torch
        if t is None:
            raise ValueError(f"{name} is required")
        if tuple(t.shape) != tuple(shape) or t.dtype != dtype or not t.is_contiguous() or t.device.type != "cuda":
            raise ValueError(f"{name}: want contiguous cuda {dtype} {tuple(shape)}, got "
                             f"{t.device} {t.dtype} {tuple(t.shape)}")

    def _inputs(self, x, W, b, h0, c0):
        torch, s = self.torch, self.spec
        op = torch.float32 if s.dtype == "f32" else torch.bfloat16
        G, B, D, H, n = s.gates, s.batch, s.input, s.hidden, s.n_steps
        if s.cell == "resmlp":
            self._check("W", W, (n, H, H), op)
            self._check("b", b, (n, H), torch.float32)
        elif s.cell == "mlp":
            w = s.widths or (H,) * (n + 1)
            self._check("W", W, (sum(w[l + 1] * w[l] for l in range(n)),), op)
            self._check("b", b, (sum(w[1:]),), torch.float32)
            self._check("h0", h0, (B, w[0]), op)
            return x, W, b, h0, None
        else:
            self._check("x", x, (n, B, D), op)
            self._check("W", W, (G * H, D + H), op)
            self._check("b", b, (G * H,), torch.float32)
        self._check("h0", h0, (B, H), op)
        if s.cell == "lstm":
            self._check("c0", c0, (B, H), torch.float32)
        return x, W, b, h0, (c0 if s.cell == "lstm" else None)

    def set(self, key: str, value: int) -> None:
        check(self.L.ambptt_set_int(self.ctx, key.encode(), int(value)))

    def calibrate(self, x, W, b, h0, c0=None) -> tuple[int, float, float]:
        x, W, b, h0, c0 = self._inputs(x, W, b, h0, c0)
        I, ta, tt = C.c_int32(), C.c_double(), C.c_double()
        check(self.L.ambptt_calibrate(self.ctx, _ptr(x), _ptr(W), _ptr(b), _ptr(h0), _ptr(c0),
                                      C.byref(I), C.byref(ta), C.byref(tt)))
        return int(I.value), float(ta.value), float(tt.value)

    def run(self, x, W, b, h0, c0=None, out: dict | None = None) -> dict:
        return self._run(self.L.ambptt_run, x, W, b, h0, c0, out)

    def run_noalloc(self, x, W, b, h0, c0=None, out: dict | None = None) -> dict:
        """ambptt_run_noalloc: the same pass with the library's static scratch
        as workspace; `out` must be given (this call allocates nothing)."""
        if out is None:
            raise ValueError("run_noalloc needs preallocated gradient buffers (out)")
        return self._run(self.L.ambptt_run_noalloc, x, W, b, h0, c0, out)

    def _run(self, fn, x, W, b, h0, c0, out) -> dict:
        torch, s = self.torch, self.spec
        x, W, b, h0, c0 = self._inputs(x, W, b, h0, c0)
        if out is None:
            f32 = dict(dtype=torch.float32, device=self.device)
            out = {"dW": torch.empty(W.shape, **f32), "db": torch.empty(b.shape, **f32),
                   "dh0": torch.empty(h0.shape, **f32),
                   "dc0": torch.empty(h0.shape, **f32) if s.cell == "lstm" else None}
        loss = C.c_double()
        st = _lib.Stats()
        check(fn(self.ctx, _ptr(x), _ptr(W), _ptr(b), _ptr(h0), _ptr(c0),
                                _ptr(out["dW"]), _ptr(out["db"]), _ptr(out["dh0"]), _ptr(out.get("dc0")),
                                C.byref(loss), C.byref(st)))
        res = dict(out)
        res["loss"] = float(loss.value)
        res["stats"] = st.as_dict()
        return res

    def set_file_tier(self, directory: str, file_slots: int) -> None:
        """A file below the pinned host tier (ambptt_set_file_tier); 0 slots removes it."""
        check(self.L.ambptt_set_file_tier(self.ctx, str(directory).encode(), int(file_slots)))

    def set_step_costs(self, costs) -> None:
        """Relative forward costs of the n steps (ambptt_set_step_costs); None removes them."""
        if costs is None:
            check(self.L.ambptt_set_step_costs(self.ctx, None, 0))
            return
        arr = (C.c_double * len(costs))(*[float(c) for c in costs])
        check(self.L.ambptt_set_step_costs(self.ctx, arr, len(costs)))

    def last_schedule_text(self) -> str:
        """The canonical text of the schedule the last run executed."""
        return _text(lambda buf, cap, need: self.L.ambptt_last_schedule_text(self.ctx, buf, cap, need))

    def close(self) -> None:
        if getattr(self, "ctx", None) is not None and self.ctx.value:
            self.L.ambptt_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        # at interpreter shutdown the HIP runtime may already be going away:
        # contexts still open then are left to the process's end
        if sys.is_finalizing():
            return
        try:
            self.close()
        except Exception:
            pass
