"""ctypes declarations of the C ABI in include/ambptt.h (marshalling only)."""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libambptt.so")

OK, EINVAL, ENOMEM, EHIP, EUNSUPPORTED, EINTERNAL = 0, -1, -2, -3, -4, -5
CELL = {"rnn": 1, "lstm": 2, "resmlp": 3, "mlp": 4}
DTYPE = {"f32": 0, "bf16": 1}
LOSS = {"half_sq_last": 0, "mean_sq_all": 1, "mean_last": 2}

EXPORTS = ["ambptt_version", "ambptt_revolve_advances", "ambptt_schedule_evals", "ambptt_schedule_text",
           "ambptt_schedule_text_starts", "ambptt_schedule_text_starts_costs", "ambptt_schedule_text_online", "ambptt_schedule_text_costs", "ambptt_schedule_text_sized",
           "ambptt_interval_from_timings", "ambptt_set_step_costs", "ambptt_set_widths",
           "ambptt_resident_program", "ambptt_query", "ambptt_last_error",
           "ambptt_create", "ambptt_bind", "ambptt_set_int", "ambptt_set_file_tier", "ambptt_calibrate", "ambptt_run", "ambptt_run_noalloc",
           "ambptt_last_schedule_text", "ambptt_destroy"]


class Problem(C.Structure):
    _fields_ = [("cell", C.c_int32), ("dtype", C.c_int32), ("loss", C.c_int32),
                ("batch", C.c_int32), ("input", C.c_int32), ("hidden", C.c_int32),
                ("n_steps", C.c_int64), ("fast_slots", C.c_int32), ("interval_min", C.c_int32),
                ("slow_slots", C.c_int64)]


class Stats(C.Structure):
    _fields_ = [("mode", C.c_int32), ("interval", C.c_int32), ("window", C.c_int32), ("path", C.c_int32),
                ("n_steps", C.c_int64), ("actions", C.c_int64), ("forward_evals", C.c_int64),
                ("adjoints", C.c_int64), ("takeshots", C.c_int64), ("takeshot_copies", C.c_int64),
                ("restores", C.c_int64), ("stores", C.c_int64), ("prefetches", C.c_int64),
                ("prefetches_elided", C.c_int64), ("bytes_d2h", C.c_int64), ("bytes_h2d", C.c_int64),
                ("compute_waits", C.c_int64), ("kernel_launches", C.c_int64),
                ("recompute_factor", C.c_double), ("schedule_us", C.c_double), ("run_us", C.c_double), ("enqueue_us", C.c_double),
                ("kernel_us", C.c_double * 6), ("kernel_samples", C.c_int64 * 6),
                ("kernel_calls", C.c_int64 * 6), ("bytes_file_w", C.c_int64), ("bytes_file_r", C.c_int64),
                ("forward_cost", C.c_double)]

    def as_dict(self) -> dict:
        d = {}
        for k, _ in self._fields_:
            v = getattr(self, k)
            d[k] = list(v) if isinstance(v, C.Array) else v
        return d


KERNEL_CLASSES = ["fwd", "pass", "adj", "hadj", "dw", "other"]


_lib = None


class AmbpttError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"ambptt status {status}: {msg}")
        self.status = status


def load():
    """Loads libambptt.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_1806_01117_amd.build`")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    L.ambptt_version.restype = C.c_char_p
    L.ambptt_last_error.restype = C.c_char_p
    L.ambptt_revolve_advances.argtypes = [i64, i32]
    L.ambptt_revolve_advances.restype = i64
    L.ambptt_schedule_evals.argtypes = [i64, i32, i64, i32, C.POINTER(i32), C.POINTER(i32)]
    L.ambptt_schedule_evals.restype = i64
    L.ambptt_schedule_text.argtypes = [i64, i32, i64, i32, C.c_char_p, sz, C.POINTER(sz)]
    L.ambptt_schedule_text.restype = C.c_int
    L.ambptt_schedule_text_starts.argtypes = [i64, i32, i64, C.POINTER(i64), i64, C.c_char_p, sz, C.POINTER(sz)]
    L.ambptt_schedule_text_starts.restype = C.c_int
    L.ambptt_schedule_text_starts_costs.argtypes = [i64, i32, i64, C.POINTER(i64), i64, C.POINTER(C.c_double), C.c_char_p,
                                                    sz, C.POINTER(sz)]
    L.ambptt_schedule_text_starts_costs.restype = C.c_int
    L.ambptt_schedule_text_online.argtypes = [i64, i32, i64, i32, C.c_char_p, sz, C.POINTER(sz)]
    L.ambptt_schedule_text_online.restype = C.c_int
    L.ambptt_interval_from_timings.argtypes = [C.c_double, C.c_double, i32, i32]
    L.ambptt_interval_from_timings.restype = i64
    L.ambptt_schedule_text_costs.argtypes = [i64, i32, i64, i32, C.POINTER(C.c_double), C.c_char_p, sz, C.POINTER(sz)]
    L.ambptt_schedule_text_costs.restype = C.c_int
    L.ambptt_schedule_text_sized.argtypes = [i64, i32, i64, i32, C.POINTER(i64), C.POINTER(C.c_double), C.c_char_p, sz,
                                             C.POINTER(sz)]
    L.ambptt_schedule_text_sized.restype = C.c_int
    L.ambptt_set_widths.argtypes = [vp, C.POINTER(i32), i64]
    L.ambptt_set_widths.restype = C.c_int
    L.ambptt_set_step_costs.argtypes = [vp, C.POINTER(C.c_double), i64]
    L.ambptt_set_step_costs.restype = C.c_int
    L.ambptt_last_schedule_text.argtypes = [vp, C.c_char_p, sz, C.POINTER(sz)]
    L.ambptt_set_file_tier.argtypes = [vp, C.c_char_p, i64]
    L.ambptt_set_file_tier.restype = C.c_int
    L.ambptt_last_schedule_text.restype = C.c_int
    L.ambptt_resident_program.argtypes = [i64, i32, i64, i32, i32, C.POINTER(i32), sz, C.POINTER(sz)]
    L.ambptt_resident_program.restype = C.c_int
    L.ambptt_query.argtypes = [C.POINTER(Problem), C.POINTER(sz), C.POINTER(sz), C.POINTER(sz)]
    L.ambptt_query.restype = C.c_int
    L.ambptt_create.argtypes = [C.POINTER(Problem), vp, C.POINTER(vp)]
    L.ambptt_create.restype = C.c_int
    L.ambptt_bind.argtypes = [vp, vp, sz, vp, sz]
    L.ambptt_bind.restype = C.c_int
    L.ambptt_set_int.argtypes = [vp, C.c_char_p, i64]
    L.ambptt_set_int.restype = C.c_int
    L.ambptt_calibrate.argtypes = [vp, vp, vp, vp, vp, vp, C.POINTER(i32), C.POINTER(C.c_double),
                                   C.POINTER(C.c_double)]
    L.ambptt_calibrate.restype = C.c_int
    L.ambptt_run.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, C.POINTER(C.c_double), C.POINTER(Stats)]
    L.ambptt_run.restype = C.c_int
    L.ambptt_run_noalloc.argtypes = L.ambptt_run.argtypes
    L.ambptt_run_noalloc.restype = C.c_int
    L.ambptt_destroy.argtypes = [vp]
    L.ambptt_destroy.restype = None
    _lib = L
    return L


def check(status: int) -> None:
    if status != OK:
        raise AmbpttError(status, load().ambptt_last_error().decode(errors="replace"))
