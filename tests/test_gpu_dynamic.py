"""GPU runs of the store policy that decides the interval starts during the
sweep (store the next state once the previous store has completed, the
non-uniform policy of Section 6).  The starts depend on timing, so each test
takes the schedule the executor reports (ambptt_last_schedule_text), checks
it with the oracle's symbolic checker (a valid two-level schedule whose
forward count is the executor's), checks the policy's own rules on its
starts, and compares the gradients with the oracle and, bit for bit, with
the fixed-interval and plain Revolve runs on the same inputs."""
import pytest

import synth
from oracle import schedule as S

from gpu_util import (TOL_BF16, TOL_F32, assert_bitwise, assert_close, assert_close_relu, device_inputs, inputs,
                      run_gpu, run_oracle)

pytestmark = pytest.mark.gpu

DYN = {"store_policy": 1}


def _case(wl):
    x, W, b, x0 = inputs(wl)
    return (x, W, b, x0), device_inputs(wl, x, W, b, x0)


def _starts(acts):
    """Interval starts of a two-level schedule: the sweep is K - 1 triples
    (snapshot, store, advance), one per stored start; the reverse opens with
    the snapshot of the last start."""
    stored = [a[3] for a in acts if a[0] == "W"]
    opening = acts[3 * len(stored)]
    assert opening[0] == "S", opening
    return stored + [opening[2]]


def _check_dynamic(res, n, s, H):
    st = res["stats"]
    head, acts = S.parse(res["schedule_text"])
    assert st["mode"] == 2 and head["mode"] == "dynamic" and (head["n"], head["s"], head["H"]) == (n, s, H)
    c = S.check(n, s, H, acts)
    assert c["evals"] == st["forward_evals"] and c["stores"] == st["stores"]
    starts = _starts(acts)
    assert S.text_from_starts(n, s, H, starts) == res["schedule_text"]
    gaps = [b - a for a, b in zip(starts, starts[1:])]
    spacing = max(1, -(-n // (H + 1)))
    assert all(g >= spacing for g in gaps[:-1]), starts  # stored starts keep the spacing
    if gaps and len(starts) - 1 < H:                     # host slots left: the sweep ends within one interval of n
        assert n - starts[-1] <= gaps[-1], starts
    assert st["interval"] == max([b - a for a, b in zip(starts, starts[1:] + [n])])
    return starts


@pytest.mark.parametrize("cell", ["lstm", "rnn"])
def test_dynamic_f32_matches_oracle_and_fixed_interval(cell):
    """fp32 cells on the per-step path (the policy never runs on the resident
    kernel): 40 steps, 3 fast slots, a host slot per step."""
    wl = synth.get("lstm_h512_t1000").with_(cell=cell, batch=20, input=32, hidden=48, n_steps=40,
                                            name=f"{cell}_dyn")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=3, slow_slots=40, interval_min=1, opts=DYN)
    starts = _check_dynamic(a, 40, 3, 40)
    assert len(starts) >= 2
    assert_close(a, want, TOL_F32)
    # the same kernels (one launch per step) with a fixed interval, and plain Revolve
    b = run_gpu(wl, dev, fast_slots=3, slow_slots=40, interval_min=3, path=1)
    assert b["stats"]["mode"] == 1
    assert_bitwise(a, b)
    c = run_gpu(wl, dev, fast_slots=3, slow_slots=0, path=1)
    assert_bitwise(a, c)


def test_dynamic_bounded_host_tier():
    """6 host slots for 50 steps: stores at least ceil(50 / 7) = 8 steps apart."""
    wl = synth.get("lstm_h512_t1000").with_(batch=16, input=16, hidden=32, n_steps=50, name="lstm_dyn_h6")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=4, slow_slots=6, interval_min=1, opts=DYN)
    starts = _check_dynamic(a, 50, 4, 6)
    assert len(starts) - 1 <= 6
    assert_close(a, want, TOL_F32)
    assert_bitwise(a, run_gpu(wl, dev, fast_slots=4, slow_slots=0, path=1))


def test_dynamic_wide_bf16():
    """The wide-batch bf16 LSTM kernels (B = 64) under the policy."""
    wl = synth.get("lstm_h2048_bf16_t10000").with_(batch=64, input=64, hidden=128, n_steps=24,
                                                   name="lstm_bf16_dyn")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=3, slow_slots=24, interval_min=1, opts=DYN)
    _check_dynamic(a, 24, 3, 24)
    assert_close(a, want, TOL_BF16)
    assert_bitwise(a, run_gpu(wl, dev, fast_slots=3, slow_slots=24, interval_min=2))


def test_dynamic_resmlp():
    wl = synth.get("resmlp_w4096_l2000_bf16").with_(batch=70, hidden=128, n_steps=19, w_scale=0.08,
                                                    name="resmlp_dyn")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=3, slow_slots=19, interval_min=1, opts=DYN)
    _check_dynamic(a, 19, 3, 19)
    assert_close_relu(a, want, TOL_BF16)
    assert_bitwise(a, run_gpu(wl, dev, fast_slots=3, slow_slots=0))


def test_dynamic_policy_is_refused_on_the_resident_path():
    import paper_1806_01117_amd as amb
    wl = synth.get("lstm_h512_t1000").with_(batch=16, input=16, hidden=32, n_steps=8, name="lstm_dyn_res")
    r = amb.Runner(amb.ProblemSpec.from_workload(wl, fast_slots=3, slow_slots=8, interval_min=1))
    try:
        r.set("path", 2)
        with pytest.raises(amb.AmbpttError):
            r.set("store_policy", 1)
    finally:
        r.close()
