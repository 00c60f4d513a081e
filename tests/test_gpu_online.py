"""GPU runs of online checkpointing (the number of steps unknown during the
forward sweep; the variant Section 1.1 names beside Revolve).  Each test runs
the schedule the oracle generates for that (n, s, H, I) (the executor reports
the text it ran), checks the executor's counters with the oracle's symbolic
checker, compares gradients with the float64 oracle, and bit for bit with a
store-all run on the same kernels (recomputation is deterministic)."""
import pytest

import synth
from oracle import schedule as S

from gpu_util import (TOL_BF16, TOL_F32, assert_bitwise, assert_close, assert_close_relu, device_inputs, inputs,
                      run_gpu, run_oracle)

pytestmark = pytest.mark.gpu

PATHS = [pytest.param(1, id="steps"), pytest.param(2, id="resident")]
ONLINE = {"online": 1}


def _case(wl):
    x, W, b, x0 = inputs(wl)
    return (x, W, b, x0), device_inputs(wl, x, W, b, x0)


def _check_online(res, n, s, H, I):
    st = res["stats"]
    assert st["mode"] == 3
    assert res["schedule_text"] == S.text_online(n, s, H, I)
    head, acts = S.parse(res["schedule_text"])
    c = S.check(n, s, H, acts)
    assert c["evals"] == st["forward_evals"] == S.schedule_online(n, s, H, I)[0]["evals"]
    assert c["stores"] == st["stores"] and c["prefetches"] == st["prefetches"]
    assert c["adjoints"] == st["adjoints"] == n


@pytest.mark.parametrize("path", PATHS)
def test_online_lstm_f32(path):
    """A reduced 512-LSTM, 53 steps: one level with 4 slots (past C(6,2) = 15,
    so the placement goes through three phases), two levels with unbounded
    and with 3 host slots (the interval doubles twice)."""
    wl = synth.get("lstm_h512_t1000").with_(n_steps=53, name="lstm_online")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    ref = run_gpu(wl, dev, fast_slots=53, slow_slots=0, path=path)
    assert ref["stats"]["forward_evals"] == 53
    assert_close(ref, want, TOL_F32)
    for s, H, I in ((4, 0, 0), (3, 53, 2), (4, 3, 2), (2, 53, 1)):
        got = run_gpu(wl, dev, path=path, fast_slots=s, slow_slots=H, interval_min=I, opts=ONLINE)
        _check_online(got, 53, s, H, max(I, 1) if H else 0)
        assert_bitwise(got, ref)


@pytest.mark.parametrize("path", PATHS)
def test_online_rnn_workload(path):
    """The 128-step tanh RNN with 4 slots and no host tier: online within
    the bound the cited work's repetition number allows, against Revolve."""
    wl = synth.get("rnn_h64_t128")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    got = run_gpu(wl, dev, path=path, opts=ONLINE)
    _check_online(got, 128, 4, 0, 0)
    assert_close(got, want, TOL_F32)
    assert_bitwise(got, run_gpu(wl, dev, path=path))


def test_online_ragged_lstm():
    """Batch not a multiple of 16, n not a multiple of the interval."""
    wl = synth.get("lstm_h512_t1000").with_(batch=5, input=16, hidden=32, n_steps=37, name="lstm_online_ragged")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    for path in (1, 2):
        got = run_gpu(wl, dev, path=path, fast_slots=3, slow_slots=4, interval_min=3, opts=ONLINE)
        _check_online(got, 37, 3, 4, 3)
        assert_close(got, want, TOL_F32)
        assert_bitwise(got, run_gpu(wl, dev, path=path, fast_slots=37, slow_slots=0))


def test_online_wide_bf16():
    """The wide-batch bf16 LSTM kernels (B = 64)."""
    wl = synth.get("lstm_h2048_bf16_t10000").with_(batch=64, input=64, hidden=128, n_steps=30,
                                                   name="lstm_bf16_online")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    got = run_gpu(wl, dev, fast_slots=3, slow_slots=30, interval_min=2, opts=ONLINE)
    _check_online(got, 30, 3, 30, 2)
    assert_close(got, want, TOL_BF16)
    assert_bitwise(got, run_gpu(wl, dev, fast_slots=30, slow_slots=0))


def test_online_resmlp():
    wl = synth.get("resmlp_w4096_l2000_bf16").with_(batch=70, hidden=128, n_steps=23, w_scale=0.08,
                                                    name="resmlp_online")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    got = run_gpu(wl, dev, fast_slots=3, slow_slots=0, opts=ONLINE)
    _check_online(got, 23, 3, 0, 0)
    assert_close_relu(got, want, TOL_BF16)
    assert_bitwise(got, run_gpu(wl, dev, fast_slots=23, slow_slots=0))


def test_online_refuses_other_policies():
    import paper_1806_01117_amd as amb
    wl = synth.get("lstm_h512_t1000").with_(batch=16, input=16, hidden=32, n_steps=8, name="lstm_online_refuse")
    r = amb.Runner(amb.ProblemSpec.from_workload(wl, fast_slots=3, slow_slots=8, interval_min=1))
    try:
        r.set("online", 1)
        with pytest.raises(amb.AmbpttError):
            r.set("store_policy", 1)
        with pytest.raises(amb.AmbpttError):
            r.set("online", 2)
    finally:
        r.close()


def test_online_lstm512_full_workload():
    """The bench workload (1000 steps, B 64, D 256, H 512, 10 slots, a host
    slot per step) under online checkpointing on the resident kernel: the
    oracle within tolerance, plain Revolve at the same 10 slots bit for bit."""
    wl = synth.get("lstm_h512_t1000")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    got = run_gpu(wl, dev, path=2, interval_min=1, opts=ONLINE)
    _check_online(got, 1000, 10, 1000, 1)
    assert got["stats"]["recompute_factor"] == 1.0
    assert_close(got, want, TOL_F32)
    assert_bitwise(got, run_gpu(wl, dev, path=2, slow_slots=0))


@pytest.mark.parametrize("rule", [0, 1])
def test_calibrated_interval_follows_the_rule(rule):
    """On the per-step path the calibrated interval is the rule's for the
    T_A and T_T that the calibration reports."""
    import paper_1806_01117_amd as amb
    wl = synth.get("lstm_h2048_bf16_t10000").with_(batch=64, input=64, hidden=128, n_steps=40, name="lstm_calib")
    host, dev = _case(wl)
    r = amb.Runner(amb.ProblemSpec.from_workload(wl, fast_slots=4, slow_slots=40, interval_min=0))
    try:
        r.set("interval_rule", rule)
        I, ta, tt = r.calibrate(*dev)
    finally:
        r.close()
    assert ta > 0 and tt > 0
    assert I == amb.interval_from_timings(ta, tt, 4, rule)
    assert 1 <= I <= max(1, -(-tt // ta))
