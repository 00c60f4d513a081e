"""GPU runs with a file below the pinned host tier (a third storage level):
the pinned slots become a ring in front of the file, states are written
behind to it and read back ahead of the reverse.  The gradients must not
change by a bit against runs with every state in pinned memory, and the
file traffic must be what the ring implies."""
import os

import pytest

import synth
from oracle import schedule as S

from gpu_util import TOL_BF16, TOL_F32, assert_bitwise, assert_close, device_inputs, inputs, run_gpu, run_oracle

pytestmark = pytest.mark.gpu


def _case(wl):
    x, W, b, x0 = inputs(wl)
    return (x, W, b, x0), device_inputs(wl, x, W, b, x0)


def _state_bytes(wl):
    B, H = wl.batch, wl.hidden
    e = 2 if wl.dtype == "bf16" else 4
    h = B * H * e
    h_pad = -(-h // 256) * 256
    return h_pad + (B * H * 4 if wl.cell == "lstm" else 0)


@pytest.mark.parametrize("ring", [1, 3])
def test_file_tier_lstm_f32(tmp_path, ring):
    """60 steps, I = 1 (every state stored): 59 states through a ring of 1 or 3
    pinned buffers; the reverse reads 59 - ring of them back from the file."""
    wl = synth.get("lstm_h512_t1000").with_(batch=20, input=32, hidden=48, n_steps=60, name="lstm_file")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=3, slow_slots=ring, interval_min=1, file_tier=(str(tmp_path), 60))
    st = a["stats"]
    assert st["mode"] == 1 and st["interval"] == 1 and st["stores"] == 59
    assert st["bytes_file_w"] == 59 * _state_bytes(wl)
    assert st["bytes_file_r"] == (59 - ring) * _state_bytes(wl)
    assert_close(a, want, TOL_F32)
    b = run_gpu(wl, dev, fast_slots=3, slow_slots=60, interval_min=1, path=1)  # all in pinned memory
    assert b["stats"]["bytes_file_w"] == 0
    assert_bitwise(a, b)
    assert not [f for f in os.listdir(tmp_path) if f.startswith("ambptt-tier-")]  # unlinked at creation


def test_file_tier_with_the_dynamic_policy_bf16(tmp_path):
    """Stores decided during the sweep, through 2 pinned buffers, wide bf16 kernels."""
    wl = synth.get("lstm_h2048_bf16_t10000").with_(batch=64, input=64, hidden=128, n_steps=30,
                                                   name="lstm_bf16_file")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    a = run_gpu(wl, dev, fast_slots=3, slow_slots=2, interval_min=1, file_tier=(str(tmp_path), 30),
                opts={"store_policy": 1})
    st = a["stats"]
    assert st["mode"] == 2 and st["bytes_file_w"] == st["stores"] * _state_bytes(wl)
    head, acts = S.parse(a["schedule_text"])
    assert head["H"] == 30 and S.check(30, 3, 30, acts)["evals"] == st["forward_evals"]
    assert_close(a, want, TOL_BF16)
    assert_bitwise(a, run_gpu(wl, dev, fast_slots=3, slow_slots=0))


def test_file_tier_errors(tmp_path):
    import paper_1806_01117_amd as amb
    wl = synth.get("lstm_h512_t1000").with_(batch=16, input=16, hidden=32, n_steps=8, name="lstm_file_err")
    r = amb.Runner(amb.ProblemSpec.from_workload(wl, fast_slots=3, slow_slots=2, interval_min=1))
    try:
        with pytest.raises(amb.AmbpttError):
            r.set_file_tier(str(tmp_path / "missing"), 8)
        r.set("path", 2)
        with pytest.raises(amb.AmbpttError):
            r.set_file_tier(str(tmp_path), 8)
    finally:
        r.close()
    r = amb.Runner(amb.ProblemSpec.from_workload(wl, fast_slots=3, slow_slots=0))
    try:
        with pytest.raises(amb.AmbpttError):  # no pinned buffer to put in front of the file
            r.set_file_tier(str(tmp_path), 8)
    finally:
        r.close()
