"""GPU runs of schedules split for unequal step costs (ambptt_set_step_costs).
The executed schedule must be the oracle's (text for text), its weighted
forward cost the oracle's, and the gradients equal to a store-all run bit for
bit and to the float64 oracle within tolerance."""
import numpy as np
import pytest

import synth
from oracle import schedule as S

from gpu_util import (TOL_BF16, TOL_F32, assert_bitwise, assert_close, assert_close_relu, device_inputs, inputs,
                      run_oracle, say)

pytestmark = pytest.mark.gpu

PATHS = [pytest.param(1, id="steps"), pytest.param(2, id="resident")]


def _costs(n, seed):
    rng = np.random.default_rng(seed)
    return [float(c) for c in rng.choice([1.0, 1.0, 1.0, 3.0, 8.0], n)]


def _run(wl, dev, costs, path=None, **kw):
    import paper_1806_01117_amd as amb
    spec = amb.ProblemSpec.from_workload(wl, **kw)
    say(wl.name, spec, "costs", costs is not None, "path", path)
    r = amb.Runner(spec)
    try:
        if path is not None:
            r.set("path", path)
        r.set_step_costs(costs)
        out = r.run(*dev)
        text = r.last_schedule_text()
    finally:
        r.close()
    res = {k: (v.float().cpu().numpy() if hasattr(v, "cpu") else v) for k, v in out.items() if v is not None}
    res["schedule_text"] = text
    if path is not None:
        assert res["stats"]["path"] == path - 1
    return res


def _case(wl):
    x, W, b, x0 = inputs(wl)
    return (x, W, b, x0), device_inputs(wl, x, W, b, x0)


@pytest.mark.parametrize("path", PATHS)
def test_costs_lstm_f32(path):
    n = 61
    wl = synth.get("lstm_h512_t1000").with_(n_steps=n, name="lstm_costs")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    ref = _run(wl, dev, None, path=path, fast_slots=n, slow_slots=0)
    assert_close(ref, want, TOL_F32)
    costs = _costs(n, 1)
    for s, H, I in ((3, 0, 0), (4, n, 4)):
        got = _run(wl, dev, costs, path=path, fast_slots=s, slow_slots=H, interval_min=I)
        head, acts = S.schedule_costs(n, s, costs, H, I)
        assert got["schedule_text"] == S.text_costs(n, s, costs, H, I)
        assert got["stats"]["forward_evals"] == head["evals"]
        assert got["stats"]["forward_cost"] == pytest.approx(head["cost"], rel=1e-12)
        assert_bitwise(got, ref)


def test_costs_wide_bf16_and_mlp():
    wl = synth.get("lstm_h2048_bf16_t10000").with_(batch=64, input=64, hidden=128, n_steps=26, name="lstm_bf16_costs")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    costs = _costs(26, 2)
    got = _run(wl, dev, costs, fast_slots=3, slow_slots=26, interval_min=3)
    assert got["schedule_text"] == S.text_costs(26, 3, costs, 26, 3)
    assert_close(got, want, TOL_BF16)
    assert_bitwise(got, _run(wl, dev, None, fast_slots=26, slow_slots=0))

    wl = synth.get("resmlp_w4096_l2000_bf16").with_(batch=70, hidden=128, n_steps=21, w_scale=0.08, name="mlp_costs")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    costs = _costs(21, 3)
    got = _run(wl, dev, costs, fast_slots=3, slow_slots=0)
    assert got["schedule_text"] == S.text_costs(21, 3, costs)
    assert_close_relu(got, want, TOL_BF16)
    assert_bitwise(got, _run(wl, dev, None, fast_slots=21, slow_slots=0))


def test_costs_argument_errors():
    import paper_1806_01117_amd as amb
    wl = synth.get("lstm_h512_t1000").with_(batch=16, input=16, hidden=32, n_steps=8, name="lstm_costs_err")
    r = amb.Runner(amb.ProblemSpec.from_workload(wl, fast_slots=3, slow_slots=8, interval_min=1))
    try:
        with pytest.raises(amb.AmbpttError):
            r.set_step_costs([1.0] * 7)            # one cost per step
        with pytest.raises(amb.AmbpttError):
            r.set_step_costs([1.0] * 7 + [-1.0])   # positive
        r.set_step_costs([1.0] * 8)
        with pytest.raises(amb.AmbpttError):
            r.set("online", 1)
        r.set_step_costs(None)
        r.set("online", 1)
    finally:
        r.close()


def test_costs_under_the_dynamic_store_policy():
    """Interval starts chosen during the sweep (store when the previous store
    completed), each interval reversed with splits for the step costs: the
    executed text is the oracle's over the same starts, the gradients equal a
    store-all run bit for bit and the oracle within tolerance."""
    n = 48
    wl = synth.get("lstm_h512_t1000").with_(batch=20, input=32, hidden=48, n_steps=n, name="lstm_dyn_costs")
    host, dev = _case(wl)
    want = run_oracle(wl, *host)
    costs = _costs(n, 4)
    import paper_1806_01117_amd as amb
    r = amb.Runner(amb.ProblemSpec.from_workload(wl, fast_slots=4, slow_slots=n, interval_min=1))
    try:
        r.set("path", 1)
        r.set("store_policy", 1)
        r.set_step_costs(costs)
        out = r.run(*dev)
        text = r.last_schedule_text()
    finally:
        r.close()
    got = {k: (v.float().cpu().numpy() if hasattr(v, "cpu") else v) for k, v in out.items() if v is not None}
    head, acts = S.parse(text)
    assert head["mode"] == "dynamic" and head["split"] == "cost"
    starts = [a[3] for a in acts if a[0] == "W"]
    opening = acts[3 * len(starts)]
    starts.append(opening[2])
    assert text == S.text_from_starts(n, 4, n, starts, costs)
    ohead, _ = S.schedule_from_starts(n, 4, n, starts, costs)
    assert got["stats"]["forward_evals"] == ohead["evals"]
    assert got["stats"]["forward_cost"] == pytest.approx(ohead["cost"], rel=1e-12)
    assert_close(got, want, TOL_F32)
    assert_bitwise(got, _run(wl, dev, None, path=1, fast_slots=n, slow_slots=0))
