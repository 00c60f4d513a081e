"""Stream ordering under late copies.  A bounded host function holds the copy
stream before every store and prefetch, and the weight-gradient stream before
every window, and each prefetch first fills its fast slot with NaN bytes: the
edges that order compute after the copies (a store after its slot's
producer, a slot overwritten only after its store, a prefetched slot read
only after the prefetch, a window's ring half reused only after the window)
are then all exercised, and a missing one would show as NaNs or as
gradients that differ from store-all.  Also the resident kernel under a
cooperative launch."""
import pytest

import synth

from gpu_util import TOL_BF16, TOL_F32, assert_bitwise, assert_close, device_inputs, inputs, run_gpu, run_oracle

pytestmark = pytest.mark.gpu


def _case(wl):
    host = inputs(wl)
    return host, device_inputs(wl, *host)


LATE = {"test_copy_delay_us": 3000, "test_poison": 1}


@pytest.mark.parametrize("policy", [0, 1], ids=["fixed", "dynamic"])
@pytest.mark.parametrize("host_waits", [0, 1], ids=["stream-waits", "host-waits"])
def test_late_copies_small_lstm(host_waits, policy):
    # the dynamic policy stores only once the previous store has landed, so
    # its copies are delayed less than the sweep takes, to leave it several
    n, delay = (40, 3000) if policy == 0 else (96, 50)
    wl = synth.get("lstm_h512_t1000").with_(batch=24, input=32, hidden=64, n_steps=n, name="lstm_late_copies")
    host, dev = _case(wl)
    ref = run_gpu(wl, dev, fast_slots=n, slow_slots=0, path=1, window=4)  # store-all, no copies, same windows
    got = run_gpu(wl, dev, fast_slots=3, slow_slots=n, interval_min=2, path=1, window=4,
                  opts=dict(test_copy_delay_us=delay, test_poison=1, host_waits=host_waits, store_policy=policy,
                            dw_stream=1))
    st = got["stats"]
    assert st["mode"] == (2 if policy else 1)
    assert st["stores"] >= 2 and st["prefetches"] - st["prefetches_elided"] >= 1, st
    assert st["compute_waits"] > 0, "no wait on a late copy was taken"
    assert_bitwise(got, ref)
    assert_close(got, run_oracle(wl, *host), TOL_F32)


def test_late_copies_wide_bf16():
    """The wide-batch bf16 kernels (host waits by default, windows in line)."""
    wl = synth.get("lstm_h2048_bf16_t10000").with_(batch=64, input=64, hidden=128, n_steps=24, name="bf16_late_copies")
    host, dev = _case(wl)
    ref = run_gpu(wl, dev, fast_slots=24, slow_slots=0)
    got = run_gpu(wl, dev, fast_slots=3, slow_slots=24, interval_min=2, opts=LATE)
    st = got["stats"]
    assert st["compute_waits"] > 0 and st["kernel_calls"][3] > 0
    assert_bitwise(got, ref)
    assert_close(got, run_oracle(wl, *host), TOL_BF16)


def test_resident_cooperative_launch():
    wl = synth.get("lstm_h512_t1000").with_(n_steps=64)
    host, dev = _case(wl)
    plain = run_gpu(wl, dev, fast_slots=3, slow_slots=64, interval_min=2, path=2, opts={"resident_cooperative": 0})
    coop = run_gpu(wl, dev, fast_slots=3, slow_slots=64, interval_min=2, path=2)  # the default launch
    assert coop["stats"]["mode"] == 1
    assert_bitwise(coop, plain)
    assert_close(coop, run_oracle(wl, *host), TOL_F32)
