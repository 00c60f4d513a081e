"""The C-ABI library on the CPU: it loads, exports what the header declares,
and its host-only calls agree with the oracle (no GPU calls here)."""
import ctypes
import os
import re

import pytest

from oracle import schedule as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def amb():
    import paper_1806_01117_amd as amb
    amb.load()
    return amb


def _declared():
    names = []
    for f in os.listdir(os.path.join(ROOT, "include")):
        if f.endswith(".h"):
            src = open(os.path.join(ROOT, "include", f)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names += re.findall(r"\b(ambptt_[a-z_0-9]+)\s*\(", src)
    return sorted(set(names))


def test_every_declared_symbol_is_exported(amb):
    lib = ctypes.CDLL(amb.LIB_PATH)
    names = _declared()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), n
    from paper_1806_01117_amd import _lib
    assert sorted(_lib.EXPORTS) == names


def test_version(amb):
    assert "gfx950" in amb.version()


def test_revolve_counts_match_oracle(amb):
    for n in list(range(1, 80)) + [128, 1000, 2000, 10000, 20000, 123457]:
        for s in (1, 2, 3, 4, 10, 16, 32, 64):
            if s == 1 and n > 5000:
                continue
            assert amb.revolve_advances(n, s) == S.advances(n, s), (n, s)
    with pytest.raises(ValueError):
        amb.revolve_advances(0, 3)


def test_schedule_text_matches_oracle_bytewise(amb):
    for n in list(range(1, 34)) + [57, 100, 128, 257, 1000]:
        for s in (1, 2, 3, 4, 7, 10):
            for H in (0, 1, 3, 2000):
                for I in (0, 1, 2, 3, 5):
                    assert amb.schedule_text(n, s, H, I) == S.text(n, s, H, I), (n, s, H, I)


@pytest.mark.parametrize("n,s,H,I", [(128, 4, 0, 0), (1000, 10, 1000, 1), (1000, 10, 1000, 2),
                                     (2000, 16, 2000, 10), (10000, 32, 10000, 5)])
def test_workload_schedules_match_oracle(amb, n, s, H, I):
    assert amb.schedule_text(n, s, H, I) == S.text(n, s, H, I)
    ev, interval, mode = amb.schedule_evals(n, s, H, I)
    head, _ = S.schedule(n, s, H, I)
    assert (ev, interval, mode) == (head["evals"], head["I"], head["mode"])


def test_schedule_text_small_buffer(amb):
    from paper_1806_01117_amd import _lib
    L = amb.load()
    need = ctypes.c_size_t(0)
    buf = ctypes.create_string_buffer(8)
    st = L.ambptt_schedule_text(10, 3, 0, 0, buf, 8, ctypes.byref(need))
    assert st == _lib.EINVAL and need.value == len(S.text(10, 3)) + 1
    assert buf.value == b""


def test_query_sizes_and_validation(amb):
    from paper_1806_01117_amd import ProblemSpec, AmbpttError, query
    spec = ProblemSpec("lstm", "f32", "mean_sq_all", 64, 256, 512, 1000, 10, 1000)
    stride, pool, ws = query(spec)
    assert stride == 2 * 64 * 512 * 4 and pool == 10 * stride and ws > 4 * 512 * 2048
    spec_rnn = ProblemSpec("rnn", "f32", "half_sq_last", 4, 32, 64, 128, 4)
    stride, pool, ws = query(spec_rnn)
    assert stride == 1024 and pool == 4 * 1024
    for bad in (dict(n_steps=0), dict(fast_slots=0), dict(batch=0), dict(slow_slots=-1)):
        with pytest.raises(AmbpttError) as e:
            query(ProblemSpec(**{**spec.__dict__, **bad}))
        assert e.value.status == -1
    with pytest.raises(AmbpttError) as e:
        query(ProblemSpec(**{**spec.__dict__, "hidden": 500}))
    assert e.value.status == -4
    # bf16 operands: sizes must be multiples of 32; state = bf16 h + fp32 c
    bf = ProblemSpec("lstm", "bf16", "mean_last", 128, 1024, 2048, 10000, 32, 10000)
    stride, pool, ws = query(bf)
    assert stride == 128 * 2048 * 2 + 128 * 2048 * 4 and pool == 32 * stride
    with pytest.raises(AmbpttError) as e:
        query(ProblemSpec(**{**bf.__dict__, "hidden": 48}))
    assert e.value.status == -4


def test_stats_struct_layout(amb):
    from paper_1806_01117_amd import _lib
    st = _lib.Stats()
    st.kernel_launches = 7
    st.kernel_us[2] = 1.5
    d = st.as_dict()
    assert d["kernel_launches"] == 7 and d["kernel_us"][2] == 1.5 and len(d["kernel_calls"]) == 6
    # int32 x4, int64 x14, double x4, double x6, int64 x12, int64 x2 (file tier), double (forward cost)
    assert ctypes.sizeof(_lib.Stats) == 16 + 14 * 8 + 4 * 8 + 6 * 8 + 12 * 8 + 2 * 8 + 8
    assert ctypes.sizeof(_lib.Problem) == 48


def test_schedule_text_over_starts_matches_oracle_bytewise(amb):
    import random
    rng = random.Random(3)
    for _ in range(400):
        n = rng.randint(2, 200)
        s = rng.randint(2, 9)
        H = rng.randint(1, 300)
        k = rng.randint(0, min(H, n - 1))
        starts = [0] + sorted(rng.sample(range(1, n), k))
        assert amb.schedule_text_starts(n, s, H, starts) == S.text_from_starts(n, s, H, starts), (n, s, H, starts)


def test_schedule_text_over_starts_rejects_bad_starts(amb):
    for n, s, H, starts in [(10, 3, 5, [1, 4]), (10, 3, 5, [0, 4, 4]), (10, 3, 5, [0, 10]), (10, 3, 1, [0, 3, 6]),
                            (10, 1, 5, [0, 5]), (10, 3, 5, [])]:
        with pytest.raises(amb.AmbpttError):
            amb.schedule_text_starts(n, s, H, starts)


def test_online_schedule_text_matches_oracle_bytewise(amb):
    for s in (1, 2, 3, 4, 6, 10):
        for H, I in ((0, 0), (1, 1), (2, 2), (3, 1), (6, 3), (10 ** 6, 2)):
            for n in list(range(1, 40)) + [63, 128, 301]:
                assert amb.schedule_text_online(n, s, H, I) == S.text_online(n, s, H, I), (n, s, H, I)


@pytest.mark.parametrize("n,s,H,I", [(128, 4, 0, 0), (1000, 10, 1000, 2), (1000, 10, 0, 0), (2000, 16, 40, 1)])
def test_online_workload_schedules_match_oracle(amb, n, s, H, I):
    assert amb.schedule_text_online(n, s, H, I) == S.text_online(n, s, H, I)
