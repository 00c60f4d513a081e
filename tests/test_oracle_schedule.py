"""Pins for the oracle's checkpointing schedules (CPU only).

The schedule oracle is pinned against things other than itself:
  * a brute-force dynamic program over every split point (the recursive
    structure of binomial checkpointing) for the least advanced-step count
    and for the set of optimal splits;
  * the textbook special cases: one slot costs l(l-1)/2 advanced steps, and
    l <= s+1 steps cost l-1 (no recomputation, memory ratio 1, Section 1.1);
  * hand-derived small schedules (tests/golden/schedules_small.txt);
  * a symbolic execution of every generated schedule;
  * the policy invariants of Sections 2-3: stream-all when I = 1, fallback
    to Revolve when no store fits, never more recomputation than Revolve.
"""
import functools
import os
import random

import pytest

from oracle import schedule as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "schedules_small.txt")


@functools.lru_cache(maxsize=None)
def dp(l: int, s: int) -> int:
    """Least advanced steps over every split point (brute force)."""
    if l == 1:
        return 0
    if s == 1:
        # chain: advance i steps from x_a for i = l-1 .. 1
        return sum(range(1, l))
    return min(m + dp(l - m, s - 1) + dp(m, s) for m in range(1, l))


def dp_argmins(l: int, s: int) -> list[int]:
    vals = [(m + dp(l - m, s - 1) + dp(m, s), m) for m in range(1, l)]
    best = min(v for v, _ in vals)
    return [m for v, m in vals if v == best]


def test_closed_form_equals_dp():
    for s in range(1, 11):
        for l in range(1, 181):
            assert S.advances(l, s) == dp(l, s), (l, s)


def test_split_range_is_exactly_the_optimal_set():
    for s in range(2, 8):
        for l in range(2, 120):
            lo, hi = S.split_range(l, s)
            ms = dp_argmins(l, s)
            assert ms == list(range(lo, hi + 1)), (l, s, lo, hi, ms)


def test_textbook_special_cases():
    for l in range(1, 60):
        assert S.advances(l, 1) == l * (l - 1) // 2
        for s in range(l - 1 if l > 1 else 1, l + 4):
            if s >= 1:
                assert S.advances(l, s) == l - 1, (l, s)


def test_recompute_grows_with_n_and_shrinks_with_s():
    # Section 3: the recompute factor increases with n and decreases with s.
    for s in (2, 5, 20):
        prev = 0.0
        for n in (10, 100, 1000, 10000):
            R = S.revolve_evals(n, s) / n
            assert R >= prev and R >= 1.0
            prev = R
    for n in (100, 1000):
        Rs = [S.revolve_evals(n, s) / n for s in range(1, 40)]
        assert all(a >= b for a, b in zip(Rs, Rs[1:]))


def _golden_cases():
    cases, cur = [], None
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        if line.startswith("case "):
            cur = [tuple(int(v) for v in line.split()[1:]), ""]
            cases.append(cur)
        else:
            cur[1] += line
    return cases


@pytest.mark.parametrize("case", _golden_cases(), ids=lambda c: "-".join(map(str, c[0])))
def test_hand_derived_golden(case):
    (n, s, H, I), want = case
    assert S.text(n, s, H, I) == want


def _grid():
    rng = random.Random(1806)
    out = []
    for n in list(range(1, 40)) + [57, 100, 128, 257]:
        for s in (1, 2, 3, 4, 7, 10):
            for H in (0, 1, 3, 1000):
                for I in (0, 1, 2, 3, 5, 8):
                    out.append((n, s, H, I))
    rng.shuffle(out)
    return out[:2500]


def test_generated_schedules_are_valid_and_counted():
    for n, s, H, I in _grid():
        head, acts = S.schedule(n, s, H, I)
        c = S.check(n, s, H, acts)
        assert c["evals"] == head["evals"], (n, s, H, I)
        plain = S.revolve_evals(n, s)
        if head["mode"] == "revolve":
            assert c["evals"] == plain
            assert c["stores"] == 0 and c["prefetches"] == 0
        else:
            assert c["evals"] < plain                # never worse than Revolve
            K = -(-n // head["I"])
            assert c["stores"] == K - 1 and c["prefetches"] == K - 1 <= H


def test_stream_all_and_memory_ratio_one():
    for n in (4, 5, 17, 100):
        # T_T <= T_A: every state streamed out, no recomputation (Section 3)
        # (from n = 4 on, two slots alone would need recomputation)
        head, acts = S.schedule(n, 2, n, 1)
        assert head["mode"] == "async" and head["I"] == 1
        assert S.check(n, 2, n, acts)["evals"] == n
        # enough fast slots for every state: recompute factor 1
        for s in (n - 1, n, n + 3):
            if s >= 1:
                head, acts = S.schedule(n, s)
                assert S.check(n, s, 0, acts)["evals"] == n


def test_fallback_to_revolve():
    # Section 3: if not even one store fits in the forward pass, plain Revolve.
    assert S.schedule(10, 3, 100, 10)[0]["mode"] == "revolve"
    assert S.schedule(10, 3, 100, 50)[0]["mode"] == "revolve"
    assert S.schedule(10, 3, 0, 1)[0]["mode"] == "revolve"
    assert S.schedule(10, 1, 100, 1)[0]["mode"] == "revolve"


def test_bounded_slow_tier_sets_the_interval():
    # K-1 stored states must fit in H slow slots
    head, acts = S.schedule(1000, 10, 99, 1)
    assert head["I"] == 10
    assert S.check(1000, 10, 99, acts)["stores"] <= 99


def test_interval_count_is_constant_in_n():
    # Section 3: with a fixed interval the recompute factor stops growing with n.
    Rs = [S.schedule(n, 8, n, 16)[0]["evals"] / n for n in (1000, 4000, 16000)]
    assert max(Rs) - min(Rs) < 0.02          # ~2.43 at I = 16, s = 8
    assert Rs[-1] < S.revolve_evals(16000, 8) / 16000


def dp_table(N: int, smax: int):
    """F[s][l] for l <= N, s <= smax by the same brute force, vectorised over m."""
    import numpy as np
    F = np.zeros((smax + 1, N + 1), np.int64)
    l = np.arange(N + 1)
    F[1] = l * (l - 1) // 2
    for s in range(2, smax + 1):
        for L in range(2, N + 1):
            m = np.arange(1, L)
            F[s, L] = np.min(m + F[s - 1, L - m] + F[s, m])
    return F


def test_workload_schedule_counts():
    # Revolve counts at the workloads' (n, s): closed form vs brute force
    F = dp_table(2000, 16)
    for n, s in ((128, 4), (1000, 10), (2000, 16), (1777, 7)):
        assert S.advances(n, s) == F[s, n]
    assert S.revolve_evals(128, 4) == 517


def _random_starts(rng, n, H):
    """Interval starts 0 = t_0 < ... < t_{K-1} < n with K - 1 <= H."""
    k = rng.randint(0, min(H, n - 1))
    return [0] + sorted(rng.sample(range(1, n), k))


def test_schedules_over_chosen_starts_are_valid_and_counted():
    """Stores decided during the sweep (Section 6): every interval layout gives
    a valid schedule whose symbolic forward count is the closed form
    t_{K-1} + sum_k F(l_k, s-1) + 1, with one store and one prefetch per start
    but the last."""
    rng = random.Random(7)
    for _ in range(1500):
        n = rng.randint(2, 60)
        s = rng.randint(2, 7)
        H = rng.randint(1, 70)
        st = _random_starts(rng, n, H)
        head, acts = S.schedule_from_starts(n, s, H, st)
        c = S.check(n, s, H, acts)
        assert c["evals"] == head["evals"] == S.dynamic_evals(n, s, st), (n, s, H, st)
        assert c["stores"] == c["prefetches"] == len(st) - 1
        assert c["adjoints"] == n


def test_uniform_starts_reproduce_the_fixed_interval_schedule():
    """Starts kI reproduce the fixed-interval two-level schedule action for action."""
    for n in (5, 9, 12, 31, 100):
        for s in (2, 3, 5):
            for I in (1, 2, 3, 7):
                head, acts = S.schedule(n, s, n, I)
                if head["mode"] != "async":
                    continue
                h2, acts2 = S.schedule_from_starts(n, s, n, list(range(0, n, I)))
                assert acts2 == acts and h2["evals"] == head["evals"], (n, s, I)


def test_chosen_starts_edge_cases():
    # one interval: no store, Revolve on s - 1 slots from x_0
    head, acts = S.schedule_from_starts(7, 3, 4, [0])
    assert head["evals"] == S.advances(7, 2) + 1 and not any(a[0] in "WP" for a in acts)
    # every state an interval start: no recomputation (R = 1)
    head, acts = S.schedule_from_starts(6, 2, 5, list(range(6)))
    assert head["evals"] == 6
    for bad in ([1, 3], [0, 3, 3], [0, 7], [0, 1, 2, 3]):
        with pytest.raises(ValueError):
            S.schedule_from_starts(7, 3, 2, bad)
    with pytest.raises(ValueError):
        S.schedule_from_starts(7, 1, 2, [0, 3])


def test_paper_model_figure():
    """Section 3's model and its figure (s = 100; classic Revolve against
    intervals I = 8, 64, 1024; only the axis, 0 to 5, is printed): intervals
    of at most s + 1 steps need no recomputation; R(I, s) never exceeds
    R(n, s) for n >= I; Revolve's factor grows with n and stays inside the
    figure's axis up to a million steps; the schedules' own count of a
    two-level pass, which includes the sweep, is never below the model's."""
    s = 100
    assert S.paper_model_R(8, s) == 1.0 and S.paper_model_R(64, s) == 1.0
    r1024 = S.paper_model_R(1024, s)
    assert 1.0 < r1024 < 2.0
    prev = 0.0
    for n in (10 ** 3, 10 ** 4, 10 ** 5, 10 ** 6):
        r = S.paper_model_R(n, s)
        assert r >= prev and r <= 5.0
        assert S.paper_model_R(1024, s) <= r or n < 1024
        prev = r
    assert abs(S.paper_model_R(10 ** 6, s) - 3.818) < 5e-4
    for n in (2000, 10 ** 4):
        for I in (8, 64, 1024):
            head, _ = S.schedule(n, s, n, I)
            assert head["evals"] / n >= S.paper_model_R(I, s) - 1e-12


def _mutate(acts, i, new):
    out = list(acts)
    out[i] = new
    return out


def test_check_rejects_planted_store_and_prefetch_mistakes():
    """The symbolic checker's Level-2 rules, each shown to fail on a planted
    mistake in a valid two-level schedule (Section 2: a stored state is the
    one its fast slot holds; a prefetch brings back what was stored)."""
    n, s, H, I = 12, 3, 100, 3
    _, acts = S.schedule(n, s, H, I)
    S.check(n, s, H, acts)  # the unmodified schedule passes
    iw = next(i for i, a in enumerate(acts) if a[0] == "W" and a[3] > 0)
    # a prefetch whose fast slot holds another state when it is issued (the
    # first one of this schedule refills a slot that still holds its state)
    held, ip = {}, None
    for i, a in enumerate(acts):
        if a[0] == "S":
            held[a[1]] = a[2]
        elif a[0] == "P":
            if ip is None and held.get(a[2]) != a[3]:
                ip = i
            held[a[2]] = a[3]
    k, h, t = acts[iw][1:]
    hp, kp, tp = acts[ip][1:]
    planted = {
        # a store from a fast slot that holds another state
        "store wrong slot": _mutate(acts, iw, ("W", 1 - k, h, t)),
        # a store that claims a state its slot does not hold
        "store wrong state": _mutate(acts, iw, ("W", k, h, t + 1)),
        # a store past the host budget
        "store beyond H": _mutate(acts, iw, ("W", k, H, t)),
        # a prefetch of a host slot that holds another state
        "prefetch wrong host slot": _mutate(acts, ip, ("P", hp + 1, kp, tp)),
        # a prefetch into a slot beyond the fast budget
        "prefetch beyond s": _mutate(acts, ip, ("P", hp, s, tp)),
        # a prefetch issued before the store that fills its host slot
        "prefetch before store": [a for a in acts if not (a[0] == "W" and a[2] == hp)],
        # a dropped prefetch: the reverse restores a state no slot holds
        "dropped prefetch": acts[:ip] + acts[ip + 1:],
    }
    for name, bad in planted.items():
        with pytest.raises(AssertionError):
            S.check(n, s, H, bad)
            pytest.fail(f"check() accepted: {name}")
