"""Pins for the oracle's online checkpointing schedules (CPU only).

Online checkpointing decides where to hold states while the number of steps
is still unknown (the variant Section 1.1 names beside Revolve).  Pinned
against things other than the generator itself:
  * hand-derived small schedules (tests/golden/schedules_online.txt);
  * the symbolic checker on every generated schedule (slots and host slots
    hold what each action claims, adjoints run n-1 .. 0 once);
  * the online property itself: every action before the sweep reaches
    x_{n-1} is the same for every longer sequence;
  * optimality where an online placement can reach it: for n <= beta(s, 2)
    the forward count equals the brute-force optimum of binomial
    checkpointing (a dynamic program over every split);
  * the least possible repetition number: no step is evaluated more often
    than the closed-form r(n, s) of binomial checkpointing allows;
  * the two-level composition: interval starts every I steps with the
    fixed-interval policy's count for all but the last interval;
  * replay on a tiny LSTM equals store-all BPTT bit for bit.
"""
import functools
import os

import numpy as np
import pytest

from oracle import bptt
from oracle import schedule as S
from oracle.cells import Cell

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "schedules_online.txt")


@functools.lru_cache(maxsize=None)
def dp(l: int, s: int) -> int:
    """Least advanced steps over every split point (brute force)."""
    if l == 1:
        return 0
    if s == 1:
        return sum(range(1, l))
    return min(m + dp(l - m, s - 1) + dp(m, s) for m in range(1, l))


def _golden_cases():
    cases, cur = [], None
    for ln in open(GOLDEN):
        if ln.startswith("#"):
            continue
        if ln.startswith("case "):
            cur = [tuple(int(v) for v in ln.split()[1:]), ""]
            cases.append(cur)
        elif cur is not None:
            cur[1] += ln
    return cases


@pytest.mark.parametrize("case", _golden_cases(), ids=lambda c: "-".join(map(str, c[0])))
def test_hand_derived_golden(case):
    (n, s, H, I), txt = case
    assert S.text_online(n, s, H, I) == txt


def _sweep_events(acts):
    """Actions of the forward sweep (before the first turn or the first
    prefetch) with advances split into single steps."""
    ev = []
    for a in acts:
        if a[0] in ("F", "P"):
            break
        if a[0] == "A":
            ev += [("A", t) for t in range(a[1], a[2])]
        else:
            ev.append(a)
    return ev


GRID = [(s, H, I) for s in (1, 2, 3, 4, 6) for H, I in ((0, 0), (1, 1), (2, 2), (3, 1), (5, 3), (1000, 2))]


@pytest.mark.parametrize("s,H,I", GRID)
def test_valid_and_counted(s, H, I):
    for n in list(range(1, 50)) + [97, 150]:
        head, acts = S.schedule_online(n, s, H, I)
        c = S.check(n, s, H, acts)
        assert c["evals"] == head["evals"], (n, s, H, I)
        # no fewer than the offline optimum in one level, than n in two
        assert c["evals"] >= (dp(n, s) + 1 if H == 0 or s == 1 else n), (n, s, H, I)


def _sweep_of_shorter(full, n):
    """The part of a longer sequence's sweep that a sequence of n steps also
    runs: up to reaching x_{n-1}, without the decision about x_{n-1} (only
    taken when step n-1 is known to exist)."""
    count = 0
    for i, e in enumerate(full):
        if e[0] == "A":
            if n == 1:
                return full[:i]
            count += 1
            if count == n - 1:
                return full[:i + 1]
    raise AssertionError("longer sequence expected")


@pytest.mark.parametrize("s,H,I", GRID)
def test_sweep_does_not_depend_on_n(s, H, I):
    N = 70
    full = _sweep_events(S.schedule_online(N, s, H, I)[1])
    for n in range(1, N):
        ev = _sweep_events(S.schedule_online(n, s, H, I)[1])
        assert ev == _sweep_of_shorter(full, n), (n, s, H, I)


def test_single_level_optimal_up_to_beta_s_2():
    for s in range(1, 11):
        for n in range(1, S.beta(s, 2) + 1):
            assert S.schedule_online(n, s)[0]["evals"] == dp(n, s) + 1, (n, s)


def _repetitions(n, acts):
    c = [0] * n
    for a in acts:
        if a[0] == "A":
            for t in range(a[1], a[2]):
                c[t] += 1
        elif a[0] == "F":
            c[a[1]] += 1
    return max(c)


def test_least_repetition_number():
    for s in range(1, 9):
        for n in range(1, 260):
            _, acts = S.schedule_online(n, s)
            assert _repetitions(n, acts) == max(1, S.revolve_r(n, s)), (n, s)


def test_overhead_over_revolve_is_bounded():
    # regression guard for the placement heuristic (not a property the
    # cited work fixes): at most 13 % more forward evaluations than the
    # offline optimum for s >= 2, and 2 % for s >= 8
    for s, bound in ((2, 1.13), (3, 1.13), (4, 1.13), (8, 1.02), (10, 1.02)):
        pol = S.OnlinePlacement(s, 0)
        for n in range(2, 1500):
            if n >= 3:
                pol.decide(n - 2)
            ev = n + pol.reverse_cost(pol.held, n - 1)
            assert ev <= bound * (dp(n, s) + 1) if n < 300 else ev <= bound * S.revolve_evals(n, s), (n, s)
            if n in (3, 50, 499, 1499):
                assert ev == S.schedule_online(n, s)[0]["evals"], (n, s)


def test_two_level_composition():
    # unbounded host tier: starts every I steps; all intervals but the last
    # cost what the fixed-interval policy charges them, the last one what the
    # single-level online placement with s - 1 slots charges a sequence of
    # its length
    for s in (2, 3, 5):
        for I in (1, 2, 3, 7):
            for n in range(1, 60):
                # starts are the multiples of I up to n-2: x_{n-1} is known
                # to be the last state when it is reached
                K = 1 + max(n - 2, 0) // I
                last = n - (K - 1) * I
                want = (K - 1) * I + (K - 1) * S.advances(I, s - 1) + S.schedule_online(last, s - 1)[0]["evals"]
                head, acts = S.schedule_online(n, s, 10 ** 6, I)
                assert head["evals"] == want, (n, s, I)
                assert [a[3] for a in acts if a[0] == "W"] == list(range(0, max(n - 1, 1), I)), (n, s, I)
    # I = 1 stores every state: no recomputation
    for n in range(1, 40):
        assert S.schedule_online(n, 3, 10 ** 6, 1)[0]["evals"] == n


def test_thinning_keeps_multiples_of_the_interval():
    for I0 in (1, 3):
        for H in (1, 2, 3, 4, 7):
            for n in range(2, 200, 7):
                _, acts = S.schedule_online(n, 4, H, I0)
                c = S.check(n, 4, H, acts)
                assert c["stores"] >= 1
                assert max(a[2] for a in acts if a[0] == "W") < H
                # the starts prefetched in the reverse, and the last start,
                # are the multiples of one interval I0 * 2^j
                starts = sorted({a[3] for a in acts if a[0] == "P"} | {0})
                if len(starts) >= 2:
                    gaps = {y - x for x, y in zip(starts, starts[1:])}
                    assert len(gaps) == 1, (H, n, starts)
                    g = gaps.pop()
                    assert g % I0 == 0 and (g // I0) & (g // I0 - 1) == 0, (H, n, g)


def _tiny_lstm(n):
    rng = np.random.default_rng(7)
    D, Hd, B = 3, 4, 2
    W = rng.uniform(-0.5, 0.5, (4 * Hd, D + Hd))
    b = rng.uniform(-0.2, 0.2, 4 * Hd)
    u = rng.standard_normal((n, B, D))
    x0 = (rng.standard_normal((B, Hd)) * 0.3, np.zeros((B, Hd)))
    cell = Cell("lstm", "mean_sq_all", B, D, Hd, W=W, b=b)
    return cell, (lambda t: u[t]), x0


@pytest.mark.parametrize("n,s,H,I", [(1, 2, 0, 0), (9, 2, 0, 0), (23, 3, 0, 0), (23, 3, 2, 2), (40, 4, 3, 3),
                                     (17, 1, 0, 0), (30, 5, 1000, 1)])
def test_replay_equals_store_all(n, s, H, I):
    cell, u_of, x0 = _tiny_lstm(n)
    want = bptt.store_all(cell, n, u_of, x0)
    _, acts = S.schedule_online(n, s, H, I)
    got = S.replay(cell, n, u_of, x0, acts)
    assert got["loss"] == want["loss"]
    for k in ("dW", "db"):
        assert np.array_equal(got[k], want[k]), k
    for a, b in zip(got["dx0"], want["dx0"]):
        assert np.array_equal(a, b)
