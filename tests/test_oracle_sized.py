"""Pins for schedules over states of different sizes (CPU only).

Sections 1.1 and 6 set states of unequal size beside Revolve's uniform ones
and would checkpoint them, inside each interval, with a one-level method for
unequal states.  The oracle's SizedSplits runs Revolve's
recursion with a memory budget in units of a common granule, the snapshots
stacked in a byte-addressed pool.  Pinned against:
  * Revolve itself: with unit sizes the schedules are the canonical ones,
    action for action (one and two levels), and with unit sizes and step
    costs those of the cost splits;
  * hand-derived lists (tests/golden/schedules_sized.txt);
  * a brute-force shortest-path search over every strategy of one memory
    level under the same byte budget (advance, snapshot if it fits, drop,
    restore, adjoint): its least cost equals the recursion's;
  * the uniform treatment (every state in a slot of the largest size),
    which it never exceeds;
  * the symbolic checker with the pool's budget and the stack layout, which
    also rejects planted mistakes;
  * a CPU replay with the MLP cell of layers of different widths, equal to
    store-all BPTT bit for bit.
"""
import heapq
import os
import random

import numpy as np
import pytest

from oracle import bptt
from oracle import schedule as S
from oracle.cells import Cell

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "schedules_sized.txt")


def _golden():
    cases, cur = [], None
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        if line.startswith("case "):
            cur = [tuple(int(v) for v in line.split()[1:]), None, ""]
            cases.append(cur)
        elif line.startswith("sizes "):
            cur[1] = [int(v) for v in line.split()[1:]]
        else:
            cur[2] += line
    return cases


@pytest.mark.parametrize("case", _golden(), ids=lambda c: "-".join(map(str, c[1])))
def test_hand_derived_golden(case):
    (n, s, H, I), sizes, want = case
    assert S.text_sized(n, s, sizes, H, I) == want


def test_unit_sizes_give_the_canonical_schedules():
    for n in list(range(1, 40)) + [64, 100]:
        for s in range(1, 7):
            for H, I in ((0, 0), (100, 2), (100, 3), (7, 1), (3, 0)):
                head, body = S.text_sized(n, s, [1] * (n + 1), H, I).split("\n", 1)
                chead, cbody = S.text(n, s, H, I).split("\n", 1)
                assert head == chead + " split=size" and body == cbody, (n, s, H, I)
    # any common size is the same as unit sizes
    assert S.text_sized(30, 4, [3] * 31, 100, 3) == S.text_sized(30, 4, [1] * 31, 100, 3)


def test_unit_sizes_with_costs_give_the_cost_splits():
    rng = random.Random(2)
    for _ in range(60):
        n, s = rng.randint(2, 40), rng.randint(1, 6)
        costs = [rng.choice([1.0, 2.0, 0.5, 4.0]) for _ in range(n)]
        a = S.text_sized(n, s, [1] * (n + 1), 0, 0, costs).split("\n", 1)[1]
        b = S.text_costs(n, s, costs).split("\n", 1)[1]
        assert a == b, (n, s, costs)


def brute_force(sizes, costs, P):
    """Least total cost of advanced steps that runs every adjoint n-1 .. 0 with
    one memory level of P units (x_0 held at the start, the live state not
    counted), over every strategy."""
    n = len(costs)
    start = (0, frozenset([0]), n - 1)
    dist = {start: 0.0}
    pq = [(0.0, 0, start)]
    tie = 1
    while pq:
        d, _, st = heapq.heappop(pq)
        if d > dist[st]:
            continue
        live, held, nxt = st
        if nxt < 0:
            return d
        moves = []
        if live is not None and live < nxt:
            moves.append(((live + 1, held, nxt), costs[live]))
        if live is not None and live not in held and sum(sizes[h] for h in held) + sizes[live] <= P:
            moves.append(((live, held | {live}, nxt), 0.0))
        for h in held:
            moves.append(((live, held - {h}, nxt), 0.0))
            moves.append(((h, held, nxt), 0.0))
        if live == nxt:
            moves.append(((None, held, nxt - 1), 0.0))
        for nst, c in moves:
            nd = d + c
            if nd < dist.get(nst, float("inf")):
                dist[nst] = nd
                heapq.heappush(pq, (nd, tie, nst))
                tie += 1
    raise AssertionError("unreachable")


def test_recursion_equals_brute_force_over_every_strategy():
    rng = random.Random(17)
    for trial in range(150):
        n = rng.randint(1, 7)
        sizes = [rng.randint(1, 3) for _ in range(n + 1)]
        costs = [float(rng.randint(1, 4)) for _ in range(n)] if trial % 2 else [1.0] * n
        P = rng.randint(sizes[0], sizes[0] + 5)
        want = brute_force(sizes, costs, P)
        ss = S.SizedSplits(sizes, costs)
        assert ss.T(0, n, P - sizes[0]) == want, (sizes, costs, P)


def test_never_worse_than_slots_of_the_largest_size():
    rng = random.Random(23)
    for _ in range(80):
        n, s = rng.randint(2, 60), rng.randint(1, 5)
        sizes = [rng.choice([1, 1, 2, 4]) for _ in range(n + 1)]
        H, I = rng.choice([(0, 0), (100, 3), (100, 5), (6, 0)])
        head, acts = S.schedule_sized(n, s, sizes, H, I)
        uni, _ = S.schedule_sized(n, s, [max(sizes)] * (n + 1), H, I)
        assert head["evals"] <= uni["evals"], (n, s, sizes, H, I)


def _random_cases(seed, count):
    rng = random.Random(seed)
    for _ in range(count):
        n, s = rng.randint(1, 50), rng.randint(1, 5)
        sizes = [rng.choice([1, 2, 3, 4]) for _ in range(n + 1)]
        H, I = rng.choice([(0, 0), (100, 2), (100, 4), (5, 0), (2, 1)])
        yield n, s, sizes, H, I


def test_sized_schedules_are_valid_within_the_pool():
    for n, s, sizes, H, I in _random_cases(29, 300):
        head, acts = S.schedule_sized(n, s, sizes, H, I)
        c = S.check_sized(n, s, H, acts, sizes, head["mode"] != "revolve")
        assert c["evals"] == head["evals"] and c["peak_units"] <= s * max(sizes)


def test_sized_schedules_over_chosen_starts():
    rng = random.Random(31)
    for _ in range(100):
        n, s = rng.randint(3, 60), rng.randint(2, 5)
        sizes = [rng.choice([1, 2, 3]) for _ in range(n + 1)]
        starts = sorted({0} | set(rng.sample(range(1, n), rng.randint(0, min(6, n - 1)))))
        head, acts = S.schedule_sized_from_starts(n, s, 100, starts, sizes)
        c = S.check_sized(n, s, 100, acts, sizes, True)
        assert c["evals"] == head["evals"] and c["stores"] == len(starts) - 1


def test_checker_rejects_planted_mistakes():
    n, s, sizes = 12, 2, [2, 1, 1, 2, 1, 1, 1, 2, 1, 1, 1, 1, 2]
    head, acts = S.schedule_sized(n, s, sizes)
    S.check_sized(n, s, 0, acts, sizes, False)
    # a snapshot one level deeper than the recursion puts it: past the pool
    i = max(i for i, a in enumerate(acts) if a[0] == "S")
    k = max(a[1] for a in acts if a[0] == "S")
    deeper = list(acts)
    deeper[i] = ("S", k + 3, acts[i][2])
    deeper = [("R", k + 3, a[2]) if a[0] == "R" and a[1] == acts[i][1] and a[2] == acts[i][2] else a for a in deeper]
    with pytest.raises(AssertionError):
        S.check_sized(n, s, 0, deeper, sizes, False)
    # a lower slot rewritten while a state above it is still to be restored
    j = next(j for j, a in enumerate(acts) if a[0] == "S" and a[1] == 2)
    moved = list(acts)
    moved.insert(j + 1, ("S", 1, acts[j][2]))
    with pytest.raises(AssertionError):
        S.check_sized(n, s, 0, moved, sizes, False)


def _mlp(widths, loss, B=2, seed=3):
    rng = np.random.default_rng(seed)
    n = len(widths) - 1
    Ws = {l: (rng.standard_normal((widths[l + 1], widths[l])) * (1.4 / np.sqrt(widths[l])),
              rng.standard_normal(widths[l + 1]) * 0.2) for l in range(n)}
    cell = Cell("mlp", loss, B, 0, max(widths), layer=lambda l: Ws[l])
    y0 = (rng.standard_normal((B, widths[0])),)
    return cell, y0


@pytest.mark.parametrize("loss", ["half_sq_last", "mean_sq_all", "mean_last"])
def test_replay_of_sized_schedules_equals_store_all(loss):
    widths = [8, 4, 12, 4, 4, 16, 8, 4, 12, 8, 4, 8, 16, 4, 8, 4, 12]
    n, B = len(widths) - 1, 2
    cell, y0 = _mlp(widths, loss, B)
    zero = np.zeros((B, 0))
    want = bptt.store_all(cell, n, lambda t: zero, y0)
    sizes = [w // 4 for w in widths]
    for s, H, I in ((1, 0, 0), (2, 0, 0), (3, 0, 0), (2, 100, 3), (3, 6, 0), (2, 100, 1)):
        head, acts = S.schedule_sized(n, s, sizes, H, I)
        got = S.replay(cell, n, lambda t: zero, y0, acts)
        assert got["loss"] == want["loss"], (s, H, I)
        for l in range(n):
            assert np.array_equal(got["dW"][l], want["dW"][l]) and np.array_equal(got["db"][l], want["db"][l])
        assert np.array_equal(got["dx0"][0], want["dx0"][0])


amb_lib = pytest.importorskip("paper_1806_01117_amd")


def test_c_abi_sized_text_equals_the_oracle():
    """The library's sized schedule builder against the oracle, byte for byte."""
    rng = random.Random(37)
    cases = list(_random_cases(41, 250))
    cases += [(n, s, [rng.choice([1, 2, 4, 8]) for _ in range(n + 1)], H, I)
              for n, s, H, I in ((90, 2, 0, 0), (120, 3, 40, 0), (64, 2, 64, 1))]
    for n, s, sizes, H, I in cases:
        costs = [rng.choice([1.0, 2.0, 0.5]) for _ in range(n)] if rng.random() < 0.3 else None
        want = S.text_sized(n, s, sizes, H, I, costs)
        assert amb_lib.schedule_text_sized(n, s, sizes, H, I, costs) == want, (n, s, sizes, H, I)


def test_c_abi_sized_errors():
    from paper_1806_01117_amd._lib import EINVAL, EUNSUPPORTED, AmbpttError
    with pytest.raises(AmbpttError) as e:
        amb_lib.schedule_text_sized(4, 2, [1, 1, 0, 1, 1])
    assert e.value.status == EINVAL
    with pytest.raises(AmbpttError) as e:    # one reversal of 400 steps on 1200 units: table too large
        amb_lib.schedule_text_sized(400, 300, [4] * 401)
    assert e.value.status == EUNSUPPORTED


def test_parts_that_fit_are_answered_without_the_recursion():
    """A part whose inner states all fit: the recursion itself splits at 1 and
    costs each step once, which is what T and split return directly."""
    rng = random.Random(43)
    for _ in range(200):
        n = rng.randint(2, 12)
        sizes = [rng.randint(1, 3) for _ in range(n + 1)]
        costs = [rng.choice([0.5, 1.0, 2.0]) for _ in range(n)] if rng.random() < 0.5 else None
        ss = S.SizedSplits(sizes, costs)
        a = rng.randint(0, n - 2)
        l = rng.randint(2, n - a)
        M = sum(sizes[a + 1:a + l]) + rng.randint(0, 2)
        assert ss.fits(a, l, M)
        v, m = ss._solve(a, l, M)
        assert m == 1 and v == pytest.approx(ss.C(a, a + l - 1), rel=1e-12)
        assert ss.split(a, l, M) == 1 and ss.T(a, l, M) == ss.C(a, a + l - 1)
        # one unit less than everything needs: the recursion must recompute
        assert not ss.fits(a, l, sum(sizes[a + 1:a + l]) - 1)


def test_store_all_over_many_states_of_different_sizes():
    """A slot for every state: the schedule advances every step once, for the
    oracle and the library alike, with no table (400 steps would need a table
    of 257 M entries; the library also over 2000)."""
    n = 400
    sizes = [4, 2, 1, 2] * (n // 4) + [4]
    txt = S.text_sized(n, n + 1, sizes)
    _, acts = S.parse(txt)
    assert sum(a[2] - a[1] for a in acts if a[0] == "A") == n - 1   # with the first turn's step: n
    assert amb_lib.schedule_text_sized(n, n + 1, sizes) == txt
    _, big = S.parse(amb_lib.schedule_text_sized(2000, 2001, [4, 2, 1, 2] * 500 + [4]))
    assert sum(a[2] - a[1] for a in big if a[0] == "A") == 1999
