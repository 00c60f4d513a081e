"""Pins for schedules split for unequal step costs (CPU only).

The paper names layers of unequal cost and size as the case Revolve does not
cover (Sections 1.1 and 6).  The oracle's WeightedSplits chooses Revolve's
split points by dynamic programming over weighted step costs.  Pinned
against:
  * Revolve itself: with equal costs the schedule is the canonical one, action
    for action (the DP's tie-break meets the closed-form split range);
  * a brute-force shortest-path search over every strategy of one memory level
    (advance, snapshot, drop, restore, adjoint; not only recursive splits) on
    tiny sequences: its least cost equals the DP's;
  * Revolve's weighted cost on the same costs, which it never exceeds;
  * the symbolic checker and a replay equal to store-all BPTT;
  * the C ABI, byte for byte.
"""
import heapq
import random

import numpy as np
import pytest

from oracle import bptt
from oracle import schedule as S
from oracle.cells import Cell

amb = pytest.importorskip("paper_1806_01117_amd")


def _actions(txt):
    return txt.split("\n", 1)[1]


def _weighted(acts, costs):
    n = len(costs)
    return sum(sum(costs[t] for t in range(a[1], a[2])) for a in acts if a[0] == "A") + costs[n - 1]


def test_equal_costs_give_the_revolve_schedule():
    for s in range(1, 7):
        for H, I in ((0, 0), (100, 2), (100, 3), (7, 1)):
            for n in list(range(1, 45)) + [80, 130]:
                got = S.text_costs(n, s, [2.0] * n, H, I)
                assert got.split("\n", 1)[0].endswith(" split=cost")
                assert _actions(got) == _actions(S.text(n, s, H, I)), (n, s, H, I)


def brute_force(costs, s):
    """Least total cost of advanced steps that runs every adjoint n-1 .. 0 in
    one memory level of s states (x_0 held at the start), over every strategy."""
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
        if live is not None and live not in held and len(held) < s:
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


def test_dp_equals_brute_force_over_every_strategy():
    rng = random.Random(11)
    for trial in range(60):
        n = rng.randint(1, 7)
        s = rng.randint(1, 3)
        costs = [float(rng.randint(1, 5)) for _ in range(n)]
        want = brute_force(costs, s)
        ws = S.WeightedSplits(costs)
        assert ws.T(0, n, s) == want, (costs, s)
        head, acts = S.schedule_costs(n, s, costs)
        assert head["cost"] == want + costs[-1] == _weighted(acts, costs)


def test_never_costlier_than_revolve():
    rng = random.Random(5)
    for trial in range(80):
        n = rng.randint(2, 70)
        s = rng.randint(2, 6)
        H, I = rng.choice([(0, 0), (100, 3), (100, 5)])
        costs = [rng.choice([1.0, 1.0, 2.0, 4.0, 0.5]) for _ in range(n)]
        head, acts = S.schedule_costs(n, s, costs, H, I)
        _, racts = S.schedule(n, s, H, I)
        c = S.check(n, s, H, acts)
        assert c["evals"] == head["evals"]
        assert head["cost"] == _weighted(acts, costs) <= _weighted(racts, costs), (n, s, H, I)


def test_a_costly_step_is_recomputed_less():
    # one step 50 times dearer than the rest: the schedule snapshots right
    # after it instead of recomputing it as Revolve's split would
    n, s = 30, 3
    costs = [1.0] * n
    costs[4] = 50.0
    ev = lambda acts: sum(1 for a in acts if a[0] == "A" and a[1] <= 4 < a[2])
    _, acts = S.schedule_costs(n, s, costs)
    _, racts = S.schedule(n, s)
    assert ev(acts) < ev(racts)


@pytest.mark.parametrize("n,s,H,I", [(23, 3, 0, 0), (31, 4, 100, 4), (17, 2, 0, 0)])
def test_replay_equals_store_all(n, s, H, I):
    rng = np.random.default_rng(2)
    D, Hd, B = 3, 4, 2
    cell = Cell("lstm", "mean_sq_all", B, D, Hd, W=rng.uniform(-0.5, 0.5, (4 * Hd, D + Hd)),
                b=rng.uniform(-0.2, 0.2, 4 * Hd))
    u = rng.standard_normal((n, B, D))
    x0 = (rng.standard_normal((B, Hd)) * 0.3, np.zeros((B, Hd)))
    costs = list(rng.choice([1.0, 3.0], n))
    _, acts = S.schedule_costs(n, s, costs, H, I)
    got = S.replay(cell, n, lambda t: u[t], x0, acts)
    want = bptt.store_all(cell, n, lambda t: u[t], x0)
    assert got["loss"] == want["loss"] and np.array_equal(got["dW"], want["dW"])
    for a, b in zip(got["dx0"], want["dx0"]):
        assert np.array_equal(a, b)


def test_c_abi_matches_oracle_bytewise():
    rng = random.Random(3)
    for trial in range(200):
        n = rng.randint(1, 60)
        s = rng.randint(1, 6)
        H = rng.choice([0, 0, 5, 100])
        I = rng.randint(0, 4)
        costs = [rng.choice([0.5, 1.0, 1.0, 2.5, 3.0]) for _ in range(n)]
        assert amb.schedule_text_costs(n, s, costs, H, I) == S.text_costs(n, s, costs, H, I), (n, s, H, I)
    with pytest.raises(amb.AmbpttError):
        amb.schedule_text_costs(3, 2, [1.0, 0.0, 1.0])


def test_c_abi_cost_errors():
    import math
    with pytest.raises(amb.AmbpttError, match="positive"):
        amb.schedule_text_costs(4, 2, [1.0, math.nan, 1.0, 1.0])
    with pytest.raises(amb.AmbpttError, match="positive"):
        amb.schedule_text_costs(4, 2, [1.0, math.inf, 1.0, 1.0])
    # one reversal of 400 steps on 10 slots: 400 * 401 * 11 entries exceed the table limit
    with pytest.raises(amb.AmbpttError, match="too large"):
        amb.schedule_text_costs(400, 10, [1.0] * 400)
    # the same steps in two levels: the intervals are the reversals
    txt = amb.schedule_text_costs(400, 10, [1.0] * 400, 400, 4)
    assert txt.startswith("ambptt-schedule v1 n=400 s=10 H=400 I=4 mode=async split=cost")


def test_costs_over_chosen_starts():
    rng = random.Random(8)
    for trial in range(60):
        n = rng.randint(2, 60)
        s = rng.randint(2, 6)
        k = rng.randint(0, min(n - 1, 8))
        starts = [0] + sorted(rng.sample(range(1, n), k))
        costs = [rng.choice([0.5, 1.0, 3.0]) for _ in range(n)]
        head, acts = S.schedule_from_starts(n, s, n, starts, costs)
        c = S.check(n, s, n, acts)
        assert c["evals"] == head["evals"] and head["cost"] == _weighted(acts, costs)
        _, racts = S.schedule_from_starts(n, s, n, starts)
        assert head["cost"] <= _weighted(racts, costs)
        eq = S.text_from_starts(n, s, n, starts, [1.0] * n)
        assert _actions(eq) == _actions(S.text_from_starts(n, s, n, starts))


def test_c_abi_costs_over_chosen_starts_bytewise():
    """The library's schedule for stores decided during the sweep with step
    costs (ambptt_schedule_text_starts_costs) against the oracle, byte for
    byte, and its error codes."""
    rng = random.Random(12)
    for trial in range(150):
        n = rng.randint(2, 60)
        s = rng.randint(2, 6)
        H = rng.choice([n, n + 3, 8])
        k = rng.randint(0, min(n - 1, H, 8))
        starts = [0] + sorted(rng.sample(range(1, n), k))
        costs = [rng.choice([0.5, 1.0, 3.0]) for _ in range(n)]
        assert amb.schedule_text_starts(n, s, H, starts, costs) == S.text_from_starts(n, s, H, starts, costs), \
            (n, s, H, starts)
    from paper_1806_01117_amd._lib import EINVAL, EUNSUPPORTED
    # an interval of 1499 steps reversed on 2 slots: 1499 * 1500 * 3 entries exceed the table limit
    with pytest.raises(amb.AmbpttError) as e:
        amb.schedule_text_starts(1500, 3, 10, [0, 1], [1.0] * 1500)
    assert e.value.status == EUNSUPPORTED
    with pytest.raises(amb.AmbpttError) as e:
        amb.schedule_text_starts(10, 3, 10, [0, 4], [1.0] * 9 + [0.0])
    assert e.value.status == EINVAL
    with pytest.raises(ValueError):
        amb.schedule_text_starts(10, 3, 10, [0, 4], [1.0] * 9)
