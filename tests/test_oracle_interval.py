"""The interval chosen from measured timings (Section 3), oracle and C ABI
(CPU only).

Rule 0 is the paper's: the smallest I whose forward sweep hides one transfer.
Rule 1 picks, among I up to that one, the interval with the least modelled
time per step.  The model is pinned against a discrete-event simulation of
the two-level pass written independently here: a host link that moves one
state at a time, two fast slots for the interval starts (a start's slot is
taken again two starts later, after its store has finished), the reverse
prefetching one interval ahead and recomputing inside each interval with
s - 1 slots.  Rule 1's interval must be (up to edge effects of the first and
last interval) the fastest in that simulation; rule 0's is never faster.
"""
import math

import pytest

from oracle import schedule as S

amb = pytest.importorskip("paper_1806_01117_amd")


def simulate(n, s, I, t_a, t_t, t_b):
    """Device time of one pass under the two-level policy with interval I."""
    K = -(-n // I)
    dev = link = 0.0
    slot_free = [0.0, 0.0]
    for k in range(K - 1):                      # sweep: start k -> slot k % 2, store, advance I steps
        dev = max(dev, slot_free[k % 2])
        end = max(dev, link) + t_t
        link = slot_free[k % 2] = end
        dev += I * t_a
    for k in range(K - 1, -1, -1):              # reverse from the last interval
        l = n - k * I if k == K - 1 else I
        pref_end = None
        if k >= 1:
            pref_end = max(dev, link) + t_t
            link = pref_end
        dev += S.advances(l, s - 1) * t_a + l * t_b + (t_a if k == K - 1 else 0.0)
        if pref_end is not None:
            dev = max(dev, pref_end)
    return dev


GRID = [(t_a, t_t, s) for t_a in (5.7, 18.0, 25.0) for t_t in (3.0, 6.4, 11.0, 40.0, 48.0, 90.0, 200.0)
        for s in (3, 10, 16, 32)]


@pytest.mark.parametrize("t_a,t_t,s", GRID)
def test_rule_matches_the_simulated_optimum(t_a, t_t, s):
    n = 3000
    strict = max(1, math.ceil(t_t / t_a))
    I1 = S.interval_from_timings(t_a, t_t, s, 1)
    I0 = S.interval_from_timings(t_a, t_t, s, 0)
    assert I0 == strict and 1 <= I1 <= I0
    sim = {I: simulate(n, s, I, t_a, t_t, 2.0 * t_a) for I in range(1, strict + 1)}
    best = min(sim.values())
    assert sim[I1] <= 1.005 * best, (I1, sim)
    assert sim[I0] >= sim[I1] * 0.999


def test_rule_edge_cases():
    assert S.interval_from_timings(10.0, 9.0, 8, 1) == 1 == S.interval_from_timings(10.0, 9.0, 8, 0)
    assert S.interval_from_timings(10.0, 0.0, 8, 1) == 1
    assert S.interval_from_timings(10.0, 35.0, 1, 1) == 4          # one slot: no two-level schedule
    assert S.interval_from_timings(6.0, 6.3, 10, 0, slack=0.05) == 1  # a 5 % slack hides the transfer


@pytest.mark.parametrize("rule", [0, 1])
def test_c_abi_matches_oracle(rule):
    for t_a in (0.5, 5.69, 18.18, 24.5, 546.0):
        for t_t in (0.0, 1.0, 6.4, 39.4, 47.9, 1000.0, 5000.0):
            for s in (1, 2, 3, 10, 32, 64):
                assert amb.interval_from_timings(t_a, t_t, s, rule) == S.interval_from_timings(t_a, t_t, s, rule), \
                    (t_a, t_t, s, rule)
    with pytest.raises(ValueError):
        amb.interval_from_timings(0.0, 1.0, 4)
