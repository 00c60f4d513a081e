"""Checkpointing schedules: Revolve and asynchronous two-level (float-free).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Vocabulary (one action per line in the canonical text):
  A t0 t1    advance the live state from x_t0 to x_t1 (t1 - t0 forward steps)
  S k t      take a snapshot: copy the live state x_t into fast slot k
  R k t      restore: the live state becomes x_t from fast slot k
  F t        first turn: forward step t = n-1 (x_n, loss, seed), then its adjoint
  Y t        adjoint of step t (needs the live state x_t and xbar_{t+1})
  W k h t    store fast slot k (holding x_t) to slow slot h, asynchronously
  P h k t    prefetch slow slot h (holding x_t) into fast slot k, asynchronously

Counting (Revolve, Griewank and Walther; the paper's R(n, s), Section 3):
  beta(s, r) = C(s + r, s).  With s slots (the one holding the interval's
  first state included) and l >= 1 steps, let r be the integer with
  beta(s, r-1) < l <= beta(s, r).  The least number of advanced steps needed
  to run the l adjoint steps is  F(l, s) = r*l - beta(s+1, r-1).
  Forward evaluations of a schedule = advanced steps + 1 (the first turn's
  forward step); the recompute factor is forward evaluations / n, so storing
  every state gives 1 (Section 1.1).

Split rule (one optimal choice among many; the paper does not fix it):
  reversing [a, a+l) with s >= 2 slots advances m steps, snapshots x_{a+m}
  into the lowest free slot, reverses [a+m, a+l) with s-1 slots, releases the
  slot, restores x_a and reverses [a, a+m) with s slots.  The optimal m form
  the range [lo, hi] with
      lo = max(1, l - beta(s-1, r), beta(s, r-2)),
      hi = min(l-1, beta(s, r-1), l - beta(s-1, r-1));
  this oracle takes m = hi.  With one slot the interval is reversed as a
  chain (restore x_a and advance i steps, for i = l-1 .. 0).  A restore is
  emitted only when the live state is not already x_a.

Asynchronous two-level policy (Section 2, with the interval of Section 3):
  interval I = max(I_min, 1, ceil(n / (H+1))) so that the K-1 stored states,
  K = ceil(n / I), fit in H slow slots.  Fast slots 0 and 1 alternately hold
  the interval starts (one being stored or prefetched while the other is in
  use); Revolve inside an interval gets the other s-1 slots (the start's slot
  included), i.e. working slots 2 .. s-1.
    forward sweep, k = 0 .. K-2:   S (k%2) kI ; W (k%2) k kI ; A kI (k+1)I
    reverse, k = K-1 .. 0, a = kI, l = n-a (last) or I, base = k%2:
       k = K-1: S base a
       k >= 1 : P (k-1) ((k-1)%2) (k-1)I        (prefetch one interval ahead)
       reverse [a, a+l) with s-1 slots
  Forward evaluations = (K-1) I + F(I_last, s-1) + 1 + (K-1) F(I, s-1).
  When H = 0, s < 2, I >= n, or this is not strictly fewer than plain
  Revolve needs with s slots, plain Revolve is used (the paper's fallback
  when not even one store fits, Section 3, generalised), so the policy never
  recomputes more than Revolve at the same fast-slot budget.

Stores when the previous transfer has completed (the non-uniform policy the
paper's conclusions propose instead of a fixed I): the interval starts
0 = t_0 < t_1 < ... < t_{K-1} < n are decided during the forward sweep, and
the same two-level rule applies with interval k = [t_k, t_{k+1}) (the last
one [t_{K-1}, n)):
    forward sweep, k = 0 .. K-2:   S (k%2) t_k ; W (k%2) k t_k ; A t_k t_{k+1}
    reverse, k = K-1 .. 0, a = t_k, l = its length, base = k%2:
       k = K-1: S base a
       k >= 1 : P (k-1) ((k-1)%2) t_{k-1}
       reverse [a, a+l) with s-1 slots
  Forward evaluations = t_{K-1} + sum_k F(l_k, s-1) + 1.  Fixed intervals are
  the case t_k = kI.

Online checkpointing (the number of steps unknown during the forward sweep,
the variant named in Section 1.1 beside Revolve): every decision about x_t is
taken when x_t is computed, knowing only that step t exists (t <= n-2); the
end of the sequence shows itself when x_{n-1} is reached.  Placement in m
fast slots from a sweep start a (our policy; the paper only cites the prior
work):
  held = [a], phase r = 1; segment j = [held_j, held_{j+1}) (the last one ends
  at the live state) may be at most cap_j = beta(m - j, r - 1) long, so that
  reversing it with the m - j slots it will have advances each step at most
  r - 1 more times; the phase-end placement P_r puts held_j at
  a + cap_0 + ... + cap_{j-1}.
  At x_t: if fewer than m states are held, hold x_t.  Otherwise the options
  are "drop held_j (j >= 1) and hold x_t", allowed when the merged segment
  fits cap_{j-1}, and "hold nothing new", allowed when the last segment
  extended to t+1 fits its cap; only options keeping every point of P_r at or
  before t are admissible.  None admissible: r += 1 and look again.  Among
  the admissible, take the least cost of reversing if the sweep ended at step
  t+1, sum_j F(l_j, m - j), then holding x_t before not, then the smallest j.
  Pinned: optimal (equal to Revolve) for n <= beta(s, 2), no step advanced
  more often than under Revolve (the least possible repetition number), and
  the forward prefix does not depend on n.
Single level (H = 0):  S 0 0, the sweep A/S of the placement with m = s in
  slots 0 .. s-1 (lowest free slot), F n-1, then the segments from the last
  down, segment j reversed with s - j slots by the split rule.
Two levels (H > 0, s >= 2): interval length I = max(I_min, 1) fixed up front.
  The sweep snapshots each interval start into fast slot 0 or 1 (alternating)
  and stores it to the lowest free host slot; inside an interval the
  placement above runs with m = s - 1 (the start's slot and working slots
  2 .. s-1).  When a start finds every host slot taken, I doubles and the
  stored starts that are not multiples of the new I give their host slots
  back (repeated while the step is still a start and nothing was freed).
  After the sweep: P of the previous start, F n-1, the last interval's
  segments, then the earlier intervals from the last down, each reversed by
  the split rule on s - 1 slots with its predecessor prefetched first (into
  the other one of slots 0, 1).

Unequal step costs (Sections 1.1 and 6 point to non-uniform layers): the
mode, interval and slots stay those above, and every reversal on two or more
slots splits where a dynamic program over the same recursion finds the least
total cost of recomputed forward steps (WeightedSplits); the header then ends
with " split=cost".

States of different sizes (the other non-uniform case of Sections 1.1 and 6;
inside an interval the paper would replace Revolve by an existing one-level
method for checkpoints of unequal size): sizes[t] is the size of x_t
in units of a common granule, and the fast memory is a byte-addressed pool of
P = s * max(sizes) units (s states of the largest size).  Checkpoints form a
stack: the snapshot taken at recursion depth k ("slot" k) sits right above
the ones below it, so its offset is the sum of their sizes (in two levels,
slots 0 and 1 are the interval starts' regions of max(sizes) units each and
the stack starts above them).  Reversing [a, a+l) with M units free beyond
x_a (SizedSplits):
    T(a, 1, M) = 0
    T(a, l, M) = min over m with sizes[a+m] <= M of
                 C(a, a+m) + T(a+m, l-m, M - sizes[a+m]) + T(a, m, M)
    (ties: the largest m), or the chain when no snapshot fits;
plain: M = P - sizes[0]; two levels: M = P - 2 max(sizes) in every interval.
The mode is the one with the smaller weighted forward cost (with unit costs:
forward evaluations), the two levels taken only when strictly cheaper.  With
unit sizes this is Revolve's recursion with M + 1 slots, and the schedules
are the canonical ones.  Header suffix " split=size".

Canonical text: a header line
  ambptt-schedule v1 n=<n> s=<s> H=<H> I=<I or 0> mode=<revolve|async|dynamic|online> [split=cost|size]
(I = 0 for revolve and dynamic, the initial interval for online, 0 when single
level) then the actions, single spaces, decimal integers, newline-terminated.
"""
from __future__ import annotations

import heapq
from math import comb

import numpy as np


def beta(s: int, r: int) -> int:
    if r < 0 or s < 0:
        return 0
    return comb(s + r, s)


def revolve_r(l: int, s: int) -> int:
    """Smallest r >= 0 with beta(s, r) >= l."""
    r = 0
    while beta(s, r) < l:
        r += 1
    return r


def advances(l: int, s: int) -> int:
    """F(l, s): least number of advanced steps to reverse l steps with s slots."""
    if l < 1 or s < 1:
        raise ValueError("need l >= 1 and s >= 1")
    r = revolve_r(l, s)
    return r * l - beta(s + 1, r - 1)


def split_range(l: int, s: int) -> tuple[int, int]:
    r = revolve_r(l, s)
    lo = max(1, l - beta(s - 1, r), beta(s, r - 2))
    hi = min(l - 1, beta(s, r - 1), l - beta(s - 1, r - 1))
    return lo, hi


def revolve_evals(n: int, s: int) -> int:
    return advances(n, s) + 1


def paper_model_R(n: int, s: int) -> float:
    """The recompute factor of the paper's performance model (Section 3):
    R(n, s) for plain Revolve over n steps; the model's asynchronous factor
    is R(I, s), the same function at the interval length (it leaves out the
    sweep that produces the stored states, which the schedules here count)."""
    return revolve_evals(n, s) / n


def choose(n: int, s: int, H: int, I_min: int) -> tuple[str, int, int]:
    """(mode, I, forward evaluations) under the policy above."""
    plain = revolve_evals(n, s)
    if H <= 0 or s < 2:
        return "revolve", 0, plain
    I = max(I_min, 1, -(-n // (H + 1)))
    if I >= n:
        return "revolve", 0, plain
    K = -(-n // I)
    last = n - (K - 1) * I
    ev = (K - 1) * I + advances(last, s - 1) + 1 + (K - 1) * advances(I, s - 1)
    if ev >= plain:
        return "revolve", 0, plain
    return "async", I, ev


def interval_from_timings(t_a: float, t_t: float, s: int, rule: int = 1, slack: float = 0.0) -> int:
    """Interval from measured times of one forward step (t_a) and of one
    state over the host link (t_t).  Rule 0 (Section 3): the smallest I whose
    sweep hides a transfer, ceil(t_t / t_a - slack).  Rule 1: over I = 1 ..
    that I, the least modelled time per step (max(I t_a, t_t) + F(I, s-1) t_a)
    / I, where a sweep interval lasts as long as its store when the link is
    slower, and the reverse recomputes F(I, s-1) of its steps; ties to the
    smaller I."""
    import math
    t_a = max(t_a, 1e-3)
    strict = max(1, math.ceil(t_t / t_a - slack))
    if rule == 0 or s < 2:
        return strict
    cost = {I: (max(I * t_a, t_t) + advances(I, s - 1) * t_a) / I for I in range(1, strict + 1)}
    return min(cost, key=lambda I: (cost[I], I))


class _Gen:
    def __init__(self, n: int):
        self.n = n
        self.out: list[tuple] = []
        self.live = None
        self.split = lambda a, l, k: split_range(l, k)[1]

    def emit(self, *a):
        self.out.append(a)

    def leaf(self, t):
        self.emit("F" if t == self.n - 1 else "Y", t)

    def restore(self, k, a):
        if self.live != a:
            self.emit("R", k, a)
            self.live = a

    def advance(self, t0, t1):
        self.emit("A", t0, t1)
        self.live = t1

    def reverse(self, a: int, l: int, s: int, base: int, free: list[int]):
        """Reverse [a, a+l) with s slots; x_a sits in slot `base`; `free` = free slot ids."""
        while True:
            if l == 1:
                self.restore(base, a)
                self.leaf(a)
                return
            if s == 1:
                for i in range(l - 1, -1, -1):
                    self.restore(base, a)
                    if i > 0:
                        self.advance(a, a + i)
                    self.leaf(a + i)
                return
            m = self.split(a, l, s)
            self.restore(base, a)
            self.advance(a, a + m)
            k = min(free)
            free.remove(k)
            self.emit("S", k, a + m)
            self.reverse(a + m, l - m, s - 1, k, free)
            free.append(k)
            l = m


def _reverse_sized(g: _Gen, ss: "SizedSplits", a: int, l: int, M: int, base: int, depth: int) -> None:
    """Reverse [a, a+l) with M units free above x_a (in slot `base`); the next
    snapshot goes to slot `depth` (the top of the stack)."""
    while True:
        if l == 1:
            g.restore(base, a)
            g.leaf(a)
            return
        m = ss.split(a, l, M)
        if m == 0:  # no snapshot fits: the chain from x_a
            for i in range(l - 1, -1, -1):
                g.restore(base, a)
                if i > 0:
                    g.advance(a, a + i)
                g.leaf(a + i)
            return
        g.restore(base, a)
        g.advance(a, a + m)
        g.emit("S", depth, a + m)
        _reverse_sized(g, ss, a + m, l - m, M - ss.z[a + m], depth, depth + 1)
        l = m


def _two_level(g: _Gen, n: int, s: int, starts: list[int], sized=None) -> None:
    """The sweep and the reverse of the two-level policy over the given
    interval starts; `sized` = (SizedSplits, M) reverses each interval with
    the sized recursion on M units above its start."""
    K = len(starts)
    ends = starts[1:] + [n]
    g.live = 0
    for k in range(K - 1):
        g.emit("S", k % 2, starts[k])
        g.emit("W", k % 2, k, starts[k])
        g.advance(starts[k], starts[k + 1])
    for k in range(K - 1, -1, -1):
        a, l, base = starts[k], ends[k] - starts[k], k % 2
        if k == K - 1:
            g.emit("S", base, a)
        if k >= 1:
            g.emit("P", k - 1, (k - 1) % 2, starts[k - 1])
        if sized is not None:
            _reverse_sized(g, sized[0], a, l, sized[1], base, 2)
        else:
            g.reverse(a, l, s - 1, base, list(range(2, s)))


def schedule(n: int, s: int, H: int = 0, I_min: int = 0) -> tuple[dict, list[tuple]]:
    """(header dict, action list) for n steps, s fast slots, H slow slots."""
    if n < 1 or s < 1 or H < 0 or I_min < 0:
        raise ValueError("need n >= 1, s >= 1, H >= 0, I_min >= 0")
    mode, I, ev = choose(n, s, H, I_min)
    g = _Gen(n)
    if mode == "revolve":
        g.emit("S", 0, 0)
        g.live = 0
        g.reverse(0, n, s, 0, list(range(1, s)))
    else:
        _two_level(g, n, s, list(range(0, n, I)))
    head = {"n": n, "s": s, "H": H, "I": I, "mode": mode, "evals": ev}
    return head, g.out


def dynamic_evals(n: int, s: int, starts: list[int]) -> int:
    ends = list(starts[1:]) + [n]
    return starts[-1] + sum(advances(e - a, s - 1) for a, e in zip(starts, ends)) + 1


def schedule_from_starts(n: int, s: int, H: int, starts: list[int], costs=None) -> tuple[dict, list[tuple]]:
    """(header dict, action list) of the two-level policy with interval starts
    decided during the sweep (stores whenever the previous one completed);
    with step costs every reversal is split by WeightedSplits."""
    starts = list(starts)
    if n < 1 or s < 2 or not starts or starts[0] != 0 or any(b <= a for a, b in zip(starts, starts[1:])) \
            or starts[-1] >= n or len(starts) - 1 > H:
        raise ValueError("need s >= 2 and starts 0 = t_0 < t_1 < ... < n with at most H + 1 of them")
    g = _Gen(n)
    if costs is not None:
        if len(costs) != n or any(not (c > 0) for c in costs):
            raise ValueError("need n positive step costs")
        ws = WeightedSplits(costs)
        g.split = lambda a, l, k: ws.split(a, l, k)
    _two_level(g, n, s, starts)
    head = {"n": n, "s": s, "H": H, "I": 0, "mode": "dynamic", "evals": dynamic_evals(n, s, starts)}
    if costs is not None:
        head["evals"] = sum(x[2] - x[1] for x in g.out if x[0] == "A") + 1
        head["cost"] = sum(ws.C(x[1], x[2]) for x in g.out if x[0] == "A") + costs[n - 1]
        head["split"] = "cost"
    return head, g.out


class OnlinePlacement:
    """Fast-slot placement for a sweep from x_a whose end is unknown (rules in
    the module docstring).  held: the times held, increasing, held[0] = a."""

    def __init__(self, m: int, a: int):
        if m < 1:
            raise ValueError("need m >= 1 slots")
        self.m, self.a, self.r = m, a, 1
        self.held = [a]

    def cap(self, j: int) -> int:
        return beta(self.m - j, self.r - 1)

    def phase_end_points(self) -> list[int]:
        pts, acc = [self.a], self.a
        for j in range(self.m - 1):
            acc += self.cap(j)
            pts.append(acc)
        return pts

    def reverse_cost(self, held: list[int], end: int) -> int:
        """Advances needed to reverse [a, end) from this placement (end = the last step's index)."""
        bounds = held + [end]
        return sum(advances(bounds[j + 1] - bounds[j], self.m - j) for j in range(len(held)))

    def decide(self, t: int):
        """x_t has been computed and step t exists.  Returns None (hold
        nothing new) or ("hold", dropped) with dropped the time given up or None."""
        if len(self.held) < self.m:
            self.held.append(t)
            return ("hold", None)
        k = len(self.held) - 1
        while True:
            must = [p for p in self.phase_end_points() if p <= t]
            opts = []
            for j in range(1, k + 1):
                nxt = self.held[j + 1] if j < k else t
                if nxt - self.held[j - 1] <= self.cap(j - 1):
                    opts.append((self.held[:j] + self.held[j + 1:] + [t], 0, j))
            if t + 1 - self.held[k] <= self.cap(k):
                opts.append((list(self.held), 1, 0))
            opts = [o for o in opts if all(p in o[0] for p in must)]
            if opts:
                held, skip, j = min(opts, key=lambda o: (self.reverse_cost(o[0], t + 1), o[1], o[2]))
                if skip:
                    return None
                dropped = self.held[j]
                self.held = held
                return ("hold", dropped)
            self.r += 1


def schedule_online(n: int, s: int, H: int = 0, I_min: int = 0) -> tuple[dict, list[tuple]]:
    """(header dict, action list) of online checkpointing over n steps; every
    action before the sweep reaches x_{n-1} is the same for every longer n."""
    if n < 1 or s < 1 or H < 0 or I_min < 0:
        raise ValueError("need n >= 1, s >= 1, H >= 0, I_min >= 0")
    two = H > 0 and s >= 2
    I0 = max(I_min, 1) if two else 0
    g = _Gen(n)
    g.live = 0
    g.emit("S", 0, 0)
    run = [0]  # first step of the advance not yet emitted

    def flush(t):
        if run[0] < t:
            g.advance(run[0], t)
        run[0] = t

    m = s - 1 if two else s
    work = list(range(2, s)) if two else list(range(1, s))
    base = 0
    slot_of = {0: 0}
    pol = OnlinePlacement(m, 0)
    starts = []  # (time, host slot) of the interval starts kept on the host
    I = I0
    if two:
        g.emit("W", 0, 0, 0)
        starts.append((0, 0))
        released, fresh = [], 1  # host slots given back (a heap), the next never used
    for t in range(1, n):
        if t == n - 1:
            break
        if two and t % I == 0:
            while not released and fresh >= H and t % I == 0:
                I *= 2
                keep = []
                for a, h in starts:
                    if a % I == 0:
                        keep.append((a, h))
                    else:
                        heapq.heappush(released, h)
                starts = keep
            if t % I == 0:
                flush(t)
                base = 1 - base
                g.emit("S", base, t)
                if released:  # the lowest free host slot
                    h = heapq.heappop(released)
                else:
                    h, fresh = fresh, fresh + 1
                g.emit("W", base, h, t)
                starts.append((t, h))
                pol = OnlinePlacement(m, t)
                slot_of = {t: base}
                continue
        d = pol.decide(t)
        if d is not None:
            used = set(slot_of.values())
            if d[1] is not None:
                used.discard(slot_of.pop(d[1]))
            k = min(x for x in work if x not in used)
            flush(t)
            g.emit("S", k, t)
            slot_of[t] = k
    flush(n - 1)
    if two and len(starts) >= 2:
        a, h = starts[-2]
        g.emit("P", h, 1 - base, a)
    g.leaf(n - 1)
    held = pol.held
    bounds = held + [n - 1]
    for j in range(len(held) - 1, -1, -1):
        l = bounds[j + 1] - bounds[j]
        if l > 0:
            busy = {slot_of[x] for x in held[:j + 1]}
            g.reverse(held[j], l, m - j, slot_of[held[j]], [x for x in work if x not in busy])
    if two:
        for k in range(len(starts) - 2, -1, -1):
            base = 1 - base
            if k >= 1:
                a, h = starts[k - 1]
                g.emit("P", h, 1 - base, a)
            a = starts[k][0]
            g.reverse(a, starts[k + 1][0] - a, s - 1, base, list(work))
    evals = sum(x[2] - x[1] for x in g.out if x[0] == "A") + 1
    head = {"n": n, "s": s, "H": H, "I": I0, "mode": "online", "evals": evals}
    return head, g.out


class WeightedSplits:
    """Optimal splits for reversing steps of unequal forward cost (the
    non-uniform case the paper's Sections 1.1 and 6 point to), by dynamic
    programming over Revolve's recursion.  costs[t] is the cost of forward
    step t.  With s slots (x_a's included) and the live state at x_a,
    reversing [a, a+l) costs
        T(a, 1, s) = 0                      (the adjoint of step a alone)
        T(a, l, 1) = sum_{i=1}^{l-1} C(a, a+i)   (restore x_a, advance i, for i = l-1 .. 1)
        T(a, l, s) = min_m  C(a, a+m) + T(a+m, l-m, s-1) + T(a, m, s)
    with C(a, b) the cost of steps a .. b-1; ties go to the largest m, so that
    equal costs give the Revolve split m = hi."""

    def __init__(self, costs):
        self.c = [float(x) for x in costs]
        self.pre = [0.0]
        for x in self.c:
            self.pre.append(self.pre[-1] + x)
        self.memo = {}

    def C(self, a: int, b: int) -> float:
        return self.pre[b] - self.pre[a]

    def T(self, a: int, l: int, s: int) -> float:
        return self._solve(a, l, s)[0]

    def split(self, a: int, l: int, s: int) -> int:
        return self._solve(a, l, s)[1]

    def _solve(self, a, l, s):
        key = (a, l, s)
        if key in self.memo:
            return self.memo[key]
        if l == 1:
            out = (0.0, 0)
        elif s == 1:
            acc = 0.0
            for i in range(1, l):
                acc += self.C(a, a + i)
            out = (acc, 0)
        else:
            best = None
            for m in range(1, l):
                v = self.C(a, a + m) + self._solve(a + m, l - m, s - 1)[0] + self._solve(a, m, s)[0]
                if best is None or v <= best[0]:
                    best = (v, m)
            out = best
        self.memo[key] = out
        return out


def schedule_costs(n: int, s: int, costs, H: int = 0, I_min: int = 0) -> tuple[dict, list[tuple]]:
    """The schedule of `schedule` (same mode, interval and slots) with every
    reversal of [a, a+l) on k >= 2 slots split where WeightedSplits puts it
    for the given step costs.  Equal costs give `schedule` itself."""
    if len(costs) != n or any(not (c > 0) for c in costs):
        raise ValueError("need n positive step costs")
    head, _ = schedule(n, s, H, I_min)
    ws = WeightedSplits(costs)
    g = _Gen(n)
    g.split = lambda a, l, k: ws.split(a, l, k)
    if head["mode"] == "revolve":
        g.emit("S", 0, 0)
        g.live = 0
        g.reverse(0, n, s, 0, list(range(1, s)))
    else:
        _two_level(g, n, s, list(range(0, n, head["I"])))
    evals = sum(x[2] - x[1] for x in g.out if x[0] == "A") + 1
    cost = sum(ws.C(x[1], x[2]) for x in g.out if x[0] == "A") + costs[n - 1]
    return dict(head, evals=evals, cost=cost, split="cost"), g.out


class SizedSplits:
    """Optimal splits when states differ in size (one-level checkpointing of
    unequal states, which Section 6 would run inside each interval and for
    which Section 1.1 cites a dynamic program): Revolve's
    recursion with a memory budget in units instead of a slot count.
    sizes[t] (t = 0 .. n) is the size of x_t in units, costs[t] the cost of
    forward step t (default 1).  With the live state at x_a and M units free
    above x_a's own checkpoint, reversing [a, a+l) costs
        T(a, 1, M) = 0
        T(a, l, M) = min over m with sizes[a+m] <= M of
                     C(a, a+m) + T(a+m, l-m, M - sizes[a+m]) + T(a, m, M)
    (x_{a+m} stays while [a+m, a+l) is reversed above it, then its units are
    free again for [a, a+m)); ties go to the largest m; when no snapshot fits
    the chain (restore x_a and advance i steps, i = l-1 .. 1) costs
    sum_{i=1}^{l-1} C(a, a+i).  A split that fits never costs more than the
    chain, so a split is always taken when one fits.  When every state of
    (a, a+l) fits in M, splitting at 1 at every level advances each step
    once and every other split costs more, so T and split answer such a part
    directly (C(a, a+l-1) and 1) without the recursion; the pins check this
    against the recursion."""

    def __init__(self, sizes, costs=None):
        self.z = [int(v) for v in sizes]
        n = len(self.z) - 1
        if n < 1 or any(v < 1 for v in self.z):
            raise ValueError("need n + 1 >= 2 positive sizes")
        self.c = [1.0] * n if costs is None else [float(x) for x in costs]
        if len(self.c) != n or any(not (x > 0) for x in self.c):
            raise ValueError("need n positive step costs")
        self.pre = [0.0]
        for x in self.c:
            self.pre.append(self.pre[-1] + x)
        self.memo = {}

    def C(self, a: int, b: int) -> float:
        return self.pre[b] - self.pre[a]

    def fits(self, a: int, l: int, M: int) -> bool:
        """Every state strictly inside [a, a+l) fits in M units at once."""
        return l <= 1 or sum(self.z[a + 1:a + l]) <= M

    def T(self, a: int, l: int, M: int) -> float:
        if self.fits(a, l, M):
            return 0.0 if l <= 1 else self.C(a, a + l - 1)
        return self._solve(a, l, M)[0]

    def split(self, a: int, l: int, M: int) -> int:
        """The split m, or 0 for the chain."""
        if self.fits(a, l, M):
            return 1
        return self._solve(a, l, M)[1]

    def _solve(self, a, l, M):
        key = (a, l, M)
        if key in self.memo:
            return self.memo[key]
        best = None
        if l == 1:
            best = (0.0, 0)
        else:
            for m in range(1, l):
                if self.z[a + m] <= M:
                    v = self.C(a, a + m) + self._solve(a + m, l - m, M - self.z[a + m])[0] + self._solve(a, m, M)[0]
                    if best is None or v <= best[0]:
                        best = (v, m)
            if best is None:
                best = (sum(self.C(a, a + i) for i in range(1, l)), 0)
        self.memo[key] = best
        return best


def _sized_result(g: _Gen, head: dict, ss: SizedSplits, n: int) -> tuple[dict, list[tuple]]:
    head["evals"] = sum(x[2] - x[1] for x in g.out if x[0] == "A") + 1
    head["cost"] = sum(ss.C(x[1], x[2]) for x in g.out if x[0] == "A") + ss.c[n - 1]
    head["split"] = "size"
    return head, g.out


def schedule_sized(n: int, s: int, sizes, H: int = 0, I_min: int = 0, costs=None) -> tuple[dict, list[tuple]]:
    """(header dict, action list) when the states x_0 .. x_n have the given
    sizes (units), in a fast pool of s * max(sizes) units and H slow slots
    (each holding any state).  Plain: the sized recursion over [0, n) with
    P - sizes[0] units above x_0.  Two levels (H > 0, s >= 2, I < n, strictly
    cheaper): the fixed-interval policy with every interval reversed by the
    sized recursion on P - 2 max(sizes) units."""
    if n < 1 or s < 1 or H < 0 or I_min < 0 or len(sizes) != n + 1:
        raise ValueError("need n >= 1, s >= 1, H >= 0, I_min >= 0 and n + 1 sizes")
    ss = SizedSplits(sizes, costs)
    zmax = max(ss.z)
    P = s * zmax
    best = ("revolve", 0, ss.T(0, n, P - ss.z[0]))
    if H > 0 and s >= 2:
        I = max(I_min, 1, -(-n // (H + 1)))
        if I < n:
            starts = list(range(0, n, I))
            ends = starts[1:] + [n]
            M = P - 2 * zmax
            c = ss.C(0, starts[-1]) + sum(ss.T(a, e - a, M) for a, e in zip(starts, ends))
            if c < best[2]:
                best = ("async", I, c)
    g = _Gen(n)
    if best[0] == "revolve":
        g.emit("S", 0, 0)
        g.live = 0
        _reverse_sized(g, ss, 0, n, P - ss.z[0], 0, 1)
    else:
        _two_level(g, n, s, list(range(0, n, best[1])), sized=(ss, P - 2 * zmax))
    return _sized_result(g, {"n": n, "s": s, "H": H, "I": best[1], "mode": best[0]}, ss, n)


def schedule_sized_from_starts(n: int, s: int, H: int, starts: list[int], sizes, costs=None):
    """The two-level policy over interval starts chosen during the sweep,
    each interval reversed by the sized recursion (the pairing Section 6
    proposes: a store as soon as the previous one has finished, and one-level
    checkpointing of unequal states inside each interval)."""
    starts = list(starts)
    if n < 1 or s < 2 or not starts or starts[0] != 0 or any(b <= a for a, b in zip(starts, starts[1:])) \
            or starts[-1] >= n or len(starts) - 1 > H or len(sizes) != n + 1:
        raise ValueError("need s >= 2, starts 0 = t_0 < t_1 < ... < n with at most H + 1 of them, n + 1 sizes")
    ss = SizedSplits(sizes, costs)
    zmax = max(ss.z)
    g = _Gen(n)
    _two_level(g, n, s, starts, sized=(ss, s * zmax - 2 * zmax))
    return _sized_result(g, {"n": n, "s": s, "H": H, "I": 0, "mode": "dynamic"}, ss, n)


def text_sized(n: int, s: int, sizes, H: int = 0, I_min: int = 0, costs=None) -> str:
    return _render(*schedule_sized(n, s, sizes, H, I_min, costs))


def text_sized_from_starts(n: int, s: int, H: int, starts, sizes, costs=None) -> str:
    return _render(*schedule_sized_from_starts(n, s, H, starts, sizes, costs))


def slot_offsets(acts: list[tuple], sizes, two_level: bool) -> list[int | None]:
    """Unit offset of every S / R / W / P action's fast slot in the stack
    layout of sized schedules (None for other actions): slot k sits above
    the states most recently snapshotted into slots below it (two levels:
    slots 0 and 1 at 0 and max(sizes), the stack from 2 max(sizes))."""
    zmax = max(sizes)
    content: dict[int, int] = {}
    out = []

    def off(k):
        if two_level and k <= 1:
            return k * zmax
        lo = 2 if two_level else 0
        assert all(j in content for j in range(lo, k)), ("a slot below slot", k, "holds no state")
        return (2 * zmax if two_level else 0) + sum(sizes[content[j]] for j in range(lo, k))

    for a in acts:
        op = a[0]
        if op in ("S", "R", "W"):
            k = a[1]
            if op == "S":
                out.append(off(k))
                content[k] = a[2]
            else:
                out.append(off(k))
        elif op == "P":
            out.append(off(a[2]))
            content[a[2]] = a[3]
        else:
            out.append(None)
    return out


def check_sized(n: int, s: int, H: int, acts: list[tuple], sizes, two_level: bool) -> dict:
    """check() plus the byte budget of the sized layout: every snapshot lies
    inside the pool of s * max(sizes) units, every state read back from a
    slot is read at the offset it was written to, and the interval starts
    fit their regions."""
    c = check(n, s_slots(acts, s), H, acts)
    zmax = max(sizes)
    P = s * zmax
    offs = slot_offsets(acts, sizes, two_level)
    written: dict[int, int] = {}
    for a, o in zip(acts, offs):
        op = a[0]
        if op == "S":
            k, t = a[1], a[2]
            assert o + sizes[t] <= P, (a, o, P)
            if two_level and k <= 1:
                assert sizes[t] <= zmax
            written[k] = o
        elif op == "P":
            assert a[2] <= 1 and two_level, a
            written[a[2]] = o
        elif op in ("R", "W"):
            assert written.get(a[1]) == o, ("slot moved under its state", a, o, written.get(a[1]))
    c["peak_units"] = max([o + sizes[a[2]] for a, o in zip(acts, offs) if a[0] == "S"] + [0])
    return c


def s_slots(acts: list[tuple], s: int) -> int:
    """Slot ids a sized schedule may use (stack depths can exceed s when the
    states are small): one more than the largest id it names, at least s."""
    ks = [a[1] for a in acts if a[0] in ("S", "R", "W")] + [a[2] for a in acts if a[0] == "P"]
    return max([s] + [k + 1 for k in ks])


def text_costs(n: int, s: int, costs, H: int = 0, I_min: int = 0) -> str:
    return _render(*schedule_costs(n, s, costs, H, I_min))


def text_online(n: int, s: int, H: int = 0, I_min: int = 0) -> str:
    return _render(*schedule_online(n, s, H, I_min))


def _render(head: dict, acts: list[tuple]) -> str:
    lines = [f"ambptt-schedule v1 n={head['n']} s={head['s']} H={head['H']} I={head['I']} mode={head['mode']}"
             + (f" split={head['split']}" if head.get("split") else "")]
    lines += [" ".join(str(v) for v in a) for a in acts]
    return "\n".join(lines) + "\n"


def text(n: int, s: int, H: int = 0, I_min: int = 0) -> str:
    return _render(*schedule(n, s, H, I_min))


def text_from_starts(n: int, s: int, H: int, starts: list[int], costs=None) -> str:
    return _render(*schedule_from_starts(n, s, H, starts, costs))


def parse(txt: str) -> tuple[dict, list[tuple]]:
    """Canonical text -> (header dict, action list)."""
    lines = txt.strip("\n").split("\n")
    f = lines[0].split()
    assert f[:2] == ["ambptt-schedule", "v1"], lines[0]
    head = {}
    for kv in f[2:]:
        k, v = kv.split("=")
        head[k] = v if k in ("mode", "split") else int(v)
    acts = []
    for ln in lines[1:]:
        p = ln.split()
        acts.append((p[0],) + tuple(int(v) for v in p[1:]))
    return head, acts


# ---------------------------------------------------------------------------

def check(n: int, s: int, H: int, acts: list[tuple]) -> dict:
    """Symbolic execution: every action reads what it claims, adjoints run n-1..0 once.

    Returns counters (forward evaluations, snapshots, ...) or raises AssertionError.
    """
    slot: dict[int, int] = {}
    host: dict[int, int] = {}
    live = 0
    nxt = n - 1
    c = dict(evals=0, advances=0, takeshots=0, restores=0, stores=0, prefetches=0, adjoints=0)
    for a in acts:
        op = a[0]
        if op == "A":
            t0, t1 = a[1], a[2]
            assert live == t0 and t0 < t1 <= nxt, a
            live = t1
            c["advances"] += t1 - t0
            c["evals"] += t1 - t0
        elif op == "S":
            k, t = a[1], a[2]
            assert 0 <= k < s and live == t, a
            slot[k] = t
            c["takeshots"] += 1
        elif op == "R":
            k, t = a[1], a[2]
            assert slot.get(k) == t, a
            live = t
            c["restores"] += 1
        elif op in ("F", "Y"):
            t = a[1]
            assert t == nxt and live == t, a
            assert (op == "F") == (t == n - 1), a
            if op == "F":
                c["evals"] += 1
            nxt -= 1
            c["adjoints"] += 1
        elif op == "W":
            k, h, t = a[1:]
            assert 0 <= h < H and slot.get(k) == t, a
            host[h] = t
            c["stores"] += 1
        elif op == "P":
            h, k, t = a[1:]
            assert 0 <= k < s and host.get(h) == t, a
            slot[k] = t
            c["prefetches"] += 1
        else:
            raise AssertionError(f"unknown action {a}")
    assert nxt == -1, "not every adjoint step ran"
    return c


def replay(cell, n: int, u_of, x0: tuple, acts: list[tuple]) -> dict:
    """Execute a schedule on the CPU with copies applied at once; returns like store_all."""
    from .bptt import Reverse

    slot: dict[int, tuple] = {}
    host: dict[int, tuple] = {}
    live = tuple(np.asarray(v, np.float64) for v in x0)
    rev = Reverse(cell, n, u_of)
    for a in acts:
        op = a[0]
        if op == "A":
            for t in range(a[1], a[2]):
                live = cell.step(t, live, u_of(t))
        elif op == "S":
            slot[a[1]] = tuple(v.copy() for v in live)
        elif op == "R":
            live = tuple(v.copy() for v in slot[a[1]])
        elif op in ("F", "Y"):
            rev.adjoint(a[1], live)
        elif op == "W":
            host[a[2]] = tuple(v.copy() for v in slot[a[1]])
        elif op == "P":
            slot[a[2]] = tuple(v.copy() for v in host[a[1]])
    return rev.result()
