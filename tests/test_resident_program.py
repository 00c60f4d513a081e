"""The resident kernel's program, compiled from the schedule by the library's
host code (ambptt_resident_program), replayed on the CPU with the oracle's
float64 cells under the kernel's own visibility rules (CPU only).

The kernel runs the program on many workgroups that meet at a barrier per
step.  Its rules, modelled here:
  * a step's output is written after its barrier and is readable by every
    workgroup from the next barrier on;
  * a prefetch's data reach the slot right after the next barrier (the
    current step has read its inputs by then) and are readable from the
    barrier after that; a second prefetch before that barrier is an error;
  * a copy is readable from the next barrier; a copy into a buffer that the
    latest step read must first wait for every workgroup to read it;
  * a store reads the slot at once and writes host memory at the next
    barrier (or at the next store or prefetch); a store flagged "staged"
    takes the slice from the output the workgroup just computed, which is
    only right when the previous entry is the forward step that wrote the
    slot.
Under those rules every program must reproduce store-all BPTT bit for bit
(the schedule decides which states are recomputed, never the arithmetic),
and its forward count must be the schedule's.
"""
import numpy as np
import pytest

from oracle import bptt
from oracle.cells import Cell

amb = pytest.importorskip("paper_1806_01117_amd")

FWD, ADJ, COPY, STORE, PREF, SYNC, END = 1, 2, 3, 4, 5, 6, 0
STAGED = 1 << 8   # store flag: the slice comes from the previous entry's output in LDS


def _cell(kind="lstm", loss="half_sq_last", B=2, D=3, H=4, seed=0):
    rng = np.random.default_rng(seed)
    G = 4 if kind == "lstm" else 1
    W = rng.standard_normal((G * H, D + H)) * 0.6
    b = rng.standard_normal(G * H) * 0.3
    cell = Cell(kind, loss, B, D, H, W=W, b=b)
    x0 = (rng.standard_normal((B, H)) * 0.5,) + ((rng.standard_normal((B, H)) * 0.5,) if G == 4 else ())
    return cell, x0, rng


def replay_program(prog, cell, n, s, u_of, x0):
    L0 = s
    buf = {L0: tuple(np.asarray(v, np.float64) for v in x0)}
    vis = {L0: 0}          # first barrier from which every workgroup may read the buffer
    last_read = {}         # barrier of the last step that read the buffer
    host = {}
    bar = 0
    pend_pref = None       # (slot, state)
    pend_store = None      # (host slot, state)
    rev = bptt.Reverse(cell, n, u_of)
    fwd = extra = 0

    def flush(reading):
        nonlocal pend_pref, pend_store
        if pend_pref is not None:
            k, st = pend_pref
            assert k != reading, "a prefetch lands in the slot the current step reads"
            buf[k], vis[k] = st, bar + 1
            pend_pref = None
        if pend_store is not None:
            host[pend_store[0]] = pend_store[1]
            pend_store = None

    ended = False
    prev = None
    for entry in prog:
        op, y, z, w = entry
        flags, op = op >> 8, op & 0xFF
        if op == STORE and flags & 1:
            assert prev is not None and prev[0] == FWD and prev[3] == z, "staged store not right after its step"
        prev = (op, y, z, w)
        assert not ended, "entries after the end"
        if op in (FWD, ADJ):
            bar += 1
            assert z in buf and vis[z] <= bar, f"step {y} reads buffer {z} before every workgroup may"
            state = buf[z]
            last_read[z] = bar
            flush(z)
            if op == FWD:
                assert w != z
                buf[w], vis[w] = cell.step(y, state, u_of(y)), bar + 1
                fwd += 1
            else:
                rev.adjoint(y, state)
                fwd += 1 if w else 0
        elif op == COPY:
            assert pend_pref is None or pend_pref[0] not in (z, w)
            if bar > 0 and last_read.get(w, 0) == bar:
                assert y >= bar, "a copy overwrites a buffer the latest step may still read"
            buf[w], vis[w] = buf[z], bar + 1
        elif op == STORE:
            assert pend_pref is None or pend_pref[0] != z
            if pend_store is not None:
                host[pend_store[0]] = pend_store[1]
            pend_store = (w, buf[z])
        elif op == PREF:
            assert pend_pref is None, "two prefetches without a barrier between them"
            if pend_store is not None:
                host[pend_store[0]] = pend_store[1]
                pend_store = None
            pend_pref = (w, host[z])
        elif op == SYNC:
            bar += 1
            extra += 1
            flush(None)
        elif op == END:
            bar += 1
            flush(None)
            ended = True
        else:
            raise AssertionError(f"unknown op {op}")
    assert ended, "program without an end"
    return rev.result(), fwd, extra


CASES = [  # n, s, H, I_min
    (1, 1, 0, 1), (2, 2, 0, 1), (5, 1, 0, 1), (9, 2, 0, 1), (40, 3, 0, 1),
    (12, 3, 100, 3), (13, 2, 13, 1), (30, 4, 30, 1), (30, 4, 30, 2), (37, 5, 37, 4),
    (50, 6, 50, 5), (64, 3, 64, 2), (25, 10, 25, 1),
]


@pytest.mark.parametrize("elide", [True, False])
@pytest.mark.parametrize("n,s,H,I", CASES)
def test_program_reproduces_store_all(n, s, H, I, elide):
    cell, x0, rng = _cell()
    us = [rng.standard_normal((2, 3)) for _ in range(n)]
    u_of = lambda t: us[t]
    prog = amb.resident_program(n, s, H, I, elide)
    got, fwd, _ = replay_program(prog, cell, n, s, u_of, x0)
    want = bptt.store_all(cell, n, u_of, x0)
    assert fwd == amb.schedule_evals(n, s, H, I)[0]
    assert got["loss"] == want["loss"]
    assert np.array_equal(got["dW"], want["dW"]) and np.array_equal(got["db"], want["db"])
    for a, b in zip(got["dx0"], want["dx0"]):
        assert np.array_equal(a, b)


def test_replayer_catches_a_misplaced_staged_store():
    cell, x0, rng = _cell()
    n, s = 30, 4
    us = [rng.standard_normal((2, 3)) for _ in range(n)]
    prog = amb.resident_program(n, s, n, 2)
    i = next(i for i, e in enumerate(prog) if e[0] == STORE | STAGED)
    broken = prog[:i - 1] + [prog[i], prog[i - 1]] + prog[i + 1:]   # the store before its step
    with pytest.raises(AssertionError):
        replay_program(broken, cell, n, s, lambda t: us[t], x0)


def test_program_rnn_and_losses():
    for kind in ("rnn", "lstm"):
        for loss in ("half_sq_last", "mean_sq_all", "mean_last"):
            cell, x0, rng = _cell(kind, loss, seed=3)
            n = 21
            us = [rng.standard_normal((2, 3)) for _ in range(n)]
            got, _, _ = replay_program(amb.resident_program(n, 4, n, 2), cell, n, 4, lambda t: us[t], x0)
            want = bptt.store_all(cell, n, lambda t: us[t], x0)
            assert got["loss"] == want["loss"] and np.array_equal(got["dW"], want["dW"])


def test_replayer_catches_a_broken_program():
    """A plausible compiler mistake (a step reading a slot whose prefetch has
    not landed) must trip the visibility rule."""
    cell, x0, rng = _cell()
    n, s = 12, 3
    us = [rng.standard_normal((2, 3)) for _ in range(n)]
    prog = amb.resident_program(n, s, 100, 3, False)
    # drop every barrier-only entry: some step then reads a prefetched slot too early
    broken = [e for e in prog if e[0] & 0xFF != SYNC]
    if len(broken) == len(prog):  # no extra barrier in this program: move a prefetch right before its reader
        i = next(i for i, e in enumerate(prog) if e[0] & 0xFF == PREF)
        k = prog[i][3]
        j = next(j for j in range(i + 1, len(prog)) if prog[j][0] & 0xFF in (FWD, ADJ) and prog[j][2] == k)
        broken = prog[:i] + prog[i + 1:j] + [prog[i]] + prog[j:]
    with pytest.raises(AssertionError):
        replay_program(broken, cell, n, s, lambda t: us[t], x0)


def test_program_entry_limits():
    prog = amb.resident_program(1000, 10, 1000, 2)
    ops = [e[0] & 0xFF for e in prog]
    staged = [e for e in prog if e[0] == STORE | STAGED]
    assert len(staged) == ops.count(STORE) - 1   # all but the first state's store come from LDS
    assert ops[-1] == END and ops.count(END) == 1
    assert ops.count(ADJ) == 1000
    assert all(0 <= e[2] < 12 and 0 <= e[3] < 1000 for e in prog if e[0] & 0xFF in (FWD, COPY))


ONLINE_CASES = [  # n, s, H, I_min
    (1, 2, 0, 1), (9, 2, 0, 1), (40, 3, 0, 1), (53, 4, 0, 1), (23, 3, 2, 2), (37, 3, 4, 3), (53, 4, 3, 2),
    (30, 2, 30, 1), (41, 5, 41, 2),
]


@pytest.mark.parametrize("elide", [True, False])
@pytest.mark.parametrize("n,s,H,I", ONLINE_CASES)
def test_online_program_reproduces_store_all(n, s, H, I, elide):
    """Programs of online schedules: held states dropped and their slots
    reused during the sweep, host slots given back and stored again."""
    from oracle import schedule as S
    cell, x0, rng = _cell(seed=5)
    us = [rng.standard_normal((2, 3)) for _ in range(n)]
    u_of = lambda t: us[t]
    prog = amb.resident_program(n, s, H, I, elide, online=True)
    got, fwd, _ = replay_program(prog, cell, n, s, u_of, x0)
    want = bptt.store_all(cell, n, u_of, x0)
    assert fwd == S.schedule_online(n, s, H, I if H else 0)[0]["evals"]
    assert got["loss"] == want["loss"]
    assert np.array_equal(got["dW"], want["dW"]) and np.array_equal(got["db"], want["db"])
    for a, b in zip(got["dx0"], want["dx0"]):
        assert np.array_equal(a, b)
