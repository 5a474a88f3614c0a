"""Host model of the fused trainer's exchange protocol (CPU).

The trainer (paper_2606_30497_amd/csrc/train_persistent.hip) runs every SGD step
of a call in one launch; its workgroups exchange tagged words through three
buffers, each double-buffered by step parity, and no writer ever waits for a
reader. Correctness rests on one claim: before any word of a parity slot is
written for step s + 2, every read of that slot for step s has completed. This
test checks the claim on the happens-before order the waits create, for every
instantiated shape, with vector clocks: event y happens after event x iff y's
clock entry for x's workgroup is at least x's index there.

Events of workgroup (gx, gb) (group gx = hidden-unit slice, rank gb = row block)
in step s, in program order (the workgroup's barriers order its waves):
  F   forward done, exchange-A words of its rows stored       A[p][gb][gx]
  RA  exchange A read: waits for F of every group's rank-gb workgroup
  LS  (workgroup (0, 0) only, s >= 1) reads the SSE words of step s - 1
  WB  exchange-B words stored (its P partial, its SSE word)   B[p][gx][*][gb]
  RB  owner role: waits for WB of every workgroup of its group
  WC  owner role: updated words stored                       C[p][gx][gb]
  RC  exchange C read: waits for WC of every workgroup of its group
with p = s mod 2. The next step's F follows RC.
"""
import itertools

import numpy as np
import pytest

# the library's shape table: (groups PX, workgroups per group PR, rows R, units U)
FUSED_SHAPES = [(8, 32, 128, 32), (8, 32, 64, 32), (8, 32, 32, 32), (4, 32, 16, 64),
                (1, 16, 16, 256), (8, 32, 32, 128), (8, 32, 16, 128),
                (8, 32, 16, 64), (2, 16, 16, 64), (1, 16, 16, 64), (1, 8, 32, 32),
                (4, 16, 16, 64), (2, 16, 16, 128), (4, 4, 16, 64), (8, 4, 32, 32),
                (8, 8, 32, 32)]

EVENTS = ("F", "RA", "LS", "WB", "RB", "WC", "RC")


def happens_before_clocks(px, pr, steps, drop_waits=()):
    """Vector clocks of every event. drop_waits: (event, ) names whose cross-
    workgroup waits are left out (used to show the check detects a violation)."""
    n = px * pr
    wg = lambda gx, gb: gx * pr + gb
    idx = {}                     # (event, w, s) -> index in w's chain
    clock = {}                   # (event, w, s) -> np.array of n ints (-1 = nothing)
    last = [None] * n
    counter = [0] * n

    def add(ev, w, s, deps):
        vc = np.full(n, -1, dtype=np.int64) if last[w] is None else clock[last[w]].copy()
        for d in deps:
            np.maximum(vc, clock[d], out=vc)
        key = (ev, w, s)
        idx[key] = counter[w]
        vc[w] = counter[w]
        counter[w] += 1
        clock[key] = vc
        last[w] = key

    for s in range(steps):
        for gx in range(px):
            for gb in range(pr):
                add("F", wg(gx, gb), s, [])
        for gx in range(px):
            for gb in range(pr):
                deps = [] if "RA" in drop_waits else [("F", wg(g2, gb), s) for g2 in range(px)]
                add("RA", wg(gx, gb), s, deps)
                if gx == 0 and gb == 0 and s >= 1:
                    add("LS", wg(0, 0), s, [])      # its words were written a step earlier
        for gx in range(px):
            for gb in range(pr):
                add("WB", wg(gx, gb), s, [])
        for gx in range(px):
            for gb in range(pr):
                deps = [] if "RB" in drop_waits else [("WB", wg(gx, b2), s) for b2 in range(pr)]
                add("RB", wg(gx, gb), s, deps)
                add("WC", wg(gx, gb), s, [])
        for gx in range(px):
            for gb in range(pr):
                deps = [] if "RC" in drop_waits else [("WC", wg(gx, b2), s) for b2 in range(pr)]
                add("RC", wg(gx, gb), s, deps)
    return idx, clock


def before(idx, clock, x, y):
    """x happens before y."""
    return clock[y][x[1]] >= idx[x]


def slot_uses(px, pr, steps, slots=2):
    """For every buffer slot and step: (writer events, reader events). slots: the
    number of step buffers (2 = the kernel's parity double buffer)."""
    wg = lambda gx, gb: gx * pr + gb
    uses = []
    for s in range(steps):
        p = s % slots
        # exchange A: slot of group gx's words for row block gb, read by every group's rank gb
        for gx, gb in itertools.product(range(px), range(pr)):
            uses.append((("A", p, gx, gb), s, [("F", wg(gx, gb), s)],
                         [("RA", wg(g2, gb), s) for g2 in range(px)]))
        # exchange B: source gb's words for owner o of group gx, read by o
        for gx, o, gb in itertools.product(range(px), range(pr), range(pr)):
            uses.append((("B", p, gx, o, gb), s, [("WB", wg(gx, gb), s)],
                         [("RB", wg(gx, o), s)]))
        # SSE words: group 0's B words, read a step late by workgroup (0, 0)
        if s + 1 < steps:
            for gb in range(pr):
                uses.append((("SSE", p, gb), s, [("WB", wg(0, gb), s)],
                             [("LS", wg(0, 0), s + 1)]))
        # exchange C: owner o's updated words, read by every workgroup of its group
        for gx, o in itertools.product(range(px), range(pr)):
            uses.append((("C", p, gx, o), s, [("WC", wg(gx, o), s)],
                         [("RC", wg(gx, gb), s) for gb in range(pr)]))
    return uses


def violations(px, pr, steps, drop_waits=(), slots=2):
    idx, clock = happens_before_clocks(px, pr, steps, drop_waits)
    by_slot = {}
    for slot, s, writers, readers in slot_uses(px, pr, steps, slots):
        by_slot.setdefault(slot, []).append((s, writers, readers))
    bad = []
    for slot, seq in by_slot.items():
        seq.sort(key=lambda t: t[0])
        for (s0, w0, r0), (s1, w1, r1) in zip(seq, seq[1:]):
            # every read of the earlier use precedes every write of the later use
            for r in r0:
                for w in w1:
                    if not before(idx, clock, r, w):
                        bad.append((slot, s0, r, w))
    return bad


@pytest.mark.parametrize("shape", FUSED_SHAPES, ids=lambda s: "%d-%d-%d-%d" % s)
def test_no_slot_is_rewritten_before_its_readers_are_done(shape):
    px, pr, _, _ = shape
    assert violations(px, pr, steps=6) == []


def test_the_check_sees_a_missing_wait():
    """A mutant of the protocol: without exchange A's wait for the other groups'
    words (RA), a group can run ahead and rewrite its exchange-A words of step
    s + 2 while another group still reads those of step s; the check reports it,
    so the passing test above is not vacuous."""
    bad = violations(8, 4, steps=6, drop_waits=("RA",))
    assert bad and all(b[0][0] in ("A", "SSE") for b in bad)


def test_which_buffers_need_two_slots():
    """With one slot per buffer instead of two: exchange A and the SSE words would
    be unsafe (a group can start step s + 1 while another group still reads the
    A words of step s), while exchanges B and C would stay safe, since every write
    of B or C for step s + 1 waits, through exchange B itself, for every reader of
    step s. The kernel double-buffers all three; for B and C that is margin, not
    a requirement."""
    bad = violations(8, 4, steps=6, slots=1)
    kinds = {b[0][0] for b in bad}
    assert "A" in kinds and "SSE" in kinds
    assert "B" not in kinds and "C" not in kinds


def test_lds_row_double_buffer():
    """Inside a workgroup: the loader waves write the rows of step s + 1 into LDS
    buffer (s + 1) mod 2 during step s, once compute wave 0 has posted that its
    forward of step s is done (an LDS flag); the compute waves read buffer s mod 2
    in step s (forward and backward operands) before the workgroup's P barrier.
    Waves and barriers as a happens-before graph: every read of a buffer precedes
    the loader's next write of it, and that write precedes the next step's reads."""
    waves = ["c0", "c1", "c2", "c3", "ld"]
    last = {w: frozenset() for w in waves}     # events known to precede each wave's next one
    ev = {}

    def add(name, w, extra=()):
        known = set(last[w]) | {name}
        for e in extra:
            known |= ev[e]
        ev[name] = frozenset(known)
        last[w] = ev[name]

    def barrier(name):
        known = set().union(*(last[w] for w in waves)) | {name}
        ev[name] = frozenset(known)
        for w in waves:
            last[w] = ev[name]

    steps = 6
    for w in waves:
        add(("init_stage", w), w)
    barrier(("start",))
    for s in range(steps):
        for c in waves[:4]:
            add(("fwd_read", c, s), c)             # forward operands of buffer s % 2
        add(("fwd_flag", s), "c0")                 # wave 0 posts its forward done
        add(("stage", s), "ld", extra=[("fwd_flag", s)])   # writes buffer (s + 1) % 2
        for c in waves[:4]:
            add(("bwd_read", c, s), c)             # backward operands of buffer s % 2
        barrier(("P", s))
        barrier(("O", s))
        barrier(("N", s))

    def before(x, y):
        return x in ev[y]

    for s in range(1, steps):
        w = ("stage", s)                           # writes buffer (s + 1) % 2 = (s - 1) % 2
        for c in waves[:4]:
            assert before(("fwd_read", c, s - 1), w) and before(("bwd_read", c, s - 1), w)
        if s + 1 < steps:
            for c in waves[:4]:
                assert before(w, ("fwd_read", c, s + 1)) and before(w, ("bwd_read", c, s + 1))
    # without the forward-done flag the loader could write during step s's reads
    # of the other buffer only after P(s - 1); the flag is what orders it after the
    # step's own forward (the check above would still pass without it, since the
    # buffers differ): the double buffer is what keeps the loader off the rows in use
    assert not before(("stage", 2), ("fwd_read", "c1", 2))
