"""The contributor-set checker itself is pinned (CPU only).

`oracle.provenance_steps` decides correctness of a step list symbolically
(Sec. 3: every rank must end with every rank's input counted exactly once).
A checker that never reports anything would pass every schedule, so it is
run here on hand-written step lists whose verdict is known: the textbook
ring AllReduce and a direct reduce-then-broadcast are correct, and each
planted fault (a hop repeated, a source listed twice, an allgather hop or a
source missing, a reduce after the allgather) must be reported with the
right kind of message.  The same faults planted in a real OptCC schedule
are reported too.
"""
import copy

import pytest

import oracle
from oracle import COPY, REDUCE


def _st(op, dst, srcs, off, ln=1):
    return dict(op=op, dst=dst, srcs=list(srcs), off=off, len=ln)


def textbook_ring(p):
    """Ring AllReduce over p coordinates (chunk j = coordinate j): chunk j
    starts at rank j and is reduced along j+1, ..., j+p-1; the last rank of
    the chain holds the sum and the allgather copies it on around the ring."""
    steps = []
    for j in range(p):
        for t in range(1, p):
            steps.append(_st(REDUCE, (j + t) % p, [(j + t - 1) % p], j))
    for j in range(p):
        for t in range(0, p - 1):
            steps.append(_st(COPY, (j + t) % p, [(j + t - 1) % p], j))
    return steps


def direct(p, n):
    """Rank 0 adds every other rank's value in one multi-source step, then
    every other rank copies the sum from rank 0."""
    return [_st(REDUCE, 0, range(1, p), 0, n)] + [_st(COPY, r, [0], 0, n) for r in range(1, p)]


@pytest.mark.parametrize("p", [3, 4, 7])
def test_correct_lists_pass(p):
    assert oracle.provenance_steps(p, p, textbook_ring(p)) == (True, "ok")
    assert oracle.provenance_steps(p, 5, direct(p, 5)) == (True, "ok")


def _verdict(p, n, steps):
    ok, msg = oracle.provenance_steps(p, n, steps)
    assert not ok
    return msg


@pytest.mark.parametrize("p", [3, 5])
def test_planted_faults_are_reported(p):
    ring = textbook_ring(p)
    # a reduce-scatter hop applied twice counts its source again
    twice = ring[:1] + ring[:1] + ring[1:]
    assert "double count" in _verdict(p, p, twice)
    # one allgather hop missing leaves a rank without the full sum
    short = ring[:-1]
    assert "misses contributions" in _verdict(p, p, short)
    # a reduce-scatter hop turned into a copy drops the destination's own value
    as_copy = copy.deepcopy(ring)
    as_copy[0]["op"] = COPY
    assert "misses contributions" in _verdict(p, p, as_copy)
    # a reduce after the allgather adds a finished sum onto a finished sum
    late = ring + [_st(REDUCE, 0, [1], 0)]
    assert "double count" in _verdict(p, p, late)
    # the direct form with a source listed twice, and with one source missing
    d = direct(p, 3)
    d[0]["srcs"].append(1)
    assert "double count" in _verdict(p, 3, d)
    d = direct(p, 3)
    d[0]["srcs"].pop()
    assert "misses contributions" in _verdict(p, 3, d)


def test_faults_in_an_optcc_schedule_are_reported():
    """The Sec. 4.2 worked example (p=5, GPU 0 at half bandwidth, k=4),
    whose unmodified steps pass."""
    n = 4 * 4 * 64
    s = oracle.Schedule(5, [0.5, 1, 1, 1, 1], n, 4)
    steps = s.steps()
    assert oracle.provenance_steps(5, n, steps) == (True, "ok")
    hop = next(i for i, st in enumerate(steps) if st["slot"] == 1)
    assert "double count" in _verdict(5, n, steps[:hop + 1] + [steps[hop]] + steps[hop + 1:])
    last_ag = max(i for i, st in enumerate(steps) if st["slot"] == 4)
    assert "misses contributions" in _verdict(5, n, steps[:last_ag] + steps[last_ag + 1:])
    up = next(i for i, st in enumerate(steps) if st["slot"] == 2)
    dropped = [st for i, st in enumerate(steps) if i != up]
    assert "misses contributions" in _verdict(5, n, dropped)
