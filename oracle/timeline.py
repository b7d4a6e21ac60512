"""Evaluated schedule of the oracle's flows in the paper's network model.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Rules (paper: "Don't Let a Few Network Failures Slow the Entire AllReduce"):
* Sec. 3 model: a healthy NIC moves one element per time unit, a NIC with
  slowdown l one element per l units; App. B.1 time weighting: a transfer that
  touches a slow NIC costs the slow rate on both ends, so a flow of len
  elements between ranks a and b lasts len * max(l_a, l_b).
* Sec. 4.1: each NIC receives at most one flow at a time; Sec. 4.2: no NIC
  sends or receives two flows at once; the straggler sends and receives at
  the same time (full duplex).  So every rank has one send and one receive
  port, each busy with at most one flow.
* Sec. 3 correctness (i): a rank transmits only data it already holds: a
  flow waits for the earlier steps of its section that wrote its source's or
  its destination's range.
* Scheduling policy (a reading of ours, the pattern figures being
  missing): non-preemptive, work-conserving list scheduling; at every event
  time the unstarted flows are scanned in priority order and each one whose
  dependencies are done and whose two ports are free starts.  Two priority
  orders are tried: (1) the serial step order; (2) pattern groups, group by
  group, each in serial order, a group being four consecutive segments, one
  per pattern (the k/4 groups that the time analyses of Sec. 4.3 and App. D
  count), or with several GPUs per server eight consecutive segments of
  every part (App. E: the overlay needs 8 | k).  The second schedule is kept
  only if its makespan is below (1 - 1e-9) times the first's.
* Several GPUs per server (App. E bandwidth model): a flow between two GPUs
  of the same server uses their NVLink lanes, not their NICs: separate send
  and receive ports per GPU, each running at (g-1) times NIC speed, so the
  flow lasts len/(g-1).  Bandwidths are then given per server.

Times are exact rationals (``fractions.Fraction``), so there are no ties to
break by tolerance (the library, in doubles, merges events closer than 1e-9 of
the current time).  The naive scan is quadratic: small schedules only.
"""
from __future__ import annotations

from fractions import Fraction as F


def slowdowns(bandwidths):
    """l_i = max(b)/b_i, read as the nearest fraction with denominator at most
    10**6: bandwidths are NIC fractions (7/8, 2/3, ...) given as doubles, so
    2/3 means l = 3/2 and simultaneous events stay simultaneous."""
    b = [F(x) for x in bandwidths]
    bmax = max(b)
    return [(bmax / x).limit_denominator(10**6) for x in b]


def rank_slowdowns(sched, bandwidths):
    """Slowdown of every rank: one bandwidth per rank, or per server when
    the schedule has g > 1 GPUs per server."""
    ell = slowdowns(bandwidths)
    g = getattr(sched, "g", 1)
    return [ell[r // g] for r in range(sched.p)] if g > 1 else ell


def flow_cost(sched, ell, a, b, ln):
    """(port kind, duration) of a flow of ln elements from rank a to rank b."""
    g = getattr(sched, "g", 1)
    if g > 1 and a // g == b // g:
        return "nvlink", F(ln, g - 1)
    return "nic", ln * max(ell[a], ell[b])


def dependencies(steps):
    """For every step, the earlier steps of its section that last wrote one of
    its sources or its destination."""
    last = {}
    deps = []
    for i, st in enumerate(steps):
        sec = (st["seg"], st["sec"])
        d = set()
        for r in list(st["srcs"]) + [st["dst"]]:
            if (r, sec) in last:
                d.add(last[(r, sec)])
        deps.append(d)
        last[(st["dst"], sec)] = i
    return deps


def pattern_group(sched, seg):
    """Group of a segment: four consecutive segments (one GPU per server), or
    eight consecutive segments of a part (several GPUs per server)."""
    if getattr(sched, "g", 1) > 1:
        return (seg % sched.k) // 8
    return seg // 4


def evaluate(sched, bandwidths):
    """(makespan, [(start, finish) per flow in flow order]): the shorter of
    the two list schedules (serial order, then pattern groups)."""
    steps = sched.steps()
    ell = rank_slowdowns(sched, bandwidths)
    deps = dependencies(steps)
    flows = []
    for i, st in enumerate(steps):
        for src in st["srcs"]:
            kind, dur = flow_cost(sched, ell, src, st["dst"], st["len"])
            flows.append((i, (kind, src), (kind, st["dst"]), dur))
    best = list_schedule(steps, deps, flows, range(len(flows)))
    groups = [pattern_group(sched, steps[i]["seg"]) for i, _, _, _ in flows]
    if len(set(groups)) > 1:
        scan = sorted(range(len(flows)), key=lambda f: (groups[f], f))
        other = list_schedule(steps, deps, flows, scan)
        if other[0] < best[0] * (1 - F(1, 10**9)):
            best = other
    return best


def list_schedule(steps, deps, flows, scan):
    """One list schedule, unstarted flows scanned in the order `scan`."""
    left = [len(st["srcs"]) for st in steps]
    done_steps = set()
    start = [None] * len(flows)
    finish = [None] * len(flows)
    send_free = {}
    recv_free = {}
    t = F(0)
    running = []
    remaining = len(flows)
    while remaining:
        for f in scan:
            i, a, b, dur = flows[f]
            if start[f] is not None or not deps[i] <= done_steps:
                continue
            if send_free.get(a, F(0)) > t or recv_free.get(b, F(0)) > t:
                continue
            start[f], finish[f] = t, t + dur
            send_free[a] = recv_free[b] = t + dur
            running.append(f)
        if not running:
            raise RuntimeError("no flow can start")
        t = min(finish[f] for f in running)
        for f in [f for f in running if finish[f] == t]:
            running.remove(f)
            remaining -= 1
            i = flows[f][0]
            left[i] -= 1
            if left[i] == 0:
                done_steps.add(i)
    return max(finish, default=F(0)), list(zip(start, finish))


def validate(sched, bandwidths, times):
    """Check a timeline against the model, whatever policy produced it:
    durations, one flow per port at a time, and data dependencies.
    Returns a list of violations (empty when valid)."""
    steps = sched.steps()
    ell = rank_slowdowns(sched, bandwidths)
    deps = dependencies(steps)
    errs = []
    flows = []
    for i, st in enumerate(steps):
        for src in st["srcs"]:
            kind, dur = flow_cost(sched, ell, src, st["dst"], st["len"])
            flows.append((i, (kind, src), (kind, st["dst"]), dur))
    if len(flows) != len(times):
        return [f"{len(times)} times for {len(flows)} flows"]
    step_end = {}
    for (i, a, b, dur), (s, e) in zip(flows, times):
        if abs(F(e) - F(s) - dur) > F(1, 10**6) * max(1, dur):
            errs.append(f"flow of step {i}: duration {e - s} != {dur}")
        step_end[i] = max(step_end.get(i, F(-1)), F(e))
    for port in ("send", "recv"):
        busy = {}
        for (i, a, b, dur), (s, e) in zip(flows, times):
            busy.setdefault(a if port == "send" else b, []).append((F(s), F(e)))
        for r, iv in busy.items():
            iv.sort()
            for (s0, e0), (s1, e1) in zip(iv, iv[1:]):
                if s1 < e0 - F(1, 10**6) * max(1, e0):
                    errs.append(f"rank {r} {port} port: overlapping flows at {s1}")
    for (i, a, b, dur), (s, e) in zip(flows, times):
        for d in deps[i]:
            if F(s) < step_end[d] - F(1, 10**6) * max(1, step_end[d]):
                errs.append(f"step {i} starts before its dependency {d} ends")
    return errs
