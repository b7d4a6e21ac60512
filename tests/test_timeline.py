"""Evaluated schedule (the plan's flows timed in the paper's network model).

Plans with one GPU per server are timed by the paper's pattern overlay
(`tests/test_timetable.py` pins it against the time analyses); here the
library's timeline of the workloads and of ragged plans is compared with the
oracle's exact run and the policy-free validator, and the validator itself is
checked by planting mistakes in a valid timeline.  Plans with several GPUs per
server are timed by list scheduling (App. E's overlay is given only as
figures), compared the same way.
"""
from fractions import Fraction as F

import numpy as np
import pytest

import oracle
from oracle import model
from oracle import timeline as T


@pytest.fixture(scope="module")
def o():
    from paper_2606_01680_amd import optcc
    return optcc


def _bw(p, slow):
    b = [1.0] * p
    for r, v in slow.items():
        b[r] = v
    return b


CASES = [
    (3, {}, 3 * 64 * 4, 4), (7, {}, 7 * 64 * 8, 8), (4, {3: 0.5}, 5000, 8), (5, {0: 0.5}, 64 * 4 * 4 * 8, 4),
    (5, {0: 2 / 3}, 52 * 64 * 4, 4), (6, {2: 0.75}, 3000, 4), (8, {7: 0.875}, 64 * 7 * 8 * 4, 8),
    (7, {0: 0.5, 1: 0.75}, 64 * 5 * 8 * 4, 8), (9, {0: 0.875, 3: 0.75, 8: 0.5}, 4000, 4),
    (6, {5: 0.25}, 64 * 5 * 4, 4),
    (6, {1: 0.5, 4: 0.875}, 64 * 4 * 12 * 2, 12), (9, {2: 0.75, 5: 0.5, 6: 0.5}, 64 * 6 * 16, 16),
]


@pytest.mark.parametrize("p,slow,n,k", CASES)
def test_timeline_equals_oracle(o, p, slow, n, k):
    bw = _bw(p, slow)
    sched = oracle.Schedule(p, bw, n, k)
    mk_ref, ref, _ = T.construction(sched, bw, asap=True)
    pl = o.optcc_plan(p, bw, n, k)
    mk, st, fi = pl.timeline()
    scale = max(1.0, float(mk_ref))
    assert abs(mk - float(mk_ref)) <= 1e-9 * scale
    assert len(st) == len(ref)
    assert np.allclose(st, [float(a) for a, _ in ref], rtol=0, atol=1e-9 * scale)
    assert np.allclose(fi, [float(b) for _, b in ref], rtol=0, atol=1e-9 * scale)
    assert T.validate(sched, bw, list(zip(st, fi))) == []


@pytest.mark.parametrize("p,slow,n,k", CASES)
def test_evaluated_respects_lower_bound(p, slow, n, k):
    """Theorems 1/2 and the tight bound hold for any correct AllReduce, so
    also for the timetable and its as-soon-as-possible run."""
    bw = _bw(p, slow)
    sched = oracle.Schedule(p, bw, n, k)
    for asap in (False, True):
        mk, _, _ = T.construction(sched, bw, asap=asap)
        assert mk >= model.lower_bound(bw, n)


def test_validator_catches_planted_mistakes():
    """The validator rejects a shortened flow, two flows on one port at once,
    and a flow that starts before the data it forwards exists."""
    p, bw, n, k = 5, [0.5, 1, 1, 1, 1], 64 * 4 * 4, 4
    sched = oracle.Schedule(p, bw, n, k)
    _, good, _ = T.construction(sched, bw)
    assert T.validate(sched, bw, good) == []
    flows = [(st["slot"], src, st["dst"]) for st in sched.steps() for src in st["srcs"]]
    # shorten the first flow
    bad = list(good)
    s, e = bad[0]
    bad[0] = (s, s + (e - s) / 2)
    assert any("duration" in x for x in T.validate(sched, bw, bad))
    # move a Stage-4 hop to time 0: its data does not exist yet, and its
    # ports are busy with Stage-1 flows
    i = next(i for i, f in enumerate(flows) if f[0] == 4)
    s, e = good[i]
    bad = list(good)
    bad[i] = (F(0), e - s)
    errs = T.validate(sched, bw, bad)
    assert any("dependency" in x for x in errs) and any("overlapping" in x for x in errs)


@pytest.mark.parametrize("w", ["p4_f32", "p8_f32", "p16_bf16", "p64_f32",
                               pytest.param("p128_f32", marks=pytest.mark.slow)])
def test_workload_evaluated_times(o, w):
    """Full-size timelines against the closed forms and bounds: one
    straggler within 0.5 % of Sec. 4.3 / App. C (the sections' whole quanta
    differ by one quantum: p4 +0.3 %, p8 and p16 below 0.01 %), several
    stragglers at or below (k+4) T_body (App. D); always above the best
    lower bound."""
    from paper_2606_01680_amd.workloads import WORKLOADS
    W = WORKLOADS[w]
    pl = o.optcc_plan(W.p, W.bandwidths, W.n, W.k)
    mk, _, _ = pl.timeline(with_flows=False)
    closed = o.optcc_model_time(pl)
    lb = o.optcc_lower_bound(W.p, W.bandwidths, W.n)
    assert mk >= lb * (1 - 1e-12)
    if pl.kind == "multi":
        assert mk <= closed * (1 + 1e-12)
    else:
        assert mk <= closed * 1.005


# ------------------------------------------------ several GPUs per server
# (q, g, {straggler server: bandwidth}, n, k): small enough for the naive
# exact-rational scan, with every section of a segment non-empty in the
# larger cases
SERVER_CASES = [
    (3, 2, {2: 0.5}, 64 * 48, 24), (3, 2, {0: 0.875}, 64 * 2 * 24 * 2, 24),
    (4, 2, {1: 0.5}, 64 * 2 * 24 * 3, 24), (3, 3, {2: 0.25}, 64 * 3 * 24 * 2, 24),
    (4, 4, {3: 0.875}, 64 * 4 * 24, 24),
]


def _sbw(q, slow):
    b = [1.0] * q
    for s, v in slow.items():
        b[s] = v
    return b


@pytest.mark.parametrize("q,g,slow,n,k", SERVER_CASES)
def test_server_timeline_equals_oracle(o, q, g, slow, n, k):
    """App. E bandwidth model: NVLink flows on their own ports at (g-1)x NIC
    speed, NIC flows as in the one-GPU model; the library's evaluation equals
    the oracle's exact one flow by flow and passes the validator."""
    bw = _sbw(q, slow)
    sched = oracle.Schedule.servers(q, g, bw, n, k)
    mk_ref, ref = T.evaluate(sched, bw)
    pl = o.optcc_plan_servers(q, g, bw, n, k)
    mk, st, fi = pl.timeline()
    scale = max(1.0, float(mk_ref))
    assert abs(mk - float(mk_ref)) <= 1e-9 * scale
    assert len(st) == len(ref)
    assert np.allclose(st, [float(a) for a, _ in ref], rtol=0, atol=1e-9 * scale)
    assert np.allclose(fi, [float(b) for _, b in ref], rtol=0, atol=1e-9 * scale)
    assert T.validate(sched, bw, list(zip(st, fi))) == []
    # Theorem 3 and its tight form hold for any correct AllReduce
    ell = model.slowdowns(bw)[0][0]
    assert mk_ref >= model.lb_servers_tight(q, g, ell, n)


def test_server_validator_uses_nvlink_ports():
    """An NVLink flow must last len/(g-1); a NIC flow between servers and an
    NVLink flow of the same rank may overlap (different ports), two NVLink
    flows of one rank may not."""
    q, g, bw, n, k = 3, 2, [1, 1, 0.5], 64 * 48, 24
    sched = oracle.Schedule.servers(q, g, bw, n, k)
    _, good = T.evaluate(sched, bw)
    assert T.validate(sched, bw, good) == []
    flows = [(src, st["dst"]) for st in sched.steps() for src in st["srcs"]]
    i = next(i for i, (a, b) in enumerate(flows) if a // g == b // g)
    s, e = good[i]
    bad = list(good)
    bad[i] = (s, s + 2 * (e - s))  # an NVLink flow at NIC speed
    assert any("duration" in x for x in T.validate(sched, bw, bad))


@pytest.mark.parametrize("w", ["q4g4_bf16", "q16g4_f32"])
def test_server_workload_evaluated_times(o, w):
    """Full-size server workloads: the evaluated makespan lies above the
    tight multi-GPU bound (App. B.3) and within 20 % of the App. E closed
    form (list scheduling does not reproduce the eight-row N-S overlay)."""
    from paper_2606_01680_amd.workloads import WORKLOADS
    W = WORKLOADS[w]
    pl = o.optcc_plan_servers(W.q, W.g, W.bandwidths, W.n, W.k)
    mk, _, _ = pl.timeline(with_flows=False)
    lb = o.optcc_lower_bound_servers(W.q, W.g, W.bandwidths, W.n)
    closed = o.optcc_model_time(pl)
    assert lb * (1 - 1e-12) <= mk <= 1.2 * closed
