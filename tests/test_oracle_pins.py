"""Pins of the oracle against what the paper and the mathematics fix.

Each test names the passage it follows.  None of them re-derives the oracle's
own formula: they check worked-example counts printed in the paper, the
definition of the result (exact integer sums, fp error bounds), symbolic
contributor sets, the paper's lemmas and closed-form limits, and brute-force
minimisation of the lower-bound programmes.
"""
import itertools
import json
import os
from fractions import Fraction as F

import numpy as np
import pytest

import oracle
from oracle import model

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _bw(p, slow):
    b = [1.0] * p
    for r, v in slow.items():
        b[r] = v
    return b


def _rand(dtype, p, n, seed):
    rng = np.random.default_rng(seed)
    if dtype == "i32":
        return rng.integers(-(2**31), 2**31, size=(p, n), dtype=np.int64).astype(np.int32)
    x = rng.standard_normal((p, n)).astype(np.float32)
    if dtype == "bf16":
        return oracle.bf16_round(x)
    if dtype == "f16":
        return oracle.f16_round(x)
    return x


# A grid of bandwidth profiles: no straggler, one straggler (l >= 2, l < 2,
# l exactly 2), several stragglers with mixed slowdowns and arbitrary ranks.
CASES = [
    (3, {}), (4, {3: 0.5}), (5, {0: 0.5}), (5, {2: 0.75}), (7, {6: 0.875}),
    (8, {1: 0.875}), (9, {4: 0.25}), (6, {0: 0.5, 5: 0.75}), (7, {1: 0.5, 2: 0.5}),
    (9, {0: 0.875, 3: 0.75, 8: 0.5}), (16, {15: 0.5}), (8, {}), (5, {4: 0.5 + 1e-9}),
]


# ------------------------------------------------------------ worked example
def test_worked_example_flow_counts():
    """Sec. 4.2: p=5, l=2, straggler GPU 0: per segment 12 Stage-1 flows,
    4 Stage-2, 4 Stage-3 and 12 Stage-4 flows (golden fixture)."""
    g = json.load(open(os.path.join(GOLD, "worked_example_p5_l2.json")))
    p, k = g["p"], g["k"]
    n = k * (p - 1) * 64 * 3
    s = oracle.Schedule(p, g["bandwidths"], n, k)
    assert s.kind == "single_ge2" and list(s.stragglers) == [0]
    # Stage of a flow: slot 1 -> S1, slot 4 -> S4; flows that leave the
    # straggler are Stage 3 (download), flows that reach it are Stage 2.
    for seg in range(k):
        cnt = {"S1": 0, "S2": 0, "S3": 0, "S4": 0}
        for st in s.steps():
            if st["seg"] != seg:
                continue
            for src in st["srcs"]:
                if st["slot"] == 1:
                    cnt["S1"] += 1
                elif st["slot"] == 4:
                    cnt["S4"] += 1
                elif src == 0:
                    cnt["S3"] += 1
                elif st["dst"] == 0:
                    cnt["S2"] += 1
                else:
                    raise AssertionError(st)
        assert cnt == g["flows_per_segment"], (seg, cnt)
    # 2(p-1) slots per stage, a straggler flow taking l=2 cells: the four
    # stages of one pattern fill 4 * 8 cells; k segments take k+1 bodies.
    ell = 2
    assert (p - 1) * ell == g["slots_per_stage"]
    assert 4 * g["slots_per_stage"] == g["slots_per_pattern"]
    assert model.optcc_single(p, ell, 1, k) == F(ell) * F(k + 1, k)
    assert (k + 1) == g["parallel_bodies"]


def test_bubble_example_split():
    """Sec. 4.2 caption + App. C at p=5, l=1.5, k=4: s'=3n/52, D=n/52; the
    data accounting n = k[(p-1)s' + D] holds and an enlarged flow lasts 2s'."""
    g = json.load(open(os.path.join(GOLD, "bubble_example_p5_l1.5.json")))
    p, k, ell = g["p"], g["k"], F(g["ell"])
    sp, d = model.bubble_split(p, ell, 1, k)
    assert sp == F(g["s_prime_over_n"]) and d == F(g["d_over_n"])
    assert k * ((p - 1) * sp + d) == 1
    assert (1 + (2 - ell) / ell) * ell * sp == F(g["enlarged_flow_duration_over_s_prime"]) * sp
    # The oracle's integer split reproduces it exactly when n is a multiple
    # of 52 quanta: every section is s' and every P2P chunk is D.
    n = 52 * 64
    s = oracle.Schedule(p, g["bandwidths"], n, k)
    assert s.kind == "single_lt2" and abs(s.ell[0] - 1.5) == 0
    for seg in range(k):
        assert s.p2p_len[seg] == d * n
        secs = {st["sec"]: st["len"] for st in s.steps() if st["seg"] == seg and st["sec"] >= 0}
        assert set(secs.values()) == {sp * n}
    # Straggler volume equals z* n, the minimiser of the tight bound (App. B.1).
    sent = sum(ln for (_, src, dst, _, ln, _) in s.flows() if src == 0)
    recv = sum(ln for (_, src, dst, _, ln, _) in s.flows() if dst == 0)
    assert sent == recv == model.straggler_volume_optimum(p, ell, n)


# ------------------------------------------------------- result definition
@pytest.mark.parametrize("p,slow", CASES)
@pytest.mark.parametrize("n,k", [(0, 4), (1, 4), (63, 4), (257, 8), (1000, 4), (64 * 41 + 7, 8)])
def test_int32_exact_and_provenance(orc, p, slow, n, k):
    """Sec. 3: every rank ends with the elementwise sum.  int32 wraps exactly,
    so any dropped, doubled or misplaced term changes the bits; the symbolic
    run checks that no REDUCE counts a rank twice."""
    s = orc.Schedule(p, _bw(p, slow), n, k)
    x = _rand("i32", p, n, 7 * p + n)
    want = orc.brute_sum("i32", x)
    y = orc.run(s, "i32", x.copy())
    assert (y == want[None, :]).all()
    if n <= 300:
        ok, msg = orc.provenance(s)
        assert ok, msg


@pytest.mark.parametrize("p,slow", CASES)
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_float_error_bound(orc, p, slow, dtype):
    """Sec. 3 result within the recursive-summation bound p u sum|x_i|
    (u = 2^-24 fp32, 2^-11 fp16, 2^-8 bf16), and every rank's buffer bitwise
    identical."""
    n, k = 64 * 37 + 5, 8
    s = orc.Schedule(p, _bw(p, slow), n, k)
    x = _rand(dtype, p, n, 11 * p)
    y = orc.run(s, dtype, x.copy())
    assert (y == y[0][None, :]).all()
    got = orc.values_f64(dtype, y[0])
    err = np.abs(got - orc.brute_sum(dtype, x))
    assert (err <= orc.tolerance(dtype, p, x)).all()


def test_bf16_rounding_matches_library():
    """bf16 narrowing is round-to-nearest-even: torch's CPU conversion is a
    library routine of the same definition (NaN excluded)."""
    import torch
    rng = np.random.default_rng(3)
    bits = rng.integers(0, 2**32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    edge = np.array([0x00000000, 0x80000000, 0x00008000, 0x00018000, 0x3f808000,
                     0x3f818000, 0x7f7fffff, 0xff7fffff, 0x7f800000, 0x0000ffff,
                     0x007fffff, 0x3f7fffff, 0x47ffffff], np.uint32)
    bits = np.concatenate([bits, edge])
    x = bits.view(np.float32)
    keep = ~np.isnan(x)
    ours = oracle.bf16_round(x[keep])
    ref = torch.from_numpy(x[keep].copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (ours == ref).all()


def test_f16_conversions_match_library():
    """fp16 narrowing is IEEE binary16 round-to-nearest-even with subnormals
    and overflow to infinity, widening is exact: torch's CPU conversions are
    library routines of the same definitions.  All 2^16 half patterns widen
    identically (NaN payloads aside) and narrow back to themselves; 2^20
    random fp32 patterns plus the boundaries (largest finite, the overflow
    midpoint 65520, the smallest normal and subnormal, the 2^-25 tie, signed
    zeros, infinities) narrow identically."""
    import torch
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = oracle.f16_to_f64(h)
    ref = torch.from_numpy(h.view(np.int16).copy()).view(torch.float16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert (np.isnan(ours) == nan).all()
    assert (ours[~nan] == ref[~nan]).all()
    assert (np.signbit(ours[~nan]) == np.signbit(ref[~nan])).all()
    assert (oracle.f16_round(ours[~nan].astype(np.float32)) == h[~nan]).all()
    rng = np.random.default_rng(4)
    bits = rng.integers(0, 2**32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    # values from 2^-30 to 2^20 hit the subnormal, normal and overflow paths often
    near = (rng.integers(97, 148, size=1 << 18).astype(np.uint32) << 23) | \
        rng.integers(0, 1 << 23, size=1 << 18).astype(np.uint32)
    edge = np.array([0x477fe000, 0x477ff000, 0x477fefff, 0x477ff001, 0x38800000, 0x387fffff,
                     0x33800000, 0x33000000, 0x33000001, 0x32ffffff, 0x00000000, 0x80000000,
                     0x7f800000, 0xff800000, 0x3f800000, 0x3f801000, 0x3f803000, 0x3f800fff],
                    np.uint32)
    x = np.concatenate([bits, near, near | 0x80000000, edge]).view(np.float32)
    x = x[~np.isnan(x)]
    ref = torch.from_numpy(x.copy()).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    assert (oracle.f16_round(x) == ref).all()


def _fold(vals):
    """Left fold of fp32 additions in the listed order: numpy's sequential
    cumulative sum (every step of the schedule adds one new value to a
    running partial, and fp32 addition is commutative, so each result is such
    a fold)."""
    return np.cumsum(np.stack(vals), axis=0, dtype=np.float32)[-1]


def _section_ranges(s):
    out = {}
    for st in s.steps():
        out.setdefault((st["seg"], st["sec"]), (st["off"], st["len"]))
    return out


@pytest.mark.parametrize("p,slow,k", [(6, {}, 4), (5, {2: 0.5}, 4), (8, {1: 0.875}, 8),
                                      (6, {0: 0.5, 5: 0.75}, 8),
                                      (9, {0: 0.875, 3: 0.75, 8: 0.5}, 8)])
def test_fp32_association_is_the_chain(orc, p, slow, k):
    """Where the stage order puts each addition (Sec. 4.1 orderings, App. C
    star, App. D folds; readings of where the stragglers' values join): the
    fp32 result on every rank equals numpy's sequential cumulative sum over
    the ranks in that order.  Ordering 1: chain from R[j], the worst
    straggler last (the other stragglers first, at R[j], for A'/C');
    ordering 2: every straggler, worst first, at R[j] before the chain; P2P
    chunk: the straggler, then R[0..P'-1]."""
    bw = _bw(p, slow)
    n = 64 * 3 * k * p + 17
    s = orc.Schedule(p, bw, n, k)
    x = _rand("f32", p, n, 5 + p)
    y = orc.run(s, "f32", x.copy())
    ring, strag, pp = list(s.ring), list(s.stragglers), s.pp
    m = len(strag)
    seen = 0
    for (seg, j), (off, ln) in _section_ranges(s).items():
        c = slice(off, off + ln)
        seen += ln
        if j < 0:
            order = strag[:1] + ring
        else:
            chain = [ring[(j + t) % pp] for t in range(pp)]
            if m <= 1:
                ordering = 1 if seg % 4 in (0, 2) else 2
            else:
                ordering = 2 if seg % 4 in (0, 1) else 1
            if ordering == 2:
                order = chain[:1] + strag + chain[1:]
            else:
                order = chain[:1] + strag[1:] + chain[1:] + strag[:1]
        want = _fold([x[r, c] for r in order])
        assert all((y[r, c].view(np.uint32) == want.view(np.uint32)).all() for r in range(p))
    assert seen == n


@pytest.mark.parametrize("q,g,slow", [(4, 3, {2: 0.5}), (3, 4, {1: 0.25}), (5, 2, {0: 0.75})])
def test_fp32_association_servers(orc, q, g, slow):
    """App. E: a server's value is the fold of its local ring from position
    g-1 down to the leader; the chain folds the collected values; type 2
    starts it with the straggler server's collected value, type 1 hands the
    healthy sum to the straggler's leader and folds forward along its ring
    (numpy's sequential cumulative sums)."""
    k = 24
    n = 64 * 2 * k * g + 33
    s = orc.Schedule.servers(q, g, _sbw(q, slow), n, k)
    x = _rand("f32", s.p, n, 9 + q * g)
    y = orc.run(s, "f32", x.copy())
    ring, sv, pp = list(s.ring), int(s.stragglers[0]), s.pp

    def rank(server, part, d):
        return server * g + (part + d) % g

    seen = 0
    for (seg, j), (off, ln) in _section_ranges(s).items():
        c = slice(off, off + ln)
        seen += ln
        part, cseg = divmod(seg, k)
        collect = [_fold([x[rank(h, part, d), c] for d in range(g - 1, -1, -1)])
                   for h in [ring[(j + t) % pp] for t in range(pp)]]
        if cseg % 4 in (0, 2):  # type 1
            want = _fold([_fold(collect)] + [x[rank(sv, part, d), c] for d in range(g)])
        else:
            straggler = _fold([x[rank(sv, part, d), c] for d in range(g - 1, -1, -1)])
            want = _fold(collect[:1] + [straggler] + collect[1:])
        assert all((y[r, c].view(np.uint32) == want.view(np.uint32)).all() for r in range(s.p))
    assert seen == n


# ------------------------------------------------------------- stage pins
def _sets_after(s, slot_hi, n):
    p = s.p
    held = [[1 << r for _ in range(n)] for r in range(p)]
    for st in s.steps():
        if st["slot"] >= slot_hi:
            continue
        for c in range(st["off"], min(st["off"] + st["len"], n)):
            if st["op"] == oracle.COPY:
                held[st["dst"]][c] = held[st["srcs"][0]][c]
            else:
                for src in st["srcs"]:
                    held[st["dst"]][c] |= held[src][c]
    return held


@pytest.mark.parametrize("p,slow", [(5, {0: 0.5}), (6, {3: 0.25}), (7, {0: 0.5, 6: 0.75})])
def test_stage_semantics(orc, p, slow):
    """Sec. 4.1: after Stage 1 of an ordering-1 section the holder has the sum
    of all healthy ranks; after Stage 2 the straggler has the global sum.  In
    ordering 2 the chain already produces the global sum (App. D for m >= 2)."""
    n, k = 64 * 4 * p, 4
    s = orc.Schedule(p, _bw(p, slow), n, k)
    full = (1 << p) - 1
    healthy = sum(1 << r for r in s.ring)
    pp = s.pp
    after1 = _sets_after(s, 2, n)
    after2 = _sets_after(s, 3, n)
    for st in s.steps():
        if st["slot"] != 1 or st["dst"] != s.ring[(st["sec"] + pp - 1) % pp]:
            continue  # the last hop of each chain writes the holder
        c = st["off"]
        holder = st["dst"]
        ordering = (1 if st["seg"] % 2 == 0 else 2) if s.m == 1 else (2 if st["seg"] % 4 < 2 else 1)
        if ordering == 1:
            extra = sum(1 << r for r in s.stragglers[1:])
            assert after1[holder][c] == healthy | extra
            assert after2[s.stragglers[0]][c] == full
        else:
            assert after1[holder][c] == full


@pytest.mark.parametrize("p,slow", CASES)
def test_lemmas_on_flows(orc, p, slow):
    """App. B lemmas on the oracle's flows: total traffic >= 2(p-1)N; every
    straggler sends and receives every coordinate at least once; and the
    time-weighted NIC load (a flow touching rank i costs l_i per element on
    both ends) is at least the best lower bound."""
    n, k = 64 * 5 * p + 13, 8
    s = orc.Schedule(p, _bw(p, slow), n, k)
    flows = s.flows()
    assert sum(f[4] for f in flows) >= 2 * (p - 1) * n
    for st_rank in s.stragglers:
        out_cov = np.zeros(n, bool)
        in_cov = np.zeros(n, bool)
        for (_, src, dst, off, ln, _) in flows:
            if src == st_rank:
                out_cov[off:off + ln] = True
            if dst == st_rank:
                in_cov[off:off + ln] = True
        assert out_cov.all() and in_cov.all()
    ell = [F(1)] * p
    bmax = max(F(b) for b in _bw(p, slow))
    for r, b in enumerate(_bw(p, slow)):
        ell[r] = bmax / F(b)
    send = [F(0)] * p
    recv = [F(0)] * p
    for (_, src, dst, _, ln, _) in flows:
        c = ln * max(ell[src], ell[dst])
        send[src] += c
        recv[dst] += c
    assert max(max(send), max(recv)) >= model.lower_bound(_bw(p, slow), n)


@pytest.mark.parametrize("p,slow,k", [(8, {7: 0.875}, 64), (16, {15: 0.5}, 128),
                                      (64, {62: 0.75, 63: 0.5}, 128),
                                      (128, {124: 0.875, 125: 0.75, 126: 0.5, 127: 0.5}, 256)])
def test_straggler_volume(orc, p, slow, k):
    """Straggler volume: N per straggler when there is no bubble filling
    (Sec. 4.1: one section in and one out per section; App. D likewise), and
    z* N for l < 2 up to one quantum per segment (App. C accounting)."""
    n = 1 << 16
    s = orc.Schedule(p, _bw(p, slow), n, k, seg_lo=0, seg_hi=4)
    # only the first 4 segments are built: volume over their elements
    n4 = int(s.seg_off[4]) if k > 4 else n
    for r in s.stragglers:
        sent = sum(ln for (_, src, dst, _, ln, _) in s.flows() if src == r)
        recv = sum(ln for (_, src, dst, _, ln, _) in s.flows() if dst == r)
        if s.kind == "single_lt2":
            want = model.straggler_volume_optimum(p, F(s.ell[r]), n4)
            assert abs(sent - want) <= 4 * p * 64 and abs(recv - want) <= 4 * p * 64
        else:
            assert sent == recv == n4


# ------------------------------------------------------------- model pins
@pytest.mark.parametrize("p", [3, 5, 8, 16, 128])
@pytest.mark.parametrize("k", [4, 64])
def test_model_limits(p, k):
    """Sec. 4.3: at l=1 the l<2 formula gives T0; at l=2 both single-straggler
    branches give 2n(k+1)/k; for l in [1,2] T/T0 <= 1 + 1/(p-1) as k grows;
    every model time is at least the best lower bound."""
    n = 1000
    assert model.optcc_single(p, F(1), n, k) == model.t0(p, n) * F(k, k)
    lt = F(2 * (p - 1)) * 2 * n / ((p - 2) * 2 + 2) * F(k + 1, k)
    assert lt == model.optcc_single(p, F(2), n, k) == 2 * n * F(k + 1, k)
    for ell in [F(1), F(9, 8), F(4, 3), F(3, 2), F(7, 4), F(2)]:
        asym = F(2 * (p - 1)) * ell / ((p - 2) * ell + 2)
        assert asym / (model.t0(p, 1)) <= 1 + F(1, p - 1)
        t = model.optcc_single(p, ell, n, k)
        assert t >= model.lb_tight_single(p, ell, n)
    for ell in [F(2), F(3), F(8)]:
        assert model.optcc_single(p, ell, n, k) >= model.lb_tight_single(p, ell, n)


def test_model_ring_is_t0():
    """No straggler: the schedule is the ring, 2(p-1)n/p (Sec. 3)."""
    for p in [3, 8, 128]:
        assert model.optcc_time([1.0] * p, 1 << 20, 64) == F(2 * (p - 1), p) * (1 << 20)
        assert model.lower_bound([2.0] * p, 10) == model.t0(p, 10)


def _minmax_lp(terms, nvar, lb=1.0):
    """min t s.t. t >= a.x + c for each (a, c), x_i >= lb: brute force by LP."""
    from scipy.optimize import linprog
    A, b = [], []
    for a, c in terms:
        A.append(list(a) + [-1.0])
        b.append(-c)
    res = linprog([0.0] * nvar + [1.0], A_ub=A, b_ub=b,
                  bounds=[(lb, None)] * nvar + [(None, None)], method="highs")
    assert res.status == 0
    return res.fun


@pytest.mark.parametrize("p", [3, 4, 8, 16, 64])
@pytest.mark.parametrize("ell", [1.05, 8 / 7, 1.5, 1.9, 2.0, 2.5, 4.0])
def test_single_lower_bounds_by_lp(p, ell):
    """App. B.1: Theorem 1 and the tight bound are the minima over x, y >= 1 of
    the max of the straggler and (time-weighted) healthy bottlenecks."""
    weak = _minmax_lp([((ell, 0), 0.0), ((0, ell), 0.0),
                       ((-1 / (p - 1), 0), 2.0), ((0, -1 / (p - 1)), 2.0)], 2)
    tight = _minmax_lp([((ell, 0), 0.0), ((0, ell), 0.0),
                        ((-1 / (p - 1), (ell - 1) / (p - 1)), 2.0),
                        (((ell - 1) / (p - 1), -1 / (p - 1)), 2.0)], 2)
    assert float(model.lb_weak_single(p, F(ell), 1)) == pytest.approx(weak, rel=1e-9)
    assert float(model.lb_tight_single(p, F(ell), 1)) == pytest.approx(tight, rel=1e-9)


@pytest.mark.parametrize("p,ells", [(8, [2.0, 4 / 3]), (64, [2.0, 4 / 3]),
                                    (128, [2.0, 2.0, 4 / 3, 8 / 7]), (10, [1.1, 1.05]),
                                    (20, [3.0, 1.5, 1.2])])
def test_multi_lower_bound_by_lp(p, ells):
    """App. B.2: Theorem 2 is the minimum over x_i >= 1 of the max of the m
    straggler bottlenecks l_i x_i and the healthy average [2(p-1)-sum x]/(p-m);
    with m = 1 it is Theorem 1."""
    m = len(ells)
    terms = []
    for i, e in enumerate(ells):
        a = [0.0] * m
        a[i] = e
        terms.append((a, 0.0))
    terms.append(([-1.0 / (p - m)] * m, 2.0 * (p - 1) / (p - m)))
    want = _minmax_lp(terms, m)
    ells_f = sorted((F(e) for e in ells), reverse=True)
    assert float(model.lb_multi(p, ells_f, 1)) == pytest.approx(want, rel=1e-9)
    assert model.lb_multi(p, [F(3, 2)], 7) == model.lb_weak_single(p, F(3, 2), 7)


def test_table1_asymptotics():
    """Table 1: relative to T0, the single-straggler bound is
    1 + (l-1)/(l p) + O(1/p^2) below 2 and l/2 + l/(2p) + O(1/p^2) above."""
    for ell in [F(5, 4), F(3, 2)]:
        for p in [10**4, 10**5]:
            r = model.lb_weak_single(p, ell, 1) / model.t0(p, 1)
            assert abs((r - 1 - (ell - 1) / (ell * p)) * p * p) < 10
    for ell in [F(5, 2), F(4)]:
        for p in [10**4, 10**5]:
            r = model.lb_weak_single(p, ell, 1) / model.t0(p, 1)
            assert abs((r - ell / 2 - ell / (2 * p)) * p * p) < 10


def test_multi_model_regimes():
    """App. D: T = (k+4) T_body -> 2(p-1)/(p-m) n for l_1 < 2 and
    (l_1 + 2(m-1)/(p-m)) n for l_1 >= 2, and never below Theorem 2."""
    n = 1
    for p, ells in [(64, [F(2), F(4, 3)]), (128, [F(2), F(2), F(4, 3), F(8, 7)]),
                    (20, [F(3, 2), F(5, 4)]), (30, [F(3), F(2)])]:
        m = len(ells)
        big = 10**9
        t = model.optcc_multi(p, ells, n, big)
        if ells[0] < 2:
            lim = F(2 * (p - 1), p - m)
        else:
            lim = max(F(2 * (p - 1), p - m), ells[0] + F(2 * (m - 1), p - m))
        assert abs(t - lim) < F(1, 10**6)
        for k in [4, 128, 256]:
            assert model.optcc_multi(p, ells, n, k) >= model.lb_multi(p, ells, n)


def test_invalid_inputs(orc):
    """Problem setting (p >= 3), k a multiple of 4 (Sec. 4.2 pipelining)."""
    with pytest.raises(orc.OracleError):
        orc.Schedule(2, [1.0, 1.0], 10, 4)
    with pytest.raises(orc.OracleError):
        orc.Schedule(4, [1.0] * 4, 10, 6)
    with pytest.raises(orc.OracleError):
        orc.Schedule(4, [1.0, 0.0, 1.0, 1.0], 10, 4)
    with pytest.raises(orc.OracleError):
        orc.Schedule(4, [1.0, 0.5, 0.5, 0.5], 10, 4)  # one healthy rank


# ------------------------------------------- several GPUs per server (App. E)
SERVER_CASES = [(3, 2, {1: 0.5}), (4, 2, {3: 0.75}), (4, 3, {0: 0.5}), (5, 4, {2: 0.25}),
                (3, 4, {2: 0.875}), (6, 2, {5: 0.5})]


def _sbw(q, slow):
    return _bw(q, slow)


@pytest.mark.parametrize("q,g,slow", SERVER_CASES)
@pytest.mark.parametrize("n", [0, 1, 63, 64 * 3 * 24 + 5, 5000])
def test_servers_int32_exact_and_provenance(orc, q, g, slow, n):
    """App. E schedule, Sec. 3 correctness: exact int32 sums on every rank and
    no rank counted twice."""
    s = orc.Schedule.servers(q, g, _sbw(q, slow), n, 24)
    assert s.kind == "servers" and s.p == q * g
    x = _rand("i32", s.p, n, 3 * q + g + n)
    y = orc.run(s, "i32", x.copy())
    assert (y == orc.brute_sum("i32", x)[None, :]).all()
    if 0 < n <= 300:
        ok, msg = orc.provenance(s)
        assert ok, msg


@pytest.mark.parametrize("q,g,slow", SERVER_CASES)
@pytest.mark.parametrize("dtype", ["f32", "bf16", "f16"])
def test_servers_float_error_bound(orc, q, g, slow, dtype):
    n = 64 * 40 + 3
    s = orc.Schedule.servers(q, g, _sbw(q, slow), n, 24)
    x = _rand(dtype, s.p, n, 5 * q + g)
    y = orc.run(s, dtype, x.copy())
    assert (y == y[0][None, :]).all()
    got = orc.values_f64(dtype, y[0])
    assert (np.abs(got - orc.brute_sum(dtype, x)) <= orc.tolerance(dtype, s.p, x)).all()


@pytest.mark.parametrize("q,g,slow", SERVER_CASES)
def test_servers_nic_volumes(orc, q, g, slow):
    """App. B.3 lemmas: every coordinate crosses server boundaries at least
    2(q-1) times, and the slow server sends and receives every coordinate;
    this schedule meets both exactly (2(q-1)N inter-server elements, N out of
    and N into the slow server)."""
    n = 64 * 2 * 24 * 3 + 7
    s = orc.Schedule.servers(q, g, _sbw(q, slow), n, 24)
    sv = int(s.stragglers[0])
    inter = sent = recv = 0
    for (_, src, dst, _, ln, _) in s.flows():
        if src // g != dst // g:
            inter += ln
            sent += ln if src // g == sv else 0
            recv += ln if dst // g == sv else 0
    assert inter == 2 * (q - 1) * n
    assert sent == n and recv == n


@pytest.mark.parametrize("q,g,slow", [(4, 3, {0: 0.5}), (5, 2, {4: 0.75})])
def test_servers_stage_semantics(orc, q, g, slow):
    """App. E: after N1 every healthy leader holds its server's local sum;
    in type 1 the end of the straggler's ring holds the global sum after N2;
    in type 2 the holder's leader holds it after S1."""
    n, k = 64 * (q - 1) * 24 * g, 24
    s = orc.Schedule.servers(q, g, _sbw(q, slow), n, k)
    sv = int(s.stragglers[0])
    full = (1 << s.p) - 1
    after = {h: _sets_after(s, h, n) for h in (2, 4, 6)}
    for seg in range(s.nseg):
        part, sg = divmod(seg, k)
        c = int(s.seg_off[seg])
        if s.seg_len[seg] == 0:
            continue
        for h in s.ring:
            leader = int(h) * g + part
            assert after[2][leader][c] == sum(1 << (int(h) * g + l) for l in range(g))
        typ = 1 if sg % 4 in (0, 2) else 2
        if typ == 1:
            end = sv * g + (part + g - 1) % g
            assert after[6][end][c] == full
        else:
            # section 0 of the segment: chain starts at ring[0], holder ring[-1]
            holder = int(s.ring[-1]) * g + part
            assert after[4][holder][c] == full


def test_servers_bounds_and_model():
    """Theorem 3 (Sec. 3 form max{2l(p-g)/(g(l(p-g)+g)), l/g} n) equals its
    App. B.3 form; g = 1 recovers Theorem 1 and the tight single bound; the
    App. E time stays within q/(q-1) of the tight bound for l < 2 as k grows
    and above it always."""
    for q, g in [(4, 2), (8, 8), (16, 4), (33, 3)]:
        p = q * g
        for ell in [F(9, 8), F(3, 2), F(2), F(3)]:
            sec3 = max(2 * ell * (p - g) / (g * (ell * (p - g) + g)), ell / g)
            assert sec3 == model.lb_servers_weak(q, g, ell, 1)
            assert model.lb_servers_tight(q, g, ell, 1) >= model.lb_servers_weak(q, g, ell, 1)
            t = model.optcc_servers(q, g, ell, 1, 10**9)
            assert t >= model.lb_servers_tight(q, g, ell, 1)
            if ell < 2:
                assert t / model.lb_servers_tight(q, g, ell, 1) < F(q, q - 1) * (1 + F(1, 10**6))
            for k in (24, 64):
                assert model.optcc_servers(q, g, ell, 1, k) >= model.lb_servers_tight(q, g, ell, 1)
    for p in [5, 9]:
        for ell in [F(3, 2), F(5, 2)]:
            assert model.lb_servers_weak(p, 1, ell, 7) == model.lb_weak_single(p, ell, 7)
            assert model.lb_servers_tight(p, 1, ell, 7) == model.lb_tight_single(p, ell, 7)


def test_servers_invalid(orc):
    with pytest.raises(orc.OracleError):
        orc.Schedule.servers(4, 2, [1, 1, 1, 1], 100, 24)  # no straggler server
    with pytest.raises(orc.OracleError):
        orc.Schedule.servers(4, 2, [1, 0.5, 0.5, 1], 100, 24)  # two
    with pytest.raises(orc.OracleError):
        orc.Schedule.servers(4, 2, [1, 0.5, 1, 1], 100, 20)  # 8 does not divide k
    with pytest.raises(orc.OracleError):
        orc.Schedule.servers(4, 2, [1, 0.5, 1, 1], 100, 16)  # k < 24
