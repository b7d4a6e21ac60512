"""Host half of the library against the oracle (no GPU needed).

Row a0 (plan) must match the oracle's independently built schedule bit for
bit: every step's slot, segment, section, operation, destination, sources in
accumulation order and element range.  Row a9 (model time and lower bound)
must match the oracle's exact rationals to fp64 rounding.
"""
import ctypes
import os
import re
import time

import numpy as np
import pytest

import oracle
from oracle import model

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def o():
    from paper_2606_01680_amd import optcc
    return optcc


def _bw(p, slow):
    b = [1.0] * p
    for r, v in slow.items():
        b[r] = v
    return b


PROFILES = [
    (3, {}), (3, {1: 0.5}), (4, {3: 0.5}), (5, {0: 0.5}), (5, {2: 0.75}), (7, {6: 0.875}),
    (8, {7: 0.875}), (8, {0: 0.25}), (9, {4: 0.5, 5: 0.5}), (6, {0: 0.5, 5: 0.75}),
    (9, {0: 0.875, 3: 0.75, 8: 0.5}), (16, {15: 0.5}), (12, {}), (10, {3: 0.5000001}),
    (6, {1: 0.9, 2: 0.8, 3: 0.7, 4: 0.6}),
    (4, {0: 0.5, 1: 0.75}), (5, {1: 0.5, 2: 0.5, 3: 0.5}), (8, {2: 0.9999999}),
    (6, {5: 0.50000001}), (6, {5: 0.5}), (256, {0: 0.5, 100: 0.875, 255: 0.75}),
]
SIZES = [(0, 4), (1, 4), (63, 4), (64, 4), (257, 8), (1000, 4), (64 * 53 + 9, 8), (5000, 12)]


def _steps_of_flows(fl):
    """Group the library's flows back into steps (sources in listed order)."""
    steps = []
    last = None
    for f in fl:
        if last is not None and f["step"] == last:
            steps[-1]["srcs"].append(int(f["src"]))
            continue
        last = f["step"]
        steps.append(dict(slot=int(f["slot"]), seg=int(f["segment"]), sec=int(f["section"]),
                          op=int(f["op"]), dst=int(f["dst"]), srcs=[int(f["src"])],
                          off=int(f["offset"]), len=int(f["length"])))
    return steps


@pytest.mark.parametrize("p,slow", PROFILES)
@pytest.mark.parametrize("n,k", SIZES)
def test_plan_equals_oracle(o, p, slow, n, k):
    bw = _bw(p, slow)
    pl = o.optcc_plan(p, bw, n, k)
    ref = oracle.Schedule(p, bw, n, k)
    assert pl.kind == ref.kind and pl.m == ref.m and pl.healthy == ref.pp
    assert list(pl.ring) == list(ref.ring)
    assert list(pl.stragglers) == list(ref.stragglers)
    assert np.array_equal(pl.slowdowns, ref.ell)
    off, ln, p2p = pl.segments()
    assert np.array_equal(off, ref.seg_off) and np.array_equal(ln, ref.seg_len)
    assert np.array_equal(p2p, ref.p2p_len)
    fl = pl.flows()
    assert len(fl) == pl.num_flows
    got = _steps_of_flows(fl)
    assert len(got) == pl.num_steps
    assert got == ref.steps()


@pytest.mark.parametrize("w", ["p4_f32", "p8_f32", "p16_bf16", "p64_f32", "p128_f32"])
def test_workload_plans_equal_oracle_counts(o, w):
    """Full-size plans: split, kinds and flow counts equal the oracle's (first
    8 segments' steps compared one by one)."""
    from paper_2606_01680_amd.workloads import WORKLOADS
    W = WORKLOADS[w]
    pl = o.optcc_plan(W.p, W.bandwidths, W.n, W.k)
    ref = oracle.Schedule(W.p, W.bandwidths, W.n, W.k, seg_lo=0, seg_hi=8)
    off, ln, p2p = pl.segments()
    assert np.array_equal(off, ref.seg_off) and np.array_equal(ln, ref.seg_len)
    assert np.array_equal(p2p, ref.p2p_len)
    fl = pl.flows()
    got = _steps_of_flows(fl[fl["segment"] < 8])
    assert got == ref.steps()
    expect_flows = {"p4_f32": 144, "p8_f32": 7168, "p16_bf16": 57600, "p64_f32": 999936,
                    "p128_f32": 8062976}
    assert pl.num_flows == expect_flows[w]


@pytest.mark.parametrize("p,slow", PROFILES + [(64, {62: 0.75, 63: 0.5}),
                                               (128, {124: 0.875, 125: 0.75, 126: 0.5, 127: 0.5})])
@pytest.mark.parametrize("n,k", [(1 << 20, 64), (12345, 8)])
def test_model_and_bound_equal_oracle(o, p, slow, n, k):
    bw = _bw(p, slow)
    pl = o.optcc_plan(p, bw, n, k)
    t = o.optcc_model_time(pl)
    assert t == pytest.approx(float(model.optcc_time(bw, n, k)), rel=1e-13)
    assert o.optcc_model_time(pl, bw) == t
    lb = o.optcc_lower_bound(p, bw, n)
    assert lb == pytest.approx(float(model.lower_bound(bw, n)), rel=1e-13)
    assert t >= lb * (1 - 1e-15)


def test_workload_model_values(o):
    """The five workloads' modeled times and bounds, in units of N, equal the
    oracle's exact rationals."""
    from paper_2606_01680_amd.workloads import WORKLOADS
    for w in WORKLOADS.values():
        if w.g > 1:  # several GPUs per server
            pl = o.optcc_plan_servers(w.q, w.g, w.bandwidths, w.n, w.k)
            ell = model.slowdowns(w.bandwidths)[0][0]
            assert o.optcc_model_time(pl) / w.n == pytest.approx(
                float(model.optcc_servers(w.q, w.g, ell, 1, w.k)), rel=1e-13)
            assert o.optcc_lower_bound_servers(w.q, w.g, w.bandwidths, w.n) / w.n == pytest.approx(
                float(model.lb_servers_tight(w.q, w.g, ell, 1)), rel=1e-13)
            continue
        pl = o.optcc_plan(w.p, w.bandwidths, w.n, w.k)
        assert o.optcc_model_time(pl) / w.n == pytest.approx(
            float(model.optcc_time(w.bandwidths, 1, w.k)), rel=1e-13)
        assert o.optcc_lower_bound(w.p, w.bandwidths, w.n) / w.n == pytest.approx(
            float(model.lower_bound(w.bandwidths, 1)), rel=1e-13)


def test_errors(o):
    with pytest.raises(o.OptccError) as e:
        o.optcc_plan(2, [1.0, 1.0], 10, 4)
    assert e.value.status == o.OPTCC_EUNSUPPORTED
    for args in [(4, [1.0] * 4, 10, 6), (4, [1.0] * 4, 10, 0), (4, [1.0] * 4, -1, 4),
                 (4, [1.0, float("nan"), 1, 1], 10, 4), (4, [1.0, 0.0, 1, 1], 10, 4),
                 (4, [1.0, -1.0, 1, 1], 10, 4), (4, [1.0, float("inf"), 1, 1], 10, 4)]:
        with pytest.raises(o.OptccError) as e:
            o.optcc_plan(*args)
        assert e.value.status == o.OPTCC_EINVAL
        assert o.optcc_last_error()
    with pytest.raises(o.OptccError) as e:
        o.optcc_plan(4, [1.0, 0.5, 0.5, 0.5], 10, 4)
    assert e.value.status == o.OPTCC_EUNSUPPORTED
    with pytest.raises(o.OptccError):
        o.optcc_plan(2000, [1.0] * 2000, 10, 4)
    pl = o.optcc_plan(4, [1, 1, 1, 0.5], 100, 4)
    with pytest.raises(o.OptccError):
        o.optcc_model_time(pl, [1, 1, 0.5, 1])  # other straggler
    with pytest.raises(o.OptccError):
        o.optcc_lower_bound(2, [1, 1], 10)
    # emulate argument checks happen before any device call
    L = o.lib()
    ptrs = (ctypes.c_void_p * 4)(16, 32, 48, 64)
    assert L.optcc_allreduce_emulate(ptrs, 5, 100, 0, pl.handle, None) == o.OPTCC_EINVAL
    assert L.optcc_allreduce_emulate(ptrs, 4, 99, 0, pl.handle, None) == o.OPTCC_EINVAL
    assert L.optcc_allreduce_emulate(ptrs, 4, 100, 7, pl.handle, None) == o.OPTCC_EINVAL
    assert L.optcc_allreduce_emulate(ptrs, 4, 100, 0, pl.handle, None) == o.OPTCC_EINVAL  # overlap
    assert "overlap" in o.optcc_last_error()
    ptrs = (ctypes.c_void_p * 4)(4096, 8192, 0, 16384)
    assert L.optcc_allreduce_emulate(ptrs, 4, 100, 0, pl.handle, None) == o.OPTCC_EINVAL
    ptrs = (ctypes.c_void_p * 4)(4097, 8192, 12288, 16384)
    assert L.optcc_allreduce_emulate(ptrs, 4, 100, 0, pl.handle, None) == o.OPTCC_EINVAL
    # a buffer whose N elements would wrap around the address space
    ptrs = (ctypes.c_void_p * 4)(4096, 8192, 12288, 2**64 - 256)
    assert L.optcc_allreduce_emulate(ptrs, 4, 100, 0, pl.handle, None) == o.OPTCC_EINVAL
    assert "address space" in o.optcc_last_error()
    ptrs = (ctypes.c_void_p * 4)(4096, 8192, 12288, 16384)
    assert L.optcc_allreduce_emulate_slots(ptrs, 4, 100, 0, pl.handle, 3, 2, 1, None) == o.OPTCC_EINVAL
    assert L.optcc_allreduce_emulate_slots(ptrs, 4, 100, 0, pl.handle, 0, 7, 1, None) == o.OPTCC_EINVAL
    assert L.optcc_allreduce_emulate_slots(ptrs, 4, 100, 0, pl.handle, 0, 6, 2, None) == o.OPTCC_EINVAL
    # an empty slot range or N = 0 is a no-op that touches no device
    assert L.optcc_allreduce_emulate_slots(ptrs, 4, 100, 0, pl.handle, 2, 2, 1, None) == 0
    pl0 = o.optcc_plan(4, [1, 1, 1, 0.5], 0, 4)
    assert L.optcc_allreduce_emulate(ptrs, 4, 0, 0, pl0.handle, None) == 0
    nulls = (ctypes.c_void_p * 4)(0, 0, 0, 0)
    assert L.optcc_allreduce_emulate(nulls, 4, 0, 0, pl0.handle, None) == 0


def test_exports_match_header(o):
    """The library exports every function include/optcc.h declares."""
    hdr = open(os.path.join(ROOT, "include", "optcc.h")).read()
    decl = set(re.findall(r"^\w[\w\s\*]*?\b(optcc_\w+)\s*\(", hdr, re.M))
    assert decl == set(o.EXPORTED)
    L = ctypes.CDLL(o.LIB_PATH)
    for name in decl:
        assert hasattr(L, name), name


def test_replanning_is_fast(o):
    """Sec. 4.3 (schedule generation complexity): closed-form rules, no search;
    re-planning after a NIC failure costs well under a millisecond per plan at
    p = 1024 (median of repeated builds; host timing)."""
    bw = [1.0] * 1024
    bw[5] = 0.75
    L = o.lib()
    arr = np.asarray(bw, np.float64)
    times = []
    for _ in range(20):
        h = ctypes.c_void_p()
        t = time.perf_counter()
        rc = L.optcc_plan(1024, arr.ctypes.data, 1 << 26, 256, ctypes.byref(h))
        times.append(time.perf_counter() - t)
        assert rc == 0
        L.optcc_plan_free(h)
    assert np.median(times) < 1e-3


def test_traffic_accounting(o):
    """Fused traffic per coordinate: every input read once; one write per
    step (p=8, one straggler: ring sections 2(p-1) writes, P2P chunk p)."""
    pl = o.optcc_plan(8, [1.0] * 7 + [0.875], 1 << 20, 64)
    r, w = pl.traffic("f32")
    assert r == 8 * 4 * (1 << 20)
    off, ln, p2p = pl.segments()
    ring = int(ln.sum() - p2p.sum())
    assert w == 4 * (14 * ring + 8 * int(p2p.sum()))
    # one launch per slot re-reads the state each slot starts from
    r6, w6 = pl.traffic("f32", launches=0)
    assert w6 == w and r6 > r
    # 16-bit types move half the bytes of the same steps
    assert pl.traffic("bf16") == pl.traffic("f16") == (r // 2, w // 2)


def test_narrow_argument_checks(o):
    """optcc_narrow_f32 validates before touching the device: negative n,
    other dtypes, NULL, misaligned and overlapping pointers and lengths past
    the end of the address space are OPTCC_EINVAL; n = 0 is a no-op."""
    L = o.lib()
    assert L.optcc_narrow_f32(None, None, -1, o.DTYPES["bf16"], None) == o.OPTCC_EINVAL
    assert L.optcc_narrow_f32(None, None, 4, o.DTYPES["f32"], None) == o.OPTCC_EINVAL
    assert L.optcc_narrow_f32(None, None, 4, o.DTYPES["f16"], None) == o.OPTCC_EINVAL
    assert "non-NULL" in o.optcc_last_error()
    assert L.optcc_narrow_f32(None, None, 0, o.DTYPES["bf16"], None) == o.OPTCC_OK
    # checked before any launch: misaligned, overlapping
    assert L.optcc_narrow_f32(0x1002, 0x9000, 4, o.DTYPES["bf16"], None) == o.OPTCC_EINVAL
    assert L.optcc_narrow_f32(0x1000, 0x1008, 4, o.DTYPES["bf16"], None) == o.OPTCC_EINVAL
    assert "overlap" in o.optcc_last_error()
    # lengths whose byte ranges would wrap around the address space
    assert L.optcc_narrow_f32(0x1000, 0x100000, 1 << 62, o.DTYPES["bf16"], None) == o.OPTCC_EINVAL
    assert "address space" in o.optcc_last_error()
    assert L.optcc_narrow_f32(0x1000, 0x100000, (1 << 63) - 1, o.DTYPES["f16"], None) == o.OPTCC_EINVAL


@pytest.mark.parametrize("p,slow", PROFILES)
def test_flow_stages_follow_the_stage_definitions(o, p, slow):
    """Every exported flow names the paper's stage it belongs to (Sec. 4.1:
    S1 and S4 run between healthy ranks, S2 ends at a straggler, S3 starts
    at one; bubble filling rides on S2 and S3, App. C), and `hop` counts the
    steps of a section within its slot: the S1 chain and the S4 allgather
    have P' - 1 hops each."""
    bw = _bw(p, slow)
    pl = o.optcc_plan(p, bw, 64 * 97 + 5, 8)
    strag = set(int(r) for r in pl.stragglers)
    fl = pl.flows()
    assert set(np.unique(fl["stage"])) <= {1, 2, 3, 4}
    for f in fl:
        st, src, dst = int(f["stage"]), int(f["src"]), int(f["dst"])
        if st in (1, 4):
            assert src not in strag and dst not in strag
            assert int(f["op"]) == (1 if st == 1 else 0)
        elif st == 2:
            assert dst in strag and src not in strag
        else:
            assert src in strag and dst not in strag
    ring = fl[(fl["section"] >= 0) & np.isin(fl["stage"], [1, 4])]
    for slot in (1, 4):
        hops = ring["hop"][ring["slot"] == slot]
        if hops.size:
            assert hops.min() == 0 and hops.max() == pl.healthy - 2
            assert np.bincount(hops).tolist() == [hops.size // (pl.healthy - 1)] * (pl.healthy - 1)


@pytest.mark.parametrize("q,g,sb", [(3, 2, {1: 0.5}), (4, 4, {0: 0.5}), (5, 3, {4: 0.875})])
def test_server_flow_stages(o, q, g, sb):
    """App. E: NVLink phases N1-N4 run between GPUs of one server, NIC stages
    S1-S4 between servers; S2 ends on the straggler server, S3 leaves it."""
    bw = [1.0] * q
    for s, v in sb.items():
        bw[s] = v
    pl = o.optcc_plan_servers(q, g, bw, 64 * 24 * 7 + 3, 24)
    sv = int(pl.stragglers[0])
    fl = pl.flows()
    assert set(np.unique(fl["stage"])) == set(range(1, 9))
    for f in fl:
        st, a, b = int(f["stage"]), int(f["src"]) // g, int(f["dst"]) // g
        if st >= 5:
            assert a == b
        else:
            assert a != b
            assert (b == sv) == (st == 2) and (a == sv) == (st == 3)


def test_segment_quanta_beyond_32_bits_refused(o):
    """The device tables index a segment's ring quanta in 32 bits: a plan
    whose segment holds 2^31 quanta or more is refused with
    OPTCC_EUNSUPPORTED before any device call (the pointers are never
    dereferenced).  Only refused cases are run here: an accepted one would
    go on to the device."""
    L = o.lib()
    for p, bw, k, nq in [(3, [1.0] * 3, 4, 4 * 2**31), (5, [1.0] * 4 + [0.5], 8, 8 * (2**31 + 5)),
                         (3, [1.0] * 3, 4, 4 * 2**31 + 3)]:
        n = 64 * nq
        pl = o.optcc_plan(p, bw, n, k)
        ptrs = (ctypes.c_void_p * p)(*[(r + 1) << 45 for r in range(p)])
        rc = L.optcc_allreduce_emulate(ptrs, p, n, 2, pl.handle, None)
        assert rc == o.OPTCC_EUNSUPPORTED and "quanta" in o.optcc_last_error()


def test_noalloc_refuses_tables_beyond_its_scratch(o):
    """optcc_allreduce_emulate_noalloc stages the plan's tables in a static
    array of OPTCC_NOALLOC_SCRATCH_BYTES: a plan whose tables need more is
    refused with OPTCC_EUNSUPPORTED before any device call (the pointers are
    never dereferenced)."""
    L = o.lib()
    n = 1 << 30  # p = 3 fp32 takes 4096-element tiles: 2^18 tiles of 16 bytes = 4 MiB
    pl = o.optcc_plan(3, [1.0] * 3, n, 4)
    ptrs = (ctypes.c_void_p * 3)(*[(r + 1) << 40 for r in range(3)])
    rc = L.optcc_allreduce_emulate_noalloc(ptrs, 3, n, 0, pl.handle, None)
    assert rc == o.OPTCC_EUNSUPPORTED
    assert "scratch" in o.optcc_last_error()
    # the argument checks of optcc_allreduce_emulate apply as well
    assert L.optcc_allreduce_emulate_noalloc(ptrs, 4, n, 0, pl.handle, None) == o.OPTCC_EINVAL
