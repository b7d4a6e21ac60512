"""GPU parity: the HIP executor against the oracle, through the C ABI.

Every case compares every element of every rank bit for bit with the
oracle's serial execution (fp32, bf16 and int32 alike: the schedule fixes the
reduction order; fp16 likewise), from small ragged cases to the full-size workloads.  Slot
prefixes check that every step is materialised in its destination buffer,
stage by stage.  Full-size runs also check properties that hold at any size
(all ranks identical, exact int32 sums, the fp error bound) and sampled
coordinates through the oracle's per-coordinate executor.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from gpu_util import bits_equal, int_view, rand_inputs, to_device, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def o():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_01680_amd import optcc
    return optcc


def _bw(p, slow):
    b = [1.0] * p
    for r, v in slow.items():
        b[r] = v
    return b


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


PROFILES = [
    (3, {}), (3, {2: 0.5}), (4, {3: 0.5}), (5, {0: 0.5}), (5, {2: 0.75}), (8, {7: 0.875}),
    (8, {3: 0.25}), (6, {0: 0.5, 5: 0.75}), (9, {0: 0.875, 3: 0.75, 8: 0.5}), (16, {15: 0.5}),
    (12, {}), (20, {1: 0.5, 2: 0.5, 19: 0.9}), (40, {5: 0.6}),
    # degenerate profiles: two healthy ranks, slowdown barely above 1, just
    # under and exactly at l = 2
    (4, {0: 0.5, 1: 0.75}), (5, {1: 0.5, 2: 0.5, 3: 0.5}), (8, {2: 0.9999999}),
    (6, {5: 0.50000001}), (6, {5: 0.5}),
]
# sizes span several tiles (at these sizes 1024 elements for 4-byte types,
# 2048 for 2-byte types), ragged tails, empty sections
SIZES = [(1, 4), (37, 4), (64, 4), (1000, 8), (2048 * 3 + 64 * 5 + 3, 8), (40000, 12)]


def _run_both(o, p, slow, n, k, dtype, seed, kind="normal", slot_end=6, launches=1):
    bw = _bw(p, slow)
    x = rand_inputs(dtype, p, n, seed, kind)
    ref = oracle.run(oracle.Schedule(p, bw, n, k), dtype, x.copy(), 0, slot_end)
    pl = o.optcc_plan(p, bw, n, k)
    d = to_device(x, dtype)
    o.optcc_allreduce_emulate_slots(d, p, n, dtype, pl, 0, slot_end, launches)
    torch.cuda.synchronize()
    return x, ref, to_host(d, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32", "f16"])
@pytest.mark.parametrize("p,slow", PROFILES)
@pytest.mark.parametrize("n,k", SIZES)
def test_small_bit_exact(o, dtype, p, slow, n, k):
    _say(f"case dtype={dtype} p={p} slow={slow} n={n} k={k}")
    x, ref, got = _run_both(o, p, slow, n, k, dtype, seed=p * 1000 + n)
    assert bits_equal(got, ref)
    if n:
        assert (got == got[0][None, :]).all()


@pytest.mark.parametrize("dtype,p,slow,n,k", [
    # 2048-element tiles (two vectors per lane) with a sub-vector tail, and
    # just below the size where they start (1024-element tiles)
    ("f32", 8, {7: 0.875}, (1 << 21) + 2048 * 3 + 64 * 5 + 3, 64),
    ("i32", 8, {7: 0.875}, (1 << 21) + 2048 * 3 + 64 * 5 + 3, 64),
    ("f32", 8, {7: 0.875}, (1 << 21) - 64 * 3 + 1, 64),
    # 4096-element tiles (fp32 p = 4; fp16 p = 6) and 8192 (bf16 p = 3)
    ("f32", 4, {3: 0.5}, (1 << 22) + 5, 8),
    ("f16", 6, {5: 0.5}, (1 << 22) + 2048 + 9, 16),
    ("bf16", 3, {2: 0.5}, (1 << 23) + 77, 8),
])
def test_tile_lengths_bit_exact(o, dtype, p, slow, n, k):
    """Every tile length the launch picks (1024 to 8192 elements: longer for
    plans that move little per element, shorter for small messages), each
    with ragged tiles at segment ends, bit for bit against the oracle."""
    _say(f"case tiles dtype={dtype} p={p} slow={slow} n={n} k={k}")
    x, ref, got = _run_both(o, p, slow, n, k, dtype, seed=5 * p + n % 97)
    assert bits_equal(got, ref)


@pytest.mark.parametrize("dtype", ["f32", "i32"])
@pytest.mark.parametrize("p,slow,n,k", [
    (8, {7: 0.875}, (1 << 20) + 12345, 64),   # 5 to 7 healthy: 1024-element tiles
    (6, {0: 0.5}, (1 << 21) + 77, 16),
    (7, {}, (1 << 20) + 3, 8),                  # no straggler: the ring
    (4, {3: 0.5}, (1 << 22) + 999, 8),          # 3 healthy: the plan's own tile length
    (9, {0: 0.875, 3: 0.75, 8: 0.5}, (1 << 20) + 64 * 5 + 1, 12),
])
def test_mid_size_short_chains_bit_exact(o, dtype, p, slow, n, k):
    """Short chains of 32-bit elements whose rank buffers total 16 MiB to
    2 GiB run one vector per lane in the identity tile order: every element
    of every rank bit for bit against the oracle, ragged tails included."""
    _say(f"case mid-size short chain dtype={dtype} p={p} slow={slow} n={n} k={k}")
    x, ref, got = _run_both(o, p, slow, n, k, dtype, seed=61 + p)
    assert bits_equal(got, ref)


@pytest.mark.parametrize("p,n", [(40, 1 << 17), (64, 1 << 18), (64, (1 << 19) + 4097),
                                 # 62 healthy ranks keep the runs up to 4,096 tiles
                                 (64, 1024 * 4000 + 3)])
def test_long_chains_one_round_of_tiles(o, p, n):
    """Long chains whose tiles fit in one round of resident workgroups take
    the identity tile order, more tiles the per-XCD runs: both bit for bit."""
    slow = {p - 1: 0.5, p - 2: 0.75}
    _say(f"case long chain p={p} n={n}")
    x, ref, got = _run_both(o, p, slow, n, 16, "f32", seed=7 + p)
    assert bits_equal(got, ref)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32", "f16"])
@pytest.mark.parametrize("p,slow", [(5, {0: 0.5}), (8, {7: 0.875}), (9, {0: 0.875, 3: 0.75, 8: 0.5}),
                                    (7, {}), (6, {1: 0.25, 2: 0.5})])
@pytest.mark.parametrize("launches", [1, 0])
def test_stage_snapshots(o, dtype, p, slow, launches):
    """After the first s slots (s = 1..6), in one fused launch or one launch
    per slot, every buffer equals the oracle's state after the same slots:
    every step's destination write is materialised."""
    n, k = 2048 * 2 + 64 * 7 + 5, 8
    for s in range(1, 7):
        _say(f"case snapshot dtype={dtype} p={p} slots=[0,{s}) launches={launches}")
        x, ref, got = _run_both(o, p, slow, n, k, dtype, seed=17 + s, slot_end=s, launches=launches)
        assert bits_equal(got, ref), f"slots [0,{s})"


@pytest.mark.parametrize("dtype,kind", [(d, k) for d in ("f32", "bf16", "f16")
                                         for k in ("denormal", "wide")] + [("f16", "overflow")])
def test_special_values(o, dtype, kind):
    """Subnormal inputs (no flush to zero on either side), values spread over
    the format's binades (heavy cancellation) and, for fp16, partial sums
    beyond the largest finite half (rounded to infinity on both sides) stay
    bit-exact."""
    for p, slow in [(5, {0: 0.5}), (8, {7: 0.875}), (9, {0: 0.875, 3: 0.75, 8: 0.5})]:
        _say(f"case special {kind} dtype={dtype} p={p}")
        x, ref, got = _run_both(o, p, slow, 5000, 8, dtype, seed=3, kind=kind)
        assert bits_equal(got, ref)
        if kind == "overflow":
            assert np.isinf(oracle.f16_to_f64(got)).any()


@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32", "f16"])
def test_unaligned_buffers(o, dtype):
    """Rank buffers that are only element-aligned take the one-element path."""
    p, n, k = 8, 3000, 8
    bw = _bw(p, {7: 0.875})
    x = rand_inputs(dtype, p, n, 5)
    ref = oracle.run(oracle.Schedule(p, bw, n, k), dtype, x.copy())
    pl = o.optcc_plan(p, bw, n, k)
    stride = n + 1  # rank r starts at 1 + r*(n+1) elements: not 16-byte aligned
    flat = torch.zeros(p * stride + 8, dtype=to_device(x[:1, :1], dtype).dtype, device="cuda:0")
    for r in range(p):
        flat[1 + r * stride: 1 + r * stride + n].copy_(to_device(x[r:r + 1], dtype)[0])
    views = [flat[1 + r * stride: 1 + r * stride + n] for r in range(p)]
    _say(f"case unaligned dtype={dtype}")
    o.optcc_allreduce_emulate(views, p, n, dtype, pl)
    torch.cuda.synchronize()
    got = np.stack([to_host(v, dtype) for v in views])
    assert bits_equal(got, ref)


def test_deterministic_and_stream(o):
    """Same inputs, same bits, on the default stream and a side stream."""
    p, n, k = 9, 50000, 8
    bw = _bw(p, {0: 0.875, 3: 0.75, 8: 0.5})
    x = rand_inputs("f32", p, n, 9)
    pl = o.optcc_plan(p, bw, n, k)
    a = to_device(x, "f32")
    b = to_device(x, "f32")
    o.optcc_allreduce_emulate(a, p, n, "f32", pl)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        o.optcc_allreduce_emulate(b, p, n, "f32", pl, stream=s)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


# ----------------------------------------------------------- full workloads
def _sample_coords(plan, n, rng, count=4096):
    """Random coordinates plus every segment's first and last element, both
    sides of each P2P chunk boundary and the vector's ends."""
    off, ln, p2p = plan.segments()
    picks = set(rng.integers(0, n, size=count).tolist())
    for g in range(len(off)):
        b, e = int(off[g]), int(off[g] + ln[g])
        for c in (b, e - 1, e - int(p2p[g]), e - int(p2p[g]) - 1):
            if 0 <= c < n:
                picks.add(c)
    picks.update([0, n - 1])
    return np.array(sorted(picks), dtype=np.int64)


WORKLOADS = ["p4_f32", "p8_f32", "p8_i32", "p16_bf16", "p16_f16", "p64_f32", "p128_f32"]
UNIT = {"f32": 2.0 ** -24, "f16": 2.0 ** -11, "bf16": 2.0 ** -8}  # unit roundoff


@pytest.mark.parametrize("name", WORKLOADS)
def test_workload_full_size(o, name):
    from paper_2606_01680_amd.workloads import WORKLOADS as W, make_inputs
    w = W[name]
    _say(f"case workload {name} p={w.p} N={w.n} dtype={w.dtype} k={w.k}")
    x = make_inputs(w, device="cuda:0")
    x0 = x.clone()
    pl = o.optcc_plan(w.p, w.bandwidths, w.n, w.k)
    o.optcc_allreduce_emulate(x, w.p, w.n, w.dtype, pl)
    torch.cuda.synchronize()
    iv = int_view(x)
    for r in range(1, w.p):  # every rank holds the same bits
        assert torch.equal(iv[r], iv[0]), r
    rng = np.random.default_rng(1234)
    coords = _sample_coords(pl, w.n, rng)
    idx = torch.from_numpy(coords).to("cuda:0")
    cols = to_host(x0[:, idx], w.dtype).copy()
    sched = oracle.Schedule(w.p, w.bandwidths, w.n, w.k)
    oracle.run_sampled(sched, w.dtype, cols, coords)
    got = to_host(x[:, idx], w.dtype)
    assert bits_equal(got, cols)
    # properties over every coordinate, chunked
    step = max(1 << 16, (1 << 28) // w.p)
    for c0 in range(0, w.n, step):
        c1 = min(w.n, c0 + step)
        if w.dtype == "i32":
            want = x0[:, c0:c1].to(torch.int64).sum(0)
            want = ((want + 2**31) % 2**32 - 2**31).to(torch.int32)
            assert torch.equal(x[0, c0:c1], want)
        else:
            xs = x0[:, c0:c1].to(torch.float64)
            err = (x[0, c0:c1].to(torch.float64) - xs.sum(0)).abs()
            assert bool((err <= w.p * UNIT[w.dtype] * xs.abs().sum(0)).all())
    # and every element of every rank against the oracle's full serial run
    _say(f"case workload {name}: full oracle run")
    full = oracle.run(sched, w.dtype, to_host(x0, w.dtype).copy())
    del x0
    got_all = to_host(x, w.dtype)
    assert bits_equal(got_all, full)


@pytest.mark.parametrize("dtype", ["i32", "f32"])
def test_replanning_between_calls(o, dtype):
    """Re-planning online (Sec. 4.3, schedule generation: closed-form rules,
    cheap enough to run when a failure is detected): a sequence of NIC-loss
    profiles on p=8 (PXN pooling: losing c of 8 NICs leaves bandwidth
    (8-c)/8, Sec. 2), one fresh plan per call on the same buffers, each
    result bit-exact against the oracle."""
    p, n, k = 8, 300000, 16
    seq = [{}, {3: 7 / 8}, {3: 6 / 8, 6: 7 / 8}, {3: 4 / 8}, {3: 2 / 8, 5: 4 / 8, 6: 6 / 8},
           {0: 7 / 8, 1: 7 / 8, 2: 7 / 8, 4: 7 / 8}, {}]
    x = rand_inputs(dtype, p, n, 77)
    d = to_device(x, dtype)
    d0 = d.clone()
    prev = None
    for slow in seq:
        bw = _bw(p, slow)
        _say(f"case replan dtype={dtype} slow={slow}")
        pl = o.optcc_plan(p, bw, n, k)
        d.copy_(d0)
        o.optcc_allreduce_emulate(d, p, n, dtype, pl)
        torch.cuda.synchronize()
        ref = oracle.run(oracle.Schedule(p, bw, n, k), dtype, x.copy())
        assert bits_equal(to_host(d, dtype), ref)
        if prev is not None:
            o.optcc_plan_free(prev)  # the previous plan's device tables go with it
        prev = pl


def test_largest_rank_count(o):
    """p = OPTCC_MAX_EMULATE_RANKS (256): every rank pointer in the kernel
    arguments; one past the limit is rejected before any launch."""
    p, n, k = o.OPTCC_MAX_EMULATE_RANKS, 20000, 8
    for dtype in ("i32", "f32"):
        _say(f"case p=256 dtype={dtype}")
        x, ref, got = _run_both(o, p, {0: 0.5, 100: 0.875, 255: 0.75}, n, k, dtype, seed=256)
        assert bits_equal(got, ref)
    big = o.optcc_plan(p + 1, [1.0] * (p + 1), 128, 4)
    d = torch.zeros((p + 1, 128), dtype=torch.float32, device="cuda:0")
    with pytest.raises(o.OptccError) as e:
        o.optcc_allreduce_emulate(d, p + 1, 128, "f32", big)
    assert e.value.status == o.OPTCC_EUNSUPPORTED


def test_empty_vector(o):
    """N = 0: a valid plan with empty segments; emulation is a no-op."""
    pl = o.optcc_plan(5, [1, 1, 0.5, 1, 1], 0, 8)
    d = torch.zeros((5, 0), dtype=torch.float32, device="cuda:0")
    o.optcc_allreduce_emulate(d, 5, 0, "f32", pl)
    torch.cuda.synchronize()


def test_first_call_inside_capture_is_refused(o):
    """A plan's first call on a device uploads its tables, so it cannot be
    captured: made during a capture it raises OPTCC_EINVAL before touching
    the device, the capture stays valid (the work around it replays), the
    buffers are untouched, and an eager call afterwards gives the oracle's
    result bit for bit."""
    p, n, k = 8, 50000, 8
    bw = _bw(p, {7: 0.875})
    dtype = "f32"
    x = rand_inputs(dtype, p, n, 41)
    ref = oracle.run(oracle.Schedule(p, bw, n, k), dtype, x.copy())
    pl = o.optcc_plan(p, bw, n, k)
    d = to_device(x, dtype)
    d0 = d.clone()
    side = torch.zeros(64, device="cuda:0")
    torch.cuda.synchronize()
    _say("case first call inside a capture")
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            side.add_(1.0)
            with pytest.raises(o.OptccError) as e:
                o.optcc_allreduce_emulate(d, p, n, dtype, pl)
            side.add_(2.0)
    assert e.value.status == o.OPTCC_EINVAL
    assert "captured" in str(e.value)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    assert (side == 3.0).all()
    assert torch.equal(int_view(d), int_view(d0))
    del g
    o.optcc_allreduce_emulate(d, p, n, dtype, pl)
    torch.cuda.synchronize()
    assert bits_equal(to_host(d, dtype), ref)


def test_graph_capture_replays(o):
    """After its first call on a device (which uploads the plan tables) an
    AllReduce is one kernel launch, so it can be captured in a HIP graph.
    Each replay, with eager restores and synchronisations in between, equals
    the eager result bit for bit."""
    p, n, k = 8, 200000, 16
    bw = _bw(p, {7: 0.875})
    pl = o.optcc_plan(p, bw, n, k)
    for dtype in ("f32", "bf16", "i32", "f16"):
        x = rand_inputs(dtype, p, n, 31)
        d = to_device(x, dtype)
        d0 = d.clone()
        o.optcc_allreduce_emulate(d, p, n, dtype, pl)  # first use: table upload
        torch.cuda.synchronize()
        eager = d.clone()
        ref = oracle.run(oracle.Schedule(p, bw, n, k), dtype, x.copy())
        assert bits_equal(to_host(eager, dtype), ref)
        g = torch.cuda.CUDAGraph()
        d.copy_(d0)
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            with torch.cuda.graph(g, stream=s):
                o.optcc_allreduce_emulate(d, p, n, dtype, pl)
        torch.cuda.synchronize()
        for rep in range(4):
            _say(f"case graph replay dtype={dtype} rep={rep}")
            d.copy_(d0)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(int_view(d), int_view(eager))
        del g


def test_captured_plan_outlives_its_python_reference(o):
    """A plan whose call was captured into a graph stays alive when the
    caller drops it (its device tables are still in the graph): replays
    after garbage collection give the eager result; freeing it explicitly is
    refused until release_captured_plans()."""
    import gc
    p, n, k = 8, 100000, 8
    bw = _bw(p, {7: 0.875})
    dtype = "f32"
    x = rand_inputs(dtype, p, n, 47)
    ref = oracle.run(oracle.Schedule(p, bw, n, k), dtype, x.copy())
    d = to_device(x, dtype)
    d0 = d.clone()
    pl = o.optcc_plan(p, bw, n, k)
    o.optcc_allreduce_emulate(d, p, n, dtype, pl)  # first use: table upload
    torch.cuda.synchronize()
    assert bits_equal(to_host(d, dtype), ref)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            o.optcc_allreduce_emulate(d, p, n, dtype, pl)
    torch.cuda.synchronize()
    with pytest.raises(RuntimeError):
        o.optcc_plan_free(pl)
    del pl
    gc.collect()
    for rep in range(3):
        _say(f"case captured plan after its reference is dropped rep={rep}")
        d.copy_(d0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert bits_equal(to_host(d, dtype), ref)
    del g
    torch.cuda.synchronize()
    o.release_captured_plans()
    gc.collect()


def test_every_small_length(o):
    """Every length from 0 to 200 and around each tile and quantum boundary up
    to three tiles, for one straggler (bubble filling), several stragglers
    and a server plan: bit for bit against the oracle."""
    lengths = sorted(set(range(0, 201)) | {b + d for b in (1984, 2048, 4096, 6144)
                                           for d in (-65, -64, -63, -1, 0, 1, 63, 64, 65)})
    profiles = [("one", 8, {7: 0.875}, None), ("multi", 9, {0: 0.875, 3: 0.75, 8: 0.5}, None),
                ("servers", 6, None, (3, 2, [1.0, 1.0, 0.5]))]
    for name, p, slow, srv in profiles:
        _say(f"case every small length {name}")
        for n in lengths:
            x = rand_inputs("i32", p, n, 7 + n)
            if srv is None:
                bw = _bw(p, slow)
                pl, sched = o.optcc_plan(p, bw, n, 8), oracle.Schedule(p, bw, n, 8)
            else:
                q, g, sbw = srv
                pl = o.optcc_plan_servers(q, g, sbw, n, 24)
                sched = oracle.Schedule.servers(q, g, sbw, n, 24)
            ref = oracle.run(sched, "i32", x.copy())
            d = to_device(x, "i32")
            o.optcc_allreduce_emulate(d, p, n, "i32", pl)
            torch.cuda.synchronize()
            assert bits_equal(to_host(d, "i32"), ref), (name, n)


def test_more_than_2g_elements_per_rank(o):
    """N = 2^31 + 4099 elements per rank (three ranks, 25.8 GB): element
    offsets beyond 32 bits.  All ranks identical, the exact wrapped int32
    sum everywhere, and sampled coordinates (segment and section ends, the
    last elements) bit for bit against the oracle."""
    p, n, k = 3, (1 << 31) + 4099, 4
    bw = [1.0, 1.0, 0.5]
    _say(f"case p=3 N={n} i32")
    g = torch.Generator(device="cuda:0")
    g.manual_seed(2606)
    x0 = torch.randint(-(1 << 30), 1 << 30, (p, n), generator=g, device="cuda:0", dtype=torch.int32)
    x = x0.clone()
    pl = o.optcc_plan(p, bw, n, k)
    o.optcc_allreduce_emulate(x, p, n, "i32", pl)
    torch.cuda.synchronize()
    for r in range(1, p):
        assert torch.equal(x[r], x[0]), r
    step = 1 << 28
    for c0 in range(0, n, step):
        c1 = min(n, c0 + step)
        want = x0[:, c0:c1].to(torch.int64).sum(0)
        want = ((want + 2**31) % 2**32 - 2**31).to(torch.int32)
        assert torch.equal(x[0, c0:c1], want), c0
    rng = np.random.default_rng(31)
    coords = _sample_coords(pl, n, rng, count=2048)
    coords = np.unique(np.concatenate([coords, np.arange(n - 300, n)]))
    idx = torch.from_numpy(coords).to("cuda:0")
    cols = to_host(x0[:, idx], "i32").copy()
    oracle.run_sampled(oracle.Schedule(p, bw, n, k), "i32", cols, coords)
    assert bits_equal(to_host(x[:, idx], "i32"), cols)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32", "f16"])
def test_fused_ranges_from_the_middle(o, dtype):
    """Any slot range [a, b), fused into one launch and started from the
    state after [0, a) (computed by the oracle), ends in the oracle's state
    after [0, b): the executor's lanes pick up mid-way state from memory
    exactly where the earlier slots left it.  One straggler with bubble
    filling, several stragglers, no straggler, and two server plans (with
    the local ring fixed at compile time, g = 2, and general, g = 3)."""
    n = 2048 * 2 + 64 * 7 + 5
    cases = [("one", 8, _bw(8, {7: 0.875}), None, 8, 6),
             ("multi", 9, _bw(9, {0: 0.875, 3: 0.75, 8: 0.5}), None, 8, 6),
             ("ring", 5, _bw(5, {}), None, 8, 6),
             ("servers g=2", 8, [1.0, 0.5, 1.0, 1.0], (4, 2), 24, 12),
             ("servers g=3", 9, [1.0, 1.0, 0.75], (3, 3), 24, 12)]
    for name, p, bw, srv, k, ns in cases:
        if srv is None:
            pl, sched = o.optcc_plan(p, bw, n, k), oracle.Schedule(p, bw, n, k)
        else:
            pl = o.optcc_plan_servers(srv[0], srv[1], bw, n, k)
            sched = oracle.Schedule.servers(srv[0], srv[1], bw, n, k)
        x = rand_inputs(dtype, p, n, 23 + p)
        for a in range(1, ns):
            start = oracle.run(sched, dtype, x.copy(), 0, a)
            for b in range(a + 1, ns + 1):
                _say(f"case fused range {name} dtype={dtype} [{a},{b})")
                want = oracle.run(sched, dtype, start.copy(), a, b)
                d = to_device(start, dtype)
                o.optcc_allreduce_emulate_slots(d, p, n, dtype, pl, a, b, 1)
                torch.cuda.synchronize()
                assert bits_equal(to_host(d, dtype), want), (name, a, b)


def test_binding_rejects_mismatched_tensors(o):
    """The binding refuses tensors whose element size or length disagrees
    with dtype and N before any pointer reaches the library: the library
    reads and writes N elements of dtype at every rank address and cannot
    see allocation sizes."""
    p, n, k = 5, 1000, 8
    pl = o.optcc_plan(p, [1, 1, 0.5, 1, 1], n, k)
    bf = torch.zeros((p, n), dtype=torch.bfloat16, device="cuda:0")
    with pytest.raises(ValueError, match="element"):
        o.optcc_allreduce_emulate(bf, p, n, "f32", pl)
    with pytest.raises(ValueError, match="element"):
        o.optcc_allreduce_emulate([bf[r] for r in range(p)], p, n, "i32", pl)
    short = [torch.zeros(n - 1, device="cuda:0") for _ in range(p)]
    with pytest.raises(ValueError, match="elements per rank"):
        o.optcc_allreduce_emulate(short, p, n, "f32", pl)
    with pytest.raises(ValueError, match="dtype"):
        o.optcc_allreduce_emulate(torch.zeros((p, n), device="cuda:0"), p, n, "f64", pl)
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_narrowing_every_fp32_pattern(o, dtype):
    """The executor's per-step rounding of an fp32 sum to bf16 / fp16 (round
    to nearest even; fp16 subnormals and overflow to infinity), through the
    library's optcc_narrow_f32, equals the oracle's C rule on all 2^32 fp32
    bit patterns.  NaN inputs: bf16 bit for bit (both sides keep the top
    payload bits and quieten), fp16 NaN for NaN (IEEE 754 leaves the payload
    of a narrowed NaN open)."""
    chunk = 1 << 27
    round_ref = oracle.bf16_round if dtype == "bf16" else oracle.f16_round
    out = torch.empty(chunk, dtype=torch.int16, device="cuda:0")
    for c in range((1 << 32) // chunk):
        if c % 8 == 0:
            _say(f"case narrow {dtype} patterns from {c * chunk:#x}")
        bits = np.arange(c * chunk, (c + 1) * chunk, dtype=np.int64).astype(np.uint32)
        x = bits.view(np.float32)
        want = round_ref(x)
        d = torch.from_numpy(x).to("cuda:0")
        o.optcc_narrow_f32(d, out, dtype)
        torch.cuda.synchronize()
        got = out.cpu().numpy().view(np.uint16)
        nan_in = (bits & 0x7fffffff) > 0x7f800000
        if dtype == "bf16":
            assert np.array_equal(got, want), c
        else:
            assert np.array_equal(got[~nan_in], want[~nan_in]), c
            g = got[nan_in]
            assert bool((((g & 0x7c00) == 0x7c00) & ((g & 0x3ff) != 0)).all()), c
    # odd lengths: the last element goes through the single-value form
    bits = np.array([0x7fa00001, 0xffc12345, 0x3f808000, 0x3f818000, 0x00000001,
                     0x7f7fffff, 0xc0490fdb], dtype=np.uint32)
    for n in (1, 3, 7):
        x = bits[:n].view(np.float32)
        want = round_ref(x)
        d = torch.from_numpy(x.copy()).to("cuda:0")
        o.optcc_narrow_f32(d, out[:n], dtype)
        torch.cuda.synchronize()
        got = out[:n].cpu().numpy().view(np.uint16)
        nan_in = (bits[:n] & 0x7fffffff) > 0x7f800000
        if dtype == "bf16":
            assert np.array_equal(got, want), n
        else:
            assert np.array_equal(got[~nan_in], want[~nan_in]), n


def test_threads_share_one_plan(o):
    """A plan is shared read-only across host threads and streams: four
    threads call a fresh plan at once (its device tables are uploaded on
    first use under the plan's lock), each on its own stream and buffers,
    and every result is bit-exact against the oracle."""
    import threading
    p, n, k = 9, 70000, 8
    bw = _bw(p, {0: 0.875, 3: 0.75, 8: 0.5})
    pl = o.optcc_plan(p, bw, n, k)
    dts = ["f32", "bf16", "i32", "f16"]
    xs = {dt: rand_inputs(dt, p, n, 300 + i) for i, dt in enumerate(dts)}
    devs = {dt: to_device(xs[dt], dt) for dt in dts}
    streams = {dt: torch.cuda.Stream() for dt in dts}
    torch.cuda.synchronize()
    errors = []
    start = threading.Barrier(len(dts))

    def work(dt):
        try:
            start.wait()
            for it in range(3):  # repeated calls reuse the uploaded tables
                with torch.cuda.stream(streams[dt]):
                    d = devs[dt]
                    o.optcc_allreduce_emulate(d, p, n, dt, pl, stream=streams[dt])
                    streams[dt].synchronize()
                    if it == 0:
                        first = d.clone()
                    d.copy_(to_device(xs[dt], dt))
                    streams[dt].synchronize()
            devs[dt] = first
        except Exception as e:  # reported by the main thread
            errors.append((dt, e))

    _say("case threads sharing one plan")
    ts = [threading.Thread(target=work, args=(dt,)) for dt in dts]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    sched = oracle.Schedule(p, bw, n, k)
    for dt in dts:
        ref = oracle.run(sched, dt, xs[dt].copy())
        assert bits_equal(to_host(devs[dt], dt), ref), dt


# Long chains (more than 32 healthy ranks, one workgroup per CU, tiles of
# one vector per lane) whose tiles outnumber the per-XCD-run limit (2,048;
# 4,096 below 90 healthy ranks) run as a persistent grid that takes tiles
# from a device counter (work stealing), every element type.  Sizes above
# the limit, ragged, two just above it.
STEAL = [(40, {5: 0.6}, 2048 * 2100 + 77, 8), (70, {3: 0.875}, 2048 * 2200 + 130, 16),
         (36, {}, 2048 * 2300 + 3, 4), (100, {7: 0.5, 60: 0.75}, 1024 * 2049 + 5, 8),
         (64, {63: 0.5, 62: 0.75}, 1024 * 4100 + 5, 16),
         # 98 healthy ranks, 2,101 tiles of 2048 2-byte elements: bf16 and fp16 steal too
         (100, {7: 0.5, 60: 0.75}, 2048 * 2100 + 9, 8)]


@pytest.mark.parametrize("p,slow,n,k", STEAL)
def test_work_stealing_launches(o, p, slow, n, k):
    """Three calls in a row of a work-stealing plan (the counters reset
    themselves at the end of each launch), fp32, int32, fp16 and bf16: the
    first result equals the oracle on every element, the others equal the
    first."""
    bw = _bw(p, slow)
    pl = o.optcc_plan(p, bw, n, k)
    sched = oracle.Schedule(p, bw, n, k)
    for dtype in ("f32", "i32", "f16", "bf16"):
        _say(f"case work stealing p={p} n={n} k={k} dtype={dtype}")
        x = rand_inputs(dtype, p, n, 90 + p)
        d = to_device(x, dtype)
        d0 = d.clone()
        first = None
        for rep in range(3):
            d.copy_(d0)
            o.optcc_allreduce_emulate(d, p, n, dtype, pl)
            torch.cuda.synchronize()
            if first is None:
                first = d.clone()
            else:
                assert torch.equal(int_view(d), int_view(first)), rep
        del d, d0
        ref = oracle.run(sched, dtype, x)
        assert bits_equal(to_host(first, dtype), ref), dtype
        del first
        torch.cuda.empty_cache()


def test_work_stealing_equals_static_order(o):
    """Work stealing changes only which workgroup runs which tile: the same
    AllReduce through the no-allocation entry point and inside a captured
    HIP graph (both keep the static tile order) gives the same bits."""
    p, n, k = 40, 2048 * 2100 + 77, 8
    bw = _bw(p, {5: 0.6})
    pl = o.optcc_plan(p, bw, n, k)
    x = rand_inputs("f32", p, n, 4242)
    d0 = to_device(x, "f32")
    d = d0.clone()
    o.optcc_allreduce_emulate(d, p, n, "f32", pl)
    torch.cuda.synchronize()
    steal = d.clone()
    d.copy_(d0)
    o.optcc_allreduce_emulate_noalloc(d, p, n, "f32", pl)
    torch.cuda.synchronize()
    assert torch.equal(int_view(d), int_view(steal))
    g = torch.cuda.CUDAGraph()
    d.copy_(d0)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            o.optcc_allreduce_emulate(d, p, n, "f32", pl)
    torch.cuda.synchronize()
    for rep in range(3):
        _say(f"case work stealing against a captured graph, replay {rep}")
        d.copy_(d0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(int_view(d), int_view(steal)), rep
    del g


def test_work_stealing_slot_ranges(o):
    """A work-stealing plan run as two slot ranges in a row, and as one
    launch per slot (each launch takes the same counter block after the one
    before has set it back to zero), equals the fused call bit for bit, and
    the oracle's stage prefix after the first range."""
    p, n, k = 40, 2048 * 2100 + 77, 8
    bw = _bw(p, {5: 0.6})
    pl = o.optcc_plan(p, bw, n, k)
    x = rand_inputs("f32", p, n, 777)
    d0 = to_device(x, "f32")
    d = d0.clone()
    o.optcc_allreduce_emulate(d, p, n, "f32", pl)
    torch.cuda.synchronize()
    fused = d.clone()
    d.copy_(d0)
    o.optcc_allreduce_emulate_slots(d, p, n, "f32", pl, 0, 2, 1)
    torch.cuda.synchronize()
    ref = oracle.run(oracle.Schedule(p, bw, n, k), "f32", x.copy(), 0, 2)
    assert bits_equal(to_host(d, "f32"), ref)
    o.optcc_allreduce_emulate_slots(d, p, n, "f32", pl, 2, 6, 1)
    torch.cuda.synchronize()
    assert torch.equal(int_view(d), int_view(fused))
    d.copy_(d0)
    o.optcc_allreduce_emulate_slots(d, p, n, "f32", pl, 0, 6, 0)
    torch.cuda.synchronize()
    assert torch.equal(int_view(d), int_view(fused))


def test_work_stealing_threads_share_one_plan(o):
    """Four host threads, each on its own stream and buffers, run one
    work-stealing plan at once, three times each: concurrent launches take
    different counter blocks, and every result equals the oracle."""
    import threading
    p, n, k = 40, 2048 * 2100 + 77, 8
    bw = _bw(p, {5: 0.6})
    pl = o.optcc_plan(p, bw, n, k)
    names = ["a", "b", "c", "d"]
    dts = {"a": "f32", "b": "i32", "c": "f32", "d": "f16"}
    xs = {nm: rand_inputs(dts[nm], p, n, 500 + i) for i, nm in enumerate(names)}
    devs = {nm: to_device(xs[nm], dts[nm]) for nm in names}
    orig = {nm: devs[nm].clone() for nm in names}
    streams = {nm: torch.cuda.Stream() for nm in names}
    o.optcc_allreduce_emulate(devs["a"].clone(), p, n, "f32", pl)  # tables uploaded first
    torch.cuda.synchronize()
    errors, out = [], {}
    start = threading.Barrier(len(names))

    def work(nm):
        try:
            start.wait()
            with torch.cuda.stream(streams[nm]):
                for it in range(3):
                    d = devs[nm]
                    d.copy_(orig[nm])
                    o.optcc_allreduce_emulate(d, p, n, dts[nm], pl, stream=streams[nm])
                    if it == 0:
                        out[nm] = d.clone()
                    elif not torch.equal(int_view(d), int_view(out[nm])):
                        errors.append((nm, it, "differs from the first call"))
                streams[nm].synchronize()
        except Exception as e:  # reported by the main thread
            errors.append((nm, e))

    _say("case threads sharing one work-stealing plan")
    ts = [threading.Thread(target=work, args=(nm,)) for nm in names]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    sched = oracle.Schedule(p, bw, n, k)
    for nm in names:
        ref = oracle.run(sched, dts[nm], xs[nm].copy())
        assert bits_equal(to_host(out[nm], dts[nm]), ref), nm


def _random_case(rng):
    """One random plan: ranks, stragglers and their bandwidths (NIC losses of
    eighths or any fraction), N, k, element type; a fifth are server plans."""
    dtype = ["f32", "bf16", "i32", "f16"][int(rng.integers(4))]
    n = int(np.exp(rng.uniform(0.0, np.log(300000))))
    def bandwidth():
        return float(rng.integers(1, 8)) / 8 if rng.random() < 0.5 else float(rng.uniform(0.2, 0.999))
    if rng.random() < 0.2:
        q, g = int(rng.integers(3, 13)), int(rng.integers(2, 10))
        bw = [1.0] * q
        bw[int(rng.integers(q))] = bandwidth()
        return dict(servers=(q, g), p=q * g, bw=bw, n=n, k=8 * int(rng.integers(3, 9)), dtype=dtype)
    p = int(rng.integers(3, 73))
    m = min(int(rng.choice([0, 1, 1, 1, 2, 3, 5])), p - 2)
    bw = [1.0] * p
    for r in rng.choice(p, size=m, replace=False):
        bw[int(r)] = bandwidth()
    return dict(servers=None, p=p, bw=bw, n=n, k=4 * int(rng.integers(1, 17)), dtype=dtype)


def test_random_plans_bit_exact(o):
    """200 seeded random plans of every kind, each bit for bit against the
    oracle on every element of every rank."""
    rng = np.random.default_rng(26060168)
    for i in range(200):
        c = _random_case(rng)
        _say(f"case random #{i}: {c}")
        if c["servers"] is None:
            pl = o.optcc_plan(c["p"], c["bw"], c["n"], c["k"])
            sched = oracle.Schedule(c["p"], c["bw"], c["n"], c["k"])
        else:
            q, g = c["servers"]
            pl = o.optcc_plan_servers(q, g, c["bw"], c["n"], c["k"])
            sched = oracle.Schedule.servers(q, g, c["bw"], c["n"], c["k"])
        x = rand_inputs(c["dtype"], c["p"], c["n"], 1000 + i)
        ref = oracle.run(sched, c["dtype"], x.copy())
        d = to_device(x, c["dtype"])
        o.optcc_allreduce_emulate(d, c["p"], c["n"], c["dtype"], pl)
        torch.cuda.synchronize()
        assert bits_equal(to_host(d, c["dtype"]), ref), i


def _random_rule_case(rng, i):
    """A random plan at the sizes where the launch rules change: short
    chains (3-8 healthy ranks) with 16 MiB to 512 MiB of rank buffers, where
    32-bit types run one vector per lane in pipelined tiles; long chains
    (33-200 ranks) with more tiles than one round of resident workgroups,
    where they take per-XCD tile runs; server plans of the same sizes."""
    def bandwidth():
        return float(rng.integers(1, 8)) / 8 if rng.random() < 0.5 else float(rng.uniform(0.2, 0.999))
    kind = ("short", "long", "servers")[i % 3]
    if kind == "servers":
        q, g = int(rng.integers(3, 17)), int(rng.choice([2, 4, 8]))
        bw = [1.0] * q
        bw[int(rng.integers(q))] = bandwidth()
        n = int(rng.integers(1 << 19, (1 << 28) // (q * g)))
        dtype = ["f32", "bf16", "i32"][int(rng.integers(3))]
        return dict(servers=(q, g), p=q * g, bw=bw, n=n, k=8 * int(rng.integers(3, 9)), dtype=dtype)
    if kind == "short":
        p = int(rng.integers(4, 10))
        m = min(int(rng.choice([0, 1, 1, 2])), p - 3)
        n = int(rng.integers((4 << 20) // p, (128 << 20) // p))
        dtype = ["f32", "i32", "f32", "bf16"][int(rng.integers(4))]
    else:
        p = int(rng.integers(33, 201))
        m = int(rng.choice([0, 1, 2, 3]))
        n = int(rng.integers(600_000, (1 << 28) // p))
        dtype = ["f32", "i32", "bf16"][int(rng.integers(3))]
    bw = [1.0] * p
    for r in rng.choice(p, size=m, replace=False):
        bw[int(r)] = bandwidth()
    return dict(servers=None, p=p, bw=bw, n=n, k=4 * int(rng.integers(2, 33)), dtype=dtype)


def test_random_plans_at_rule_sizes(o):
    """18 seeded random plans at mid and large sizes (up to 2^28 elements in
    all), each bit for bit against the oracle's full serial run on every
    element of every rank."""
    rng = np.random.default_rng(1680)
    for i in range(18):
        c = _random_rule_case(rng, i)
        _say(f"case rule-size random #{i}: p={c['p']} n={c['n']} k={c['k']} "
             f"dtype={c['dtype']} servers={c['servers']} bw={sorted(set(c['bw']))}")
        if c["servers"] is None:
            pl = o.optcc_plan(c["p"], c["bw"], c["n"], c["k"])
            sched = oracle.Schedule(c["p"], c["bw"], c["n"], c["k"])
        else:
            q, g = c["servers"]
            pl = o.optcc_plan_servers(q, g, c["bw"], c["n"], c["k"])
            sched = oracle.Schedule.servers(q, g, c["bw"], c["n"], c["k"])
        x = rand_inputs(c["dtype"], c["p"], c["n"], 7000 + i)
        d = to_device(x, c["dtype"])
        o.optcc_allreduce_emulate(d, c["p"], c["n"], c["dtype"], pl)
        torch.cuda.synchronize()
        got = to_host(d, c["dtype"])
        del d
        ref = oracle.run(sched, c["dtype"], x)
        assert bits_equal(got, ref), i
        del x, got, ref
        torch.cuda.empty_cache()


THREE_PER_CU_CASES = [
    # 6-7 healthy ranks at the 512 MiB edge of the three-workgroups-per-CU
    # launch: just above (three per CU), just below (four per CU), and
    # element-aligned buffers above it (four per CU, one element per access)
    ("p=8 at 0.875, fp32, 512 MiB", 8, {7: 0.875}, 1 << 24, "f32"),
    ("p=8 at 0.875, fp32, 512 MiB - 128 B", 8, {7: 0.875}, (1 << 24) - 4, "f32"),
    ("p=7 at 0.5, int32, 512 MiB + 80 B", 7, {6: 0.5}, 19173964, "i32"),
    ("p=9, two stragglers, fp32, odd N", 9, {7: 0.5, 8: 0.5}, (1 << 24) + 1, "f32"),
    # bf16 chains of 13-32 healthy ranks (three per CU at any size) and
    # just outside that range
    ("p=14 at 0.5, bf16, 13 healthy", 14, {13: 0.5}, 3 << 20, "bf16"),
    ("p=13 at 0.5, bf16, 12 healthy", 13, {12: 0.5}, 3 << 20, "bf16"),
    ("p=33 at 0.75, bf16, 32 healthy", 33, {0: 0.75}, (1 << 20) + 8, "bf16"),
    ("p=16 at 0.5, bf16, odd N", 16, {15: 0.5}, (1 << 21) + 3, "bf16"),
    # fp32/int32 chains of 11-32 healthy ranks from 1 GiB of buffers run one
    # workgroup per CU; 10 healthy ranks and smaller buffers keep two
    ("p=12 at 0.5, fp32, 11 healthy, 1 GiB", 12, {11: 0.5}, 22369624, "f32"),
    ("p=11 at 0.5, int32, 10 healthy, 1 GiB", 11, {10: 0.5}, 24403352, "i32"),
    ("p=16 at 0.875, fp32, 1 GiB - 256 B", 16, {15: 0.875}, (1 << 24) - 4, "f32"),
    ("p=33 at 0.5, int32, 32 healthy, 1 GiB + 7 KiB", 33, {32: 0.5}, 8134464, "i32"),
    ("p=16 at 0.5, fp32, odd N, 1 GiB + 64 B", 16, {15: 0.5}, (1 << 24) + 1, "f32"),
    ("p=16, three stragglers, fp32, 1 GiB (two per CU)", 16, {0: 0.5, 1: 0.75, 15: 0.875},
     1 << 24, "f32"),
    ("p=16 ring, int32, 1 GiB", 16, {}, 1 << 24, "i32"),
]


@pytest.mark.parametrize("case", THREE_PER_CU_CASES, ids=[c[0] for c in THREE_PER_CU_CASES])
def test_three_workgroups_per_cu_edges(o, case):
    """Plans on both sides of the launch rules that change the workgroups
    per CU (three: short fp32/int32 chains from 512 MiB of rank buffers and
    bf16 chains of 13-32 healthy ranks; one: fp32/int32 chains of 11-32
    healthy ranks from 1 GiB): every element of every rank bit for bit
    against the oracle's full serial run."""
    label, p, strag, n, dtype = case
    _say(f"case three-per-CU edge: {label}: p={p} n={n} dtype={dtype}")
    bw = _bw(p, strag)
    pl = o.optcc_plan(p, bw, n, 64)
    x = rand_inputs(dtype, p, n, 4242 + p)
    d = to_device(x, dtype)
    o.optcc_allreduce_emulate(d, p, n, dtype, pl)
    torch.cuda.synchronize()
    got = to_host(d, dtype)
    del d
    ref = oracle.run(oracle.Schedule(p, bw, n, 64), dtype, x)
    assert bits_equal(got, ref), label
    del x, got, ref
    torch.cuda.empty_cache()


WIDE_WINDOW_CASES = [
    # 32-bit chains of more than 32 healthy ranks keep 24 hop loads in flight
    # from 2^23 elements per rank (16-byte-aligned buffers); just below, with
    # element-aligned buffers and for bf16 they keep 16
    ("p=34 at 0.5, fp32, 2^23 (24 loads)", 34, {33: 0.5}, 1 << 23, "f32"),
    ("p=34 at 0.5, int32, 2^23 - 4 (16 loads)", 34, {33: 0.5}, (1 << 23) - 4, "i32"),
    ("p=40, two stragglers, int32, 2^23 + 4 (24 loads)", 40, {38: 0.5, 39: 0.75},
     (1 << 23) + 4, "i32"),
    ("p=34 at 0.5, fp32, odd N (one element per access)", 34, {33: 0.5}, (1 << 23) + 1, "f32"),
    ("p=64 at 0.875 (P2P chunks), fp32, 2^23 (24 loads)", 64, {63: 0.875}, 1 << 23, "f32"),
    ("p=34 at 0.5, bf16, 2^23 (16 loads)", 34, {33: 0.5}, 1 << 23, "bf16"),
]


@pytest.mark.parametrize("case", WIDE_WINDOW_CASES, ids=[c[0] for c in WIDE_WINDOW_CASES])
def test_wide_hop_window_edges(o, case):
    """Long chains on both sides of the launch rule that selects the kernel
    with the deeper hop-load window (32-bit elements, at least 2^23 per
    rank, 16-byte-aligned buffers): every element of every rank bit for bit
    against the oracle's full serial run."""
    label, p, strag, n, dtype = case
    _say(f"case wide hop window edge: {label}: p={p} n={n} dtype={dtype}")
    bw = _bw(p, strag)
    pl = o.optcc_plan(p, bw, n, 64)
    x = rand_inputs(dtype, p, n, 2424 + p)
    d = to_device(x, dtype)
    o.optcc_allreduce_emulate(d, p, n, dtype, pl)
    torch.cuda.synchronize()
    got = to_host(d, dtype)
    del d
    ref = oracle.run(oracle.Schedule(p, bw, n, 64), dtype, x)
    assert bits_equal(got, ref), label
    del x, got, ref
    torch.cuda.empty_cache()


def test_random_large_short_chains(o):
    """Four seeded random plans of 6-8 healthy ranks with 480 MiB to 1.9 GiB
    of rank buffers (the range where 6-7 healthy ranks launch at three
    workgroups per CU and 8 take two vectors per lane), fp32 and int32, one
    or two stragglers: every element of every rank bit for bit against the
    oracle's full serial run."""
    rng = np.random.default_rng(2606)
    for i in range(4):
        p = int(rng.integers(7, 10))
        m = 1 if p < 9 else int(rng.integers(1, 3))
        bw = [1.0] * p
        for r in rng.choice(p, size=m, replace=False):
            bw[int(r)] = float(rng.integers(1, 8)) / 8
        dtype = ("f32", "i32")[i % 2]
        lo, hi = (480 << 20) // (4 * p), (1900 << 20) // (4 * p)
        n = int(rng.integers(lo, hi)) // 4 * 4 + int(rng.integers(0, 4))
        k = 4 * int(rng.integers(4, 33))
        _say(f"case large short chain #{i}: p={p} n={n} k={k} dtype={dtype} bw={sorted(set(bw))}")
        pl = o.optcc_plan(p, bw, n, k)
        x = rand_inputs(dtype, p, n, 9100 + i)
        d = to_device(x, dtype)
        o.optcc_allreduce_emulate(d, p, n, dtype, pl)
        torch.cuda.synchronize()
        got = to_host(d, dtype)
        del d
        ref = oracle.run(oracle.Schedule(p, bw, n, k), dtype, x)
        assert bits_equal(got, ref), i
        del x, got, ref
        torch.cuda.empty_cache()


def test_one_graph_of_several_allreduces(o):
    """Several AllReduces with different plans and element types (bubble
    filling, several stragglers, a 40-rank chain launched at one workgroup
    per CU, a server plan, fp16) captured in one HIP graph, as a training
    step would capture its gradient buckets.  Every replay, with eager
    restores and synchronisations in between, equals the oracle bit for bit."""
    specs = [("one", 8, _bw(8, {7: 0.875}), None, 60000, 16, "f32"),
             ("multi", 9, _bw(9, {0: 0.875, 3: 0.75, 8: 0.5}), None, 30000, 8, "bf16"),
             ("long", 40, _bw(40, {5: 0.6}), None, 50000, 8, "f32"),
             ("servers", 6, [1.0, 1.0, 0.5], (3, 2), 40000, 24, "i32"),
             ("fp16", 5, _bw(5, {0: 0.5}), None, 20000, 8, "f16")]
    cases = []
    for name, p, bw, srv, n, k, dt in specs:
        if srv is None:
            pl, sched = o.optcc_plan(p, bw, n, k), oracle.Schedule(p, bw, n, k)
        else:
            pl = o.optcc_plan_servers(srv[0], srv[1], bw, n, k)
            sched = oracle.Schedule.servers(srv[0], srv[1], bw, n, k)
        x = rand_inputs(dt, p, n, 500 + p)
        d = to_device(x, dt)
        cases.append((name, p, n, dt, pl, oracle.run(sched, dt, x.copy()), d, d.clone()))
    for name, p, n, dt, pl, ref, d, d0 in cases:  # first use: table upload
        o.optcc_allreduce_emulate(d, p, n, dt, pl)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    for c in cases:
        c[6].copy_(c[7])
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for name, p, n, dt, pl, ref, d, d0 in cases:
                o.optcc_allreduce_emulate(d, p, n, dt, pl)
    torch.cuda.synchronize()
    for rep in range(3):
        _say(f"case one graph of several AllReduces rep={rep}")
        for c in cases:
            c[6].copy_(c[7])
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, p, n, dt, pl, ref, d, d0 in cases:
            assert bits_equal(to_host(d, dt), ref), (name, rep)
    del g
