"""Several GPUs per server (App. E): host rows against the oracle, and the
HIP executor against the oracle bit for bit.

The library's server plan must equal the oracle's independently built
schedule step for step (slot, segment, section, operation, destination,
source, range); its model time and lower bound must equal the oracle's exact
rationals.  On the GPU every element of every rank must equal the oracle's
serial execution, after the whole AllReduce and after every prefix of the
twelve stage slots (fused or one launch per slot).
"""
import ctypes
import sys

import numpy as np
import pytest

import oracle
from oracle import model
from test_plan_parity import _steps_of_flows


@pytest.fixture(scope="module")
def o():
    from paper_2606_01680_amd import optcc
    return optcc


def _sbw(q, slow):
    b = [1.0] * q
    for s, v in slow.items():
        b[s] = v
    return b


# (q, g, {straggler server: bandwidth})
PROFILES = [
    (3, 2, {2: 0.5}), (3, 2, {0: 0.875}), (4, 4, {1: 0.875}), (5, 3, {0: 0.5}), (3, 8, {2: 0.25}),
    (4, 2, {3: 0.5000001}), (6, 5, {2: 0.75}), (16, 4, {15: 0.5}), (32, 4, {31: 0.875}),
    (64, 4, {7: 0.5}),
]
SIZES = [(0, 24), (1, 24), (63, 24), (64 * 7 + 5, 32), (5000, 24), (64 * 24 * 3 * 2 + 17, 48)]


@pytest.mark.parametrize("q,g,slow", PROFILES)
@pytest.mark.parametrize("n,k", SIZES)
def test_server_plan_equals_oracle(o, q, g, slow, n, k):
    bw = _sbw(q, slow)
    pl = o.optcc_plan_servers(q, g, bw, n, k)
    ref = oracle.Schedule.servers(q, g, bw, n, k)
    assert pl.kind == "servers" == ref.kind
    assert (pl.p, pl.g, pl.q, pl.m, pl.healthy) == (q * g, g, q, 1, q - 1)
    assert pl.num_segments == g * k == ref.nseg and pl.num_slots == 12
    assert list(pl.ring) == list(ref.ring) and list(pl.stragglers) == list(ref.stragglers)
    assert np.array_equal(pl.slowdowns, ref.ell)
    off, ln, p2p = pl.segments()
    assert np.array_equal(off, ref.seg_off) and np.array_equal(ln, ref.seg_len)
    assert not p2p.any()
    fl = pl.flows()
    assert len(fl) == pl.num_flows == pl.num_steps
    assert _steps_of_flows(fl) == ref.steps()


@pytest.mark.parametrize("q,g,slow", PROFILES)
@pytest.mark.parametrize("n,k", [(1 << 20, 32), (12345, 24)])
def test_server_model_and_bound_equal_oracle(o, q, g, slow, n, k):
    bw = _sbw(q, slow)
    pl = o.optcc_plan_servers(q, g, bw, n, k)
    ell = model.slowdowns(bw)[0][0]
    t = o.optcc_model_time(pl)
    assert t == pytest.approx(float(model.optcc_servers(q, g, ell, n, k)), rel=1e-13)
    assert o.optcc_model_time(pl, bw) == t
    lb = o.optcc_lower_bound_servers(q, g, bw, n)
    assert lb == pytest.approx(float(model.lb_servers_tight(q, g, ell, n)), rel=1e-13)
    assert t >= lb
    # the fault-free optimum and the one-GPU bound as the g = 1 case
    assert o.optcc_lower_bound_servers(q, g, [1.0] * q, n) == pytest.approx(
        float(model.t0_servers(q * g, g, n)), rel=1e-13)
    assert o.optcc_lower_bound_servers(q, 1, bw, n) == pytest.approx(
        o.optcc_lower_bound(q, bw, n), rel=1e-13)


def test_server_traffic(o):
    """Fused: every input read once, one write per step: p reads and 2(p-1)
    writes per coordinate; one launch per slot re-reads each slot's state."""
    q, g, n = 16, 4, 1 << 20
    pl = o.optcc_plan_servers(q, g, _sbw(q, {15: 0.5}), n, 32)
    for dt, es in (("f32", 4), ("bf16", 2), ("i32", 4), ("f16", 2)):
        r, w = pl.traffic(dt)
        assert r == q * g * n * es and w == 2 * (q * g - 1) * n * es
    r0, w0 = pl.traffic("f32", launches=0)
    assert w0 == 2 * (q * g - 1) * n * 4 and r0 > q * g * n * 4


def test_server_errors(o):
    def code(*a):
        with pytest.raises(o.OptccError) as e:
            o.optcc_plan_servers(*a)
        return e.value.status
    assert code(2, 4, [1, 0.5], 100, 24) == o.OPTCC_EINVAL            # q < 3
    assert code(4, 1, [1, 1, 1, 0.5], 100, 24) == o.OPTCC_EINVAL      # g = 1 is optcc_plan
    assert code(4, 2, [1, 1, 1, 0.5], 100, 20) == o.OPTCC_EINVAL      # k < 24
    assert code(4, 2, [1, 1, 1, 0.5], 100, 28) == o.OPTCC_EINVAL      # 8 does not divide k
    assert code(4, 2, [1, 1, 1, 0.0], 100, 24) == o.OPTCC_EINVAL
    assert code(4, 2, [1, 1, 1, 1], 100, 24) == o.OPTCC_EUNSUPPORTED  # no straggler server
    assert code(4, 2, [1, 1, 0.5, 0.5], 100, 24) == o.OPTCC_EUNSUPPORTED
    assert code(300, 4, [1.0] * 299 + [0.5], 100, 24) == o.OPTCC_EUNSUPPORTED
    pl = o.optcc_plan_servers(4, 2, [1, 1, 1, 0.5], 100, 24)
    with pytest.raises(o.OptccError):
        o.optcc_model_time(pl, [1, 1, 0.5, 1])  # another straggler server
    L = o.lib()
    ptrs = (ctypes.c_void_p * 8)(*[4096 * (i + 1) for i in range(8)])
    assert L.optcc_allreduce_emulate_slots(ptrs, 8, 100, 0, pl.handle, 0, 13, 1, None) == o.OPTCC_EINVAL
    assert L.optcc_allreduce_emulate(ptrs, 4, 100, 0, pl.handle, None) == o.OPTCC_EINVAL
    with pytest.raises(o.OptccError):
        o.optcc_lower_bound_servers(4, 2, [1, 0.5, 1, 0.5], 100)


# ------------------------------------------------------------------ GPU
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _run_both(o, q, g, slow, n, k, dtype, seed, slot_end=12, launches=1, kind="normal"):
    torch = _gpu()
    from gpu_util import rand_inputs, to_device, to_host
    bw = _sbw(q, slow)
    x = rand_inputs(dtype, q * g, n, seed, kind)
    ref = oracle.run(oracle.Schedule.servers(q, g, bw, n, k), dtype, x.copy(), 0, slot_end)
    pl = o.optcc_plan_servers(q, g, bw, n, k)
    d = to_device(x, dtype)
    o.optcc_allreduce_emulate_slots(d, q * g, n, dtype, pl, 0, slot_end, launches)
    torch.cuda.synchronize()
    return x, ref, to_host(d, dtype)


# every server size with a compile-time local ring (2..8) and the general lane (12)
GPU_PROFILES = [(3, 2, {2: 0.5}), (4, 4, {1: 0.875}), (5, 3, {0: 0.5}), (3, 8, {2: 0.25}),
                (6, 5, {2: 0.75}), (16, 4, {15: 0.5}), (9, 3, {4: 0.875}), (4, 6, {0: 0.5}),
                (3, 7, {1: 0.875}), (3, 12, {2: 0.5})]
GPU_SIZES = [(1, 24), (37, 24), (2048 * 3 + 64 * 5 + 3, 24), (40000, 32)]


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32", "f16"])
@pytest.mark.parametrize("q,g,slow", GPU_PROFILES)
@pytest.mark.parametrize("n,k", GPU_SIZES)
def test_server_small_bit_exact(o, dtype, q, g, slow, n, k):
    from gpu_util import bits_equal
    _say(f"case servers dtype={dtype} q={q} g={g} slow={slow} n={n} k={k}")
    x, ref, got = _run_both(o, q, g, slow, n, k, dtype, seed=q * 100 + g * 10 + n)
    assert bits_equal(got, ref)
    assert (got == got[0][None, :]).all()


@pytest.mark.gpu
@pytest.mark.parametrize("dtype,q,g,slow,n,k", [
    # 2048-element tiles, two vectors per lane, a sub-vector tail
    ("f32", 4, 2, {3: 0.5}, (1 << 21) + 2048 * 3 + 64 * 5 + 3, 24),
    ("i32", 4, 2, {3: 0.5}, (1 << 21) + 2048 * 3 + 64 * 5 + 3, 24),
    # 4096-element tiles (2-byte elements, six ranks)
    ("bf16", 3, 2, {2: 0.5}, (1 << 22) + 77, 24),
    ("f16", 3, 2, {0: 0.875}, (1 << 22) + 2048 + 9, 24),
])
def test_server_tile_lengths_bit_exact(o, dtype, q, g, slow, n, k):
    """Server plans at sizes where the launch takes 2048- or 4096-element
    tiles (the small-message rule does not shorten them), bit for bit
    against the oracle."""
    from gpu_util import bits_equal
    _say(f"case servers tiles dtype={dtype} q={q} g={g} slow={slow} n={n} k={k}")
    x, ref, got = _run_both(o, q, g, slow, n, k, dtype, seed=q * 100 + g * 10 + n % 89)
    assert bits_equal(got, ref)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype,q,g,slow,n", [
    # at most 32 ranks, 32-bit elements, from 1 GiB of buffers: one
    # workgroup per CU with 4 or more GPUs per server, two with 2
    ("f32", 4, 4, {3: 0.5}, (1 << 24) + 4),
    ("i32", 8, 2, {0: 0.5}, (1 << 24) + 8),
    ("f32", 4, 4, {1: 0.875}, (1 << 24) - 4),
])
def test_server_occupancy_edges(o, dtype, q, g, slow, n):
    """Server plans around the 1 GiB edge of the one-workgroup-per-CU
    launch, bit for bit against the oracle on every element."""
    from gpu_util import bits_equal
    _say(f"case servers occupancy dtype={dtype} q={q} g={g} slow={slow} n={n}")
    x, ref, got = _run_both(o, q, g, slow, n, 24, dtype, seed=q * 7 + g)
    assert bits_equal(got, ref)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32", "f16"])
@pytest.mark.parametrize("q,g,slow", [(3, 2, {2: 0.5}), (4, 3, {1: 0.875}), (5, 4, {0: 0.5})])
@pytest.mark.parametrize("launches", [1, 0])
def test_server_stage_snapshots(o, dtype, q, g, slow, launches):
    """After the first s of the twelve slots, fused or one launch per slot,
    every buffer equals the oracle's state after the same slots: every
    step's destination write is materialised."""
    from gpu_util import bits_equal
    n, k = 2048 * 2 + 64 * 7 + 5, 24
    for s in range(1, 13):
        _say(f"case server snapshot dtype={dtype} q={q} g={g} slots=[0,{s}) launches={launches}")
        x, ref, got = _run_both(o, q, g, slow, n, k, dtype, seed=29 + s, slot_end=s,
                                launches=launches)
        assert bits_equal(got, ref), f"slots [0,{s})"


@pytest.mark.gpu
@pytest.mark.parametrize("dtype,kind", [(d, k) for d in ("f32", "bf16", "f16")
                                         for k in ("denormal", "wide")] + [("f16", "overflow")])
def test_server_special_values(o, dtype, kind):
    from gpu_util import bits_equal, half_equal_nan
    for q, g, slow in [(3, 2, {2: 0.5}), (4, 4, {1: 0.875})]:
        _say(f"case server special {kind} dtype={dtype} q={q} g={g}")
        x, ref, got = _run_both(o, q, g, slow, 5000, 24, dtype, seed=3, kind=kind)
        if kind == "overflow":
            # opposite infinities meet where two partial sums are added (a
            # collected server sum and the chain's partial): IEEE 754 leaves
            # the sign and payload of that NaN open, so NaN positions must
            # agree and every other element bit for bit
            assert half_equal_nan(got, ref)
            assert np.isinf(oracle.f16_to_f64(got)).any()
        else:
            assert bits_equal(got, ref)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32", "f16"])
def test_server_unaligned_buffers(o, dtype):
    """Rank buffers that are only element-aligned take the one-element path."""
    torch = _gpu()
    from gpu_util import bits_equal, rand_inputs, to_device, to_host
    q, g, n, k = 4, 3, 3000, 24
    bw = _sbw(q, {2: 0.5})
    p = q * g
    x = rand_inputs(dtype, p, n, 5)
    ref = oracle.run(oracle.Schedule.servers(q, g, bw, n, k), dtype, x.copy())
    pl = o.optcc_plan_servers(q, g, bw, n, k)
    stride = n + 1
    flat = torch.zeros(p * stride + 8, dtype=to_device(x[:1, :1], dtype).dtype, device="cuda:0")
    for r in range(p):
        flat[1 + r * stride: 1 + r * stride + n].copy_(to_device(x[r:r + 1], dtype)[0])
    views = [flat[1 + r * stride: 1 + r * stride + n] for r in range(p)]
    _say(f"case server unaligned dtype={dtype}")
    o.optcc_allreduce_emulate(views, p, n, dtype, pl)
    torch.cuda.synchronize()
    got = np.stack([to_host(v, dtype) for v in views])
    assert bits_equal(got, ref)


SERVER_WORKLOADS = ["q4g4_bf16", "q16g4_f32", "q32g4_f32"]


@pytest.mark.gpu
@pytest.mark.parametrize("name", SERVER_WORKLOADS)
def test_server_workload_full_size(o, name):
    """Full-size server workloads: all ranks identical, within the error
    bound of the exact sum, and every element equal to the oracle's serial
    execution."""
    torch = _gpu()
    from gpu_util import bits_equal, to_host
    from paper_2606_01680_amd.workloads import WORKLOADS as W, make_inputs
    w = W[name]
    _say(f"case server workload {name} q={w.q} g={w.g} N={w.n} dtype={w.dtype} k={w.k}")
    x = make_inputs(w, device="cuda:0")
    x0 = x.clone()
    pl = o.optcc_plan_servers(w.q, w.g, w.bandwidths, w.n, w.k)
    o.optcc_allreduce_emulate(x, w.p, w.n, w.dtype, pl)
    torch.cuda.synchronize()
    iv = x.view(torch.int16) if x.element_size() == 2 else x.view(torch.int32)
    for r in range(1, w.p):
        assert torch.equal(iv[r], iv[0]), r
    step = max(1 << 16, (1 << 28) // w.p)
    for c0 in range(0, w.n, step):
        c1 = min(w.n, c0 + step)
        xs = x0[:, c0:c1].to(torch.float64)
        err = (x[0, c0:c1].to(torch.float64) - xs.sum(0)).abs()
        u = {"f32": 2.0 ** -24, "f16": 2.0 ** -11, "bf16": 2.0 ** -8}[w.dtype]
        assert bool((err <= w.p * u * xs.abs().sum(0)).all())
    _say(f"case server workload {name}: full oracle run")
    full = oracle.run(oracle.Schedule.servers(w.q, w.g, w.bandwidths, w.n, w.k), w.dtype,
                      to_host(x0, w.dtype).copy())
    del x0
    assert bits_equal(to_host(x, w.dtype), full)


@pytest.mark.gpu
def test_server_graph_capture_replays(o):
    """A server-plan AllReduce is one kernel launch after its first call, so
    it can be captured in a HIP graph; every replay (eager restores and
    synchronisations in between) equals the eager result bit for bit."""
    torch = _gpu()
    from gpu_util import bits_equal, rand_inputs, to_device, to_host
    q, g, n, k = 4, 4, 200000, 24
    bw = _sbw(q, {1: 0.875})
    p = q * g
    pl = o.optcc_plan_servers(q, g, bw, n, k)
    for dtype in ("f32", "bf16", "i32", "f16"):
        x = rand_inputs(dtype, p, n, 41)
        d = to_device(x, dtype)
        d0 = d.clone()
        o.optcc_allreduce_emulate(d, p, n, dtype, pl)  # first use: table upload
        torch.cuda.synchronize()
        eager = d.clone()
        ref = oracle.run(oracle.Schedule.servers(q, g, bw, n, k), dtype, x.copy())
        assert bits_equal(to_host(eager, dtype), ref)
        gr = torch.cuda.CUDAGraph()
        d.copy_(d0)
        torch.cuda.synchronize()
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            with torch.cuda.graph(gr, stream=s):
                o.optcc_allreduce_emulate(d, p, n, dtype, pl)
        torch.cuda.synchronize()
        iv = torch.int16 if d.element_size() == 2 else torch.int32
        for rep in range(3):
            _say(f"case server graph replay dtype={dtype} rep={rep}")
            d.copy_(d0)
            torch.cuda.synchronize()
            gr.replay()
            torch.cuda.synchronize()
            assert torch.equal(d.view(iv), eager.view(iv))
        del gr


@pytest.mark.gpu
def test_server_graph_capture_of_a_stealing_plan(o):
    """A server plan whose eager launches take work stealing (96 ranks, more
    than 4096 tiles) keeps the per-XCD runs when captured in a HIP graph:
    every replay equals the eager result and the oracle bit for bit."""
    torch = _gpu()
    from gpu_util import bits_equal, rand_inputs, to_device, to_host
    q, g, n, k, dtype = 24, 4, (1 << 23) + (1 << 20) + 8, 64, "bf16"
    bw = _sbw(q, {23: 0.5})
    p = q * g
    pl = o.optcc_plan_servers(q, g, bw, n, k)
    x = rand_inputs(dtype, p, n, 43)
    d = to_device(x, dtype)
    d0 = d.clone()
    o.optcc_allreduce_emulate(d, p, n, dtype, pl)
    torch.cuda.synchronize()
    eager = d.clone()
    ref = oracle.run(oracle.Schedule.servers(q, g, bw, n, k), dtype, x.copy())
    assert bits_equal(to_host(eager, dtype), ref)
    gr = torch.cuda.CUDAGraph()
    d.copy_(d0)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        with torch.cuda.graph(gr, stream=s):
            o.optcc_allreduce_emulate(d, p, n, dtype, pl)
    torch.cuda.synchronize()
    for rep in range(2):
        _say(f"case server graph replay of a stealing plan rep={rep}")
        d.copy_(d0)
        torch.cuda.synchronize()
        gr.replay()
        torch.cuda.synchronize()
        assert torch.equal(d.view(torch.int16), eager.view(torch.int16))
    # eager again after the capture: stealing, same bits
    d.copy_(d0)
    o.optcc_allreduce_emulate(d, p, n, dtype, pl)
    torch.cuda.synchronize()
    assert torch.equal(d.view(torch.int16), eager.view(torch.int16))
    del gr, d, d0, eager
    torch.cuda.empty_cache()


@pytest.mark.gpu
@pytest.mark.parametrize("q,g", [(32, 8), (4, 64), (128, 2)])
def test_server_largest_rank_count(o, q, g):
    """p = q g = 256 ranks, the executor's limit: 32 servers x 8 GPUs and
    128 x 2 (local ring fixed at compile time) and 4 servers x 64 GPUs (the
    general lane, the largest g), bit for bit against the oracle."""
    from gpu_util import bits_equal
    slow = {q - 1: 0.5} if q > 4 else {1: 0.875}
    for dtype in ("i32", "f32"):
        _say(f"case servers p=256 q={q} g={g} dtype={dtype}")
        x, ref, got = _run_both(o, q, g, slow, 20000, 24, dtype, seed=q * 7 + g)
        assert bits_equal(got, ref)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype,q,g,slow,n", [
    # 90 or more ranks, more than 4096 tiles (2048 from 120 ranks),
    # 16-byte-aligned buffers: work stealing; fewer tiles, element-aligned
    # buffers or fewer ranks: the per-XCD runs
    ("bf16", 24, 4, {23: 0.5}, (1 << 23) + (1 << 20) + 8),
    ("bf16", 32, 4, {5: 0.875}, (1 << 23) + (1 << 21) + 16),
    ("f32", 45, 2, {44: 0.5}, (1 << 23) + 2048 * 3 + 4),
    ("bf16", 24, 4, {23: 0.5}, 1 << 22),
    ("bf16", 24, 4, {23: 0.5}, (1 << 23) + (1 << 20) + 1),
    ("bf16", 22, 4, {21: 0.5}, (1 << 23) + (1 << 20) + 8),
    # from 120 ranks the bound is 2048 tiles
    ("f32", 32, 4, {31: 0.875}, (1 << 22) + (1 << 20) + 4),
    ("bf16", 30, 4, {29: 0.5}, (1 << 22) + (1 << 20) + 8),
    ("bf16", 29, 4, {28: 0.5}, (1 << 22) + (1 << 20) + 8),
    ("bf16", 32, 4, {31: 0.5}, 1 << 21),
])
def test_server_work_stealing(o, dtype, q, g, slow, n):
    """Server plans on both sides of the work-stealing rule (90 or more
    ranks, more than 4096 tiles of 2048 elements, more than 2048 from 120
    ranks, 16-byte-aligned buffers):
    three calls on one plan, the first two from the same inputs (the device
    counter block of the first is reset for the second), the third on the
    second's output, each bit for bit against the oracle on every
    element."""
    torch = _gpu()
    from gpu_util import bits_equal, rand_inputs, to_device, to_host
    _say(f"case servers work stealing dtype={dtype} q={q} g={g} slow={slow} n={n}")
    bw = _sbw(q, slow)
    k = 64
    x = rand_inputs(dtype, q * g, n, q * 31 + g, "normal")
    ref = oracle.run(oracle.Schedule.servers(q, g, bw, n, k), dtype, x.copy())
    pl = o.optcc_plan_servers(q, g, bw, n, k)
    for call in range(2):
        d = to_device(x, dtype)
        o.optcc_allreduce_emulate(d, q * g, n, dtype, pl)
        torch.cuda.synchronize()
        got = to_host(d, dtype)
        assert bits_equal(got, ref), f"call {call}"
    ref2 = oracle.run(oracle.Schedule.servers(q, g, bw, n, k), dtype, ref.copy())
    o.optcc_allreduce_emulate(d, q * g, n, dtype, pl)
    torch.cuda.synchronize()
    assert bits_equal(to_host(d, dtype), ref2), "call 2"
    del d
    torch.cuda.empty_cache()
