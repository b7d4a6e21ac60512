"""The no-allocation entry point against the allocating one (MI355X).

optcc_allreduce_emulate_noalloc stages the plan's tables in the library's
static per-GPU scratch array instead of device memory of their own.  Called
through the C ABI, it must give exactly the bits of optcc_allreduce_emulate
on the same inputs (and both the oracle's), on calls in a row whose plans
differ, each later one smaller than the first, so that the array holds the
previous call's tables when the next one stages its own.
"""
import ctypes
import sys

import numpy as np
import pytest
import torch

import oracle
from gpu_util import bits_equal, rand_inputs, to_device, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def o():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_01680_amd import optcc
    return optcc


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _bw(p, slow):
    b = [1.0] * p
    for r, v in slow.items():
        b[r] = v
    return b


def _ptrs(d):
    p = d.shape[0]
    base, stride = d.data_ptr(), d.stride(0) * d.element_size()
    return (ctypes.c_void_p * p)(*[base + r * stride for r in range(p)])


# (name, p, straggler bandwidths or server shape, N, k, dtype): each call
# after the first moves less data than the first and has another plan
CALLS = [
    ("p8 one straggler l<2, f32", 8, {7: 0.875}, None, 1_000_003, 16, "f32"),
    ("p5 one straggler l=2, bf16", 5, {0: 0.5}, None, 70_001, 8, "bf16"),
    ("p9 three stragglers, i32", 9, {0: 0.875, 3: 0.75, 8: 0.5}, None, 123_457, 8, "i32"),
    ("3x2 servers, f16", 6, None, (3, 2, [1.0, 1.0, 0.5]), 50_000, 24, "f16"),
    ("p8 again, smaller N, f32", 8, {7: 0.875}, None, 300_001, 16, "f32"),
]


def test_noalloc_equals_emulate(o):
    L = o.lib()
    for i, (name, p, slow, srv, n, k, dtype) in enumerate(CALLS):
        _say(f"case no-alloc call {i}: {name} N={n}")
        if srv is None:
            bw = _bw(p, slow)
            pl = o.optcc_plan(p, bw, n, k)
            sched = oracle.Schedule(p, bw, n, k)
        else:
            q, g, sbw = srv
            pl = o.optcc_plan_servers(q, g, sbw, n, k)
            sched = oracle.Schedule.servers(q, g, sbw, n, k)
        x = rand_inputs(dtype, p, n, 900 + i)
        ref = oracle.run(sched, dtype, x.copy())
        a = to_device(x, dtype)
        b = a.clone()
        s = torch.cuda.current_stream().cuda_stream
        rc = L.optcc_allreduce_emulate(_ptrs(a), p, n, o.DTYPES[dtype], pl.handle,
                                       ctypes.c_void_p(s))
        assert rc == 0, o.optcc_last_error()
        rc = L.optcc_allreduce_emulate_noalloc(_ptrs(b), p, n, o.DTYPES[dtype], pl.handle,
                                               ctypes.c_void_p(s))
        assert rc == 0, o.optcc_last_error()
        torch.cuda.synchronize()
        got_a, got_b = to_host(a, dtype), to_host(b, dtype)
        assert bits_equal(got_b, got_a), name
        assert bits_equal(got_b, ref), name
        if i == 0:
            first = n * p
        else:
            assert n * p < first


def test_noalloc_back_to_back_on_one_stream(o):
    """Two calls queued back to back on one stream, the second on a smaller
    input with another plan, before any synchronisation: stream order keeps
    each call's tables until its kernel has read them."""
    L = o.lib()
    cases = [(8, {7: 0.875}, 400_000, 16, "f32", 31), (6, {0: 0.5, 5: 0.75}, 90_001, 8, "f32", 32)]
    devs, refs, plans = [], [], []
    s = torch.cuda.current_stream().cuda_stream
    for p, slow, n, k, dtype, seed in cases:
        bw = _bw(p, slow)
        x = rand_inputs(dtype, p, n, seed)
        refs.append(oracle.run(oracle.Schedule(p, bw, n, k), dtype, x.copy()))
        plans.append(o.optcc_plan(p, bw, n, k))
        devs.append(to_device(x, dtype))
    torch.cuda.synchronize()
    _say("case no-alloc back to back")
    for (p, slow, n, k, dtype, _), d, pl in zip(cases, devs, plans):
        rc = L.optcc_allreduce_emulate_noalloc(_ptrs(d), p, n, o.DTYPES[dtype], pl.handle,
                                               ctypes.c_void_p(s))
        assert rc == 0, o.optcc_last_error()
    torch.cuda.synchronize()
    for (p, slow, n, k, dtype, _), d, ref in zip(cases, devs, refs):
        assert bits_equal(to_host(d, dtype), ref)
