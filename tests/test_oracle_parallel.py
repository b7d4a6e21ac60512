"""The oracle's all-cores executor gives the serial executor's bits (CPU).

`oracle.run_parallel` shares the segments out among OpenMP threads; since a
step touches only its own segment's coordinates and each segment's steps
keep their serial order, every coordinate sees the same operations in the
same order as `oracle.run`.  Checked bit for bit on every plan kind, every
element type, partial slot ranges and thread counts from 1 to more threads
than segments.
"""
import numpy as np
import pytest

import oracle

PLANS = [
    ("ring", lambda n: oracle.Schedule(5, [1.0] * 5, n, 8)),
    ("one, l >= 2", lambda n: oracle.Schedule(6, [1, 1, 0.5, 1, 1, 1], n, 8)),
    ("one, l < 2", lambda n: oracle.Schedule(8, [1.0] * 7 + [0.875], n, 12)),
    ("several", lambda n: oracle.Schedule(9, [0.875, 1, 1, 0.75, 1, 1, 1, 1, 0.5], n, 8)),
    ("servers", lambda n: oracle.Schedule.servers(4, 3, [1.0, 0.5, 1.0, 1.0], n, 24)),
]


def _inputs(dtype, p, n, seed):
    rng = np.random.default_rng(seed)
    if dtype == "i32":
        return rng.integers(-(2**31), 2**31, size=(p, n), dtype=np.int64).astype(np.int32)
    x = rng.standard_normal((p, n)).astype(np.float32)
    if dtype == "f32":
        return x
    return oracle.bf16_round(x) if dtype == "bf16" else oracle.f16_round(x)


@pytest.mark.parametrize("name,make", PLANS, ids=[p[0] for p in PLANS])
@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32", "f16"])
def test_parallel_equals_serial(name, make, dtype):
    n = 64 * 301 + 17
    s = make(n)
    x = _inputs(dtype, s.p, n, 7)
    want = oracle.run(s, dtype, x.copy())
    for threads in (1, 3, 8, 64):
        got = oracle.run_parallel(s, dtype, x.copy(), threads)
        assert np.array_equal(got.view(np.uint8), want.view(np.uint8)), (name, dtype, threads)
    hi = s.num_slots // 2
    want = oracle.run(s, dtype, x.copy(), 0, hi)
    got = oracle.run_parallel(s, dtype, x.copy(), 4, 0, hi)
    assert np.array_equal(got.view(np.uint8), want.view(np.uint8))


def test_parallel_rejects_bad_arguments():
    s = oracle.Schedule(4, [1, 1, 1, 0.5], 100, 4)
    x = np.zeros((4, 100), np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.run_parallel(s, "f32", x, 0)
