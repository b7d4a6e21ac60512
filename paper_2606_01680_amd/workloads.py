"""Named workloads and seeded synthetic inputs.

This module only draws numbers: it holds none of the schedule's arithmetic and
is shared by the tests, the benchmark and the smoke check.  The paper's own
workloads are data-parallel gradient buffers of hundreds of MB to several GB
per rank, simulated without values; the value distributions below stand in for
real gradients.

Seeds: rank r of workload w draws from ``manual_seed(2606 + 1000 * w + r)``.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

TORCH_DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16, "i32": torch.int32,
                "f16": torch.float16}
ESIZE = {"f32": 4, "bf16": 2, "i32": 4, "f16": 2}


@dataclass(frozen=True)
class Workload:
    name: str
    index: int          # seed block
    p: int              # ranks (q servers x g GPUs when g > 1)
    bandwidths: tuple   # one entry per rank (per server when g > 1), healthy = 1.0
    n: int              # elements per rank
    k: int              # segments ("n_chunks"; per part when g > 1)
    dtype: str
    values: str         # value recipe, see make_inputs
    note: str = field(default="", compare=False)
    g: int = 1          # GPUs per server

    @property
    def q(self) -> int:
        return self.p // self.g


def _bw(p, slow):
    b = [1.0] * p
    for r, v in slow.items():
        b[r] = v
    return tuple(b)


WORKLOADS = {
    "p4_f32": Workload("p4_f32", 0, 4, _bw(4, {3: 0.5}), 65536, 8, "f32", "normal",
                       "rank 3 at 50% bandwidth"),
    "p8_f32": Workload("p8_f32", 1, 8, _bw(8, {7: 0.875}), 1 << 26, 64, "f32", "normal",
                       "one of 8 NICs lost on rank 7"),
    "p8_i32": Workload("p8_i32", 1, 8, _bw(8, {7: 0.875}), 1 << 26, 64, "i32", "uniform_2p20",
                       "int32 run of the p=8 workload"),
    "p16_bf16": Workload("p16_bf16", 2, 16, _bw(16, {15: 0.5}), 1 << 26, 128, "bf16",
                         "normal_1e-2", "rank 15 at 50% bandwidth"),
    # the p = 16 workload with IEEE fp16 gradients (loss-scaled mixed precision)
    "p16_f16": Workload("p16_f16", 8, 16, _bw(16, {15: 0.5}), 1 << 26, 128, "f16",
                        "normal_1e-2", "fp16 run of the p=16 workload"),
    "p64_f32": Workload("p64_f32", 3, 64, _bw(64, {62: 0.75, 63: 0.5}), 1 << 24, 128, "f32",
                        "normal_zeros1pct", "two stragglers"),
    "p128_f32": Workload("p128_f32", 4, 128,
                         _bw(128, {124: 0.875, 125: 0.75, 126: 0.5, 127: 0.5}), 1 << 24, 256,
                         "f32", "student_t3_1e-3", "four stragglers"),
    # several GPUs per server (App. E), like the paper's g = 4 experiments:
    # the straggler server loses 4 of its 8 NICs (l = 2) or 1 of 8 (l = 8/7)
    "q16g4_f32": Workload("q16g4_f32", 5, 64, _bw(16, {15: 0.5}), 1 << 24, 128, "f32", "normal",
                          "16 servers x 4 GPUs, server 15 at 50% bandwidth", g=4),
    "q32g4_f32": Workload("q32g4_f32", 6, 128, _bw(32, {31: 0.875}), 1 << 24, 128, "f32",
                          "normal", "32 servers x 4 GPUs, server 31 lost 1 of 8 NICs", g=4),
    "q4g4_bf16": Workload("q4g4_bf16", 7, 16, _bw(4, {0: 0.5}), 1 << 26, 128, "bf16",
                          "normal_1e-2", "4 servers x 4 GPUs, server 0 at 50% bandwidth", g=4),
}


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def make_rank(values: str, dtype: str, n: int, seed: int, device) -> torch.Tensor:
    """One rank's input vector.

    normal            N(0, 1)
    normal_1e-2       N(0, 1) * 1e-2, rounded to the dtype (bf16, fp16:
                      torch's round-to-nearest-even)
    normal_zeros1pct  N(0, 1), each element independently set to +0.0 with
                      probability 0.01
    student_t3_1e-3   z / sqrt(chi2_3 / 3) * 1e-3 with chi2_3 a sum of three
                      squared standard normals
    uniform_2p20      integers uniform on [-2**20, 2**20] inclusive
    denormal          fp32 values around the smallest normal, half subnormal
    """
    g = _gen(device, seed)
    td = TORCH_DTYPES[dtype]
    if values == "uniform_2p20":
        x = torch.randint(-(1 << 20), (1 << 20) + 1, (n,), generator=g, device=device,
                          dtype=torch.int64)
        return x.to(td)
    if dtype == "i32":
        raise ValueError("integer workloads use uniform_2p20")
    if values == "normal":
        x = torch.randn(n, generator=g, device=device)
    elif values == "normal_1e-2":
        x = torch.randn(n, generator=g, device=device) * 1e-2
    elif values == "normal_zeros1pct":
        x = torch.randn(n, generator=g, device=device)
        z = torch.rand(n, generator=g, device=device) < 0.01
        x = torch.where(z, torch.zeros_like(x), x)
    elif values == "student_t3_1e-3":
        z = torch.randn(n, generator=g, device=device)
        c = torch.randn(3, n, generator=g, device=device).pow(2).sum(0)
        x = z / torch.sqrt(c / 3.0) * 1e-3
    elif values == "denormal":
        x = torch.randn(n, generator=g, device=device) * 1.2e-38
    else:
        raise ValueError(f"unknown value recipe {values!r}")
    return x.to(td)


def make_inputs(w: Workload, device="cpu", n: int | None = None) -> torch.Tensor:
    """[p, N] contiguous inputs of workload w (optionally truncated to n)."""
    n = w.n if n is None else n
    out = torch.empty((w.p, n), dtype=TORCH_DTYPES[w.dtype], device=device)
    for r in range(w.p):
        out[r].copy_(make_rank(w.values, w.dtype, n, 2606 + 1000 * w.index + r, device))
    return out


def custom(p, bandwidths, n, k, dtype="f32", values="normal", index=100, name="custom"):
    return Workload(name, index, p, tuple(float(b) for b in bandwidths), n, k, dtype, values)
