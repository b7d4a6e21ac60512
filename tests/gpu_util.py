"""Helpers for the GPU tests: moving seeded inputs between numpy (oracle
side) and torch device tensors (library side)."""
import numpy as np
import torch

TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "i32": torch.int32, "f16": torch.float16}
HALF = ("bf16", "f16")  # 16-bit types: numpy holds their bit patterns as uint16


def to_device(x: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype in HALF:
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(TORCH[dtype])
    else:
        t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to("cuda:0").contiguous()


def to_host(t: torch.Tensor, dtype: str) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if dtype in HALF:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def int_view(t: torch.Tensor) -> torch.Tensor:
    """Bit patterns of a device tensor, for bitwise comparisons."""
    return t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32)


def rand_inputs(dtype: str, p: int, n: int, seed: int, kind: str = "normal") -> np.ndarray:
    """Seeded host inputs for small parity cases.  For fp16, "denormal" and
    "wide" are scaled to the half format (around its smallest normal 2^-14,
    and over its whole exponent range) and "overflow" puts values near the
    largest finite half (65504) so that partial sums overflow to infinity."""
    rng = np.random.default_rng(seed)
    if dtype == "i32":
        return rng.integers(-(2**31), 2**31, size=(p, n), dtype=np.int64).astype(np.int32)
    half = dtype == "f16"
    if kind == "denormal":
        x = (rng.standard_normal((p, n)) * (6.1e-5 if half else 1.2e-38)).astype(np.float32)
    elif kind == "wide":
        lo, hi = (-26, 14) if half else (-60, 60)
        x = (rng.standard_normal((p, n)) * np.exp2(rng.integers(lo, hi, size=(p, n)))).astype(np.float32)
    elif kind == "overflow":
        x = (rng.uniform(-1.0, 1.0, (p, n)) * 65504.0).astype(np.float32)
    else:
        x = rng.standard_normal((p, n)).astype(np.float32)
    import oracle
    if dtype == "bf16":
        return oracle.bf16_round(x)
    if half:
        return oracle.f16_round(x)
    return x


def bits_equal(a: np.ndarray, b: np.ndarray) -> bool:
    return a.shape == b.shape and a.dtype == b.dtype and np.array_equal(
        a.view(np.uint8), b.view(np.uint8))


def half_equal_nan(a: np.ndarray, b: np.ndarray) -> bool:
    """fp16 bit patterns equal, except that a NaN matches any NaN."""
    nan_a = ((a & 0x7c00) == 0x7c00) & ((a & 0x3ff) != 0)
    nan_b = ((b & 0x7c00) == 0x7c00) & ((b & 0x3ff) != 0)
    return a.shape == b.shape and np.array_equal(nan_a, nan_b) and np.array_equal(a[~nan_a], b[~nan_b])
