"""Helpers for the GPU tests: moving seeded inputs between numpy (oracle
side) and torch device tensors (library side)."""
import numpy as np
import torch

TORCH = {"f32": torch.float32, "bf16": torch.bfloat16, "i32": torch.int32}


def to_device(x: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to("cuda:0").contiguous()


def to_host(t: torch.Tensor, dtype: str) -> np.ndarray:
    t = t.detach().cpu().contiguous()
    if dtype == "bf16":
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def rand_inputs(dtype: str, p: int, n: int, seed: int, kind: str = "normal") -> np.ndarray:
    """Seeded host inputs for small parity cases."""
    rng = np.random.default_rng(seed)
    if dtype == "i32":
        return rng.integers(-(2**31), 2**31, size=(p, n), dtype=np.int64).astype(np.int32)
    if kind == "denormal":
        x = (rng.standard_normal((p, n)) * 1.2e-38).astype(np.float32)
    elif kind == "wide":
        x = (rng.standard_normal((p, n)) * np.exp2(rng.integers(-60, 60, size=(p, n)))).astype(np.float32)
    else:
        x = rng.standard_normal((p, n)).astype(np.float32)
    if dtype == "bf16":
        import oracle
        return oracle.bf16_round(x)
    return x


def bits_equal(a: np.ndarray, b: np.ndarray) -> bool:
    return a.shape == b.shape and a.dtype == b.dtype and np.array_equal(
        a.view(np.uint8), b.view(np.uint8))
