"""Helpers shared by the parity tests: moving the same bytes to both sides and
the error measures of the parity bar.  No FP8 arithmetic here."""
from __future__ import annotations

import numpy as np
import torch

# Parity bar for the matmuls: relative Frobenius error against the oracle's
# fp64-accumulated result rounded to the same output type.
REL_F_TOL = 1e-3


def np_bits(t: torch.Tensor) -> np.ndarray:
    """CPU view of a bf16 tensor as uint16 patterns, or of an fp32 tensor as float32."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.numpy()
    if t.dtype == torch.uint8:
        return t.numpy()
    raise TypeError(t.dtype)


def as_f64(a: np.ndarray) -> np.ndarray:
    """bf16 patterns (uint16) or float32 -> float64 values."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def rel_f(got: np.ndarray, ref: np.ndarray) -> float:
    g, r = as_f64(got), as_f64(ref)
    den = np.linalg.norm(r)
    num = np.linalg.norm(g - r)
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return float(num / den)


def sample_rows(n: int, k: int, seed: int) -> np.ndarray:
    """k distinct sorted row indices of [0, n), always including the first
    and the last row (the ragged tail of a tiled kernel)."""
    if n <= k:
        return np.arange(n)
    rng = np.random.default_rng(seed)
    rows = rng.choice(np.arange(1, n - 1), size=k - 2, replace=False)
    return np.sort(np.concatenate([[0, n - 1], rows]))


def i32(t: torch.Tensor) -> int:
    return int(t.item())


def u32(t: torch.Tensor) -> int:
    return int(t.item()) & 0xFFFFFFFF
