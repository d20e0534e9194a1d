"""Helpers shared by the GPU parity tests (device plumbing and comparison only)."""
import numpy as np
import pytest
import torch

TOL = 2e-3   # relative L2 error bound for fp32-accumulated outputs

needs_gpu = pytest.mark.skipif(not torch.cuda.is_available(), reason="needs an MI355X")


def rel_l2(y, yo) -> float:
    y = np.asarray(y, dtype=np.float64)
    yo = np.asarray(yo, dtype=np.float64)
    den = np.linalg.norm(yo)
    num = np.linalg.norm(y - yo)
    return float(num / den) if den > 0 else float(num)


def stream():
    return torch.cuda.current_stream()


def zeros_u8(n):
    return torch.zeros(max(1, n), dtype=torch.uint8, device="cuda")


def f32_bits(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float32).view(np.uint32)


def sample_rows(M, n=64, seed=0):
    """First, last and n spread rows of an M-row matrix."""
    if M <= n + 2:
        return np.arange(M)
    rng = np.random.default_rng(seed + M)
    return np.unique(np.concatenate([[0, 1, M - 2, M - 1], rng.choice(M, n, replace=False)]))
