"""Helpers shared by the GPU parity tests (device transfer and error norms)."""
import sys

import numpy as np


def torch_mod():
    import torch

    return torch


def gpu_available() -> bool:
    try:
        torch = torch_mod()
        return torch.cuda.is_available()
    except Exception:
        return False


def to_dev(x: np.ndarray):
    """complex64 -> complex64 tensor; (.., 2) float16 pairs -> float16 tensor."""
    torch = torch_mod()
    if x.dtype == np.complex64:
        return torch.from_numpy(np.ascontiguousarray(x)).cuda()
    if x.dtype == np.float16:
        return torch.from_numpy(np.ascontiguousarray(x)).cuda()
    raise TypeError(x.dtype)


def to_host(t) -> np.ndarray:
    return t.cpu().numpy()


def widen(y: np.ndarray) -> np.ndarray:
    """Stored result -> complex128 (binary16 pairs are widened exactly)."""
    if y.dtype == np.float16:
        y = y.astype(np.float64)
        return y[..., 0] + 1j * y[..., 1]
    return y.astype(np.complex128)


def rel_rows(y: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per-transform relative L2 error ||y - ref|| / ||ref|| over the last axis."""
    num = np.sqrt((np.abs(y - ref) ** 2).sum(-1))
    den = np.sqrt((np.abs(ref) ** 2).sum(-1))
    return num / den


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()
