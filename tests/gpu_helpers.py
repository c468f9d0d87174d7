"""Shared helpers for the GPU parity tests (host <-> device marshalling and
comparison utilities; no arithmetic of the method lives here)."""

from __future__ import annotations

import numpy as np
import torch

DEV = "cuda:0"


def dev(a: np.ndarray, dtype=None) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    """uint16 bf16 bit patterns -> a bfloat16 GPU tensor with exactly those bits."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def host(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy()
    return t.cpu().numpy()


def qkv_dev(wl):
    if wl.dtype == "bf16":
        return dev_bf16(wl.q), dev_bf16(wl.k), dev_bf16(wl.v)
    return dev(wl.q), dev(wl.k), dev(wl.v)


def sample_rows(Lq: int, n: int, seed: int = 0) -> np.ndarray:
    """First, last and ragged-tail rows plus a seeded random sample."""
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 31, 32, 127, 128, Lq // 2, Lq - 129, Lq - 128, Lq - 2, Lq - 1]
    fixed = [r for r in fixed if 0 <= r < Lq]
    rest = rng.choice(Lq, size=min(n, Lq), replace=False)
    return np.unique(np.concatenate([fixed, rest])).astype(np.int64)


def same_bits_f32(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Elementwise: identical fp32 values, NaN equal to NaN."""
    a = np.asarray(a, np.float32)
    b = np.asarray(b, np.float32)
    return (a.view(np.uint32) == b.view(np.uint32)) | (np.isnan(a) & np.isnan(b))


_HIP = None


def read_device(ptr: int, nbytes: int) -> np.ndarray:
    """Bytes at a raw device pointer (after the work producing them has finished)."""
    global _HIP
    import ctypes
    if _HIP is None:
        _HIP = ctypes.CDLL("libamdhip64.so")
        _HIP.hipMemcpy.restype = ctypes.c_int
        _HIP.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    out = np.empty(nbytes, np.uint8)
    if nbytes:
        assert _HIP.hipMemcpy(out.ctypes.data, ptr, nbytes, 2) == 0  # device to host
    return out
