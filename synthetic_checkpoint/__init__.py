"""Seeded synthetic checkpoint values, shared by the GPU path's tests and the oracle.

This module only makes input data. It holds none of the resharding method's
arithmetic: no layouts, no plan, no casts. The method's casts (fp32 -> bf16
round-to-nearest-even, bf16 -> fp8 e4m3) live in the oracle and in the HIP
kernels; values here are produced directly in the trainer's dtype.

Definition (the same on every device, bit for bit):

  key_t       = mix32((25442 * 1000003 + t) mod 2^32)          t = checkpoint tensor index
  a, b        = mix32((2n) ^ key_t), mix32((2n + 1) ^ key_t)   n = row-major flat element index
  s           = lo16(a) + hi16(a) + lo16(b) + hi16(b)          Irwin-Hall sum of four u16, in [0, 262140]
  x (fp32)    = fp32(s - 131070) * SCALE                       one IEEE fp32 multiply
  bf16 value  = the high 16 bits of x's fp32 encoding          (truncation, a generator choice)

mix32 is a three-round xor-shift-multiply finaliser with multipliers below
2^31, so every intermediate product fits in a signed 64-bit integer on any
backend. SCALE makes the standard deviation 0.02: the sum of four independent
uniforms on {0..65535} has variance 4 * (65536^2 - 1) / 12.

torch (CPU or GPU, bulk) and numpy (CPU, any subset of indices) evaluate the
same integer expression and the same single fp32 multiply, so both give
identical bits.
"""

from __future__ import annotations

import math

import numpy as np

__all__ = [
    "SEED_BASE",
    "SCALE",
    "tensor_key",
    "values_numpy",
    "values_torch",
    "DTYPE_BYTES",
]

SEED_BASE = 25442 * 1000003
_M32 = 0xFFFFFFFF
_C1 = 0x21F0AAAD
_C2 = 0x735A2D97
SCALE = np.float32(0.02 / math.sqrt(4.0 * (65536.0 ** 2 - 1.0) / 12.0))

DTYPE_BYTES = {"f32": 4, "bf16": 2}


def _mix32_int(x: int) -> int:
    x &= _M32
    x ^= x >> 16
    x = (x * _C1) & _M32
    x ^= x >> 15
    x = (x * _C2) & _M32
    x ^= x >> 15
    return x


def tensor_key(t: int) -> int:
    """32-bit key of checkpoint tensor number ``t``."""
    return _mix32_int((SEED_BASE + int(t)) & _M32)


def _mix32_np(x: np.ndarray) -> np.ndarray:
    x = x ^ (x >> 16)
    x = (x * _C1) & _M32
    x = x ^ (x >> 15)
    x = (x * _C2) & _M32
    x = x ^ (x >> 15)
    return x


def values_numpy(t: int, flat_index, dtype: str) -> np.ndarray:
    """Raw bit patterns of tensor ``t`` at the given row-major flat indices.

    Returns uint32 codes for ``dtype == "f32"`` and uint16 codes for ``"bf16"``.
    """
    n = np.asarray(flat_index, dtype=np.int64)
    if n.size and (n.min() < 0 or n.max() >= (1 << 31)):
        raise ValueError("flat index out of range")
    key = np.int64(tensor_key(t))
    a = _mix32_np(((2 * n) & _M32) ^ key)
    b = _mix32_np(((2 * n + 1) & _M32) ^ key)
    s = (a & 0xFFFF) + (a >> 16) + (b & 0xFFFF) + (b >> 16)
    x = (s - 131070).astype(np.float32) * SCALE
    bits = x.view(np.uint32)
    if dtype == "f32":
        return bits
    if dtype == "bf16":
        return (bits >> 16).astype(np.uint16)
    raise ValueError(f"unsupported trainer dtype {dtype!r}")


def values_torch(t: int, rows: int, cols: int, dtype: str, device="cpu", start: int = 0, count: int | None = None):
    """Tensor ``t`` (shape [rows, cols]) in the trainer dtype, built with torch ops.

    With ``start``/``count`` only the flat range [start, start+count) is built
    and returned as a 1-D tensor. Integer work is done in int64 chunks so that
    very large tensors do not need eight bytes of scratch per element at once.
    """
    import torch

    numel = rows * cols
    if count is None:
        count = numel - start
    if start < 0 or start + count > numel or numel >= (1 << 31):
        raise ValueError("range out of tensor")
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]
    out = torch.empty(count, dtype=tdt, device=device)
    key = tensor_key(t)
    scale = torch.tensor(float(SCALE), dtype=torch.float32, device=device)
    chunk = 1 << 26
    for c0 in range(0, count, chunk):
        c1 = min(count, c0 + chunk)
        n = torch.arange(start + c0, start + c1, dtype=torch.int64, device=device)
        a = _mix32_t(((2 * n) & _M32) ^ key)
        b = _mix32_t(((2 * n + 1) & _M32) ^ key)
        del n
        s = (a & 0xFFFF) + (a >> 16) + (b & 0xFFFF) + (b >> 16)
        del a, b
        x = (s - 131070).to(torch.float32) * scale
        del s
        if dtype == "f32":
            out[c0:c1] = x
        else:
            hi = (x.view(torch.int32) >> 16).to(torch.int16)
            out[c0:c1] = hi.view(torch.bfloat16)
    if count == numel and start == 0:
        return out.view(rows, cols)
    return out


def _mix32_t(x):
    x = x ^ (x >> 16)
    x = (x * _C1) & _M32
    x = x ^ (x >> 15)
    x = (x * _C2) & _M32
    x = x ^ (x >> 15)
    return x
