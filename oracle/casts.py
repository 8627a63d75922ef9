"""Number-format conversions, written from the format definitions.

The paper assumes trainer and rollout precisions match and leaves conversion
to future work (Sec. 5, "Precision mismatch"); the workloads here add two
conversions in the assembly step:

* fp32 -> bf16, IEEE 754 round-to-nearest, ties to even. bf16 is the upper
  half of the binary32 encoding (1 sign, 8 exponent, 7 fraction bits).
* bf16/fp32 -> fp8 E4M3FN (OCP 8-bit floating point: 1 sign, 4 exponent bits
  with bias 7, 3 fraction bits, subnormals, no infinities, S.1111.111 is NaN,
  largest finite 448), round to nearest, ties to even, with a 128x128 blockwise
  scale: amax = max|x| over the block, s = fp32(amax) / 448 (IEEE fp32
  division; s = 1 when amax = 0), q = E4M3FN(fp32(x) / s).

Rounding is done by comparing exact distances to the two neighbouring
representable values (float64 holds every fp32, bf16 and E4M3 value and every
difference used here exactly), which is the definition of round-to-nearest.
Inputs must be finite.
"""

from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0


def bf16_to_f32(bits16: np.ndarray) -> np.ndarray:
    """bf16 codes -> fp32 codes (exact widening)."""
    return bits16.astype(np.uint32) << 16


def _bf16_value_unbounded(code: np.ndarray) -> np.ndarray:
    """Value of a non-negative bf16 code, reading the all-ones exponent as one
    more binade (so 0x7F80 stands for 2**128, the overflow threshold)."""
    e = (code >> 7).astype(np.int64)
    m = (code & 0x7F).astype(np.float64)
    sub = e == 0
    val = np.where(sub, m * 2.0 ** -133, (1.0 + m / 128.0) * np.exp2((e - 127).astype(np.float64)))
    return val


def f32_to_bf16(bits32: np.ndarray) -> np.ndarray:
    """fp32 codes -> bf16 codes, IEEE round to nearest even; overflow gives +-inf."""
    u = np.asarray(bits32, dtype=np.uint32)
    if np.any((u & 0x7F800000) == 0x7F800000):
        raise ValueError("non-finite input")
    sign = (u >> 31).astype(np.uint16)
    mag = u & 0x7FFFFFFF
    x = mag.view(np.float32).astype(np.float64)
    lo = (mag >> 16).astype(np.uint16)          # largest bf16 magnitude <= |x|
    hi = lo + np.uint16(1)                      # next magnitude up (0x7F80 = overflow)
    d_lo = x - _bf16_value_unbounded(lo)
    d_hi = _bf16_value_unbounded(hi) - x
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & ((lo & 1) == 1))
    code = np.where(pick_hi, hi, lo).astype(np.uint16)
    return code | (sign << np.uint16(15))


def _e4m3_table():
    """Values of the non-negative finite E4M3FN codes 0x00..0x7E (ascending)."""
    vals = []
    for c in range(0x7F):
        e, m = c >> 3, c & 7
        vals.append(m * 2.0 ** -9 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7))
    return np.array(vals, dtype=np.float64)


E4M3_VALUES = _e4m3_table()


def f64_to_e4m3(x: np.ndarray) -> np.ndarray:
    """Exact real values (float64 holding fp32 numbers) -> E4M3FN codes, round to
    nearest even. |x| must be below 464, the midpoint past the largest finite."""
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("non-finite input")
    a = np.abs(x)
    if np.any(a >= 464.0):
        raise ValueError("outside the finite E4M3FN rounding range")
    hi = np.searchsorted(E4M3_VALUES, a, side="left")      # first code with value >= a
    hi = np.minimum(hi, 0x7E)
    lo = np.where(E4M3_VALUES[hi] > a, hi - 1, hi)
    lo = np.maximum(lo, 0)
    d_lo = a - E4M3_VALUES[lo]
    d_hi = E4M3_VALUES[np.minimum(lo + 1, 0x7E)] - a
    exact = d_lo == 0
    up = ~exact & (lo < 0x7E) & ((d_hi < d_lo) | ((d_hi == d_lo) & ((lo & 1) == 1)))
    code = np.where(up, lo + 1, lo).astype(np.uint8)
    sign = np.signbit(x).astype(np.uint8) << 7
    return code | sign


def e4m3_to_f64(codes: np.ndarray) -> np.ndarray:
    c = np.asarray(codes, dtype=np.uint8)
    mag = c & 0x7F
    if np.any(mag == 0x7F):
        raise ValueError("NaN code")
    v = E4M3_VALUES[mag]
    return np.where(c >> 7, -v, v)


def block_scale(amax_f32: np.float32) -> np.float32:
    """s = fp32(amax) / 448 (IEEE fp32 division); 1 for an all-zero block."""
    a = np.float32(amax_f32)
    if a == 0:
        return np.float32(1.0)
    return np.float32(a / np.float32(E4M3_MAX))


def quantize_block(x_f32: np.ndarray):
    """One block of fp32 values -> (E4M3FN codes, fp32 scale)."""
    x = np.asarray(x_f32, dtype=np.float32)
    amax = np.float32(np.max(np.abs(x))) if x.size else np.float32(0)
    s = block_scale(amax)
    q = (x / s).astype(np.float32)            # elementwise IEEE fp32 division
    return f64_to_e4m3(q.astype(np.float64)), s


def quantize_matrix(x_f32: np.ndarray, block: int):
    """[rows, cols] fp32 matrix -> (codes [rows, cols], scales [ceil(rows/B), ceil(cols/B)]),
    blocks tiling the matrix from (0, 0); edge blocks are partial."""
    rows, cols = x_f32.shape
    nbr, nbc = -(-rows // block), -(-cols // block)
    codes = np.empty((rows, cols), dtype=np.uint8)
    scales = np.empty((nbr, nbc), dtype=np.float32)
    for bi in range(nbr):
        for bj in range(nbc):
            sl = (slice(bi * block, min(rows, (bi + 1) * block)), slice(bj * block, min(cols, (bj + 1) * block)))
            codes[sl], scales[bi, bj] = quantize_block(x_f32[sl])
    return codes, scales
