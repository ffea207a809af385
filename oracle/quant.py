"""FP8 (e4m3) weights for the FP8-weight variant.  This is not the paper's
precision: the method is orthogonal to quantization (Sec. 1), and the
variant exists to halve the weight bytes that normal steps stream.
Test infrastructure (part of the oracle): only tests, the smoke check and
the bench's CPU baseline use it.

Format (OCP FP8 E4M3): 1 sign bit, 4 exponent bits (bias 7), 3 mantissa
bits; exponent field 0 holds subnormals m * 2^-9; no infinities; the
largest finite magnitude is 448 (code 0x7E); 0x7F / 0xFF are NaN.

Quantization of a weight matrix W [N, K] (bf16 values), per output row n:
    s_n = max_k |W[n, k]| / 448            (float32; 1 for an all-zero row)
    q[n, k] = the e4m3 value nearest to W[n, k] / s_n (the quotient in
              float32), ties to the even code; magnitudes above 448 take 448
and the weight the model uses is q[n, k] * s_n (exact in float64).
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0


def e4m3_value(codes) -> np.ndarray:
    """Decode e4m3 codes (uint8) to float64 from the format definition."""
    c = np.asarray(codes, dtype=np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 7).astype(np.float64)
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7))
    mag = np.where((c & 0x7F) == 0x7F, np.nan, mag)
    return sign * mag


# the 127 finite non-negative values, codes 0x00..0x7E, in increasing order
_POS_CODES = np.arange(0x7F, dtype=np.int64)
_POS_VALUES = e4m3_value(_POS_CODES)
assert np.all(np.diff(_POS_VALUES) > 0)


def e4m3_encode(x) -> np.ndarray:
    """Nearest e4m3 code to each float32 value (ties to the even code, which
    is the even mantissa), saturating at 448; the sign of -0.0 is kept."""
    x = np.asarray(x, dtype=np.float32)
    ax = np.minimum(np.abs(x).astype(np.float64), E4M3_MAX)
    hi = np.clip(np.searchsorted(_POS_VALUES, ax, side="left"), 0, len(_POS_VALUES) - 1)
    lo = np.maximum(hi - 1, 0)
    d_lo = ax - _POS_VALUES[lo]
    d_hi = _POS_VALUES[hi] - ax
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (_POS_CODES[hi] % 2 == 0))
    code = np.where(pick_hi, _POS_CODES[hi], _POS_CODES[lo])
    return (code | np.where(np.signbit(x), 0x80, 0)).astype(np.uint8)


def quantize_rows(w) -> tuple:
    """(codes uint8 [N, K], scales float32 [N]) of a weight matrix, per row."""
    w = np.asarray(w, dtype=np.float32)
    amax = np.abs(w).max(axis=1)
    scale = np.where(amax > 0, amax / np.float32(E4M3_MAX), np.float32(1.0)).astype(np.float32)
    return e4m3_encode(w / scale[:, None]), scale


def dequantize_rows(codes, scale) -> np.ndarray:
    """The weights the FP8 model computes with, float64 [N, K]."""
    return e4m3_value(codes) * np.asarray(scale, dtype=np.float64)[:, None]
