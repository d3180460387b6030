"""OCP FP8 E4M3 ("e4m3fn") codec and 1x128 block quantisation, from the format
definition.  Test infrastructure only (see package docstring).

The paper runs routed experts in FP8 for GLM-5.3 (Section 4.1, "Models and
environments") and states that the layout transform packs activations
"together with their quantization metadata" and that an activation and
quantization step sits between the two expert GEMMs (Appendix C, "Grouped FFN
invocations").  It does not state the block size or scale rule; the reading
used here is one float32 scale per (row, 128 consecutive channels),
scale = amax / 448 (1 for an all-zero block), codes = e4m3(value / scale)
rounded to nearest, ties to even, saturating at +-448.  Both divisions are
float32 IEEE divisions (the precision the kernel works in).

E4M3 (OCP 8-bit floating point, "fn" variant): 1 sign bit, 4 exponent bits
with bias 7, 3 mantissa bits; exponent field 0 encodes subnormals
m * 2^-9; the all-ones pattern S.1111.111 is NaN; there are no infinities;
the largest finite magnitude is 1.75 * 2^8 = 448.
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0
BLOCK = 128


def decode(codes) -> np.ndarray:
    """float64 values of uint8 e4m3fn codes (NaN for 0x7F / 0xFF)."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    exp = (c >> 3) & 0xF
    man = c & 0x7
    sub = man.astype(np.float64) * 2.0 ** -9                     # exp field 0
    nor = (1.0 + man / 8.0) * np.exp2(exp.astype(np.float64) - 7.0)
    val = np.where(exp == 0, sub, nor)
    val = np.where((exp == 0xF) & (man == 0x7), np.nan, val)
    return sign * val


def _finite_table():
    """Sorted non-negative finite magnitudes and their codes (0x00..0x7E)."""
    codes = np.arange(0, 0x7F, dtype=np.uint8)
    return decode(codes), codes


_MAGS, _CODES = _finite_table()


def encode(values) -> np.ndarray:
    """Round float values to e4m3fn codes: nearest finite value, ties to the
    code with an even mantissa, magnitudes above 448 saturate to 448, NaN
    maps to 0x7F.  Zero keeps its sign bit."""
    v = np.asarray(values, dtype=np.float64)
    a = np.abs(v)
    sat = np.minimum(a, E4M3_MAX)
    hi = np.searchsorted(_MAGS, sat, side="left")        # first mag >= a
    hi = np.clip(hi, 0, len(_MAGS) - 1)
    lo = np.clip(hi - 1, 0, len(_MAGS) - 1)
    d_lo = sat - _MAGS[lo]
    d_hi = _MAGS[hi] - sat
    take_hi = (d_hi < d_lo) | ((d_hi == d_lo) & ((_CODES[hi] & 1) == 0))
    idx = np.where(take_hi, hi, lo)
    code = _CODES[idx].astype(np.uint8)
    code = np.where(np.signbit(v), code | 0x80, code).astype(np.uint8)
    return np.where(np.isnan(v), np.uint8(0x7F), code).astype(np.uint8)


def quantize_blocks(x32: np.ndarray):
    """1x128 block quantisation of float32 rows [n][c] (c divisible by 128).

    Returns (codes uint8 [n][c], scales float32 [n][c/128]) with
    scale = amax/448 in float32 (1 when amax is 0) and code = e4m3(x/scale),
    the division done in float32.
    """
    x32 = np.asarray(x32, dtype=np.float32)
    n, c = x32.shape
    assert c % BLOCK == 0
    xb = x32.reshape(n, c // BLOCK, BLOCK)
    amax = np.abs(xb).max(axis=2)
    scale = np.where(amax > 0, (amax / np.float32(E4M3_MAX)).astype(np.float32),
                     np.float32(1.0)).astype(np.float32)
    ratio = (xb / scale[:, :, None]).astype(np.float32)
    codes = encode(ratio).reshape(n, c)
    return codes, scale


def dequantize_blocks(codes: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """float64 values of 1x128 block-quantised rows."""
    n, c = codes.shape
    v = decode(codes).reshape(n, c // BLOCK, BLOCK)
    return (v * scale.astype(np.float64)[:, :, None]).reshape(n, c)


def dequantize_weight(codes: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """float64 values of one [rows][cols] weight matrix with one scale per
    128x128 block (scale shape [rows/128][cols/128])."""
    r, c = codes.shape
    # the values of all 256 codes, looked up per element (the same values as
    # decode() of each code; a weight matrix has tens of millions of codes)
    v = _code_values()[np.asarray(codes, dtype=np.uint8)].reshape(r // BLOCK, BLOCK,
                                                                 c // BLOCK, BLOCK)
    return (v * scale.astype(np.float64)[:, None, :, None]).reshape(r, c)


_VALUES = None


def _code_values() -> np.ndarray:
    """decode() of codes 0..255, computed once."""
    global _VALUES
    if _VALUES is None:
        _VALUES = decode(np.arange(256, dtype=np.uint8))
    return _VALUES
