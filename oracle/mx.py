"""OCP Microscaling (MX) formats used by the MXFP4 expert path, written from
the format definitions.  Test infrastructure only (see package docstring).

The paper keeps the routed-expert weights of its DeepSeek-V4 models in MXFP4
(Section 4.1, "Models and environments") and, for quantised experts, places
an activation-quantisation step between the two expert GEMMs (Appendix C,
"Grouped FFN invocations").  It states no block size, scale rule or
activation format; the readings used here are those of the OCP Microscaling
Formats (MX) v1.0 specification:

* an MX block is 32 consecutive elements along the contraction (K) axis that
  share one E8M0 scale X = 2^(code - 127);
* MXFP4 elements are E2M1: 1 sign bit, 2 exponent bits with bias 1, 1
  mantissa bit; exponent field 0 encodes the subnormal m * 0.5, so the
  magnitudes are 0, 0.5, 1, 1.5, 2, 3, 4, 6; two elements per byte, the
  element with the even index in the low nibble;
* activations and h are MXFP8 (E4M3 elements, ``oracle.fp8``) quantised with
  the specification's conversion: shared exponent
  floor(log2(amax)) - emax_elem, emax_elem = 8 for E4M3, clamped to the
  E8M0 range (an all-zero block gets code 0), each element
  e4m3(v / X) rounded to nearest, ties to even, saturating at +-448.
  floor(log2(amax)) is taken from the float32 amax.
"""
from __future__ import annotations

import numpy as np

from . import fp8 as _fp8

BLOCK = 32
E4M3_EMAX = 8
_E2M1_MAG = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def e2m1_decode(codes) -> np.ndarray:
    """float64 values of 4-bit E2M1 codes (0..15) from the field layout."""
    c = np.asarray(codes).astype(np.int64)
    sign = np.where(c & 0x8, -1.0, 1.0)
    exp = (c >> 1) & 0x3
    man = (c & 0x1).astype(np.float64)
    sub = man * 0.5                                          # exponent field 0
    nor = (1.0 + man / 2.0) * np.exp2(exp.astype(np.float64) - 1.0)
    return sign * np.where(exp == 0, sub, nor)


def e8m0_decode(codes) -> np.ndarray:
    """float64 values 2^(c - 127) of E8M0 scale codes (0xFF is NaN)."""
    c = np.asarray(codes).astype(np.int64)
    v = np.exp2(c.astype(np.float64) - 127.0)
    return np.where(c == 0xFF, np.nan, v)


def unpack_fp4(packed) -> np.ndarray:
    """uint8 [..., n] holding two E2M1 codes each -> int codes [..., 2n];
    element 2j is the low nibble of byte j."""
    p = np.asarray(packed, dtype=np.uint8)
    out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), np.int64)
    out[..., 0::2] = p & 0x0F
    out[..., 1::2] = p >> 4
    return out


def dequantize_mxfp4(packed, scales) -> np.ndarray:
    """float64 [rows][K] of an MXFP4 matrix stored as packed codes
    [rows][K/2] and E8M0 scales [rows][K/32] (blocks along K)."""
    v = e2m1_decode(unpack_fp4(packed))
    rows, K = v.shape
    s = e8m0_decode(scales)
    assert s.shape == (rows, K // BLOCK)
    return (v.reshape(rows, K // BLOCK, BLOCK) * s[:, :, None]).reshape(rows, K)


def _floor_log2_f32(a32: np.ndarray) -> np.ndarray:
    """floor(log2(a)) of non-negative float32 values; -127 for 0 (and
    anything below the normal range clamps there later)."""
    m, e = np.frexp(a32.astype(np.float64))     # a = m * 2^e, 0.5 <= m < 1
    return np.where(a32 > 0, e - 1, -127)


def quantize_mxfp8(x32: np.ndarray):
    """MXFP8 (E4M3) quantisation of float32 rows [n][c] (c divisible by 32)
    along the row.  Returns (codes uint8 [n][c], scale codes uint8 [n][c/32])."""
    x32 = np.asarray(x32, dtype=np.float32)
    n, c = x32.shape
    assert c % BLOCK == 0
    xb = x32.reshape(n, c // BLOCK, BLOCK)
    amax = np.abs(xb).max(axis=2)
    shared = _floor_log2_f32(amax) - E4M3_EMAX
    scode = np.clip(shared + 127, 0, 254).astype(np.uint8)
    ratio = xb.astype(np.float64) / e8m0_decode(scode)[:, :, None]  # exact: power of two
    codes = _fp8.encode(ratio).reshape(n, c)                          # saturates at 448
    return codes, scode


def dequantize_mxfp8(codes, scode) -> np.ndarray:
    """float64 values of MXFP8 rows (codes [n][c], scale codes [n][c/32])."""
    codes = np.asarray(codes, np.uint8)
    n, c = codes.shape
    v = _fp8.decode(codes).reshape(n, c // BLOCK, BLOCK)
    return (v * e8m0_decode(scode)[:, :, None]).reshape(n, c)
