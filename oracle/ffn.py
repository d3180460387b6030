"""Routed-expert output of one MoE layer on this GPU, in float64.
Test infrastructure only (see package docstring).

What is computed (Appendix C, "Grouped FFN invocations" and "Output return
and combine"; Section 3.2):

    y[r,t] = sum over slots s ascending with local expert e = id[r,t,s] >= 0 of
             w[r,t,s] * ( (silu(x[r,t] Wg[e]) * (x[r,t] Wu[e])) Wd[e] )

with silu(z) = z / (1 + exp(-z)).  The expert FFN is two GEMMs with the
activation (and, for FP8 models, a quantisation) between them; each routed
contribution is weighted by its routing coefficient exactly once and summed
at the source token.  Tokens with no local slot get y = 0.  Nothing here
depends on how tokens were chunked, batched or ordered on arrival.

Readings where the paper is silent:

* the activation is SwiGLU (silu on the gate projection, times the up
  projection), no clamp -- the paper never names it;
* ``h_mode`` mirrors the dtype the second GEMM consumes: None keeps h in
  float64, "bf16" rounds h to bfloat16 (nearest, ties to even), "fp8"
  rounds h to float32 then quantises it per (row, 128 columns) exactly like
  the activations (see ``oracle.fp8``), "mxfp8" rounds h to float32 then
  quantises it to MXFP8 per (row, 32 columns) (see ``oracle.mx``);
* ``x_mode`` "fp8" quantises each input row per 128 channels before the
  first GEMM (the "activations with their quantization metadata" the layout
  transform packs), "mxfp8" to MXFP8 per 32 channels, else inputs are used
  exactly;
* ``y_mode`` "bf16" rounds each weighted expert output w * y to bfloat16
  before the slot-order sum (the dtype in which an expert-parallel combine
  returns outputs to their source); None keeps it in float64;
* the result is rounded once to float32 at the end.
"""
from __future__ import annotations

import numpy as np

from . import fp8 as _fp8
from . import mx as _mx


def bf16_bits_to_f64(bits) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64: bf16 is the upper half of
    an IEEE binary32 pattern."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def round_bf16(v) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value (ties to even),
    returned as float64.  bfloat16 keeps 8 significant bits, normal
    exponents down to 2^-126 (quantum 2^-133 below that)."""
    v = np.asarray(v, dtype=np.float64)
    _, e = np.frexp(v)                        # v = m * 2^e, 0.5 <= |m| < 1
    e = np.maximum(e, -125)
    q = np.ldexp(v, 8 - e)                    # 8 significant bits before the point
    return np.ldexp(np.rint(q), e - 8)        # rint: nearest, ties to even


def silu(z):
    return z / (1.0 + np.exp(-z))


def expert_ffn(x: np.ndarray, wg: np.ndarray, wu: np.ndarray, wd: np.ndarray,
               h_mode=None) -> np.ndarray:
    """One expert on rows x [n][d]: GEMM (gate, up), SwiGLU, GEMM (down)."""
    g = x @ wg
    u = x @ wu
    h = silu(g) * u
    if h_mode == "bf16":
        h = round_bf16(h)
    elif h_mode == "fp8":
        codes, scale = _fp8.quantize_blocks(h.astype(np.float32))
        h = _fp8.dequantize_blocks(codes, scale)
    elif h_mode == "mxfp8":
        codes, scode = _mx.quantize_mxfp8(h.astype(np.float32))
        h = _mx.dequantize_mxfp8(codes, scode)
    elif h_mode is not None:
        raise ValueError(h_mode)
    return h @ wd


class ExpertBank:
    """float64 expert weights in math orientation, decoded once per expert.

    kind "f32": float32 arrays; "bf16": uint16 bit patterns; "fp8": uint8
    e4m3 codes with one float32 scale per 128x128 block.
    gate/up are [E][d][I], down is [E][I][d]; fp8 scales are
    [E][d/128][I/128] and [E][I/128][d/128].
    kind "mxfp4": stored output-major with K packed, as MX checkpoints keep
    linear layers: gate/up codes [E][I][d/2] with E8M0 scales [E][I][d/32],
    down codes [E][d][I/2] with scales [E][d][I/32]; decoded and transposed
    to math orientation here.
    """

    def __init__(self, kind, w_gate, w_up, w_down, s_gate=None, s_up=None, s_down=None):
        self.kind = kind
        self.w = (w_gate, w_up, w_down)
        self.s = (s_gate, s_up, s_down)
        self._cache = {}

    def _dec(self, a, s):
        if self.kind == "f32":
            return np.asarray(a, np.float32).astype(np.float64)
        if self.kind == "bf16":
            return bf16_bits_to_f64(a)
        if self.kind == "fp8":
            return _fp8.dequantize_weight(np.asarray(a, np.uint8), np.asarray(s, np.float32))
        if self.kind == "mxfp4":
            return _mx.dequantize_mxfp4(np.asarray(a, np.uint8), np.asarray(s, np.uint8)).T
        raise ValueError(self.kind)

    def __call__(self, e: int):
        if e not in self._cache:
            self._cache[e] = tuple(
                self._dec(w[e], None if s is None else s[e]) for w, s in zip(self.w, self.s))
        return self._cache[e]


def decode_rows(x, kind) -> np.ndarray:
    """Input rows -> float64 (kind "f32": float32 values, "bf16": bit patterns)."""
    if kind == "bf16":
        return bf16_bits_to_f64(x)
    return np.asarray(x, np.float32).astype(np.float64)


def routed_output(x64: np.ndarray, ids: np.ndarray, w: np.ndarray, bank, n_experts: int,
                  h_mode=None, x_mode=None, y_mode=None, group: int = 1024) -> np.ndarray:
    """y for token rows x64 [n][d] (float64) with local ids [n][k] (-1 =
    remote) and coefficients w [n][k]; returns float32 [n][d]."""
    x64 = np.asarray(x64, np.float64)
    ids = np.asarray(ids)
    w = np.asarray(w, np.float32).astype(np.float64)
    n, d = x64.shape
    k = ids.shape[1]
    out = np.zeros((n, d), np.float32)
    for lo in range(0, n, group):
        hi = min(n, lo + group)
        xg = x64[lo:hi]
        if x_mode == "fp8":
            codes, scale = _fp8.quantize_blocks(xg.astype(np.float32))
            xg = _fp8.dequantize_blocks(codes, scale)
        elif x_mode == "mxfp8":
            codes, scode = _mx.quantize_mxfp8(xg.astype(np.float32))
            xg = _mx.dequantize_mxfp8(codes, scode)
        elif x_mode is not None:
            raise ValueError(x_mode)
        idg, wgt = ids[lo:hi], w[lo:hi]
        contrib = np.zeros((hi - lo, k, d), np.float64)
        for e in range(n_experts):
            rows, slots = np.nonzero(idg == e)
            if rows.size == 0:
                continue
            wg_, wu_, wd_ = bank(e)
            y = wgt[rows, slots][:, None] * expert_ffn(xg[rows], wg_, wu_, wd_, h_mode)
            if y_mode == "bf16":
                y = round_bf16(y)
            elif y_mode is not None:
                raise ValueError(y_mode)
            contrib[rows, slots] = y
        acc = np.zeros((hi - lo, d), np.float64)
        for s in range(k):                         # ascending slot order
            m = idg[:, s] >= 0
            acc[m] = acc[m] + contrib[m, s]
        out[lo:hi] = acc.astype(np.float32)
    return out


def brute_force_token(x, ids, w, wg, wu, wd, h_round=None):
    """Scalar triple loops for one token (pure Python floats), for tiny
    shapes only.  wg/wu/wd: per-expert nested lists or arrays in math
    orientation.  h_round: optional scalar rounding applied to each h."""
    d = len(x)
    y = [0.0] * d
    for s, e in enumerate(ids):
        if e < 0:
            continue
        I = len(wg[e][0])
        h = []
        for j in range(I):
            g = sum(float(x[i]) * float(wg[e][i][j]) for i in range(d))
            u = sum(float(x[i]) * float(wu[e][i][j]) for i in range(d))
            hv = g / (1.0 + np.exp(-g)) * u
            h.append(h_round(hv) if h_round else hv)
        for c in range(d):
            yc = sum(h[j] * float(wd[e][j][c]) for j in range(I))
            y[c] += float(w[s]) * yc
    return y
