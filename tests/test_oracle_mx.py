"""Pins for the oracle's MX formats (CPU only).

E2M1 decode is checked against the hand-derived code table of the OCP MX
specification (tests/golden/e2m1_values.txt), E8M0 against torch's
float8_e8m0fnu, the packed MXFP4 matrix decode against a scalar loop over
that table, and MXFP8 quantisation against torch's float8_e4m3fn cast and the
defining property of the shared exponent (block amax / X in [256, 512)).
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import ffn, mx

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e2m1_values.txt")


def _table():
    t = {}
    for line in open(GOLDEN):
        line = line.split("#")[0].split()
        if line:
            t[int(line[0])] = float(line[1])
    assert sorted(t) == list(range(16))
    return t


def test_e2m1_decode_matches_code_table():
    t = _table()
    got = mx.e2m1_decode(np.arange(16))
    for c in range(16):
        assert got[c] == t[c] and math.copysign(1, got[c]) == math.copysign(1, t[c]), c


def test_e8m0_decode_matches_torch():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e8m0fnu).to(torch.float64).numpy()
    ours = mx.e8m0_decode(codes)
    nan = np.isnan(ref)
    assert nan.tolist() == [c == 255 for c in range(256)]
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])


def test_unpack_low_nibble_first():
    b = np.array([[0x21, 0xF0, 0x7A]], np.uint8)
    assert mx.unpack_fp4(b).tolist() == [[1, 2, 0, 15, 10, 7]]


def _loop_dequant(packed, scales, table):
    rows, half = packed.shape
    out = np.zeros((rows, 2 * half))
    for r in range(rows):
        for k in range(2 * half):
            nib = (int(packed[r, k // 2]) >> (4 * (k % 2))) & 15
            out[r, k] = table[nib] * 2.0 ** (int(scales[r, k // 32]) - 127)
    return out


def test_dequantize_mxfp4_matches_scalar_loop():
    rng = np.random.default_rng(3)
    packed = rng.integers(0, 256, size=(5, 48), dtype=np.uint8)        # K = 96
    scales = rng.integers(110, 140, size=(5, 3), dtype=np.uint8)
    assert np.array_equal(mx.dequantize_mxfp4(packed, scales),
                          _loop_dequant(packed, scales, _table()))


def _rand_rows(rng, n, c):
    x = rng.standard_normal((n, c)).astype(np.float32)
    # spread block magnitudes over many binades, include exact powers of two
    x *= np.exp2(rng.integers(-20, 20, size=(n, c // 32, 1))).repeat(32, axis=2).reshape(n, c)
    x[0, :32] = 0.0
    x[1, 32:64] = 0.0
    x[1, 40] = 256.0
    x[2, :32] = np.float32(2.0 ** -130)     # float32 subnormal block
    return x


def test_mxfp8_shared_exponent_property():
    rng = np.random.default_rng(5)
    x = _rand_rows(rng, 12, 256)
    codes, sc = mx.quantize_mxfp8(x)
    assert codes.dtype == np.uint8 and sc.shape == (12, 8)
    for r in range(12):
        for b in range(8):
            amax = float(np.abs(x[r, 32 * b:32 * b + 32]).max())
            X = 2.0 ** (int(sc[r, b]) - 127)
            if amax == 0.0:
                assert sc[r, b] == 0
            elif amax >= 2.0 ** -119:        # shared exponent above the E8M0 floor
                assert 256.0 <= amax / X < 512.0, (r, b, amax, X)
            else:
                assert sc[r, b] == 0


def test_mxfp8_elements_match_torch_cast():
    rng = np.random.default_rng(6)
    x = _rand_rows(rng, 16, 512)
    codes, sc = mx.quantize_mxfp8(x)
    X = np.exp2(sc.astype(np.float64) - 127).repeat(32, axis=1)
    ratio = np.clip(x.astype(np.float64) / X, -448.0, 448.0)
    ref = torch.from_numpy(ratio.astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8)
    got = codes.copy()
    # torch keeps the sign of zero; so does the oracle
    assert np.array_equal(got, ref.numpy())


def test_mxfp8_error_bound_and_saturation():
    rng = np.random.default_rng(8)
    x = _rand_rows(rng, 16, 256)
    codes, sc = mx.quantize_mxfp8(x)
    deq = mx.dequantize_mxfp8(codes, sc)
    X = np.exp2(sc.astype(np.float64) - 127).repeat(32, axis=1)
    ratio = np.abs(x.astype(np.float64)) / X
    normal = (ratio >= 2.0 ** -6) & (ratio <= 448.0)
    err = np.abs(deq - x)
    assert (err[normal] <= 2.0 ** -4 * np.abs(x[normal]) + 0.0).all()
    sat = ratio > 448.0
    assert sat.any()
    assert np.array_equal(np.abs(deq[sat]), 448.0 * X[sat])


def test_mxfp8_power_of_two_invariance():
    rng = np.random.default_rng(9)
    x = rng.standard_normal((4, 128)).astype(np.float32)
    c0, s0 = mx.quantize_mxfp8(x)
    for j in (-5, 3, 17):
        c1, s1 = mx.quantize_mxfp8((x * np.float32(2.0 ** j)).astype(np.float32))
        assert np.array_equal(c0, c1)
        assert np.array_equal(s1.astype(int), s0.astype(int) + j)


def _torch_mxfp8(v):
    """MXFP8 by search: the smallest power of two X with amax / X < 512,
    elements by torch's e4m3 cast of the saturated ratio."""
    v = np.asarray(v, np.float32)
    out = np.zeros(v.shape)
    for r in range(v.shape[0]):
        for b in range(v.shape[1] // 32):
            blk = v[r, 32 * b:32 * b + 32].astype(np.float64)
            amax = np.abs(blk).max()
            e = -127
            while amax / 2.0 ** e >= 512.0:
                e += 1
            q = torch.from_numpy(np.clip(blk / 2.0 ** e, -448, 448).astype(np.float32))
            out[r, 32 * b:32 * b + 32] = q.to(torch.float8_e4m3fn).to(torch.float64).numpy() * 2.0 ** e
    return out


def test_ffn_mxfp4_weights_brute_force():
    # MXFP4 expert bank vs the scalar-loop decode fed to the brute-force token
    # loop: catches a transposed operand or a swapped nibble order
    rng = np.random.default_rng(12)
    E, d, I, k = 3, 64, 96, 2
    wg = rng.integers(0, 256, size=(E, I, d // 2), dtype=np.uint8)
    wu = rng.integers(0, 256, size=(E, I, d // 2), dtype=np.uint8)
    wd = rng.integers(0, 256, size=(E, d, I // 2), dtype=np.uint8)
    sg = rng.integers(118, 124, size=(E, I, d // 32), dtype=np.uint8)
    su = rng.integers(118, 124, size=(E, I, d // 32), dtype=np.uint8)
    sd = rng.integers(118, 124, size=(E, d, I // 32), dtype=np.uint8)
    bank = ffn.ExpertBank("mxfp4", wg, wu, wd, sg, su, sd)
    t = _table()
    dec = [(_loop_dequant(wg[e], sg[e], t).T, _loop_dequant(wu[e], su[e], t).T,
            _loop_dequant(wd[e], sd[e], t).T) for e in range(E)]
    x = rng.standard_normal((4, d))
    ids = np.array([[0, 2], [1, -1], [-1, -1], [2, 1]])
    w = rng.random((4, k)).astype(np.float32)
    got = ffn.routed_output(x, ids, w, bank, E)
    for n in range(4):
        ref = ffn.brute_force_token(x[n], ids[n], w[n], [q[0] for q in dec], [q[1] for q in dec],
                                    [q[2] for q in dec])
        np.testing.assert_allclose(got[n], np.array(ref, np.float32), rtol=1e-5, atol=1e-6)


def test_ffn_mxfp8_modes_match_search_quantiser():
    rng = np.random.default_rng(13)
    d, I = 64, 64
    wg, wu = rng.standard_normal((d, I)) * 0.1, rng.standard_normal((d, I)) * 0.1
    wd = rng.standard_normal((I, d)) * 0.1
    x = rng.standard_normal((6, d)).astype(np.float32).astype(np.float64)
    got = ffn.expert_ffn(_torch_mxfp8(x), wg, wu, wd, h_mode="mxfp8")
    h = ffn.silu(_torch_mxfp8(x) @ wg) * (_torch_mxfp8(x) @ wu)
    ref = _torch_mxfp8(h.astype(np.float32)) @ wd
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-14)
    # x_mode quantises the rows exactly like the search quantiser
    ids = np.zeros((6, 1), np.int64)
    bank = ffn.ExpertBank("f32", wg[None].astype(np.float32), wu[None].astype(np.float32),
                          wd[None].astype(np.float32))
    wg32, wu32, wd32 = bank(0)
    y = ffn.routed_output(x, ids, np.ones((6, 1), np.float32), bank, 1, h_mode="mxfp8",
                          x_mode="mxfp8")
    xq = _torch_mxfp8(x)
    hq = _torch_mxfp8((ffn.silu(xq @ wg32) * (xq @ wu32)).astype(np.float32))
    np.testing.assert_allclose(y, (hq @ wd32).astype(np.float32), rtol=1e-6, atol=1e-7)
