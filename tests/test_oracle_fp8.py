"""Pins for the oracle's e4m3 codec and 1x128 block quantisation (CPU only).

The codec is checked against hand-derived codes from the OCP FP8 definition
(tests/golden/e4m3_codes.txt), against torch's float8_e4m3fn on every code and
on the rounding midpoints, and against properties of round-to-nearest-even.
"""
import math
import os

import numpy as np
import pytest
import torch

from oracle import fp8

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_codes():
    rows = []
    with open(os.path.join(GOLDEN, "e4m3_codes.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            c, v = line.split()
            rows.append((int(c, 16), float(v)))
    return rows


def test_decode_hand_derived_codes():
    for code, val in _golden_codes():
        got = fp8.decode(np.array([code], np.uint8))[0]
        if math.isnan(val):
            assert math.isnan(got), hex(code)
        else:
            assert got == val and math.copysign(1, got) == math.copysign(1, val), hex(code)


def test_decode_all_codes_match_torch():
    codes = np.arange(256, dtype=np.uint8)
    ours = fp8.decode(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.nanmax(ours) == 448.0 and np.nanmin(ours) == -448.0


def test_encode_roundtrip_every_finite_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    assert np.array_equal(fp8.encode(fp8.decode(codes)), codes)


def test_encode_midpoints_ties_to_even_and_match_torch():
    mags = fp8.decode(np.arange(0, 0x7F, dtype=np.uint8))
    mids = (mags[:-1] + mags[1:]) / 2
    got = fp8.encode(mids)
    lo_code = np.arange(0, 0x7E, dtype=np.uint8)
    expect = np.where(lo_code % 2 == 0, lo_code, lo_code + 1).astype(np.uint8)
    assert np.array_equal(got, expect)
    ref = torch.from_numpy(mids.astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(got, ref)
    # just off the midpoint rounds to the nearer side
    eps = np.spacing(mids.astype(np.float32)).astype(np.float64)
    assert np.array_equal(fp8.encode(mids - eps), lo_code)
    assert np.array_equal(fp8.encode(mids + eps), lo_code + 1)


def test_encode_random_in_range_matches_torch():
    rng = np.random.default_rng(5)
    v = np.concatenate([rng.standard_normal(20000) * s for s in (1e-3, 0.05, 1.0, 30.0, 150.0)])
    v = np.clip(v, -448, 448).astype(np.float32)
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(fp8.encode(v), ref)


def test_encode_saturates_and_nan():
    got = fp8.encode(np.array([449.0, 464.0, 470.0, 1e9, -1e9, np.nan, -0.0]))
    assert got.tolist() == [0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0x7F, 0x80]


def test_quantize_blocks_error_bound_and_scale():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((7, 512)) * rng.uniform(0.01, 10, (7, 1))).astype(np.float32)
    x[3, 128:256] = 0.0                                # all-zero block
    codes, scale = fp8.quantize_blocks(x)
    assert scale.dtype == np.float32 and scale.shape == (7, 4)
    assert scale[3, 1] == 1.0 and not codes[3, 128:256].any()
    # the block maximum lands exactly on the largest code
    xb = np.abs(x.reshape(7, 4, 128))
    amax_pos = xb.argmax(axis=2)
    cb = codes.reshape(7, 4, 128)
    for r in range(7):
        for b in range(4):
            if b == 1 and r == 3:
                continue
            assert cb[r, b, amax_pos[r, b]] & 0x7F == 0x7E
            assert scale[r, b] == np.float32(xb[r, b].max() / np.float32(448.0))
    deq = fp8.dequantize_blocks(codes, scale)
    # e4m3 keeps 4 significant bits: normal values within 2^-4 relative;
    # subnormal range (below 2^-6 * scale) within half a quantum 2^-10 * scale
    s_full = np.repeat(scale.astype(np.float64), 128, axis=1)
    err = np.abs(deq - x)
    bound = np.maximum(np.abs(x) * 2.0 ** -4, s_full * 2.0 ** -10)
    assert np.all(err <= bound * (1 + 1e-9))


def test_quantize_blocks_lossless_on_representable_rows():
    # rows made of e4m3 values times a power of two, each block containing
    # +-448 * 2^j, quantise without loss
    rng = np.random.default_rng(2)
    vals = fp8.decode(rng.integers(0, 0x7F, size=(3, 256)).astype(np.uint8))
    vals[:, 0] = 448.0
    vals[:, 128] = -448.0
    x = (vals * 2.0 ** -5).astype(np.float32)
    codes, scale = fp8.quantize_blocks(x)
    assert np.all(scale == np.float32(2.0 ** -5))
    assert np.array_equal(fp8.dequantize_blocks(codes, scale), x.astype(np.float64))


def test_dequantize_weight_block_scales_and_orientation():
    rng = np.random.default_rng(3)
    codes = rng.integers(0, 0x7E, size=(256, 384)).astype(np.uint8)
    scale = rng.uniform(0.5, 2, size=(2, 3)).astype(np.float32)
    w = fp8.dequantize_weight(codes, scale)
    # element (i, j) uses block (i // 128, j // 128)
    for i, j in [(0, 0), (127, 128), (128, 127), (255, 383), (130, 300)]:
        assert w[i, j] == fp8.decode(codes[i:i + 1, j])[0] * float(scale[i // 128, j // 128])
