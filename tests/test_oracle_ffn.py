"""Pins for the float64 routed-expert oracle (CPU only): scalar brute force on
tiny shapes, closed forms (zero expert, identity-permutation expert), one-hot
coefficients, linearity, all-remote routing, bf16 rounding and fp8 modes."""
import math

import numpy as np
import pytest
import torch

from oracle import ffn, fp8
from paper_2609_33252_amd import workload as W


def _silu(z):
    return z / (1.0 + math.exp(-z))


def _tiny(seed, d=16, I=8, E=3, k=2, n=6, remote=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, d))
    wg = rng.standard_normal((E, d, I)) * 0.3
    wu = rng.standard_normal((E, d, I)) * 0.3
    wd = rng.standard_normal((E, I, d)) * 0.3
    ids = np.stack([rng.permutation(E)[:k] for _ in range(n)]).astype(np.int32)
    if remote:
        ids[rng.random((n, k)) < 0.3] = -1
    w = rng.uniform(0.1, 1.0, (n, k)).astype(np.float32)
    return x, wg, wu, wd, ids, w


def _bank64(wg, wu, wd):
    return lambda e: (wg[e], wu[e], wd[e])


@pytest.mark.parametrize("seed", range(4))
def test_oracle_matches_scalar_brute_force(seed):
    x, wg, wu, wd, ids, w = _tiny(seed)
    got = ffn.routed_output(x, ids, w, _bank64(wg, wu, wd), 3)
    for t in range(x.shape[0]):
        ref = ffn.brute_force_token(x[t], ids[t], w[t], wg, wu, wd)
        np.testing.assert_allclose(got[t], np.float32(ref), rtol=1e-6, atol=1e-9)


def test_oracle_float64_before_final_rounding():
    # compare in float64 by scaling: the brute force and the vectorised
    # oracle agree to ~1e-12 before the final float32 rounding
    x, wg, wu, wd, ids, w = _tiny(11)
    h = ffn.expert_ffn(x[:2], wg[0], wu[0], wd[0])
    for t in range(2):
        ref = ffn.brute_force_token(x[t], [0], [1.0], wg, wu, wd)
        np.testing.assert_allclose(h[t], ref, rtol=1e-12, atol=1e-13)


def test_bf16_h_mode_matches_brute_force_with_scalar_rounding():
    x, wg, wu, wd, ids, w = _tiny(7)
    got = ffn.routed_output(x, ids, w, _bank64(wg, wu, wd), 3, h_mode="bf16")

    def rb(v):  # scalar bf16 rounding through torch (float64 -> bf16)
        return float(torch.tensor(v, dtype=torch.float64).to(torch.bfloat16).double())

    for t in range(x.shape[0]):
        ref = ffn.brute_force_token(x[t], ids[t], w[t], wg, wu, wd, h_round=rb)
        np.testing.assert_allclose(got[t], np.float32(ref), rtol=1e-6, atol=1e-9)


def test_round_bf16_definition():
    rng = np.random.default_rng(4)
    v32 = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    ours = ffn.round_bf16(v32.astype(np.float64))
    ref = torch.from_numpy(v32).to(torch.bfloat16).double().numpy()
    assert np.array_equal(ours, ref)
    # results are bf16 values: low 16 bits of the float32 pattern are zero
    assert not (ours.astype(np.float32).view(np.uint32) & 0xFFFF).any()
    # exact ties go to the even neighbour: 1 + 2^-8 lies between 1 and 1 + 2^-7
    assert ffn.round_bf16(np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8]))[:].tolist() == [1.0, 1 + 2 ** -6]


def test_zero_expert_gives_exact_zero():
    x, wg, wu, wd, ids, w = _tiny(3, remote=False)
    for which in range(3):
        ws = [wg.copy(), wu.copy(), wd.copy()]
        ws[which][:] = 0.0
        out = ffn.routed_output(x, ids, w, _bank64(*ws), 3, h_mode="bf16")
        assert not out.any()


@pytest.mark.parametrize("beta", [0.5, 2.0])
def test_identity_permutation_expert_closed_form(beta):
    # d = I, Wu = P, Wg = beta P, Wd = P^T for a permutation matrix P that is
    # a single d-cycle (not an involution): y_i = w * bf16(silu(beta x_i) x_i)
    d, n = 32, 5
    rng = np.random.default_rng(0)
    pi = np.roll(np.arange(d), 1)                       # j -> pi[j]
    P = np.zeros((d, d))
    P[pi, np.arange(d)] = 1.0                           # (x P)_j = x_{pi[j]}
    x = rng.standard_normal((n, d))
    ids = np.zeros((n, 1), np.int32)
    w = np.full((n, 1), 0.75, np.float32)
    bank = lambda e: (beta * P, P, P.T.copy())
    got = ffn.routed_output(x, ids, w, bank, 1, h_mode="bf16")
    for t in range(n):
        for i in range(d):
            hv = _silu(beta * x[t, i]) * x[t, i]
            hb = float(torch.tensor(hv, dtype=torch.float64).to(torch.bfloat16).double())
            assert got[t, i] == np.float32(0.75 * hb)


def test_one_hot_coefficients_select_one_expert_and_slot_order():
    x, wg, wu, wd, ids, w = _tiny(5, remote=False, k=3, E=4)
    for s in range(3):
        w1 = np.zeros_like(w)
        w1[:, s] = 1.0
        out = ffn.routed_output(x, ids, w1, _bank64(wg, wu, wd), 4)
        for t in range(x.shape[0]):
            e = ids[t, s]
            ref = ffn.expert_ffn(x[t:t + 1], wg[e], wu[e], wd[e])[0]
            np.testing.assert_array_equal(out[t], ref.astype(np.float32))


def test_linearity_in_down_weights_and_coefficients():
    x, wg, wu, wd, ids, w = _tiny(9)
    base = ffn.routed_output(x, ids, w, _bank64(wg, wu, wd), 3, h_mode="bf16")
    two_wd = ffn.routed_output(x, ids, w, _bank64(wg, wu, 2 * wd), 3, h_mode="bf16")
    two_w = ffn.routed_output(x, ids, 2 * w, _bank64(wg, wu, wd), 3, h_mode="bf16")
    np.testing.assert_array_equal(two_wd, 2 * base)
    np.testing.assert_array_equal(two_w, 2 * base)


def test_all_remote_routing_gives_zero_and_each_contribution_once():
    x, wg, wu, wd, ids, w = _tiny(6)
    out = ffn.routed_output(x, np.full_like(ids, -1), w, _bank64(wg, wu, wd), 3)
    assert not out.any()
    # a token routed twice to the same expert with coefficients a, b equals
    # once with a + b (each contribution counted exactly once, none dropped)
    ids2 = np.zeros((x.shape[0], 2), np.int32)
    w2 = np.stack([np.full(x.shape[0], 0.25), np.full(x.shape[0], 0.5)], 1).astype(np.float32)
    a = ffn.routed_output(x, ids2, w2, _bank64(wg, wu, wd), 3)
    b = ffn.routed_output(x, ids2[:, :1], np.full((x.shape[0], 1), 0.75, np.float32),
                          _bank64(wg, wu, wd), 3)
    np.testing.assert_allclose(a, b, rtol=1e-6)


def test_fp8_modes_lossless_on_representable_inputs():
    # inputs and weights built from e4m3 values with power-of-two scales: the
    # fp8 input quantisation and the weight dequantisation are exact, so the
    # fp8 x-mode equals the exact mode
    rng = np.random.default_rng(8)
    d, I, n = 256, 128, 4
    xv = fp8.decode(rng.integers(0, 0x7E, (n, d)).astype(np.uint8))
    xv[:, 0], xv[:, 128] = 448.0, -448.0
    x = xv * 2.0 ** -6
    def wq(r, c):
        codes = rng.integers(0, 0xFE, (r, c)).astype(np.uint8)
        codes[(codes & 0x7F) == 0x7F] = 0
        s = (2.0 ** rng.integers(-9, -5, (r // 128, c // 128))).astype(np.float32)
        return codes, s
    (cg, sg), (cu, su), (cd, sd) = wq(d, I), wq(d, I), wq(I, d)
    bank = ffn.ExpertBank("fp8", cg[None], cu[None], cd[None], sg[None], su[None], sd[None])
    ids = np.zeros((n, 1), np.int32)
    w = np.ones((n, 1), np.float32)
    exact = ffn.routed_output(x, ids, w, bank, 1)
    xq = ffn.routed_output(x, ids, w, bank, 1, x_mode="fp8")
    np.testing.assert_array_equal(exact, xq)
    # and the h quantisation mode stays within e4m3 precision of exact h
    hq = ffn.routed_output(x, ids, w, bank, 1, x_mode="fp8", h_mode="fp8")
    rel = np.linalg.norm(hq - exact) / np.linalg.norm(exact)
    assert 0 < rel < 0.08


def test_workload_banks_decode_stored_dtypes():
    wl = W.generate("tiny", 0)
    bank = ffn.ExpertBank("f32", wl.w_gate.numpy(), wl.w_up.numpy(), wl.w_down.numpy())
    assert bank(3)[0].dtype == np.float64
    np.testing.assert_array_equal(bank(3)[2], wl.w_down[3].numpy().astype(np.float64))
    wl2 = W.generate("fp8_fetch_d6144", 0, d=256, I=256, R=1, T=64, E=2, Eg=16)
    bank2 = ffn.ExpertBank("fp8", wl2.w_gate.numpy(), wl2.w_up.numpy(), wl2.w_down.numpy(),
                           wl2.s_gate.numpy(), wl2.s_up.numpy(), wl2.s_down.numpy())
    ref = (wl2.w_gate[1].view(torch.float8_e4m3fn).double()
           * wl2.s_gate[1].double().repeat_interleave(128, 0).repeat_interleave(128, 1)).numpy()
    np.testing.assert_array_equal(bank2(1)[0], ref)
    bits = wl2.x.view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ffn.bf16_bits_to_f64(bits), wl2.x.double().numpy())


def test_bf16_y_mode_rounds_each_weighted_contribution():
    # each w * y rounded to bf16 (torch's cast, per scalar) and summed in slot
    # order: the oracle's y_mode against the brute-force token loop
    x, wg, wu, wd, ids, w = _tiny(21)
    got = ffn.routed_output(x, ids, w, _bank64(wg, wu, wd), 3, y_mode="bf16")

    def rb(v):
        return float(torch.tensor(v, dtype=torch.float64).to(torch.bfloat16).double())

    for t in range(x.shape[0]):
        ref = np.zeros(x.shape[1])
        for s, e in enumerate(ids[t]):
            if e < 0:
                continue
            y = ffn.brute_force_token(x[t], [e], [1.0], wg, wu, wd)
            ref += np.array([rb(float(w[t, s]) * v) for v in y])
        np.testing.assert_allclose(got[t], np.float32(ref), rtol=1e-6, atol=1e-9)
    # and it differs from the unrounded result by at most 2^-8 (the unit
    # roundoff of 8 significant bits) per contribution
    exact = ffn.routed_output(x, ids, w, _bank64(wg, wu, wd), 3)
    bound = np.zeros_like(exact, dtype=np.float64)
    for t in range(x.shape[0]):
        for s, e in enumerate(ids[t]):
            if e >= 0:
                y = np.array(ffn.brute_force_token(x[t], [e], [w[t, s]], wg, wu, wd))
                bound[t] += 2.0 ** -8 * np.abs(y)
    assert (np.abs(got.astype(np.float64) - exact) <= bound + 1e-6).all()
    assert not np.array_equal(got, exact)
