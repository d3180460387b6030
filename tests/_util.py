"""Shared helpers for the parity tests: oracle references for a workload and
the tolerance checks.  Inputs come from the seeded generator only."""
import numpy as np
import torch

from oracle import ffn
from paper_2609_33252_amd import workload as W

# Elementwise bound for bf16 inputs with float32 accumulation, and the
# relative-RMS bound for the e4m3 path (both from the target tolerance of the
# routed-expert path); the MXFP4 path quantises activations and h to e4m3
# like the e4m3 path and takes the same bound.
BF16_ATOL, BF16_RTOL = 1e-2, 1e-2
FP8_REL_RMS = 4e-2
F32_REL_RMS = 1e-2


def np_bits(t):
    if t is None:
        return None
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def modes(wl):
    w = wl.cfg["w"]
    if w == W.FP8:
        return "fp8", "fp8", "fp8"
    if w == W.MXFP4:
        return "mxfp4", "mxfp8", "mxfp8"
    if w == W.BF16:
        return "bf16", "bf16", None
    return "f32", None, None


def bank(wl):
    kind, _, _ = modes(wl)
    return ffn.ExpertBank(kind, *[np_bits(t) for t in (wl.w_gate, wl.w_up, wl.w_down)],
                          *[np_bits(t) for t in (wl.s_gate, wl.s_up, wl.s_down)])


def reference(wl, tokens=None, bank_=None):
    """Oracle output.  tokens: None (all R*T rows, float32 [R][T][d]) or an
    array of (replica, token) pairs (float32 [n][d])."""
    c = wl.cfg
    kind, h_mode, x_mode = modes(wl)
    bank_ = bank_ or bank(wl)
    xk = "bf16" if c["x"] == W.BF16 else "f32"
    if tokens is None:
        x = ffn.decode_rows(np_bits(wl.x).reshape(c["R"] * c["T"], c["d"]), xk)
        ids = wl.topk_local.reshape(-1, c["k"])
        w = wl.topk_w.reshape(-1, c["k"])
        out = ffn.routed_output(x, ids, w, bank_, c["E"], h_mode=h_mode, x_mode=x_mode,
                                y_mode="bf16")
        return out.reshape(c["R"], c["T"], c["d"])
    tokens = np.asarray(tokens)
    r, t = tokens[:, 0], tokens[:, 1]
    xb = np_bits(wl.x)[r, t]
    x = ffn.decode_rows(xb, xk)
    return ffn.routed_output(x, wl.topk_local[r, t], wl.topk_w[r, t], bank_, c["E"],
                             h_mode=h_mode, x_mode=x_mode, y_mode="bf16")


def compare(wl, got, ref):
    """Assert the target tolerance; returns (max abs err, relative RMS)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    rel = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))
    kind, _, _ = modes(wl)
    if kind in ("fp8", "mxfp4"):
        assert rel <= FP8_REL_RMS, f"{kind} relative RMS {rel:.3e}"
    else:
        bad = err > BF16_ATOL + BF16_RTOL * np.abs(ref)
        assert not bad.any(), (f"{int(bad.sum())} elements outside tolerance, max err "
                               f"{err.max():.3e}, rel RMS {rel:.3e}")
        if kind == "f32":
            assert rel <= F32_REL_RMS, f"relative RMS {rel:.3e}"
    return float(err.max()), rel
