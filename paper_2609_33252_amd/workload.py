"""Seeded synthetic MoE-prefill workloads for the streamFFN routed-expert path.

This module only draws inputs: expert weights, hidden rows, top-k routing,
combine coefficients, the chunk arrival schedule and the set of experts whose
weights live in a separate (donor) region.  It holds none of the FFN, routing,
batching or combine arithmetic of the method; the CPU oracle and the HIP
library both consume what it returns.

The shapes follow the paper's evaluation models (Table 1: routed experts per
layer, experts per token, expert intermediate size) at one expert-parallel
rank's share; d_model is not stated in the paper and is a workload choice.

Random streams: ``numpy.random.SeedSequence(seed).spawn(6)`` in the order
weights, hidden, routing, combine logits, arrival schedule, fetched experts.
Large draws are split into fixed row blocks, each with its own spawned child
seed, so results do not depend on the number of threads used to draw them.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np
import torch

F32, BF16, FP8, MXFP4 = "f32", "bf16", "fp8_e4m3_b128", "mxfp4"
FP8_BLOCK = 128
FP8_MAX = 448.0

# Workload presets.  Keys: d (d_model), I (expert intermediate size),
# E (local experts), Eg (global experts), k (top-k), R (replicas),
# T (token slots per replica), cpr (chunks per replica), zipf (None =
# uniform routing), w/x (weight / hidden dtype), arrival (schedule kind),
# skew (per-replica finish-time scales), fetch_frac (share of local experts
# whose weights must be fetched from a donor region).
PRESETS = {
    "tiny": dict(d=256, I=128, E=8, Eg=8, k=2, R=2, T=256, cpr=2, zipf=None,
                 w=F32, x=F32, arrival="order", skew=None, fetch_frac=0.0),
    "sync_d4096": dict(d=4096, I=2048, E=8, Eg=64, k=8, R=4, T=2048, cpr=1, zipf=None,
                       w=BF16, x=BF16, arrival="simultaneous", skew=None, fetch_frac=0.0),
    "zipf_stream_d7168": dict(d=7168, I=2048, E=8, Eg=256, k=8, R=8, T=4096, cpr=8, zipf=1.2,
                              w=BF16, x=BF16, arrival="lognormal", skew=None, fetch_frac=0.0),
    "zipf_imbalanced_d7168": dict(d=7168, I=2048, E=8, Eg=256, k=8, R=8, T=4096, cpr=8, zipf=1.2,
                                  w=BF16, x=BF16, arrival="lognormal", skew="straggler0",
                                  fetch_frac=0.0),
    "fp8_fetch_d6144": dict(d=6144, I=2560, E=16, Eg=160, k=8, R=8, T=8192, cpr=1, zipf=1.5,
                            w=FP8, x=BF16, arrival="simultaneous", skew=None, fetch_frac=0.25),
    # DeepSeek-V4-Flash's routed experts at one EP8 rank's share (Table 1:
    # 256 routed experts, 6 per token, intermediate 2048; MXFP4 weights,
    # Section 4.1), balanced routing, eight chunks per replica
    "mxfp4_dsv4flash_d4096": dict(d=4096, I=2048, E=32, Eg=256, k=6, R=8, T=8192, cpr=8,
                                  zipf=None, w=MXFP4, x=BF16, arrival="lognormal", skew=None,
                                  fetch_frac=0.0),
}
# The five numbered configurations in order.
CONFIG_ORDER = ["tiny", "sync_d4096", "zipf_stream_d7168", "zipf_imbalanced_d7168",
                "fp8_fetch_d6144"]

_ROW_BLOCK = 1 << 20  # elements per independently seeded draw block


@dataclasses.dataclass
class Chunk:
    """One routed-token chunk as delivered by a replica's dispatch lane."""
    replica: int
    chunk_index: int          # position of this chunk within its replica
    token_idx: np.ndarray     # int32 [n]: token slot within the replica
    arrival_ms: float         # arrival time relative to the schedule origin

    @property
    def n_rows(self) -> int:
        return int(self.token_idx.shape[0])


@dataclasses.dataclass
class Workload:
    name: str
    cfg: dict
    seed: int
    # expert weights in math orientation; bf16/f32 as torch CPU tensors,
    # fp8 as uint8 codes (OCP e4m3fn) plus float32 128x128 block scales;
    # mxfp4 output-major with K packed: uint8 code pairs plus E8M0 scales
    w_gate: torch.Tensor      # [E][d][I]; mxfp4 [E][I][d/2]
    w_up: torch.Tensor        # [E][d][I]; mxfp4 [E][I][d/2]
    w_down: torch.Tensor      # [E][I][d]; mxfp4 [E][d][I/2]
    s_gate: Optional[torch.Tensor]  # fp8: [E][d/128][I/128]; mxfp4 [E][I][d/32]
    s_up: Optional[torch.Tensor]
    s_down: Optional[torch.Tensor]  # fp8: [E][I/128][d/128]; mxfp4 [E][d][I/32]
    x: torch.Tensor           # [R][T][d] hidden rows (bf16 or f32)
    topk_global: np.ndarray   # int32 [R][T][k] global expert ids, slot order
    topk_local: np.ndarray    # int32 [R][T][k] local id or -1 (remote)
    topk_w: np.ndarray        # float32 [R][T][k] combine coefficients
    chunks: list              # list[Chunk] in submission (arrival) order
    fetched: list             # local expert ids resident only in the donor region

    # convenience views -------------------------------------------------
    @property
    def R(self):
        return self.cfg["R"]

    @property
    def T(self):
        return self.cfg["T"]

    def chunk_rows(self, c: Chunk):
        """(x rows, local ids, weights) for one chunk, as CPU arrays/tensors."""
        return (self.x[c.replica][torch.from_numpy(c.token_idx).long()],
                self.topk_local[c.replica][c.token_idx],
                self.topk_w[c.replica][c.token_idx])

    def chunk_pairs(self, c: Chunk) -> int:
        return int((self.topk_local[c.replica][c.token_idx] >= 0).sum())

    @property
    def n_pairs(self) -> int:
        return int((self.topk_local >= 0).sum())

    @property
    def delivered(self) -> np.ndarray:
        """bool [R][T]: token has at least one local slot."""
        return (self.topk_local >= 0).any(axis=2)


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _normal(ss: np.random.SeedSequence, n: int, scale: float) -> np.ndarray:
    """n float32 N(0, scale^2) draws, block-seeded (thread-count independent)."""
    out = np.empty(n, np.float32)
    nblk = (n + _ROW_BLOCK - 1) // _ROW_BLOCK
    kids = ss.spawn(nblk)

    def fill(b):
        sl = out[b * _ROW_BLOCK:min(n, (b + 1) * _ROW_BLOCK)]
        np.random.default_rng(kids[b]).standard_normal(out=sl, dtype=np.float32)
        if scale != 1.0:
            sl *= np.float32(scale)

    if nblk == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nblk)))
    return out


def _bytes(ss: np.random.SeedSequence, n: int, lo: int, hi: int) -> np.ndarray:
    """n uint8 draws uniform in [lo, hi), block-seeded like _normal."""
    out = np.empty(n, np.uint8)
    nblk = (n + _ROW_BLOCK - 1) // _ROW_BLOCK
    kids = ss.spawn(nblk)

    def fill(b):
        sl = out[b * _ROW_BLOCK:min(n, (b + 1) * _ROW_BLOCK)]
        sl[:] = np.random.default_rng(kids[b]).integers(lo, hi, size=sl.shape[0], dtype=np.uint8)

    if nblk == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nblk)))
    return out


def _mxfp4_matrix(ss: np.random.SeedSequence, E: int, rows: int, K: int):
    """MXFP4 weights drawn directly in the checkpoint format: uniform code
    bytes (every e2m1 value equally likely) and E8M0 scales 2^-8 or 2^-7,
    an element RMS of about 0.018.  rows x K, blocks of 32 along K."""
    c_ss, s_ss = ss.spawn(2)
    codes = _bytes(c_ss, E * rows * K // 2, 0, 256).reshape(E, rows, K // 2)
    scales = _bytes(s_ss, E * rows * K // 32, 119, 121).reshape(E, rows, K // 32)
    return torch.from_numpy(codes), torch.from_numpy(scales)


def _to_dtype(a: np.ndarray, dt: str) -> torch.Tensor:
    t = torch.from_numpy(a)
    if dt == BF16:
        return t.to(torch.bfloat16)  # round-to-nearest-even
    return t.clone()


def _fp8_blocks(w: np.ndarray):
    """Block-quantise [E][rows][cols] float32 weights to e4m3 codes + scales.

    This is the checkpoint format the expert weights arrive in (one float32
    scale per 128x128 block, scale = block amax / 448, or 1 for an all-zero
    block); the conversion uses torch's float8_e4m3fn cast.
    """
    E, r, c = w.shape
    assert r % FP8_BLOCK == 0 and c % FP8_BLOCK == 0
    t = torch.from_numpy(w).view(E, r // FP8_BLOCK, FP8_BLOCK, c // FP8_BLOCK, FP8_BLOCK)
    amax = t.abs().amax(dim=(2, 4))                       # [E][rb][cb] float32
    s = torch.where(amax > 0, amax / torch.tensor(FP8_MAX, dtype=torch.float32),
                    torch.ones_like(amax))
    q = (t / s[:, :, None, :, None]).to(torch.float8_e4m3fn)
    codes = q.view(torch.uint8).reshape(E, r, c).contiguous()
    return codes, s.contiguous()


def _route(ss: np.random.SeedSequence, R: int, T: int, Eg: int, k: int, zipf):
    """Top-k global expert ids per token via Gumbel-top-k on log popularity.

    Popularity is uniform, or Zipf(s) over popularity ranks, with a seeded
    permutation mapping rank -> global expert id.  Slot order is the order of
    the perturbed scores (largest first).
    """
    perm_ss, gum_ss = ss.spawn(2)
    if zipf is None:
        logp = np.zeros(Eg, np.float64)
    else:
        ranks = np.arange(1, Eg + 1, dtype=np.float64)
        p = ranks ** (-float(zipf))
        p /= p.sum()
        rank_to_id = np.random.default_rng(perm_ss).permutation(Eg)
        logp = np.empty(Eg, np.float64)
        logp[rank_to_id] = np.log(p)
    n = R * T
    ids = np.empty((n, k), np.int32)
    blk = 65536
    kids = gum_ss.spawn((n + blk - 1) // blk)
    for b in range((n + blk - 1) // blk):
        lo, hi = b * blk, min(n, (b + 1) * blk)
        g = np.random.default_rng(kids[b]).gumbel(size=(hi - lo, Eg))
        sc = g + logp[None, :]
        top = np.argpartition(-sc, k - 1, axis=1)[:, :k]
        order = np.argsort(-np.take_along_axis(sc, top, axis=1), axis=1, kind="stable")
        ids[lo:hi] = np.take_along_axis(top, order, axis=1)
    return ids.reshape(R, T, k)


def _softmax_f32(logits: np.ndarray) -> np.ndarray:
    z = logits - logits.max(axis=-1, keepdims=True)
    e = np.exp(z, dtype=np.float32)
    return (e / e.sum(axis=-1, keepdims=True, dtype=np.float32)).astype(np.float32)


def _arrivals(ss, cfg, n_chunks_total):
    R, cpr = cfg["R"], cfg["cpr"]
    rng = np.random.default_rng(ss)
    kind = cfg["arrival"]
    if kind == "simultaneous":
        return np.zeros((R, cpr)), None
    if kind == "order":
        return np.zeros((R, cpr)), rng.permutation(R * cpr)
    # lognormal(0, 0.5) ms gaps, cumulative, scaled per replica
    gaps = rng.lognormal(mean=0.0, sigma=0.5, size=(R, cpr))
    if cfg["skew"] == "straggler0":
        s = np.empty(R)
        s[0] = 2.0
        s[1:] = rng.uniform(1.0, 1.5, size=R - 1)
    else:
        s = np.ones(R)
    return s[:, None] * np.cumsum(gaps, axis=1), None


def generate(name: str = "tiny", seed: int = 0, **overrides) -> Workload:
    """Draw one workload.  ``overrides`` may shrink R, T, cpr (chunks per
    replica) or change any preset key, keeping the distributions."""
    if isinstance(name, int):
        name = CONFIG_ORDER[name - 1]
    cfg = dict(PRESETS[name])
    cfg.update(overrides)
    d, I, E, Eg, k, R, T, cpr = (cfg[x] for x in ("d", "I", "E", "Eg", "k", "R", "T", "cpr"))
    assert T % cpr == 0, "token slots must split evenly into chunks"
    ss_w, ss_x, ss_r, ss_l, ss_a, ss_f = np.random.SeedSequence(seed).spawn(6)

    # weights: N(0, 0.02) float32 draws, then stored in the config dtype
    # (MXFP4: drawn directly as codes and scales)
    wg_ss, wu_ss, wd_ss = ss_w.spawn(3)
    s_gate = s_up = s_down = None
    if cfg["w"] == MXFP4:
        w_gate, s_gate = _mxfp4_matrix(wg_ss, E, I, d)
        w_up, s_up = _mxfp4_matrix(wu_ss, E, I, d)
        w_down, s_down = _mxfp4_matrix(wd_ss, E, d, I)
    else:
        wg = _normal(wg_ss, E * d * I, 0.02).reshape(E, d, I)
        wu = _normal(wu_ss, E * d * I, 0.02).reshape(E, d, I)
        wd = _normal(wd_ss, E * I * d, 0.02).reshape(E, I, d)
        if cfg["w"] == FP8:
            w_gate, s_gate = _fp8_blocks(wg)
            w_up, s_up = _fp8_blocks(wu)
            w_down, s_down = _fp8_blocks(wd)
        else:
            w_gate, w_up, w_down = (_to_dtype(a, cfg["w"]) for a in (wg, wu, wd))
        del wg, wu, wd

    x = _to_dtype(_normal(ss_x, R * T * d, 1.0), cfg["x"]).view(R, T, d)

    topk_global = _route(ss_r, R, T, Eg, k, cfg["zipf"])
    topk_local = np.where(topk_global < E, topk_global, -1).astype(np.int32)
    logits = np.random.default_rng(ss_l).standard_normal((R, T, k), dtype=np.float32)
    topk_w = _softmax_f32(logits)

    times, order = _arrivals(ss_a, cfg, R * cpr)
    delivered = (topk_local >= 0).any(axis=2)
    per = T // cpr
    chunks = []
    for r in range(R):
        for j in range(cpr):
            slots = np.arange(j * per, (j + 1) * per, dtype=np.int32)
            tok = slots[delivered[r, slots]]
            chunks.append(Chunk(replica=r, chunk_index=j, token_idx=tok,
                                arrival_ms=float(times[r, j])))
    if order is not None:
        chunks = [chunks[i] for i in order]
    else:
        chunks.sort(key=lambda c: (c.arrival_ms, c.replica, c.chunk_index))

    fetched = []
    if cfg["fetch_frac"] > 0:
        nf = int(round(cfg["fetch_frac"] * E))
        fetched = sorted(int(v) for v in
                         np.random.default_rng(ss_f).choice(E, size=nf, replace=False))

    return Workload(name=name, cfg=cfg, seed=seed, w_gate=w_gate, w_up=w_up, w_down=w_down,
                    s_gate=s_gate, s_up=s_up, s_down=s_down, x=x, topk_global=topk_global,
                    topk_local=topk_local, topk_w=topk_w, chunks=chunks, fetched=fetched)
