"""Replay a seeded workload through libcep on one GPU.

Uploads the expert weights, builds the donor region for experts whose
weights must be fetched, uploads every chunk, and replays a layer: opens it,
optionally issues the one weight fetch on a side stream, submits the chunks in
arrival order (optionally waiting for each chunk's scheduled arrival time and
recording an arrival event for it), and closes it with the combine barrier.
Torch provides device memory, streams and events only; all arithmetic of the
path runs in libcep's kernels.
"""
from __future__ import annotations

import time

import numpy as np
import torch

from . import cep
from . import workload as W

_DT = {W.F32: cep.CEP_F32, W.BF16: cep.CEP_BF16, W.FP8: cep.CEP_FP8_E4M3_B128,
       W.MXFP4: cep.CEP_MXFP4}


class DeviceChunk:
    __slots__ = ("replica", "n_rows", "n_pairs", "token_idx", "x", "ids", "w", "arrival_ms")


class Runner:
    """One libcep context holding one workload's experts and chunks."""

    def __init__(self, wl: W.Workload, n_streams: int = 4, record_routing: bool = False,
                 max_pairs=None, use_fetch: bool = True, device: str = "cuda"):
        self.wl = wl
        c = wl.cfg
        self.device = torch.device(device)
        self.use_fetch = use_fetch and bool(wl.fetched)
        scaled = c["w"] in (W.FP8, W.MXFP4)
        # a batch never holds more pairs than the layer: size every stream
        # slot's scratch for the layer's pairs (0 would size it for R*T*k)
        if max_pairs is None:
            max_pairs = max(1, wl.n_pairs)
        self.cfg = cep.make_config(
            d_model=c["d"], d_ff=c["I"], n_local_experts=c["E"], top_k=c["k"],
            max_replicas=c["R"], max_tokens_per_replica=c["T"], w_dtype=_DT[c["w"]],
            x_dtype=_DT[c["x"]], n_streams=n_streams, max_pairs_per_batch=max_pairs,
            fetch_buffer_bytes=0, record_routing=1 if record_routing else 0)
        blob = cep.cep_packed_expert_bytes(self.cfg)
        if blob == 0:
            raise ValueError("workload shape rejected by libcep")
        self.blob_bytes = blob
        if self.use_fetch:
            self.cfg.fetch_buffer_bytes = blob * len(wl.fetched)
        dev = self.device
        wg, wu, wd = (t.to(dev) for t in (wl.w_gate, wl.w_up, wl.w_down))
        sg = su = sd = None
        if scaled:
            sg, su, sd = (t.to(dev) for t in (wl.s_gate, wl.s_up, wl.s_down))
        weights = cep.make_weights(wg, wu, wd, sg, su, sd)
        stream = torch.cuda.current_stream(dev)
        resident = None
        if self.use_fetch:
            resident = [0 if e in wl.fetched else 1 for e in range(c["E"])]
            # the donor region: packed blobs of the fetched experts, in a
            # separate allocation (what a donor GPU holds)
            self.donor = torch.empty(blob * len(wl.fetched), dtype=torch.uint8, device=dev)
            for i, e in enumerate(wl.fetched):
                cep.cep_pack_experts(self.cfg, weights, e, 1, self.donor.data_ptr() + i * blob,
                                     stream)
        self.ctx = cep.cep_init_experts(self.cfg, weights, resident, stream)
        torch.cuda.synchronize(dev)
        del wg, wu, wd, sg, su, sd, weights

        # token rows land in one receive buffer, chunk after chunk in arrival
        # order (as a dispatch writes them into its registered receive
        # region); each chunk's x is a view of it
        n_recv = sum(ch.n_rows for ch in wl.chunks)
        self.recv = torch.empty(max(1, n_recv), c["d"], dtype=wl.x.dtype, device=dev)
        self.chunks = []
        r0 = 0
        for ch in wl.chunks:
            x, ids, w = wl.chunk_rows(ch)
            dc = DeviceChunk()
            dc.replica = ch.replica
            dc.n_rows = ch.n_rows
            dc.n_pairs = int((ids >= 0).sum())
            dc.token_idx = torch.from_numpy(ch.token_idx.astype(np.int32)).to(dev)
            dc.x = self.recv[r0:r0 + ch.n_rows]
            dc.x.copy_(x)
            r0 += ch.n_rows
            dc.ids = torch.from_numpy(np.ascontiguousarray(ids, np.int32)).to(dev)
            dc.w = torch.from_numpy(np.ascontiguousarray(w, np.float32)).to(dev)
            dc.arrival_ms = ch.arrival_ms
            self.chunks.append(dc)
        self.chunks_per_replica = [0] * c["R"]
        for ch in wl.chunks:
            self.chunks_per_replica[ch.replica] += 1
        self.out = torch.zeros(c["R"], c["T"], c["d"], dtype=torch.float32, device=dev)
        self.side = torch.cuda.Stream(dev)
        self.dispatch = torch.cuda.Stream(dev)
        self.gen = 0
        self.arrival_events = []

    @property
    def n_pairs(self) -> int:
        return sum(ch.n_pairs for ch in self.chunks)

    def run(self, policy=cep.CEP_WAIT_ALL, theta=1, n_streams=1, order=None, timed=False,
            time_scale=1.0, arrival_events=False, out=None, stream=None, inputs_ready=False,
            fetch_mode=None):
        """Replay one layer; returns the library's done event handle.

        order: optional permutation of chunk indices (submission order).
        timed: wait until each chunk's scheduled arrival (scaled) on the host.
        inputs_ready: the chunk inputs are resident and no work on the caller's
            stream writes them (steady-state replay of the same layer), so the
            chunks carry no arrival event.
        fetch_mode: cep_fetch_mode of this and later layers (None: unchanged).
        """
        out = self.out if out is None else out
        stream = torch.cuda.current_stream(self.device) if stream is None else stream
        ctx = self.ctx
        cep.cep_set_policy(ctx, policy, theta, n_streams)
        if fetch_mode is not None:
            cep.cep_set_fetch_mode(ctx, fetch_mode)
        self.gen += 1
        cep.cep_begin_layer(ctx, self.gen, self.chunks_per_replica, out)
        if self.use_fetch:
            self.fetch_ready = cep.cep_weight_fetch(
                ctx, list(self.wl.fetched),
                [self.donor.data_ptr() + i * self.blob_bytes for i in range(len(self.wl.fetched))],
                self.side)
        seq = range(len(self.chunks)) if order is None else order
        # chunk inputs and `out` were written on the caller's stream: every
        # chunk becomes valid only after that work
        if inputs_ready and not (timed or arrival_events):
            ready = None
            self.arrival_events = []
        else:
            ready = torch.cuda.Event(enable_timing=True)
            ready.record(stream)
            self.dispatch.wait_event(ready)
            self.arrival_events = [ready]
        t0 = time.perf_counter()
        for i in seq:
            ch = self.chunks[i]
            ev = ready
            if timed:
                due = t0 + ch.arrival_ms * time_scale * 1e-3
                while time.perf_counter() < due:
                    pass
            if timed or arrival_events:
                ev = torch.cuda.Event(enable_timing=True)
                ev.record(self.dispatch)
                self.arrival_events.append(ev)
            cep.cep_submit_chunk(ctx, self.gen, ch.replica, ch.n_rows, ch.n_pairs, ch.token_idx,
                                 ch.x, ch.ids, ch.w, ev)
        return cep.cep_combine(ctx, stream)

    def run_subset(self, indices, stream=None):
        """One wait-all layer over the chunks `indices` (in that order) only,
        with resident inputs: a single grouped invocation of their pairs."""
        ctx = self.ctx
        stream = torch.cuda.current_stream(self.device) if stream is None else stream
        cpr = [0] * len(self.chunks_per_replica)
        for i in indices:
            cpr[self.chunks[i].replica] += 1
        cep.cep_set_policy(ctx, cep.CEP_WAIT_ALL, 1, 1)
        self.gen += 1
        cep.cep_begin_layer(ctx, self.gen, cpr, self.out)
        for i in indices:
            ch = self.chunks[i]
            cep.cep_submit_chunk(ctx, self.gen, ch.replica, ch.n_rows, ch.n_pairs, ch.token_idx,
                                 ch.x, ch.ids, ch.w, None)
        return cep.cep_combine(ctx, stream)

    def stats(self):
        return cep.cep_get_stats(self.ctx)

    def close(self):
        if getattr(self, "ctx", None):
            cep.cep_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

