"""Benchmark of the streamFFN routed-expert path on one MI355X.

Default run (one JSON line), every input seeded, synthetic and resident in
HBM before the timed region:

* headline -- the e4m3 workload: d_model 6144, expert d_ff 2560, 16 local
  experts of 160, top-8 with Zipf(1.5) popularity, 8 replicas x 8192 tokens
  (bf16 rows), e4m3 weights with 128x128 float32 block scales, 4 of the 16
  experts resident only in a donor region and copied once per layer on a
  side stream (their tiles gated by the copy).  One step is one layer
  through the whole path: open the layer, issue the weight fetch, submit
  every chunk (wait-all: one batch), histogram/scan/permute and e4m3 row
  quantisation, grouped GEMM1 with SwiGLU and h re-quantisation, grouped
  GEMM2, combine, layer barrier.  value = routed-expert FFN TFLOP/s =
  6 * d_model * d_ff * (local pairs) per step / time per step;
* roofline of the dominant kernel (the e4m3 grouped GEMM1, both launches of
  a layer: the resident experts' and, after the copy, the fetched
  experts'), from HIP events around each launch on the batch stream;
* fetch: how long the fetched experts' tiles waited for the copy, and the
  layer time against the same layer reading the fetched experts' weights in
  place from the donor region (no copy, the same launches);
* the 4096-wide bf16 workload (4 replicas x 2048 tokens, top-8 of 64, 8
  local experts, all chunks at once): TFLOP/s and its GEMM1 roofline;
* the straggler workload (d_model 7168, 8 replicas x 4096 tokens in 64
  chunks with lognormal gaps, replica 0 finishing 2x later): time to last
  chunk done and exposed tail under wait-all and under the threshold
  theta(0.9) on timed arrivals;
* the CPU oracle (float64 numpy) on a bounded sample of every workload, on
  all host threads and on one.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu]
       python bench.py --workload NAME [--policy wait_all|per_chunk|threshold --theta N
                       --streams S]       (one workload only)
       python bench.py --sweep | --matched-work | --calibrate-theta | --oewf-sim
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "routed-expert FFN TFLOP/s (% MFMA peak) + time-to-last-chunk-done, 1 GPU"
HEADLINE = "fp8_fetch_d6144"
# dense MFMA TFLOP/s, MI355X.  MXFP4 weights meet MXFP8 activations in one
# block-scaled MFMA, which issues at the fp8 rate when either operand is e4m3.
PEAK = {"bf16": 2500.0, "fp8": 5000.0, "mxfp4": 5000.0}
HBM_PEAK_GBS = 8000.0
# launch threshold theta(0.9) of the straggler workload, from the calibration
# (bench.py --calibrate-theta: the smallest profiled count at 0.9 of peak)
THETA_09 = 8192
# Measured HBM traffic of the dominant kernel (GEMM1) per launch: rocprofv3
# FETCH_SIZE x 2.0 + WRITE_SIZE x 1.0 KiB (factors from a 1 GiB copy), keyed
# by workload, valid only while the GEMM sources hash to the recorded sha1
# prefix (the report is null once the kernel changes).
GEMM_SOURCES = {
    "bf16": ["paper_2609_33252_amd/csrc/gemm_bf16.hip", "paper_2609_33252_amd/csrc/gemm_common.h"],
    "fp8": ["paper_2609_33252_amd/csrc/gemm_fp8.hip", "paper_2609_33252_amd/csrc/gemm_common.h"],
    "mxfp4": ["paper_2609_33252_amd/csrc/gemm_mx.hip", "paper_2609_33252_amd/csrc/gemm_common.h"],
}
TRAFFIC_BYTES = {  # workload -> (GEMM family, sha1 prefix of its sources, bytes per launch)
    "fp8_fetch_d6144": ("fp8", "41923e0288b7", 1833528987),
    "sync_d4096": ("bf16", "c12c043df95d", 504261285),
    "zipf_imbalanced_d7168/per_chunk": ("bf16", "c12c043df95d", 507424984),
    "mxfp4_dsv4flash_d4096": ("mxfp4", "a63161e27ae7", 1375766455),
}


def gemm_source_hash(dtype):
    import hashlib
    m = hashlib.sha1()
    for p in GEMM_SOURCES[dtype]:
        with open(os.path.join(ROOT, p), "rb") as f:
            m.update(f.read())
    return m.hexdigest()[:12]


def measured_traffic(workload):
    entry = TRAFFIC_BYTES.get(workload)
    if entry is None:
        return None
    dtype, sha, nbytes = entry
    return nbytes if gemm_source_hash(dtype) == sha else None


POLICIES = {"wait_all": 0, "per_chunk": 1, "threshold": 2}


def describe(cfg, name):
    return (f"{name}: d_model={cfg['d']}, d_ff={cfg['I']}, {cfg['E']} local experts of "
            f"{cfg['Eg']}, top-{cfg['k']} {'uniform' if cfg['zipf'] is None else 'Zipf(%s)' % cfg['zipf']}, "
            f"{cfg['R']} replicas x {cfg['T']} tokens, {cfg['R'] * cfg['cpr']} chunks, "
            f"{cfg['w']} weights" + (f", {len(cfg.get('_fetched', []))} experts fetched"
                                     if cfg.get('_fetched') else ""))


def dtype_of(wl):
    from paper_2609_33252_amd import workload as W
    return {W.FP8: "fp8", W.MXFP4: "mxfp4"}.get(wl.cfg["w"], "bf16")


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


_BANKS = {}


def cpu_oracle_rate(wl, budget_s, threads=None):
    """The CPU oracle as it stands (float64 numpy, the plain definition) on a
    bounded sample of the workload's delivered tokens (seeded order, batches
    doubling from 64 tokens, until budget_s of oracle time); threads: BLAS
    threads (None = all).  Returns the cpu_baseline record in TFLOP/s."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits
    from oracle import ffn
    import torch

    c = wl.cfg

    def bits(t):
        return None if t is None else (t.view(torch.int16).numpy().view(np.uint16)
                                       if t.dtype == torch.bfloat16 else t.numpy())
    kind = {"f32": "f32", "bf16": "bf16", "fp8_e4m3_b128": "fp8", "mxfp4": "mxfp4"}[c["w"]]
    # one decoded copy of the weights per workload (decoding is not timed)
    bank = _BANKS.get(id(wl))
    if bank is None:
        bank = _BANKS[id(wl)] = ffn.ExpertBank(
            kind, bits(wl.w_gate), bits(wl.w_up), bits(wl.w_down), bits(wl.s_gate),
            bits(wl.s_up), bits(wl.s_down))
    h_mode = {"f32": None, "bf16": "bf16", "fp8": "mxfp8", "mxfp4": "mxfp8"}[kind]
    x_mode = {"fp8": "mxfp8", "mxfp4": "mxfp8"}.get(kind)
    deliv = np.argwhere(wl.delivered)
    rng = np.random.default_rng(0)
    deliv = deliv[rng.permutation(len(deliv))]
    for e in range(c["E"]):      # decode weights outside the timed sample
        bank(e)
    # one untimed call first: starts the BLAS threads
    sel = deliv[:8]
    ffn.routed_output(ffn.decode_rows(bits(wl.x)[sel[:, 0], sel[:, 1]],
                                      "bf16" if c["x"] == "bf16" else "f32"),
                      wl.topk_local[sel[:, 0], sel[:, 1]], wl.topk_w[sel[:, 0], sel[:, 1]], bank,
                      c["E"], h_mode=h_mode, x_mode=x_mode)
    from contextlib import nullcontext
    with (threadpool_limits(limits=threads) if threads else nullcontext()):
        used = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        done_pairs, t_total, n_tok, step = 0, 0.0, 0, 64
        while t_total < budget_s and n_tok < len(deliv):
            sel = deliv[n_tok:n_tok + step]
            xb = bits(wl.x)[sel[:, 0], sel[:, 1]]
            ids = wl.topk_local[sel[:, 0], sel[:, 1]]
            w = wl.topk_w[sel[:, 0], sel[:, 1]]
            t0 = time.perf_counter()
            x = ffn.decode_rows(xb, "bf16" if c["x"] == "bf16" else "f32")
            ffn.routed_output(x, ids, w, bank, c["E"], h_mode=h_mode, x_mode=x_mode)
            t_total += time.perf_counter() - t0
            done_pairs += int((ids >= 0).sum())
            n_tok += len(sel)
            step = min(step * 2, 1024)
    flops = 6.0 * c["d"] * c["I"] * done_pairs
    return {"value": round(flops / t_total / 1e12, 5), "unit": "TFLOP/s", "cores": int(used),
            "kind": "oracle",
            "sample": f"{n_tok} delivered tokens ({done_pairs} pairs) of {wl.name}, float64 "
                      f"numpy, {t_total:.1f} s"}


def sweep(args):
    """Timed replay of a streaming workload under each launch policy: one
    JSON line per policy (mean over --steps layers after --warmup)."""
    import numpy as np
    import torch
    from paper_2609_33252_amd import cep, harness, streaming, workload as W

    wl = W.generate(args.workload, 0)
    c = wl.cfg
    run = harness.Runner(wl, n_streams=4)
    flops = 6.0 * c["d"] * c["I"] * run.n_pairs
    plan = [("wait_all", 1, 1), ("per_chunk", 1, 1), ("per_chunk", 1, 4)]
    thetas = [int(t) for t in args.thetas.split(",")]
    plan += [("threshold", t, s) for t in thetas for s in (1, 4)]
    # GEMM1 weight bytes of each expert (gate and up), and the local experts
    # each chunk touches: a batch streams the weights of every expert it
    # touches once, so GEMM1's weight rate is the streaming roofline figure
    w1_bytes = 2 * c["I"] * c["d"] * {W.BF16: 2, W.F32: 2, W.FP8: 1}.get(c["w"], 0.5)
    touched = [set(int(e) for e in np.unique(wl.topk_local[ch.replica][ch.token_idx]) if e >= 0)
               for ch in wl.chunks]
    base = None
    for name, theta, streams in plan:
        pol = POLICIES[name]
        res, wbytes, g1ms = [], 0.0, 0.0
        for i in range(args.warmup + args.steps):
            run.run(policy=pol, theta=theta, n_streams=streams, timed=True,
                    time_scale=args.time_scale)
            torch.cuda.synchronize()
            if i >= args.warmup:
                st = run.stats()
                res.append(streaming.layer_metrics(st, flops))
                for b in st["batches"]:
                    ex = set().union(*touched[b["first_chunk"]:b["first_chunk"] + b["n_chunks"]])
                    wbytes += len(ex) * w1_bytes
                    g1ms += b["gemm1_ms"]
        m = streaming.mean_metrics(res)
        if g1ms > 0:
            m["gemm1_weight_tbps"] = round(wbytes / (g1ms * 1e-3) / 1e12, 3)
            m["gemm1_weight_frac_hbm"] = round(wbytes / (g1ms * 1e-3) / 1e12 / (HBM_PEAK_GBS / 1e3), 4)
        if name == "wait_all":
            base = m
        line = {"workload": args.workload, "policy": name, "theta": theta, "streams": streams,
                "time_scale": args.time_scale, "local_pairs": run.n_pairs, **m}
        if base and m.get("busy_tflops") and base.get("busy_tflops"):
            line["ffn_efficiency_vs_wait_all"] = m["busy_tflops"] / base["busy_tflops"]
            line["exposed_tail_vs_wait_all"] = m["exposed_tail_ms"] / base["exposed_tail_ms"]
        print(json.dumps(line), flush=True)
    cep.cep_get_status(run.ctx)
    run.close()


def matched_work(args):
    """Matched-work FFN throughput: the same layer (same weights, same
    per-expert token counts) run as one wait-all invocation and as streamed
    invocations (per chunk, or threshold theta) on 1..4 streams, inputs
    resident and no arrival timing, so only the batching and the stream
    overlap differ.  One JSON line per (policy, theta, streams) with the
    layer's throughput and its ratio to wait-all on one stream."""
    import torch
    from paper_2609_33252_amd import cep, harness, workload as W

    wl = W.generate(args.workload, 0)
    c = wl.cfg
    run = harness.Runner(wl, n_streams=4)
    flops = 6.0 * c["d"] * c["I"] * run.n_pairs
    thetas = [int(t) for t in args.thetas.split(",")]
    plan = [("wait_all", 1, 1)] + [("per_chunk", 1, s) for s in (1, 2, 4)]
    plan += [("threshold", t, s) for t in thetas for s in (1, 2, 4)]
    cep.cep_set_phase_timing(run.ctx, False)

    def layer_ms(pol, theta, streams):
        for _ in range(args.warmup):
            run.run(policy=pol, theta=theta, n_streams=streams, inputs_ready=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            run.run(policy=pol, theta=theta, n_streams=streams, inputs_ready=True)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / args.steps * 1e3

    # the GPU reaches its steady clocks only after some layers: a warm-up
    # well beyond --warmup comes first; then wait-all is timed before and
    # after the others and the base is the mean of the two, so drift over
    # the run does not favour either side
    for _ in range(max(20, 4 * args.warmup)):
        run.run(policy=cep.CEP_WAIT_ALL, theta=1, n_streams=1, inputs_ready=True)
    first = layer_ms(cep.CEP_WAIT_ALL, 1, 1)
    runs = []
    for name, theta, streams in plan[1:]:
        ms = layer_ms(POLICIES[name], theta, streams)
        runs.append((name, theta, streams, cep.cep_get_batch_count(run.ctx), ms))
    last = layer_ms(cep.CEP_WAIT_ALL, 1, 1)
    base = flops / ((first + last) / 2) / 1e9
    runs = [("wait_all", 1, 1, 1, (first + last) / 2)] + runs
    for name, theta, streams, n_batches, ms in runs:
        tflops = flops / ms / 1e9
        line = {"workload": args.workload, "policy": name, "theta": theta,
                "streams": streams, "batches": n_batches, "ms_per_layer": round(ms, 4),
                "tflops": round(tflops, 2), "throughput_vs_wait_all": round(tflops / base, 4)}
        if name == "wait_all":
            line["wait_all_first_last_ms"] = [round(first, 4), round(last, 4)]
        print(json.dumps(line), flush=True)
    cep.cep_get_status(run.ctx)
    run.close()


def calibrate_theta(args):
    """Launch-threshold calibration: FFN throughput of one grouped invocation
    against its expert-token count N (prefixes of the streaming workload's
    chunks in arrival order, wait-all over each prefix), the library's
    profile of it, theta(rho) and F(N).  One JSON line per profiled count,
    one per held-out count (F(N) prediction vs measured), and a summary."""
    import statistics

    import torch
    from paper_2609_33252_amd import cep, harness, workload as W

    wl = W.generate(args.workload, 0, cpr=args.cal_cpr)
    c = wl.cfg
    run = harness.Runner(wl, n_streams=1)
    order = sorted(range(len(run.chunks)), key=lambda i: run.chunks[i].arrival_ms)
    cum, tot = [], 0
    for i in order:
        tot += run.chunks[i].n_pairs
        cum.append(tot)

    def measure(m):
        # batch span (routing .. combine) of a layer over the first m+1 chunks
        sub = order[:m + 1]
        span = []
        for it in range(args.warmup + args.steps):
            run.run_subset(sub)
            torch.cuda.synchronize()
            if it >= args.warmup:
                b = run.stats()["batches"][0]
                span.append(b["end_ms"] - b["start_ms"])
        return statistics.median(span)

    def prefix_for(target):
        return next(m for m, v in enumerate(cum) if v >= target)

    # profiled prefixes: N ~ 16 x 2^(j/2) up to all pairs, plus the last
    # prefix below and the first at or above each count where the library
    # changes its row tile (64 and 256 rows per local expert on average), so
    # that the piecewise-linear profile does not cut across those steps
    picks = set()
    target = 16.0
    while True:
        picks.add(prefix_for(min(int(target), tot)))
        if target >= tot:
            break
        target *= 2 ** 0.5
    for per_expert in (64, 256):
        step = per_expert * c["E"]
        if step <= tot:
            m_at = prefix_for(step)
            picks.add(m_at)
            if m_at > 0:
                picks.add(m_at - 1)
    counts, tput = [], []
    for m in sorted(picks):
        if counts and cum[m] <= counts[-1]:
            continue
        ms = measure(m)
        counts.append(cum[m])
        tput.append(cum[m] / ms)
        print(json.dumps({"profile_n": cum[m], "ms": round(ms, 5),
                          "pairs_per_ms": round(cum[m] / ms, 2),
                          "tflops": round(6.0 * c["d"] * c["I"] * cum[m] / ms / 1e9, 2)}),
              flush=True)
    prof = cep.FfnProfile(counts, tput)
    blob_bytes = run.blob_bytes
    # held-out counts (geometric midpoints): model F(N) against measurement
    errs = []
    for a, b in zip(counts, counts[1:]):
        m = prefix_for(int((a * b) ** 0.5))
        if cum[m] in (a, b):
            continue
        ms = measure(m)
        pred = prof.latency(cum[m])
        errs.append(abs(pred - ms) / ms)
        print(json.dumps({"heldout_n": cum[m], "measured_ms": round(ms, 5),
                          "model_ms": round(pred, 5), "rel_err": round(errs[-1], 4)}),
              flush=True)
    line = {"workload": args.workload, "chunks_per_replica": args.cal_cpr, "rho": args.rho,
            "theta": prof.theta(args.rho), "peak_pairs_per_ms": round(prof.peak, 2),
            "eta": {str(n): round(prof.eta(n), 4) for n in counts},
            "heldout_mean_rel_err": round(sum(errs) / len(errs), 4) if errs else None}
    print(json.dumps(line), flush=True)
    prof.close()
    cep.cep_get_status(run.ctx)
    run.close()
    return counts, tput, blob_bytes


def oewf_sim(args):
    """OEWF coordinator on simulated imbalanced layers, with the FFN latency
    model measured on this GPU (the --calibrate-theta profile) and this
    workload's expert size: layer completion with and without weight
    fetching, commits, and the coordinator's call latency."""
    import numpy as np

    from paper_2609_33252_amd import cep, layer_sim

    counts, tput, blob = calibrate_theta(args)
    prof = cep.FfnProfile(counts, tput)
    rng = np.random.default_rng(0)
    R, E = 8, 8
    bw = args.fetch_gbps * 1e6          # bytes per ms
    budget = args.fetch_experts * blob
    ratios, commits, improved = [], 0, 0
    t_calls, n_calls = 0.0, 0

    class Timed:
        def __init__(self, co):
            self.co = co

        def __getattr__(self, name):
            f = getattr(self.co, name)

            def g(*a, **k):
                nonlocal t_calls, n_calls
                t0 = time.perf_counter()
                out = f(*a, **k)
                t_calls += time.perf_counter() - t0
                n_calls += 1
                return out
            return g

    for _ in range(args.oewf_layers):
        attn, disp, tok, _ = layer_sim.random_layer(rng, R, E)
        b = np.full(E, blob, dtype=np.int64)
        co = cep.Coordinator(R, prof)
        base, final, c, _ = layer_sim.simulate(Timed(co), prof.latency, attn, disp, tok, b,
                                               budget=budget, bw=bw, rng=rng)
        co.close()
        ratios.append(final / base)
        commits += c
        improved += final < base * (1 - 1e-9)
    line = {"oewf_layers": args.oewf_layers, "ranks": R, "experts_per_rank": E,
            "expert_bytes": blob, "fetch_budget_experts": args.fetch_experts,
            "fetch_gbps": args.fetch_gbps,
            "layer_time_ratio_mean": round(float(np.mean(ratios)), 4),
            "layer_time_ratio_min": round(float(np.min(ratios)), 4),
            "layer_time_ratio_max": round(float(np.max(ratios)), 4),
            "layers_improved": improved, "commits": commits,
            "coordinator_call_us": round(t_calls / max(n_calls, 1) * 1e6, 2)}
    print(json.dumps(line), flush=True)
    prof.close()


# ------------------------------------------------------------- default run
def batch_pairs(wl, st, fetched):
    """(pairs of resident experts, pairs of fetched experts, experts touched
    by each) of every batch of one layer's statistics."""
    import numpy as np
    out = []
    fset = np.asarray(sorted(fetched), dtype=np.int64)
    for b in st["batches"]:
        ids = np.concatenate([
            wl.topk_local[wl.chunks[c].replica][wl.chunks[c].token_idx].ravel()
            for c in range(b["first_chunk"], b["first_chunk"] + b["n_chunks"])])
        ids = ids[ids >= 0]
        is_f = np.isin(ids, fset) if (b["fetched"] and len(fset)) else np.zeros(len(ids), bool)
        out.append((int((~is_f).sum()), int(is_f.sum()),
                    len(np.unique(ids[~is_f])), len(np.unique(ids[is_f]))))
    return out


def gemm1_roofline(wl, stats, fetched, dtype, workload_key):
    """Roofline of the grouped GEMM1 over every GEMM1 launch of the layers in
    `stats` (the resident experts', and the fetched experts' after the copy,
    both on the batch stream and never overlapping): achieved = mean
    algorithmic work per launch / mean launch duration (HIP events around
    the launches on the batch stream)."""
    from paper_2609_33252_amd import workload as W
    c = wl.cfg
    elem = {W.BF16: 2, W.F32: 2, W.FP8: 1}.get(c["w"], 0.5)
    xel = 2 if dtype == "bf16" else 1
    flops = bytes_ = dur = 0.0
    n = 0
    for st in stats:
        for b, (pr, pf, er, ef) in zip(st["batches"], batch_pairs(wl, st, fetched)):
            for pairs, experts, ms in ((pr, er, b["gemm1_ms"]),
                                       (pf, ef, b["fetched_gemm1_ms"] if b["fetched"] else -1)):
                if ms < 0:
                    continue
                flops += 4.0 * c["d"] * c["I"] * pairs
                # gate/up weights of every expert the launch touches (each
                # streamed once), the launch's rows in and h out
                bytes_ += experts * 2.0 * c["I"] * c["d"] * elem + pairs * (c["d"] + c["I"]) * xel
                dur += ms
                n += 1
    f1, b1, ms1 = flops / n, bytes_ / n, dur / n
    hbm = b1 / (HBM_PEAK_GBS * 1e9) > f1 / (PEAK[dtype] * 1e12)
    kern = {"bf16": "k_gemm_bf16", "fp8": "k_gemm_fp8", "mxfp4": "k_gemm_mx"}[dtype]
    r = {"kernel": f"{kern}<SwiGLU> (grouped gate/up GEMM, every launch of the layer)",
         "launches": n, "launch_ms": round(ms1, 4), "traffic": measured_traffic(workload_key)}
    if hbm:
        a = b1 / (ms1 * 1e-3) / 1e9
        r.update(bound="hbm", achieved=round(a, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                 frac=round(a / HBM_PEAK_GBS, 4), bytes_per_launch=round(b1))
    else:
        a = f1 / (ms1 * 1e-3) / 1e12
        r.update(bound="mfma", achieved=round(a, 2), peak=PEAK[dtype], unit="TFLOP/s",
                 frac=round(a / PEAK[dtype], 4), flop_per_launch=f1)
    return {k: r[k] for k in ("bound", "achieved", "peak", "unit", "frac", "traffic", "kernel",
                              "launches", "launch_ms") + (("bytes_per_launch",) if hbm else
                                                          ("flop_per_launch",))}


def timed_layers(run, warmup, steps, **kw):
    """Wall time per layer (ms) of `steps` layers after `warmup`, bracketed
    by device synchronisation; per-phase events off."""
    import torch
    from paper_2609_33252_amd import cep
    cep.cep_set_phase_timing(run.ctx, False)
    for _ in range(warmup):
        run.run(**kw)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        run.run(**kw)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / steps * 1e3
    from paper_2609_33252_amd import cep as _c
    _c.cep_get_status(run.ctx)
    cep.cep_set_phase_timing(run.ctx, True)
    return ms


def phase_layers(run, steps, **kw):
    """Statistics of `steps` layers with per-phase events."""
    out = []
    for _ in range(steps):
        run.run(**kw)
        out.append(run.stats())
    return out


def mean(v):
    return sum(v) / len(v)


def full_bench(args):
    import torch
    from paper_2609_33252_amd import cep, harness, streaming, workload as W

    torch.cuda.set_device(0)
    K, Wm = args.steps, args.warmup
    line = {}

    # ---- headline: e4m3 workload with the weight fetch, wait-all
    wl = W.generate(HEADLINE, 0)
    c = wl.cfg
    run = harness.Runner(wl, n_streams=1)
    P = run.n_pairs
    flops = 6.0 * c["d"] * c["I"] * P
    kw = dict(policy=cep.CEP_WAIT_ALL, inputs_ready=True)
    ms = timed_layers(run, Wm, K, **kw)
    value = flops / (ms * 1e-3) / 1e12
    st = phase_layers(run, K, **kw)
    fetched = list(wl.fetched)
    phases = {k: round(mean([sum(b[k] for b in s["batches"]) for s in st]), 4)
              for k in ("route_ms", "gemm1_ms", "gemm2_ms", "combine_ms", "fetched_gemm1_ms",
                        "fetched_gemm2_ms")}
    copy_ms = [s["fetch"]["end_ms"] - s["fetch"]["start_ms"] for s in st]
    fbytes = st[0]["fetch"]["bytes"]
    # the fetched experts' tiles follow the resident experts' GEMM2 on the
    # batch stream: they waited for the copy from GEMM2's end to their start
    wait = [max(0.0, b["fetched_start_ms"] - (b["start_ms"] + b["route_ms"] + b["gemm1_ms"] +
                                              b["gemm2_ms"]))
            for s in st for b in s["batches"] if b["fetched"]]
    roof = gemm1_roofline(wl, st, fetched, "fp8", HEADLINE)
    # the same layer reading the fetched experts' weights in place: the same
    # launches without the copy
    ms_in = timed_layers(run, Wm, K, fetch_mode=cep.CEP_FETCH_IN_PLACE, **kw)
    cep.cep_set_fetch_mode(run.ctx, cep.CEP_FETCH_COPY)
    cep.cep_get_status(run.ctx)
    run.close()
    del run
    c = dict(c, _fetched=fetched)
    line.update({
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": K, "warmup": Wm, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp8", "data": "synthetic",
        "config": {"workload": describe(c, HEADLINE), "local_pairs": P, "policy": "wait_all",
                   "streams": 1, "global_batch": c["R"] * c["T"], "seq_len": c["T"],
                   "parallelism": "ep_share_1gpu"},
        "pct_mfma_peak": round(100 * value / PEAK["fp8"], 2),
        "phases_ms": phases,
        "roofline": roof,
        "fetch": {"experts": len(fetched), "bytes": fbytes,
                  "copy_ms": round(mean(copy_ms), 4),
                  "copy_gbps": round(fbytes / (mean(copy_ms) * 1e-3) / 1e9, 1),
                  "fetched_tiles_waited_ms": round(mean(wait), 4),
                  "layer_ms_with_copy": round(ms, 4),
                  "layer_ms_in_place": round(ms_in, 4),
                  "copy_cost_ms": round(ms - ms_in, 4),
                  "note": "with_copy: the headline layer; in_place: the fetched experts read "
                          "from the donor region, same launches, no copy (both wall time per "
                          "layer); waited: fetched tiles' start minus the resident GEMM2 end"},
    })
    print(json.dumps({"progress": "headline", "value": line["value"]}), file=sys.stderr,
          flush=True)

    # ---- 4096-wide bf16 workload, all chunks at once
    wl2 = W.generate("sync_d4096", 0)
    c2 = wl2.cfg
    run = harness.Runner(wl2, n_streams=1)
    ms2 = timed_layers(run, Wm, K, **kw)
    st2 = phase_layers(run, K, **kw)
    f2 = 6.0 * c2["d"] * c2["I"] * run.n_pairs
    cep.cep_get_status(run.ctx)
    line["sync_d4096"] = {
        "workload": describe(c2, "sync_d4096"), "local_pairs": run.n_pairs,
        "ms_per_layer": round(ms2, 4), "tflops": round(f2 / (ms2 * 1e-3) / 1e12, 2),
        "pct_mfma_peak": round(100 * f2 / (ms2 * 1e-3) / 1e12 / PEAK["bf16"], 2),
        "phases_ms": {k: round(mean([sum(b[k] for b in s["batches"]) for s in st2]), 4)
                      for k in ("route_ms", "gemm1_ms", "gemm2_ms", "combine_ms")},
        "roofline": gemm1_roofline(wl2, st2, [], "bf16", "sync_d4096")}
    run.close()
    del run
    print(json.dumps({"progress": "sync_d4096"}), file=sys.stderr, flush=True)

    # ---- timed arrivals: wait-all against theta(0.9) and the smaller launch
    # thresholds of the comparison (theta 1024 / 4096 pairs per launch and
    # per-chunk batches)
    def timed_policies(run, flop, policies):
        res = {}
        for name, pol, theta, ns in policies:
            ms_ = []
            for i in range(1 + args.timed_layers):
                run.run(policy=pol, theta=theta, n_streams=ns, timed=True)
                torch.cuda.synchronize()
                if i:
                    ms_.append(streaming.layer_metrics(run.stats(), flop))
            m = streaming.mean_metrics(ms_)
            res[name] = {"batches": m["batches"],
                         "time_to_last_chunk_done_ms": round(m["time_to_last_chunk_done_ms"], 4),
                         "last_arrival_ms": round(m["last_arrival_ms"], 4),
                         "exposed_tail_ms": round(m["exposed_tail_ms"], 4),
                         "chunk_latency_p50_ms": round(m["chunk_latency_ms"]["p50"], 4),
                         "chunk_latency_p95_ms": round(m["chunk_latency_ms"]["p95"], 4),
                         "busy_tflops": round(m["busy_tflops"], 2)}
        return res
    WA = ("wait_all", cep.CEP_WAIT_ALL, 1, 1)
    TH = (f"theta_{THETA_09}", cep.CEP_THRESHOLD, THETA_09, 2)
    PC = ("per_chunk", cep.CEP_PER_CHUNK, 1, 2)

    # the lognormal-arrival workload without a straggler (each replica's
    # eight chunks arrive with lognormal gaps)
    wl3 = W.generate("zipf_stream_d7168", 0)
    run = harness.Runner(wl3, n_streams=2)
    res3 = timed_policies(run, 6.0 * wl3.cfg["d"] * wl3.cfg["I"] * run.n_pairs, (WA, TH, PC))
    cep.cep_get_status(run.ctx)
    run.close()
    del run

    # the straggler workload
    wl4 = W.generate("zipf_imbalanced_d7168", 0)
    c4 = wl4.cfg
    run = harness.Runner(wl4, n_streams=2)
    f4 = 6.0 * c4["d"] * c4["I"] * run.n_pairs
    res = timed_policies(run, f4, (WA, TH, ("theta_4096", cep.CEP_THRESHOLD, 4096, 2),
                                   ("theta_1024", cep.CEP_THRESHOLD, 1024, 2), PC))
    # matched work (the same layer, inputs resident, no arrival timing):
    # wait-all on one stream against theta(0.9) on two streams and per-chunk
    # batches, wait-all timed before and after the others; then the
    # per-chunk batches' GEMM1 against the HBM roofline (weight streaming)
    def mw_ms(pol, theta, ns, n=5):
        for _ in range(2):
            run.run(policy=pol, theta=theta, n_streams=ns, inputs_ready=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n):
            run.run(policy=pol, theta=theta, n_streams=ns, inputs_ready=True)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / n * 1e3
    cep.cep_set_phase_timing(run.ctx, False)
    for _ in range(10):
        run.run(policy=cep.CEP_WAIT_ALL, inputs_ready=True)
    first = mw_ms(cep.CEP_WAIT_ALL, 1, 1)
    mw_th = mw_ms(cep.CEP_THRESHOLD, THETA_09, 2)
    mw_pc = mw_ms(cep.CEP_PER_CHUNK, 1, 1)
    base = (first + mw_ms(cep.CEP_WAIT_ALL, 1, 1)) / 2
    cep.cep_set_phase_timing(run.ctx, True)
    st_pc = []
    for i in range(3):
        run.run(policy=cep.CEP_PER_CHUNK, n_streams=1, inputs_ready=True)
        torch.cuda.synchronize()
        if i:
            st_pc.append(run.stats())
    line["matched_work"] = {
        "note": "same layer, inputs resident, no arrival timing; ms per layer",
        "wait_all_ms": round(base, 4), f"theta_{THETA_09}_2_streams_ms": round(mw_th, 4),
        "per_chunk_ms": round(mw_pc, 4),
        f"theta_{THETA_09}_throughput_vs_wait_all": round(base / mw_th, 4),
        "per_chunk_throughput_vs_wait_all": round(base / mw_pc, 4)}
    line["streaming_roofline"] = gemm1_roofline(wl4, st_pc, [], "bf16",
                                                "zipf_imbalanced_d7168/per_chunk")
    cep.cep_get_status(run.ctx)
    run.close()
    del run
    wa, th = res["wait_all"], res[f"theta_{THETA_09}"]
    line["time_to_last_chunk_done"] = {
        "workload": describe(c4, "zipf_imbalanced_d7168"), "local_pairs": wl4.n_pairs,
        "arrivals": "timed: lognormal(0, 0.5) ms gaps, replica 0 scaled 2x, others U[1, 1.5]x",
        "layers": args.timed_layers, **res,
        "exposed_tail_ratio": round(th["exposed_tail_ms"] / wa["exposed_tail_ms"], 4),
        "busy_tflops_ratio": round(th["busy_tflops"] / wa["busy_tflops"], 4)}
    wa3, th3 = res3["wait_all"], res3[f"theta_{THETA_09}"]
    line["time_to_last_chunk_done_no_straggler"] = {
        "workload": describe(wl3.cfg, "zipf_stream_d7168"), "local_pairs": wl3.n_pairs,
        "arrivals": "timed: lognormal(0, 0.5) ms gaps, no straggler",
        "layers": args.timed_layers, **res3,
        "exposed_tail_ratio": round(th3["exposed_tail_ms"] / wa3["exposed_tail_ms"], 4),
        "busy_tflops_ratio": round(th3["busy_tflops"] / wa3["busy_tflops"], 4)}
    print(json.dumps({"progress": "straggler"}), file=sys.stderr, flush=True)

    # ---- targets of the path, as measured here
    line["targets"] = {
        "bf16_gemm1_mfma_frac_ge_0.60": line["sync_d4096"]["roofline"]["frac"] >= 0.60,
        "fp8_gemm1_mfma_frac": roof["frac"],
        "streaming_hbm_frac_ge_0.70": line["streaming_roofline"]["frac"] >= 0.70,
        "streaming_lowers_exposed_tail": (th["exposed_tail_ms"] < wa["exposed_tail_ms"] and
                                          th3["exposed_tail_ms"] < wa3["exposed_tail_ms"])}

    # ---- the CPU oracle
    if not args.no_cpu:
        per = {}
        gens = {HEADLINE: wl, "sync_d4096": wl2, "zipf_stream_d7168": wl3,
                "zipf_imbalanced_d7168": wl4}
        for name in W.CONFIG_ORDER:
            w_ = gens.get(name) or W.generate(name, 0)
            per[name] = {"all_threads": cpu_oracle_rate(w_, args.cpu_budget),
                         "one_thread": cpu_oracle_rate(w_, args.cpu_budget / 2, threads=1)}
            _BANKS.clear()
        line["cpu_baseline"] = per[HEADLINE]["all_threads"]
        line["cpu_baseline_per_config"] = {
            "cpu_model": cpu_model(), "affinity_cpus": len(os.sched_getaffinity(0)), **per}
    print(json.dumps(line), flush=True)


def single_workload(args):
    """One workload (--workload): the line of full_bench's headline for it."""
    import torch
    from paper_2609_33252_amd import cep, harness, workload as W

    torch.cuda.set_device(0)
    wl = W.generate(args.workload, 0)
    c = wl.cfg
    run = harness.Runner(wl, n_streams=max(1, args.streams), use_fetch=not args.no_fetch)
    pol = POLICIES[args.policy]
    dtype = dtype_of(wl)
    kw = dict(policy=pol, theta=args.theta, n_streams=args.streams, inputs_ready=True)
    ms = timed_layers(run, args.warmup, args.steps, **kw)
    flops = 6.0 * c["d"] * c["I"] * run.n_pairs
    value = flops / (ms * 1e-3) / 1e12
    st = phase_layers(run, args.steps, **kw)
    fetched = list(wl.fetched) if run.use_fetch else []
    key = args.workload if args.policy == "wait_all" else f"{args.workload}/{args.policy}"
    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": describe(dict(c, _fetched=fetched), args.workload),
                   "local_pairs": run.n_pairs, "policy": args.policy, "theta": args.theta,
                   "streams": args.streams, "global_batch": c["R"] * c["T"], "seq_len": c["T"],
                   "parallelism": "ep_share_1gpu"},
        "pct_mfma_peak": round(100 * value / PEAK[dtype], 2),
        "phases_ms": {k: round(mean([sum(b[k] for b in s["batches"]) for s in st]), 4)
                      for k in ("route_ms", "gemm1_ms", "gemm2_ms", "combine_ms")},
        "roofline": gemm1_roofline(wl, st, fetched, dtype, key),
    }
    cep.cep_get_status(run.ctx)
    run.close()
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_oracle_rate(wl, args.cpu_budget)
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None,
                    help="run one workload only (default: the full run described above)")
    ap.add_argument("--policy", default="wait_all", choices=list(POLICIES))
    ap.add_argument("--theta", type=int, default=1)
    ap.add_argument("--streams", type=int, default=1)
    ap.add_argument("--no-fetch", action="store_true",
                    help="--workload: keep every expert resident")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-budget", type=float, default=2.0,
                    help="seconds of oracle time per workload and thread setting")
    ap.add_argument("--timed-layers", type=int, default=3,
                    help="timed-arrival layers per policy of the straggler workload")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run device-to-device copies of MIB MiB (counter calibration)")
    ap.add_argument("--sweep", action="store_true",
                    help="timed-arrival replay under every launch policy (one JSON line each)")
    ap.add_argument("--thetas", default="32,64,128,256,512,1024,2048,4096")
    ap.add_argument("--time-scale", type=float, default=1.0,
                    help="scale of the arrival schedule in --sweep (1 = as generated)")
    ap.add_argument("--matched-work", action="store_true",
                    help="wait-all vs streamed invocations on identical resident inputs")
    ap.add_argument("--calibrate-theta", action="store_true",
                    help="profile FFN throughput vs expert-token count; theta(rho) and F(N)")
    ap.add_argument("--rho", type=float, default=0.9)
    ap.add_argument("--cal-cpr", type=int, default=64,
                    help="chunks per replica of the calibration workload (finer prefixes)")
    ap.add_argument("--oewf-sim", action="store_true",
                    help="calibrate, then run the OEWF coordinator on simulated layers")
    ap.add_argument("--oewf-layers", type=int, default=200)
    ap.add_argument("--fetch-gbps", type=float, default=153.0,
                    help="donor-to-helper copy bandwidth (one xGMI link)")
    ap.add_argument("--fetch-experts", type=int, default=4,
                    help="fetch buffer capacity in experts (byte budget B_h)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the library has no multi-GPU path "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        import torch
        n = args.calibrate_copy << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "copies": args.steps}))
        return

    from paper_2609_33252_amd import cep
    if not os.path.exists(cep.LIB_PATH):
        from paper_2609_33252_amd import build
        build.build()
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.sweep or args.matched_work or args.calibrate_theta or args.oewf_sim:
        if args.workload is None:
            args.workload = "zipf_imbalanced_d7168"
        fn = (oewf_sim if args.oewf_sim else calibrate_theta if args.calibrate_theta
              else matched_work if args.matched_work else sweep)
        fn(args)
        return
    if args.workload is not None:
        single_workload(args)
        return
    full_bench(args)


if __name__ == "__main__":
    main()
