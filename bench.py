"""Benchmark of the streamFFN routed-expert path on one MI355X.

Workload (the synchronous-EP shape): d_model 4096, expert d_ff 2048, 8 local
experts, 4 replicas x 2048 tokens routed top-8 over 64 experts uniformly, one
chunk per replica, all arriving together, bf16 weights and tokens.  One step
is one layer through the whole path: open the layer, submit every chunk (the
launch policy forms the batch), histogram/scan/permute, grouped GEMM1 with
SwiGLU, grouped GEMM2, combine, layer barrier.  Inputs are resident in HBM
before the timed region.

value = routed-expert FFN TFLOP/s = 6 * d_model * d_ff * (local pairs) per
step / time per step.  The JSON line also carries the roofline of the
dominant kernel (grouped GEMM1, timed with HIP events on its own stream) and
the CPU oracle's throughput on a bounded sample.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
       [--workload NAME] [--policy wait_all|per_chunk|threshold --theta N --streams S]
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
# dense MFMA TFLOP/s, MI355X.  MXFP4 weights meet MXFP8 activations in one
# block-scaled MFMA, which issues at the fp8 rate when either operand is e4m3.
PEAK = {"bf16": 2500.0, "fp8": 5000.0, "mxfp4": 5000.0}
HBM_PEAK_GBS = 8000.0
# Measured HBM traffic of the dominant kernel (GEMM1) per batch: rocprofv3
# FETCH_SIZE x 2.0 + WRITE_SIZE x 1.0 KiB (factors from a 1 GiB copy), keyed
# by workload, valid only while the GEMM sources hash to the recorded sha1
# prefix (the report is null once the kernel changes).
GEMM_SOURCES = {
    "bf16": ["paper_2609_33252_amd/csrc/gemm_bf16.hip", "paper_2609_33252_amd/csrc/gemm_common.h"],
    "mxfp4": ["paper_2609_33252_amd/csrc/gemm_mx.hip", "paper_2609_33252_amd/csrc/gemm_common.h"],
}
TRAFFIC_BYTES = {  # workload -> (GEMM family, sha1 prefix of its sources, bytes per batch)
    "sync_d4096": ("bf16", "c3b56bd685eb", 504303616),
    "zipf_imbalanced_d7168/per_chunk": ("bf16", "c3b56bd685eb", 473822208),
    "mxfp4_dsv4flash_d4096": ("mxfp4", "52e124864ab3", 1369075712),
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
            f"{cfg['w']} weights")


def cpu_baseline(wl, budget_s=12.0):
    """The CPU oracle as it stands, on a bounded sample of the same workload's
    delivered tokens; returns TFLOP/s over the pairs it computed."""
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import ffn
    import torch

    c = wl.cfg

    def bits(t):
        return None if t is None else (t.view(torch.int16).numpy().view(np.uint16)
                                       if t.dtype == torch.bfloat16 else t.numpy())
    kind = {"f32": "f32", "bf16": "bf16", "fp8_e4m3_b128": "fp8", "mxfp4": "mxfp4"}[c["w"]]
    bank = ffn.ExpertBank(kind, bits(wl.w_gate), bits(wl.w_up), bits(wl.w_down),
                          bits(wl.s_gate), bits(wl.s_up), bits(wl.s_down))
    h_mode = {"f32": None, "bf16": "bf16", "fp8": "fp8", "mxfp4": "mxfp8"}[kind]
    x_mode = {"fp8": "fp8", "mxfp4": "mxfp8"}.get(kind)
    deliv = np.argwhere(wl.delivered)
    rng = np.random.default_rng(0)
    deliv = deliv[rng.permutation(len(deliv))]
    for e in range(c["E"]):      # decode weights outside the timed sample
        bank(e)
    done_pairs, t_total, n_tok, step = 0, 0.0, 0, 64
    while t_total < budget_s and n_tok < len(deliv):
        sel = deliv[n_tok:n_tok + step]
        xb = bits(wl.x)[sel[:, 0], sel[:, 1]]
        ids = wl.topk_local[sel[:, 0], sel[:, 1]]
        w = wl.topk_w[sel[:, 0], sel[:, 1]]
        t0 = time.perf_counter()
        x = ffn.decode_rows(xb, "bf16" if c["x"] == "bf16" else "f32")
        ffn.routed_output(x, ids, w, bank, c["E"], h_mode=h_mode, x_mode=x_mode, y_mode="bf16")
        t_total += time.perf_counter() - t0
        done_pairs += int((ids >= 0).sum())
        n_tok += len(sel)
        step = min(step * 2, 1024)
    flops = 6.0 * c["d"] * c["I"] * done_pairs
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": flops / t_total / 1e12, "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{n_tok} delivered tokens ({done_pairs} pairs) of the same workload, "
                      f"float64 numpy, {t_total:.1f} s"}


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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="sync_d4096")
    ap.add_argument("--policy", default="wait_all", choices=list(POLICIES))
    ap.add_argument("--theta", type=int, default=1)
    ap.add_argument("--streams", type=int, default=1)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
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
    if args.oewf_sim:
        if args.workload == "sync_d4096":
            args.workload = "zipf_imbalanced_d7168"
        oewf_sim(args)
        return
    if args.calibrate_theta:
        if args.gpus != 1:
            print("bench.py runs on one GPU only", file=sys.stderr)
            sys.exit(2)
        if args.workload == "sync_d4096":
            args.workload = "zipf_imbalanced_d7168"
        calibrate_theta(args)
        return
    if args.matched_work:
        if args.gpus != 1:
            print("bench.py runs on one GPU only", file=sys.stderr)
            sys.exit(2)
        if args.workload == "sync_d4096":
            args.workload = "zipf_imbalanced_d7168"
        matched_work(args)
        return
    if args.sweep:
        if args.gpus != 1:
            print("bench.py runs on one GPU only", file=sys.stderr)
            sys.exit(2)
        if args.workload == "sync_d4096":
            args.workload = "zipf_imbalanced_d7168"
        sweep(args)
        return
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
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the library has no multi-GPU path "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_33252_amd import cep, harness, workload as W

    if not os.path.exists(cep.LIB_PATH):
        from paper_2609_33252_amd import build
        build.build()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)

    wl = W.generate(args.workload, 0)
    c = wl.cfg
    run = harness.Runner(wl, n_streams=max(1, args.streams))
    pol = POLICIES[args.policy]
    flops_step = 6.0 * c["d"] * c["I"] * run.n_pairs
    dtype = {W.FP8: "fp8", W.MXFP4: "mxfp4"}.get(c["w"], "bf16")

    # the chunk inputs are generated once and resident in HBM: steady-state
    # layers carry no arrival events (the library orders each layer after the
    # previous one's batches itself)
    def step():
        run.run(policy=pol, theta=args.theta, n_streams=args.streams, inputs_ready=True)

    # timed steps without per-phase events (instrumentation, not work); the
    # phase pass below turns them back on
    cep.cep_set_phase_timing(run.ctx, False)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    cep.cep_get_status(run.ctx)
    cep.cep_set_phase_timing(run.ctx, True)
    ms_step = elapsed / args.steps * 1e3
    value = flops_step / (elapsed / args.steps) / 1e12

    # kernel phases of each step, from HIP events on the batch stream
    ph = {"route_ms": [], "gemm1_ms": [], "gemm2_ms": [], "combine_ms": [], "last_done_ms": []}
    for _ in range(args.steps):
        step()
        st = run.stats()
        for key in ("route_ms", "gemm1_ms", "gemm2_ms", "combine_ms"):
            ph[key].append(sum(b[key] for b in st["batches"]))
        ph["last_done_ms"].append(max(b["end_ms"] for b in st["batches"]))
    avg = {k: sum(v) / len(v) for k, v in ph.items()}
    n_launch = len(st["batches"])
    g1_flops = 4.0 * c["d"] * c["I"] * run.n_pairs / n_launch
    g1_ms = avg["gemm1_ms"] / n_launch
    # algorithmic bytes of GEMM1 per launch: the gate/up weights of every
    # local expert a batch touches (each streamed once), the batch's rows in
    # and h out
    import numpy as np
    elem = {W.BF16: 2, W.F32: 2, W.FP8: 1}.get(c["w"], 0.5)
    xel = 2 if dtype == "bf16" else 1
    touched = [set(int(e) for e in np.unique(wl.topk_local[ch.replica][ch.token_idx]) if e >= 0)
               for ch in wl.chunks]
    g1_bytes = sum(len(set().union(*touched[b["first_chunk"]:b["first_chunk"] + b["n_chunks"]]))
                   for b in st["batches"]) * 2.0 * c["I"] * c["d"] * elem / n_launch
    g1_bytes += run.n_pairs * (c["d"] + c["I"]) * xel / n_launch
    # the roofline that bounds a launch: MFMA time vs HBM time at peak
    hbm_bound = g1_bytes / (HBM_PEAK_GBS * 1e9) > g1_flops / (PEAK[dtype] * 1e12)
    traffic = measured_traffic(args.workload if args.policy == "wait_all"
                               else f"{args.workload}/{args.policy}")
    kernel = ("k_gemm_%s<SwiGLU> (grouped gate/up GEMM; %s)" %
              ({"mxfp4": "mx"}.get(dtype, dtype),
               "64-row weight-streaming tiles" if hbm_bound else
               "256-row tiles, bf16 plus 64-row remainder tiles when planned"))
    if hbm_bound:
        achieved = g1_bytes / (g1_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "kernel": kernel, "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": traffic, "launch_ms": round(g1_ms, 4),
                    "bytes_per_launch": round(g1_bytes)}
    else:
        achieved = g1_flops / (g1_ms * 1e-3) / 1e12
        roofline = {"bound": "mfma", "kernel": kernel, "achieved": round(achieved, 2),
                    "peak": PEAK[dtype], "unit": "TFLOP/s", "frac": round(achieved / PEAK[dtype], 4),
                    "traffic": traffic, "launch_ms": round(g1_ms, 4), "flop_per_launch": g1_flops}
    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": describe(c, args.workload), "local_pairs": run.n_pairs,
                   "policy": args.policy, "theta": args.theta, "streams": args.streams,
                   "global_batch": c["R"] * c["T"], "seq_len": c["T"], "parallelism": "ep_share_1gpu"},
        "pct_mfma_peak": round(100 * value / PEAK[dtype], 2),
        "time_to_last_chunk_done_ms": round(avg["last_done_ms"], 4),
        "phases_ms": {k: round(v, 4) for k, v in avg.items() if k != "last_done_ms"},
        "roofline": roofline,
    }
    run.close()
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
