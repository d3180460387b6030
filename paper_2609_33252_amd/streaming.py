"""Timing metrics of one replayed layer, from the library's layer statistics.

The statistics (``cep_get_stats``) give, on one GPU clock with the layer's
origin at ``cep_begin_layer``: every batch's start/end and chunk range, and
every chunk's arrival.  From them:

* time to last chunk done: end of the last batch;
* exposed tail: last batch end minus last chunk arrival (the FFN time the
  layer still waits for once every replica has dispatched -- what
  asynchronous execution shortens, Section 3.2);
* per-chunk latency: end of the batch holding the chunk minus its arrival;
* busy time: length of the union of the batches' [start, end] intervals, and
  the aggregate TFLOP/s of the layer's routed-expert work over it (a
  timed-arrival counterpart of the matched-work FFN efficiency comparison of
  Section 4.3, which bench.py --matched-work runs on resident inputs).
"""
from __future__ import annotations


def union_length(intervals) -> float:
    """Total length covered by a set of [a, b] intervals."""
    total, cur_a, cur_b = 0.0, None, None
    for a, b in sorted(intervals):
        if cur_b is None or a > cur_b:
            if cur_b is not None:
                total += cur_b - cur_a
            cur_a, cur_b = a, b
        else:
            cur_b = max(cur_b, b)
    if cur_b is not None:
        total += cur_b - cur_a
    return total


def percentile(vals, q):
    if not vals:
        return None
    v = sorted(vals)
    pos = (len(v) - 1) * q / 100.0
    lo = int(pos)
    hi = min(lo + 1, len(v) - 1)
    return v[lo] + (v[hi] - v[lo]) * (pos - lo)


def layer_metrics(stats: dict, flops: float) -> dict:
    """Metrics of one layer (times in ms); flops = routed-expert work of the
    layer (6 * d * I * local pairs)."""
    batches = stats["batches"]
    chunks = stats["chunks"]
    if not batches:
        return {"batches": 0}
    done = {}
    for b in batches:
        for c in range(b["first_chunk"], b["first_chunk"] + b["n_chunks"]):
            done[c] = b["end_ms"]
    arrivals = [c["arrival_ms"] for c in chunks]
    last_done = max(b["end_ms"] for b in batches)
    last_arrival = max(arrivals) if arrivals else 0.0
    lat = [done[i] - chunks[i]["arrival_ms"] for i in done
           if chunks[i]["pairs"] > 0 and chunks[i]["arrival_ms"] >= 0]
    busy = union_length([(b["start_ms"], b["end_ms"]) for b in batches])
    return {
        "batches": len(batches),
        "time_to_last_chunk_done_ms": last_done,
        "last_arrival_ms": last_arrival,
        "exposed_tail_ms": last_done - last_arrival,
        "chunk_latency_ms": {"p50": percentile(lat, 50), "p95": percentile(lat, 95),
                             "max": max(lat) if lat else None},
        "busy_ms": busy,
        "busy_tflops": flops / (busy * 1e-3) / 1e12 if busy > 0 else None,
        "phases_ms": {k: sum(b[k] for b in batches)
                      for k in ("route_ms", "gemm1_ms", "gemm2_ms", "combine_ms")},
    }


def mean_metrics(runs: list) -> dict:
    """Element-wise mean of layer_metrics dicts (nested dicts averaged too)."""
    out = {}
    for k in runs[0]:
        vals = [r[k] for r in runs]
        if isinstance(vals[0], dict):
            out[k] = mean_metrics(vals)
        elif all(isinstance(v, (int, float)) for v in vals):
            out[k] = sum(vals) / len(vals)
        else:
            out[k] = vals[0]
    return out
