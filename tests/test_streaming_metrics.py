"""Host-side timing metrics of a replayed layer (CPU only, synthetic stats)."""
import pytest

from paper_2609_33252_amd import streaming as S


def test_union_length():
    assert S.union_length([]) == 0
    assert S.union_length([(0, 1), (2, 3)]) == 2
    assert S.union_length([(0, 2), (1, 3), (5, 6), (5.5, 5.7)]) == 4
    assert S.union_length([(3, 4), (0, 10)]) == 10


def test_layer_metrics_hand_example():
    stats = {"batches": [
        {"first_chunk": 0, "n_chunks": 2, "start_ms": 1.0, "end_ms": 2.0, "route_ms": .1,
         "gemm1_ms": .5, "gemm2_ms": .3, "combine_ms": .1},
        {"first_chunk": 2, "n_chunks": 1, "start_ms": 1.5, "end_ms": 4.0, "route_ms": .1,
         "gemm1_ms": 1., "gemm2_ms": 1., "combine_ms": .4}],
        "chunks": [{"pairs": 10, "arrival_ms": 0.5}, {"pairs": 0, "arrival_ms": 0.9},
                   {"pairs": 5, "arrival_ms": 3.0}]}
    m = S.layer_metrics(stats, flops=3e9)  # 3 GFLOP over 3 ms busy = 1 TFLOP/s
    assert m["time_to_last_chunk_done_ms"] == 4.0
    assert m["last_arrival_ms"] == 3.0
    assert m["exposed_tail_ms"] == 1.0
    # chunk latencies: 2.0-0.5 and 4.0-3.0 (the empty chunk has none)
    assert m["chunk_latency_ms"]["max"] == 1.5
    assert m["chunk_latency_ms"]["p50"] == pytest.approx(1.25)
    assert m["busy_ms"] == 3.0
    assert m["busy_tflops"] == pytest.approx(1.0)
    assert m["phases_ms"]["gemm1_ms"] == pytest.approx(1.5)
    mm = S.mean_metrics([m, m])
    assert mm["exposed_tail_ms"] == 1.0 and mm["chunk_latency_ms"]["max"] == 1.5


def test_percentile():
    assert S.percentile([], 50) is None
    assert S.percentile([4, 1, 3, 2], 50) == 2.5
    assert S.percentile([1, 2, 3, 4, 5], 95) == pytest.approx(4.8)
