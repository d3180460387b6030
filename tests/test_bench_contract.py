"""Host-side parts of the benchmark contract (no GPU needed).

* more than one GPU is refused with a message and a nonzero status before
  anything touches a device;
* the measured HBM traffic of the dominant kernel is reported only while
  the GEMM sources hash to the value recorded with the counters, and is
  null once a source changes.
"""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_multi_gpu_request_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_reported_only_for_the_measured_sources(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("kernel v1\n")
    monkeypatch.setitem(bench.GEMM_SOURCES, "probe", [str(src)])
    sha = bench.gemm_source_hash("probe")
    assert len(sha) == 12
    monkeypatch.setitem(bench.TRAFFIC_BYTES, "probe_workload", ("probe", sha, 12345))
    assert bench.measured_traffic("probe_workload") == 12345
    src.write_text("kernel v2\n")  # the kernel changed since the counters were taken
    assert bench.gemm_source_hash("probe") != sha
    assert bench.measured_traffic("probe_workload") is None
    assert bench.measured_traffic("no_such_workload") is None


def test_recorded_traffic_entries_name_known_families():
    for wl, (family, sha, nbytes) in bench.TRAFFIC_BYTES.items():
        assert family in bench.GEMM_SOURCES, wl
        assert len(sha) == 12 and int(sha, 16) >= 0, wl
        assert nbytes > 0, wl
