"""Launch-threshold calibration and the FFN latency model (oracle).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Section 3.2, "Launch threshold": FFN throughput is profiled against the
expert-token count; theta is the smallest *profiled* count whose throughput
reaches a target fraction rho of the observed peak.  Section 3.3, Eq.
(ffn-throughput-latency): the FFN latency of N expert tokens is
F(N) = N / (eta(N) * P_peak), with eta(N) in (0, 1] the throughput normalised
to the profile's observed peak P_peak.

Readings (the paper gives no formula for counts between or outside the
profiled ones):

* between two profiled counts, eta is linear in N;
* below the smallest profiled count n_0 the latency is that of n_0 (a launch
  costs at least that much): eta(N) = eta(n_0) * N / n_0, so F(N) = F(n_0);
* above the largest profiled count eta stays at its last value (saturated).

Throughput is in expert tokens per unit time, so F is in that time unit.
"""
from __future__ import annotations

import numpy as np


def _check(n, tput):
    n = np.asarray(n, dtype=np.int64)
    tput = np.asarray(tput, dtype=np.float64)
    if n.ndim != 1 or n.shape != tput.shape or len(n) == 0:
        raise ValueError("profile needs equal-length, non-empty count and throughput lists")
    if (n <= 0).any() or (np.diff(n) <= 0).any():
        raise ValueError("profiled counts must be positive and strictly increasing")
    if not np.isfinite(tput).all() or (tput <= 0).any():
        raise ValueError("profiled throughputs must be positive and finite")
    return n, tput


def peak(n, tput) -> float:
    """P_peak: the largest observed throughput of the profile."""
    _, tput = _check(n, tput)
    return float(tput.max())


def eta_table(n, tput) -> np.ndarray:
    """eta at the profiled counts: throughput / observed peak."""
    _, tput = _check(n, tput)
    return tput / tput.max()


def theta(n, tput, rho: float) -> int:
    """Smallest profiled count whose normalised throughput is >= rho."""
    n, _ = _check(n, tput)
    if not (0.0 < rho <= 1.0):
        raise ValueError("rho must lie in (0, 1]")
    eta = eta_table(n, tput)
    for ni, ei in zip(n, eta):  # ascending counts: the first hit is the smallest
        if ei >= rho:
            return int(ni)
    raise AssertionError("eta reaches 1 at the peak, so some count qualifies")


def eta_at(n, tput, N: int) -> float:
    """eta(N) with the readings above (N >= 1)."""
    n, _ = _check(n, tput)
    if N < 1:
        raise ValueError("N must be >= 1")
    eta = eta_table(n, tput)
    if N <= n[0]:
        return float(eta[0] * N / n[0])
    # numpy.interp: linear between neighbours, constant past the last point
    return float(np.interp(float(N), n.astype(np.float64), eta))


def latency(n, tput, N: int) -> float:
    """F(N) = N / (eta(N) * P_peak); F(0) = 0."""
    if N == 0:
        _check(n, tput)
        return 0.0
    return N / (eta_at(n, tput, N) * peak(n, tput))
