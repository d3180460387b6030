"""Launch-threshold calibration and FFN latency model: the oracle against the
paper's definitions (a hand-worked example, closed forms, invariants), then
the library's host implementation against the oracle.  No GPU needed."""
import math
import os

import numpy as np
import pytest

from oracle import calibration as C
from paper_2609_33252_amd import cep

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "theta_profile_example.txt")


def _golden():
    counts = tput = None
    thetas, lats = [], []
    for line in open(GOLDEN):
        line = line.split("#")[0].split()
        if not line:
            continue
        if line[0] == "counts":
            counts = [int(v) for v in line[1:]]
        elif line[0] == "tput":
            tput = [float(v) for v in line[1:]]
        elif line[0] == "theta":
            thetas.append((float(line[1]), int(line[2])))
        elif line[0] == "latency":
            lats.append((int(line[1]), float(line[2])))
    return counts, tput, thetas, lats


# ------------------------------------------------------------ oracle pins
def test_oracle_worked_example():
    n, t, thetas, lats = _golden()
    assert C.peak(n, t) == 100.0
    for rho, want in thetas:
        assert C.theta(n, t, rho) == want, rho
    for N, want in lats:
        assert C.latency(n, t, N) == pytest.approx(want, rel=1e-14, abs=0), N


def test_oracle_constant_throughput_closed_form():
    # a flat profile: eta = 1 everywhere at and above n_0, theta = n_0 for any
    # rho, F(N) = N / P
    n, P = [16, 64, 256, 1024], 7.5
    t = [P] * 4
    for rho in (0.01, 0.5, 0.9, 1.0):
        assert C.theta(n, t, rho) == 16
    for N in (16, 17, 100, 256, 5000):
        assert C.latency(n, t, N) == pytest.approx(N / P, rel=1e-15)
    # below n_0 the latency is F(n_0)
    assert C.latency(n, t, 3) == pytest.approx(16 / P, rel=1e-15)


def test_oracle_latency_bound_profile_closed_form():
    # throughput proportional to N (a fixed launch cost 1/c): eta = N / n_last
    # is linear, so its interpolation is exact and F(N) = 1/c for every N
    c = 0.25
    n = [8, 32, 100, 333, 1000]
    t = [c * v for v in n]
    for N in (1, 8, 9, 50, 100, 777, 1000, 4000):
        want = 1 / c if N <= 1000 else N / (c * 1000)
        assert C.latency(n, t, N) == pytest.approx(want, rel=1e-13), N
    assert C.theta(n, t, 0.3) == 333  # first count with N / 1000 >= 0.3
    assert C.theta(n, t, 0.1) == 100


def test_oracle_invariants_random_profiles():
    rng = np.random.default_rng(7)
    for _ in range(50):
        k = int(rng.integers(1, 12))
        n = np.cumsum(rng.integers(1, 500, size=k))
        t = rng.uniform(0.1, 10.0, size=k)
        eta = C.eta_table(n, t)
        assert eta.max() == 1.0 and (eta > 0).all()
        # theta is non-decreasing in rho and always a profiled count
        prev = 0
        for rho in np.linspace(0.01, 1.0, 25):
            th = C.theta(n, t, float(rho))
            assert th in n and th >= prev
            i = list(n).index(th)
            assert eta[i] >= rho and (eta[:i] < rho).all()
            prev = th
        # eta at profiled counts equals the table; F is positive
        for i, ni in enumerate(n):
            assert C.eta_at(n, t, int(ni)) == pytest.approx(eta[i], rel=1e-15)
            assert C.latency(n, t, int(ni)) == pytest.approx(ni / (eta[i] * t.max()), rel=1e-14)


def test_oracle_rejects_bad_profiles():
    for n, t in (([], []), ([4, 4], [1, 1]), ([0, 4], [1, 1]), ([1, 2], [1, 0]),
                 ([1, 2], [1, float("nan")])):
        with pytest.raises(ValueError):
            C.peak(n, t)
    with pytest.raises(ValueError):
        C.theta([1, 2], [1, 2], 0.0)
    with pytest.raises(ValueError):
        C.theta([1, 2], [1, 2], 1.5)


# ------------------------------------------------------ library vs oracle
@pytest.fixture(scope="module")
def lib_loaded():
    if not os.path.exists(cep.LIB_PATH):
        from paper_2609_33252_amd import build
        build.build()
    return cep.lib()


def test_library_worked_example(lib_loaded):
    n, t, thetas, lats = _golden()
    p = cep.FfnProfile(n, t)
    assert p.peak == 100.0
    for rho, want in thetas:
        assert p.theta(rho) == want
    for N, want in lats:
        assert p.latency(N) == pytest.approx(want, rel=1e-14, abs=0)
    p.close()


def test_library_matches_oracle_random_profiles(lib_loaded):
    rng = np.random.default_rng(11)
    for _ in range(100):
        k = int(rng.integers(1, 16))
        n = np.cumsum(rng.integers(1, 2000, size=k)).astype(np.int64)
        t = rng.uniform(0.01, 1000.0, size=k)
        p = cep.FfnProfile(n.tolist(), t.tolist())
        assert p.peak == C.peak(n, t)
        for rho in rng.uniform(1e-3, 1.0, size=8).tolist() + [1.0]:
            assert p.theta(rho) == C.theta(n, t, rho)
        for N in [0, 1, int(n[0]), int(n[-1]), int(n[-1]) * 3] + \
                rng.integers(1, int(n[-1]) + 10, size=8).tolist():
            got, want = p.latency(int(N)), C.latency(n, t, int(N))
            assert math.isclose(got, want, rel_tol=1e-12, abs_tol=0), (N, got, want)
            if N >= 1:
                assert math.isclose(p.eta(int(N)), C.eta_at(n, t, int(N)), rel_tol=1e-12)
        p.close()


def test_library_rejects_bad_profiles(lib_loaded):
    for n, t in (([], []), ([4, 4], [1.0, 1.0]), ([0, 4], [1.0, 1.0]), ([1, 2], [1.0, 0.0]),
                 ([1, 2], [1.0, float("inf")])):
        with pytest.raises(cep.CepError) as e:
            cep.FfnProfile(n, t)
        assert e.value.status == cep.CEP_EINVAL
        assert cep.cep_last_error(None)
    p = cep.FfnProfile([1, 2], [1.0, 2.0])
    for rho in (0.0, -1.0, 1.5, float("nan")):
        with pytest.raises(cep.CepError):
            p.theta(rho)
    with pytest.raises(cep.CepError):
        p.eta(0)
    with pytest.raises(cep.CepError):
        p.latency(-1)
    p.close()
