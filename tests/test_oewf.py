"""OEWF coordinator: the oracle against a hand-worked example and closed
forms, the library against the oracle, and the non-degradation chain of
Appendix E on simulated layers.  No GPU needed."""
import math
import os

import numpy as np
import pytest

from oracle import calibration as C
from oracle import oewf as O
from paper_2609_33252_amd import cep
from tests import oewf_sim as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "oewf_example.txt")


def _parse():
    prof, ranks, steps = None, [], []
    for raw in open(GOLDEN):
        line = raw.split("#")[0].strip()
        if not line:
            continue
        key = line.split()[0]
        if key == "profile":
            a, b = line[len("profile"):].split("|")
            prof = ([int(v) for v in a.split()], [float(v) for v in b.split()])
        elif key == "rank":
            v = line.split()[1:]
            ranks.append((int(v[0]), int(v[1]), float(v[2]), float(v[3]), int(v[4]), float(v[5])))
        elif key == "select":
            parts = [p.strip() for p in line.split("|")]
            h = int(parts[0].split()[-1])
            tok = [[int(x) for x in row.split()] for row in parts[1][len("tokens"):].split(";")]
            b = [int(x) for x in parts[2].split()[1:]]
            budget = int(parts[3].split()[1])
            steps.append(("select", h, tok, b, budget))
        elif key == "admit":
            v = line.split()
            steps.append(("admit", int(v[2]), float(v[4])))
        elif key == "expect":
            v = line.split()[1:]
            steps.append(("expect", v))
    return prof, ranks, steps


def _kv(v):
    out, key = {}, None
    for tok in v:
        try:
            x = float(tok)
            out.setdefault(key, []).append(x)
        except ValueError:
            key = tok
    return out


def _run_golden(make, sel_fields):
    prof, ranks, steps = _parse()
    co = make(prof)
    for r, ia, A, D, N, T in ranks:
        co.set_rank(r, ia, A, D, N, T)
    plan = dec = None
    before = None
    for st in steps:
        if st[0] == "select":
            before = co.makespan()
            plan = co.select(st[1], st[2], st[3], st[4])
        elif st[0] == "admit":
            dec = co.evaluate(plan, st[1], st[2])
            co.commit(dec)
        else:
            kv = _kv(st[1])
            if "donor" in kv:
                donor, experts, tokens, nbytes = sel_fields(plan)
                assert donor == kv["donor"][0] and experts == [int(x) for x in kv["experts"]]
                assert tokens == [int(x) for x in kv["tokens"]] and nbytes == kv["bytes"][0]
            if "admit" in kv:
                assert bool(dec.admit) == bool(kv["admit"][0])
                for f in ("Td", "Th", "Td2", "Th2", "alpha"):
                    assert getattr(dec, f) == pytest.approx(kv[f][0], rel=1e-14, abs=1e-15), f
            if "makespan_before" in kv:
                assert before == pytest.approx(kv["makespan_before"][0], rel=1e-14)
                assert co.makespan() == pytest.approx(kv["makespan_after"][0], rel=1e-14)


def _oracle(prof):
    return S.OracleAdapter(O.Plan(4, prof[0], prof[1]))


def _oracle_fields(p):
    return p.donor, list(p.experts), list(p.tokens), p.bytes


def _lib_fields(p):
    n = p.n_experts
    return p.donor, [p.experts[i] for i in range(n)], [p.tokens[i] for i in range(n)], p.bytes


# ------------------------------------------------------------ oracle pins
def test_oracle_worked_example():
    _run_golden(_oracle, _oracle_fields)


def test_oracle_alpha_closed_forms():
    # s_h = T_h: the reassigned work runs after the helper's own (alpha = 1,
    # T_h' = T_h + F); s_h + F <= T_h: fully hidden (alpha = 0, T_h' = T_h)
    n, t = [10, 100], [1.0, 4.0]
    F = lambda N: C.latency(n, t, N)
    pl = O.Plan(2, n, t)
    pl.set_rank(0, False, 0, 0, 0, 200.0)
    pl.set_rank(1, True, 10.0, 2.0, 400, 0.0)
    p = pl.select_weights(0, [[0], [300]], [5], 10)
    assert F(300) == 75.0
    d = pl.evaluate(p, 300, 200.0)
    assert d.alpha == 1.0 and d.Th2 == 200.0 + F(300)
    d = pl.evaluate(p, 300, 200.0 - F(300))
    assert d.alpha == 0.0 and d.Th2 == 200.0
    d = pl.evaluate(p, 0, 3.0)
    assert not d.admit and d.Td2 == d.Td and d.Th2 == d.Th
    assert not pl.commit(d)


def test_oracle_selection_rules():
    pl = O.Plan(3, [1, 2], [1.0, 1.0])
    pl.set_rank(0, False, 0, 0, 0, 1.0)
    pl.set_rank(1, True, 5.0, 0.0, 10, 0.0)   # T = 5 + 10
    pl.set_rank(2, True, 5.0, 0.0, 10, 0.0)   # tie: lowest rank wins
    p = pl.select_weights(0, [[0, 0, 0], [3, 6, 1], [9, 9, 9]], [3, 6, 1], 7)
    # donor 1: ratios 1, 1, 1 -> ascending ids; 3 fits (R 4), 6 does not -> stop
    assert p.donor == 1 and p.experts == [0] and p.bytes == 3
    with pytest.raises(RuntimeError):
        pl.select_weights(0, [[0] * 3] * 3, [1, 1, 1], 10)
    # no candidate donor: nothing selected
    q = O.Plan(2, [1], [1.0])
    q.set_rank(1, False, 0, 0, 0, 1.0)
    assert q.select_weights(0, [[1], [1]], [1], 5) is None


def test_oracle_commit_fallbacks():
    pl = O.Plan(2, [1, 10], [1.0, 2.0])
    pl.set_rank(0, False, 0, 0, 0, 100.0)
    pl.set_rank(1, True, 50.0, 1.0, 40, 0.0)
    p = pl.select_weights(0, [[0], [40]], [1], 1)
    d = pl.evaluate(p, 40, 0.0)
    assert d.admit
    # the donor's entry changed since the evaluation: no commit
    pl.set_rank(1, True, 49.0, 1.0, 40, 0.0)
    assert not pl.commit(d)
    d = pl.evaluate(p, 40, 0.0)
    assert not pl.commit(d, donor_submitted=True)
    assert pl.commit(d)
    assert pl.ranks[1].N == 0
    assert not pl.commit(pl.evaluate(p, 0, 0.0))  # plan already claimed / nothing moves


def test_oracle_non_degradation_chain():
    rng = np.random.default_rng(3)
    n, t = [16, 128, 1024, 8192], [8.0, 48.0, 250.0, 400.0]
    F = lambda N: C.latency(n, t, N)
    improved = 0
    for _ in range(60):
        R, E = int(rng.integers(2, 9)), int(rng.integers(1, 9))
        attn, disp, tok, b = S.random_layer(rng, R, E)
        co = S.OracleAdapter(O.Plan(R, n, t))
        base, final, commits, trail = S.simulate(co, F, attn, disp, tok, b, budget=150,
                                                 bw=20.0, rng=rng)
        assert final <= base * (1 + 1e-12)
        prev = base
        for m in trail:  # every accepted update is non-increasing
            assert m <= prev * (1 + 1e-12)
            prev = m
        improved += final < base * (1 - 1e-9)
    assert improved > 0  # the policy does act on imbalanced layers


# ------------------------------------------------------ library vs oracle
@pytest.fixture(scope="module")
def lib_loaded():
    if not os.path.exists(cep.LIB_PATH):
        from paper_2609_33252_amd import build
        build.build()
    return cep.lib()


def test_library_worked_example(lib_loaded):
    _run_golden(lambda prof: cep.Coordinator(4, cep.FfnProfile(*prof)), _lib_fields)


def test_library_matches_oracle_random(lib_loaded):
    rng = np.random.default_rng(5)
    for it in range(80):
        R, E = int(rng.integers(2, 10)), int(rng.integers(1, 12))
        k = int(rng.integers(1, 6))
        n = np.cumsum(rng.integers(1, 3000, size=k)).tolist()
        t = rng.uniform(1.0, 500.0, size=k).tolist()
        prof = cep.FfnProfile(n, t)
        lib = cep.Coordinator(R, prof)
        ora = O.Plan(R, n, t)
        for r in range(R):
            args = (bool(rng.random() < 0.6), float(rng.uniform(0, 20)), float(rng.uniform(0, 3)),
                    int(rng.integers(0, 5000)), float(rng.uniform(0, 40)))
            lib.set_rank(r, *args)
            ora.set_rank(r, *args)
        assert lib.makespan() == pytest.approx(ora.makespan(), rel=1e-12)
        for h in rng.permutation(R).tolist():
            tok = (rng.integers(0, 400, size=(R, E)) * (rng.random((R, E)) < 0.5)).tolist()
            b = rng.integers(1, 60, size=E).tolist()
            budget = int(rng.integers(0, 150))
            pl = lib.select(h, tok, b, budget)
            po = ora.select_weights(h, tok, b, budget)
            if po is None:
                assert pl.n_experts == 0
                continue
            assert _lib_fields(pl) == _oracle_fields(po)
            ntr_max = min(sum(po.tokens), ora.ranks[po.donor].N)
            ntr = int(rng.integers(0, ntr_max + 1))
            s_h = float(rng.uniform(0, ora.ranks[h].T))
            dl, do = lib.evaluate(pl, ntr, s_h), ora.evaluate(po, ntr, s_h)
            assert bool(dl.admit) == bool(do.admit)
            for f in ("Td", "Th", "Td2", "Th2", "alpha"):
                assert math.isclose(getattr(dl, f), getattr(do, f), rel_tol=1e-12, abs_tol=1e-12)
            if rng.random() < 0.2:  # an update between test and commit: both fall back
                r = int(rng.integers(0, R))
                args = (False, 0.0, 0.0, int(rng.integers(0, 5000)), float(rng.uniform(0, 40)))
                lib.set_rank(r, *args)
                ora.set_rank(r, *args)
            sub = bool(rng.random() < 0.1)
            assert lib.commit(dl, sub) == ora.commit(do, sub)
            for r in range(R):
                assert lib.completion(r) == pytest.approx(ora.completion(r), rel=1e-12, abs=1e-12)
        lib.close()
        prof.close()


def test_library_non_degradation_chain(lib_loaded):
    rng = np.random.default_rng(9)
    n, t = [16, 128, 1024, 8192], [8.0, 48.0, 250.0, 400.0]
    prof = cep.FfnProfile(n, t)
    F = prof.latency
    for mode in ("random", "zero", "serial"):
        for _ in range(40):
            R, E = int(rng.integers(2, 9)), int(rng.integers(1, 9))
            attn, disp, tok, b = S.random_layer(rng, R, E)
            co = cep.Coordinator(R, prof)
            base, final, commits, trail = S.simulate(co, F, attn, disp, tok, b, budget=150,
                                                     bw=20.0, rng=rng, s_mode=mode)
            assert final <= base * (1 + 1e-12)
            prev = base
            for m in trail:
                assert m <= prev * (1 + 1e-12)
                prev = m
            co.close()
    prof.close()


def test_library_rejects_bad_arguments(lib_loaded):
    prof = cep.FfnProfile([1, 10], [1.0, 2.0])
    with pytest.raises(cep.CepError):
        cep.Coordinator(0, prof)
    co = cep.Coordinator(2, prof)
    with pytest.raises(cep.CepError):
        co.set_rank(2, True, 0, 0, 0, 0)
    with pytest.raises(cep.CepError):
        co.set_rank(0, True, -1.0, 0, 0, 0)
    co.set_rank(0, False, 0, 0, 0, 5.0)
    co.set_rank(1, True, 3.0, 0, 10, 0)
    with pytest.raises(cep.CepError):
        co.select(0, [[1], [1]], [0], 5)          # expert bytes must be > 0
    p = co.select(0, [[0], [10]], [1], 5)
    assert p.n_experts == 1 and p.donor == 1
    with pytest.raises(cep.CepError) as e:
        co.select(0, [[0], [10]], [1], 5)         # one decision per layer
    assert e.value.status == cep.CEP_EBUSY
    with pytest.raises(cep.CepError):
        co.evaluate(p, 11, 0.0)                   # more than the plan's tokens
    with pytest.raises(cep.CepError):
        co.evaluate(p, 5, 6.0)                    # s_h beyond T_h(S)
    d = co.evaluate(p, 10, 0.0)
    co.begin_layer()                              # a new layer: stale decision
    assert not co.commit(d)
    with pytest.raises(cep.CepError):
        co.evaluate(p, 10, 0.0)                   # the plan record is gone
    co.close()
    prof.close()
