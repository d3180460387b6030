"""Pins for the routing-metadata oracle and the batch-composition oracle
(CPU only): brute force, invariants, special cases and a hand-worked example
of the launch-threshold rule (tests/golden/policy_theta_example.txt)."""
import os

import numpy as np
import pytest

from oracle import policy, routing
from paper_2609_33252_amd import workload as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_batch(rng, n_chunks, E, k, p_remote=0.3, max_rows=40):
    out = []
    for _ in range(n_chunks):
        n = int(rng.integers(0, max_rows))
        ids = rng.integers(0, E, size=(n, k)).astype(np.int32)
        ids[rng.random((n, k)) < p_remote] = -1
        out.append(ids)
    return out


def _check_invariants(m, chunk_ids, E, A):
    flat = np.concatenate([c.reshape(-1) for c in chunk_ids]) if chunk_ids else np.zeros(0)
    P = int((flat >= 0).sum())
    assert m["cnt"].sum() == P
    assert m["off"][0] == 0 and m["off"][-1] == P
    assert np.all(np.diff(m["off"]) == m["cnt"])
    assert np.all(np.diff(m["off_pad"]) % A == 0)
    assert np.all(np.diff(m["off_pad"]) >= m["cnt"])
    assert np.all(np.diff(m["off_pad"]) < m["cnt"] + A)
    # perm_src is a bijection onto the valid pairs, grouped by expert
    assert sorted(m["perm_src"].tolist()) == np.nonzero(flat >= 0)[0].tolist()
    for e in range(E):
        seg = m["perm_src"][m["off"][e]:m["off"][e + 1]]
        assert np.all(flat[seg] == e)
        assert np.all(np.diff(seg) > 0)              # stable
        # inverse map: unpadded row q of expert e sits at padded row off_pad[e] + q
        assert np.array_equal(m["pos_of"][seg], m["off_pad"][e] + np.arange(len(seg)))
    assert np.all(m["pos_of"][flat < 0] == -1)


@pytest.mark.parametrize("seed", range(12))
def test_routing_matches_stable_sort_brute_force(seed):
    rng = np.random.default_rng(seed)
    E = int(rng.integers(1, 17))
    k = int(rng.integers(1, 9))
    A = int(rng.choice([1, 16, 64, 128, 256]))
    chunks = _rand_batch(rng, int(rng.integers(0, 6)), E, k)
    m = routing.batch_routing(chunks, E, A)
    b = routing.brute_force_routing(chunks, E, A)
    for key in m:
        assert np.array_equal(m[key], b[key]), key
    _check_invariants(m, chunks, E, A)


def test_routing_special_cases():
    E, A = 4, 8
    # empty batch
    m = routing.batch_routing([], E, A)
    assert m["cnt"].tolist() == [0] * E and m["perm_src"].size == 0
    # all remote
    m = routing.batch_routing([np.full((5, 3), -1, np.int32)], E, A)
    assert m["off_pad"].tolist() == [0] * (E + 1) and np.all(m["pos_of"] == -1)
    # a single expert: identity permutation, aligned end
    ids = np.full((9, 2), 2, np.int32)
    m = routing.batch_routing([ids[:4], ids[4:]], E, A)
    assert m["perm_src"].tolist() == list(range(18))
    assert m["off_pad"].tolist() == [0, 0, 0, 24, 24]
    # hand example: rows [[1,0],[0,-1],[1,1]], A=2
    m = routing.batch_routing([np.array([[1, 0], [0, -1]]), np.array([[1, 1]])], 2, 2)
    assert m["cnt"].tolist() == [2, 3]
    assert m["off"].tolist() == [0, 2, 5]
    assert m["off_pad"].tolist() == [0, 2, 6]
    assert m["perm_src"].tolist() == [1, 2, 0, 4, 5]
    assert m["pos_of"].tolist() == [2, 0, 1, -1, 3, 4]


def test_routing_generated_workload_full_size():
    wl = W.generate("zipf_stream_d7168", 0, d=128, I=128)   # routing is shape-independent
    chunks = [wl.topk_local[c.replica][c.token_idx] for c in wl.chunks[:9]]
    m = routing.batch_routing(chunks, wl.cfg["E"], 128)
    b = routing.brute_force_routing(chunks, wl.cfg["E"], 128)
    for key in m:
        assert np.array_equal(m[key], b[key]), key
    _check_invariants(m, chunks, wl.cfg["E"], 128)


def _golden_policy():
    pairs, cases = None, []
    with open(os.path.join(GOLDEN, "policy_theta_example.txt")) as f:
        for line in f:
            t = line.split()
            if not t or t[0].startswith("#"):
                continue
            if t[0] == "pairs":
                pairs = [int(v) for v in t[1:]]
            else:
                theta = int(t[1])
                batches = [[int(c) for c in b.split(",")] for b in t[3:]]
                cases.append((theta, batches))
    return pairs, cases


def test_policy_hand_worked_example():
    pairs, cases = _golden_policy()
    for theta, expect in cases:
        assert policy.batches(pairs, policy.THRESHOLD, theta) == expect, theta
    assert policy.batches(pairs, policy.WAIT_ALL) == [[0, 2, 3, 4, 5]]
    assert policy.batches(pairs, policy.PER_CHUNK) == [[0], [2], [3], [4], [5]]


def _threshold_property(pairs, theta, batches):
    """Independent characterisation of THRESHOLD (no cap, no flush): the
    batches partition the non-empty chunks in order; every batch but the last
    reaches theta and would not have reached it without its last chunk."""
    nonempty = [i for i, p in enumerate(pairs) if p > 0]
    assert [c for b in batches for c in b] == nonempty
    for b in batches[:-1]:
        s = sum(pairs[c] for c in b)
        assert s >= theta and s - pairs[b[-1]] < theta
    if batches:
        last = batches[-1]
        assert sum(pairs[c] for c in last) - pairs[last[-1]] < theta


@pytest.mark.parametrize("seed", range(20))
def test_policy_random_sequences(seed):
    rng = np.random.default_rng(seed)
    pairs = [int(v) if rng.random() > 0.2 else 0 for v in rng.integers(1, 50, size=int(rng.integers(0, 30)))]
    theta = int(rng.integers(1, 200))
    b = policy.batches(pairs, policy.THRESHOLD, theta)
    _threshold_property(pairs, theta, b)
    assert policy.batches(pairs, policy.THRESHOLD, 1) == policy.batches(pairs, policy.PER_CHUNK)
    wa = policy.batches(pairs, policy.WAIT_ALL)
    nonempty = [i for i, p in enumerate(pairs) if p > 0]
    assert wa == ([nonempty] if nonempty else [])


def test_policy_flush_expected_count_and_cap():
    # explicit flush launches what is pending; nothing pending -> no batch
    assert policy.batches([3, "flush", "flush", 4], policy.WAIT_ALL) == [[0], [1]]
    # the final flush waits for the expected chunk count
    assert policy.batches([3, 4], policy.THRESHOLD, 100, n_expected=3) == []
    assert policy.batches([3, 4, 0], policy.THRESHOLD, 100, n_expected=3) == [[0, 1]]
    # a capacity launches pending work before overflowing
    assert policy.batches([3, 4, 5], policy.WAIT_ALL, cap=8) == [[0, 1], [2]]
    with pytest.raises(ValueError):
        policy.batches([9], policy.WAIT_ALL, cap=8)
