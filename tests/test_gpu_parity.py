"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

* routing metadata and batch composition: bit-exact, every config
* outputs: elementwise tolerance (bf16, f32 inputs) or relative RMS (fp8),
  at reduced token counts over all rows and at full size on sampled tokens
* closed forms on the GPU: identity-permutation expert, zero expert;
  exact linearity in the coefficients and the down weights; one-hot
  coefficients equal routing to that slot alone
* invariance: chunking, submission order, policy and stream count do not
  change the output (bitwise); a fetched expert equals a resident one
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import policy as opol
from oracle import routing as orout
from paper_2609_33252_amd import cep, harness, workload as W

from . import _util as U

pytestmark = pytest.mark.gpu

# token counts small enough for the oracle over every row, at the real
# d_model / d_ff of each configuration, spanning several M tiles per expert
REDUCED = {
    "tiny": {},
    "sync_d4096": dict(T=512),
    "zipf_stream_d7168": dict(T=512, cpr=4),
    "zipf_imbalanced_d7168": dict(T=512, cpr=4),
    "fp8_fetch_d6144": dict(T=256, cpr=2),
}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cep.lib()
    torch.cuda.set_device(0)


def _out(run):
    torch.cuda.synchronize()
    cep.cep_get_status(run.ctx)
    return run.out.cpu().numpy()


# ------------------------------------------------------------- routing
@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_routing_and_batches_bit_exact(name):
    # routing does not depend on d / d_ff: full token counts, small widths
    small = dict(d=256, I=128)
    wl = W.generate(name, 0, **small)
    run = harness.Runner(wl, n_streams=3, record_routing=True, use_fetch=True)
    theta = max(1, wl.n_pairs // 5)
    run.run(policy=cep.CEP_THRESHOLD, theta=theta, n_streams=3)
    torch.cuda.synchronize()
    cep.cep_get_status(run.ctx)
    pairs_seq = [ch.n_pairs for ch in run.chunks]
    expect = opol.batches(pairs_seq, opol.THRESHOLD, theta)
    nb = cep.cep_get_batch_count(run.ctx)
    assert nb == len(expect)
    E, k = wl.cfg["E"], wl.cfg["k"]
    for b in range(nb):
        m = cep.cep_get_batch_routing(run.ctx, b, E, k)
        got_chunks = [int(c) for c in m["chunks"] if run.chunks[int(c)].n_pairs > 0]
        assert got_chunks == expect[b]
        ids = [wl.topk_local[wl.chunks[c].replica][wl.chunks[c].token_idx]
               for c in m["chunks"]]
        ref = orout.batch_routing(ids, E, m["align"])
        for key in ("cnt", "off", "off_pad", "perm_src", "pos_of"):
            assert np.array_equal(m[key], ref[key]), (b, key)
    run.close()


def test_policies_match_batch_oracle():
    wl = W.generate("zipf_stream_d7168", 0, d=256, I=128)
    run = harness.Runner(wl, n_streams=4, record_routing=True)
    seq = [ch.n_pairs for ch in run.chunks]
    for pol, theta, ns in ((cep.CEP_WAIT_ALL, 1, 1), (cep.CEP_PER_CHUNK, 1, 2),
                           (cep.CEP_THRESHOLD, 32, 4), (cep.CEP_THRESHOLD, 4096, 2)):
        run.run(policy=pol, theta=theta, n_streams=ns)
        torch.cuda.synchronize()
        want = opol.batches(seq, {0: opol.WAIT_ALL, 1: opol.PER_CHUNK, 2: opol.THRESHOLD}[pol],
                            theta)
        got = []
        for b in range(cep.cep_get_batch_count(run.ctx)):
            m = cep.cep_get_batch_routing(run.ctx, b, wl.cfg["E"], wl.cfg["k"])
            got.append([int(c) for c in m["chunks"] if seq[int(c)] > 0])
        assert got == want, (pol, theta)
        st = run.stats()
        assert [b["slot"] for b in st["batches"]] == [i % ns for i in range(len(want))]
    run.close()


# ------------------------------------------------------------- outputs
@pytest.mark.parametrize("name", W.CONFIG_ORDER)
def test_outputs_match_oracle_reduced(name):
    wl = W.generate(name, 0, **REDUCED[name])
    run = harness.Runner(wl, n_streams=2)
    run.run(policy=cep.CEP_THRESHOLD, theta=max(1, wl.n_pairs // 3), n_streams=2)
    got = _out(run)
    run.close()
    mx, rel = U.check(wl, got)
    assert not got[~wl.delivered].any()
    print(f"{name}: pairs={wl.n_pairs} max_abs={mx:.3e} rel_rms={rel:.3e}")


@pytest.mark.parametrize("name", ["sync_d4096", "zipf_stream_d7168", "fp8_fetch_d6144"])
def test_full_size_sampled_tokens(name):
    wl = W.generate(name, 0)
    run = harness.Runner(wl, n_streams=1)
    run.run(policy=cep.CEP_WAIT_ALL)
    got = _out(run)
    run.close()
    rng = np.random.default_rng(1)
    deliv = np.argwhere(wl.delivered)
    pick = deliv[rng.choice(len(deliv), size=24, replace=False)]
    # include tokens routed to the hottest and coldest local experts
    cnt = np.bincount(wl.topk_local[wl.topk_local >= 0], minlength=wl.cfg["E"])
    for e in (int(cnt.argmax()), int(np.argmin(np.where(cnt > 0, cnt, 1 << 30)))):
        rt = np.argwhere((wl.topk_local == e).any(axis=2))
        pick = np.vstack([pick, rt[-2:]])
    mx, rel = U.check(wl, got[pick[:, 0], pick[:, 1]], tokens=pick)
    assert not got[~wl.delivered].any()
    print(f"{name} full: pairs={wl.n_pairs} sampled={len(pick)} max_abs={mx:.3e} rel={rel:.3e}")


# --------------------------------------------------------- closed forms
def _custom(d, I, E, wg, wu, wd, R=2, T=256):
    wl = W.generate("sync_d4096", 3, d=d, I=I, E=E, Eg=E + 2, k=2, R=R, T=T)
    wl.w_gate, wl.w_up, wl.w_down = wg, wu, wd
    return wl


@pytest.mark.parametrize("beta", [0.5, 2.0])
def test_identity_permutation_expert_closed_form(beta):
    d = I = 256
    pi = np.roll(np.arange(d), 3)
    P = np.zeros((d, d), np.float32)
    P[pi, np.arange(d)] = 1.0
    wg = torch.from_numpy(np.stack([beta * P] * 2)).to(torch.bfloat16)
    wu = torch.from_numpy(np.stack([P] * 2)).to(torch.bfloat16)
    wd = torch.from_numpy(np.stack([P.T.copy()] * 2)).to(torch.bfloat16)
    wl = _custom(d, I, 2, wg, wu, wd)
    run = harness.Runner(wl, n_streams=1)
    run.run(policy=cep.CEP_PER_CHUNK)
    got = _out(run)
    run.close()
    x = wl.x.double().numpy()
    h = x * (beta * x) / (1 + np.exp(-beta * x))
    hb = torch.from_numpy(h).to(torch.bfloat16).double().numpy()
    wsum = np.where(wl.topk_local >= 0, wl.topk_w, 0).astype(np.float64)
    # every local slot contributes w * h: y = sum_s w_s * bf16(h)
    ref = np.zeros_like(x)
    for s in range(wl.cfg["k"]):
        ref += wsum[:, :, s:s + 1] * hb
    err = np.abs(got - ref)
    # h is rounded to bf16 on both sides; float32 silu may move it by one ulp
    assert np.all(err <= 2.0 ** -7 * np.abs(ref) * wl.cfg["k"] + 1e-6), err.max()


def test_zero_down_weights_give_exact_zero():
    wl = W.generate("sync_d4096", 4, T=256)
    wl.w_down = torch.zeros_like(wl.w_down)
    run = harness.Runner(wl)
    run.run(policy=cep.CEP_THRESHOLD, theta=500, n_streams=2)
    got = _out(run)
    run.close()
    assert not got.any()


# ------------------------------------------------------------ invariance
def _run_threshold(wl):
    run = harness.Runner(wl, n_streams=2)
    run.run(policy=cep.CEP_THRESHOLD, theta=max(1, wl.n_pairs // 3), n_streams=2)
    got = _out(run)
    run.close()
    return got


def test_linearity_in_coefficients_and_down_weights_bitwise():
    # doubling every routing coefficient, or the down weights, doubles the
    # output exactly: a factor of two commutes with every rounding on the
    # path (bf16 products, f32 sums, the bf16 output rows, the f32 combine)
    wl = W.generate("zipf_stream_d7168", 2, d=1024, I=512, T=512, cpr=4)
    a = _run_threshold(wl)
    assert np.abs(a).max() > 0
    b = _run_threshold(dataclasses.replace(wl, topk_w=wl.topk_w * 2))
    assert np.array_equal(b, 2 * a)
    c = _run_threshold(dataclasses.replace(wl, w_down=wl.w_down * 2))
    assert np.array_equal(c, 2 * a)


def test_one_hot_coefficients_equal_dropped_slots_bitwise():
    # coefficients one-hot on each token's first local slot give the bits of
    # routing the token to that slot alone: the other slots add exact zeros
    wl = W.generate("zipf_stream_d7168", 3, d=1024, I=512, T=512, cpr=4)
    ids = wl.topk_local
    local = ids >= 0
    first = np.argmax(local, axis=2)
    one = np.zeros_like(wl.topk_w)
    np.put_along_axis(one, first[..., None], 1.0, axis=2)
    one[~local] = 0.0
    only = np.where(one > 0, ids, -1).astype(ids.dtype)
    a = _run_threshold(dataclasses.replace(wl, topk_w=one))
    wl_b = dataclasses.replace(wl, topk_local=only, topk_w=one)
    b = _run_threshold(wl_b)
    assert wl_b.n_pairs < wl.n_pairs
    assert np.array_equal(a, b)
    U.check(wl_b, b)


def test_chunking_order_policy_streams_invariance_bitwise():
    wl = W.generate("zipf_imbalanced_d7168", 0, T=512, cpr=8)
    run = harness.Runner(wl, n_streams=4)
    outs = []
    rng = np.random.default_rng(0)
    for pol, theta, ns, order in ((cep.CEP_WAIT_ALL, 1, 1, None),
                                  (cep.CEP_PER_CHUNK, 1, 4, None),
                                  (cep.CEP_THRESHOLD, 200, 3, None),
                                  (cep.CEP_THRESHOLD, 700, 2, list(rng.permutation(len(run.chunks))))):
        run.out.zero_()
        run.run(policy=pol, theta=theta, n_streams=ns, order=order)
        outs.append(_out(run))
    run.close()
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])


def test_large_and_small_m_tiles_agree_bitwise():
    # one wait-all batch has >= 256 rows per expert (256-row M tile); single
    # chunks have ~125 (64-row M tile): same K order, same bits
    wl = W.generate("sync_d4096", 1, T=1024)
    assert wl.n_pairs >= 256 * wl.cfg["E"]
    assert max(wl.chunk_pairs(c) for c in wl.chunks) < 256 * wl.cfg["E"]
    run = harness.Runner(wl, n_streams=2, record_routing=True)
    run.run(policy=cep.CEP_WAIT_ALL)
    a = _out(run)
    m = cep.cep_get_batch_routing(run.ctx, 0, wl.cfg["E"], wl.cfg["k"])
    assert m["align"] == 256
    run.out.zero_()
    run.run(policy=cep.CEP_PER_CHUNK, n_streams=2)
    b = _out(run)
    m = cep.cep_get_batch_routing(run.ctx, 0, wl.cfg["E"], wl.cfg["k"])
    assert m["align"] == 64
    run.close()
    assert np.array_equal(a, b)
    U.check(wl, a)


def test_var_tiles_agree_bitwise():
    # 64-row bf16 batches with at least 64 pairs per local expert run both
    # GEMMs in 128-row tiles, an expert's last tile a 64-row half when at
    # most 64 rows remain: a hot expert spans several tiles and ends in a
    # half tile.  Same K order as the wait-all batch's 256-row tiles and the
    # per-chunk batches' 64-row tiles, so the same bits.
    wl = W.generate("zipf_imbalanced_d7168", 6, d=1024, I=512, R=8, T=4096, cpr=4)
    E, k = wl.cfg["E"], wl.cfg["k"]
    run = harness.Runner(wl, n_streams=2, record_routing=True)
    run.run(policy=cep.CEP_WAIT_ALL)
    a = _out(run)
    assert cep.cep_get_batch_routing(run.ctx, 0, E, k)["align"] == 256
    small = var_multi_half = 0
    for pol, theta in ((cep.CEP_PER_CHUNK, 1), (cep.CEP_THRESHOLD, 300),
                       (cep.CEP_THRESHOLD, 600), (cep.CEP_THRESHOLD, 1200)):
        run.out.zero_()
        run.run(policy=pol, theta=theta, n_streams=2)
        b = _out(run)
        assert np.array_equal(a, b), theta
        for i in range(cep.cep_get_batch_count(run.ctx)):
            m = cep.cep_get_batch_routing(run.ctx, i, E, k)
            if m["align"] != 64:
                continue
            c = m["cnt"]
            if c.sum() < 64 * E:
                small += 1
            else:
                var_multi_half += int(((c > 128) & (c % 128 > 0) & (c % 128 <= 64)).any())
    run.close()
    assert small > 0 and var_multi_half > 0, (small, var_multi_half)
    U.check(wl, a)


def test_var_tiles_packed_rows_agree_bitwise():
    # f32 rows are packed to bf16, so GEMM1 reads the packed copy: the
    # wait-all batch (1536 pairs, 180-212 rows per expert: a 128-row tile,
    # then a half or a second full tile) runs the 128-row tiles, single
    # chunks (384 pairs) the 64-row tiles
    wl = W.generate("tiny", 1, R=2, T=384)
    E, k = wl.cfg["E"], wl.cfg["k"]
    assert 64 * E <= wl.n_pairs < 256 * E
    assert max(wl.chunk_pairs(c) for c in wl.chunks) < 64 * E
    run = harness.Runner(wl, n_streams=2, record_routing=True)
    run.run(policy=cep.CEP_WAIT_ALL)
    a = _out(run)
    c = cep.cep_get_batch_routing(run.ctx, 0, E, k)["cnt"]
    assert (c > 128).all() and (c % 128 <= 64).any() and (c % 128 > 64).any(), c
    run.out.zero_()
    run.run(policy=cep.CEP_PER_CHUNK, n_streams=2)
    b = _out(run)
    run.close()
    assert np.array_equal(a, b)
    U.check(wl, a)


def test_stream_tiles_by_rows_agree_bitwise():
    # Weight-streaming bf16 batches (fewer than 64 pairs per local expert:
    # single chunks of the straggler shape, a hot expert of 100-150 rows
    # beside experts of a few rows) run both GEMMs over their 64-row tiles
    # listed by rows, most first, one work item per workgroup, waves of
    # padding rows loading no rows; resident and fetched experts have lists
    # of their own.  Same K order as the wait-all batch: the same bits.
    wl = W.generate("zipf_imbalanced_d7168", 8, d=1024, I=512, fetch_frac=0.25)
    E, k = wl.cfg["E"], wl.cfg["k"]
    assert wl.fetched
    run = harness.Runner(wl, n_streams=2, record_routing=True)
    run.run(policy=cep.CEP_WAIT_ALL)
    a = _out(run)
    run.out.zero_()
    run.run(policy=cep.CEP_PER_CHUNK, n_streams=2)
    b = _out(run)
    fetched = np.zeros(E, bool)
    fetched[list(wl.fetched)] = True
    mixed = 0
    for i in range(cep.cep_get_batch_count(run.ctx)):
        m = cep.cep_get_batch_routing(run.ctx, i, E, k)
        c = m["cnt"]
        assert m["align"] == 64 and c.sum() < 64 * E
        # several tiles of one expert, tiles of a few rows, resident and
        # fetched experts with pairs
        mixed += int(c.max() > 64 and ((c > 0) & (c <= 16)).any() and
                     (c[fetched] > 0).any() and (c[~fetched] > 0).any())
    run.close()
    assert mixed > 0
    assert np.array_equal(a, b)
    U.check(wl, a)


def test_remainder_tiles_agree_bitwise():
    # Full-size wait-all batch: two experts overflow 4 full 256-row tiles by a
    # few rows, which the tile plan runs as 64-row remainder tiles next to the
    # 256-row tiles (fewer full-tile rounds on a 256-CU device).  Per-chunk
    # batches use 64-row tiles only.  Same K order, same bits.
    wl = W.generate("sync_d4096", 0)
    cnt = np.bincount(wl.topk_local[wl.topk_local >= 0], minlength=wl.cfg["E"])
    assert any(0 < c % 256 <= 128 for c in cnt)
    run = harness.Runner(wl, n_streams=1)
    run.run(policy=cep.CEP_WAIT_ALL)
    a = _out(run)
    run.out.zero_()
    run.run(policy=cep.CEP_PER_CHUNK)
    b = _out(run)
    run.close()
    assert np.array_equal(a, b)


def test_fetched_experts_equal_resident_bitwise():
    wl = W.generate("fp8_fetch_d6144", 0, T=256, cpr=2)
    a = harness.Runner(wl, n_streams=2, use_fetch=True)
    a.run(policy=cep.CEP_THRESHOLD, theta=600, n_streams=2)
    ga = _out(a)
    st = a.stats()
    assert "fetch" in st and st["fetch"]["bytes"] == len(wl.fetched) * a.blob_bytes
    assert all(b["fetched"] for b in st["batches"])
    a.close()
    b = harness.Runner(wl, n_streams=1, use_fetch=False)
    b.run(policy=cep.CEP_WAIT_ALL)
    gb = _out(b)
    b.close()
    assert np.array_equal(ga, gb)


def test_fetched_bf16_experts_equal_resident_bitwise():
    # bf16 rows are read in place by GEMM1 on the helper stream too
    wl = W.generate("zipf_stream_d7168", 0, d=1024, I=512, E=8, Eg=32, T=512, cpr=4,
                    fetch_frac=0.25)
    assert wl.fetched
    a = harness.Runner(wl, n_streams=3, use_fetch=True)
    a.run(policy=cep.CEP_THRESHOLD, theta=300, n_streams=3)
    ga = _out(a)
    assert all(b["fetched"] for b in a.stats()["batches"])
    a.close()
    b = harness.Runner(wl, n_streams=1, use_fetch=False)
    b.run(policy=cep.CEP_WAIT_ALL)
    gb = _out(b)
    b.close()
    assert np.array_equal(ga, gb)
    U.check(wl, gb)


# ----------------------------------------------------------- error paths
def test_error_paths():
    wl = W.generate("tiny", 0)
    run = harness.Runner(wl, n_streams=2)
    ctx = run.ctx
    ch = run.chunks[0]
    E = pytest.raises
    with E(cep.CepError) as e:  # no open layer
        cep.cep_submit_chunk(ctx, 1, 0, ch.n_rows, ch.n_pairs, ch.token_idx, ch.x, ch.ids, ch.w)
    assert e.value.status == cep.CEP_ESTATE
    cep.cep_begin_layer(ctx, 7, run.chunks_per_replica, run.out)
    with E(cep.CepError) as e:  # wrong generation
        cep.cep_submit_chunk(ctx, 8, 0, ch.n_rows, ch.n_pairs, ch.token_idx, ch.x, ch.ids, ch.w)
    assert e.value.status == cep.CEP_ESTATE
    with E(cep.CepError) as e:  # replica out of range
        cep.cep_submit_chunk(ctx, 7, 5, ch.n_rows, ch.n_pairs, ch.token_idx, ch.x, ch.ids, ch.w)
    assert e.value.status == cep.CEP_EINVAL
    with E(cep.CepError) as e:  # more pairs than rows * k
        cep.cep_submit_chunk(ctx, 7, 0, 1, 5, ch.token_idx, ch.x, ch.ids, ch.w)
    assert e.value.status == cep.CEP_EINVAL
    with E(cep.CepError) as e:  # rows not 16-byte aligned (checked before any read)
        cep.cep_submit_chunk(ctx, 7, 0, 1, 1, ch.token_idx, ch.x.view(-1)[1:], ch.ids, ch.w)
    assert e.value.status == cep.CEP_EINVAL and "aligned" in str(e.value)
    with E(cep.CepError) as e:  # policy change inside a layer
        cep.cep_set_policy(ctx, cep.CEP_PER_CHUNK)
    assert e.value.status == cep.CEP_ESTATE
    with E(cep.CepError) as e:  # fetch beyond the (zero-byte) buffer
        cep.cep_weight_fetch(ctx, [0], [run.out.data_ptr()])
    assert e.value.status == cep.CEP_ENOMEM
    cep.cep_weight_fetch(ctx, [], [])  # the one decision: empty
    with E(cep.CepError) as e:  # no second fetch decision in a layer
        cep.cep_weight_fetch(ctx, [], [])
    assert e.value.status == cep.CEP_EBUSY
    cep.cep_flush(ctx)  # nothing pending: no-op
    with E(cep.CepError) as e:  # chunks still expected
        cep.cep_combine(ctx)
    assert e.value.status == cep.CEP_ESTATE
    for c in run.chunks:
        cep.cep_submit_chunk(ctx, 7, c.replica, c.n_rows, c.n_pairs, c.token_idx, c.x, c.ids, c.w)
    with E(cep.CepError) as e:  # all expected chunks already in
        cep.cep_submit_chunk(ctx, 7, 0, ch.n_rows, ch.n_pairs, ch.token_idx, ch.x, ch.ids, ch.w)
    assert e.value.status == cep.CEP_ESTATE
    cep.cep_combine(ctx)
    torch.cuda.synchronize()
    cep.cep_get_status(ctx)

    # device-side checks: an id outside [-1, E) and a wrong pair count
    bad = ch.ids.clone()
    bad[0, 0] = wl.cfg["E"] + 3
    cep.cep_begin_layer(ctx, 9, [1, 0], run.out)
    cep.cep_submit_chunk(ctx, 9, 0, ch.n_rows, ch.n_pairs, ch.token_idx, ch.x, bad, ch.w)
    cep.cep_combine(ctx)
    with E(cep.CepError) as e:
        cep.cep_get_status(ctx)
    assert e.value.status == cep.CEP_EINVAL and "expert id" in str(e.value)
    cep.cep_get_status(ctx)  # cleared
    run.close()


def test_phase_timing_switch_keeps_results():
    wl = W.generate("tiny", 0)
    run = harness.Runner(wl, n_streams=2)
    run.run(policy=cep.CEP_THRESHOLD, theta=300, n_streams=2)
    a = _out(run)
    st = run.stats()
    assert all(b["gemm1_ms"] >= 0 for b in st["batches"])
    cep.cep_set_phase_timing(run.ctx, False)
    run.out.zero_()
    run.run(policy=cep.CEP_THRESHOLD, theta=300, n_streams=2)
    b = _out(run)
    st = run.stats()
    assert all(x["route_ms"] == -1 and x["gemm1_ms"] == -1 for x in st["batches"])
    assert all(x["start_ms"] == -1 and x["end_ms"] >= 0 for x in st["batches"])
    run.close()
    assert np.array_equal(a, b)


def test_all_remote_chunk_launches_nothing():
    wl = W.generate("tiny", 0)
    run = harness.Runner(wl)
    ch = run.chunks[0]
    ids = torch.full_like(ch.ids, -1)
    run.out.fill_(3.0)
    cep.cep_begin_layer(run.ctx, 1, [1, 0], run.out)
    cep.cep_submit_chunk(run.ctx, 1, ch.replica, ch.n_rows, 0, ch.token_idx, ch.x, ids, ch.w)
    cep.cep_combine(run.ctx)
    torch.cuda.synchronize()
    cep.cep_get_status(run.ctx)
    assert cep.cep_get_batch_count(run.ctx) == 0
    assert torch.all(run.out == 3.0)
    run.close()


def test_fp8_persistent_tiles_odd_k_steps_all_rows():
    # The persistent 8-wave e4m3 tiles over more tiles than workgroups (each
    # workgroup runs several, prefetching the next one's first stage during
    # the epilogue) with an odd number of K steps in GEMM2 (I = 640: five),
    # so that a tile's last step uses ring buffer 0, the buffer the next
    # tile's first stage fills: every row against the oracle, and bitwise
    # equal to per-chunk batches on the 4-wave 128-row tile.
    wl = W.generate("fp8_fetch_d6144", 11, d=1024, I=640, E=4, Eg=16, R=4, T=4096, cpr=64)
    E, k = wl.cfg["E"], wl.cfg["k"]
    run = harness.Runner(wl, n_streams=1, record_routing=True, use_fetch=False)
    run.run(policy=cep.CEP_WAIT_ALL)
    a = _out(run)
    m = cep.cep_get_batch_routing(run.ctx, 0, E, k)
    assert m["align"] == 256
    m_tiles = int(sum((c + 255) // 256 for c in m["cnt"]))
    assert m_tiles * (wl.cfg["d"] // 256) > 256, m["cnt"]  # GEMM2 tiles > workgroups
    mx, rel = U.check(wl, a)
    run.out.zero_()
    run.run(policy=cep.CEP_PER_CHUNK)
    b = _out(run)
    aligns = {cep.cep_get_batch_routing(run.ctx, i, E, k)["align"]
              for i in range(cep.cep_get_batch_count(run.ctx))}
    run.close()
    assert aligns == {128}
    assert np.array_equal(a, b)
    print(f"fp8 persistent tiles, odd K steps: pairs={wl.n_pairs} max_abs={mx:.3e} rel={rel:.3e}")


def test_fp8_whole_groups_per_xcd_all_rows():
    # 141 M tiles of 256 rows with 4 column tiles in GEMM1: eighteen groups of
    # eight M tiles, the last partial, so that the persistent GEMM1 gives each
    # XCD whole groups (two or three) instead of contiguous shares.  Every
    # row against the oracle; the two per-replica batches (about 71 M tiles
    # each) bitwise equal to the wait-all batch.
    wl = W.generate("fp8_fetch_d6144", 5, d=512, I=512, E=4, Eg=8, k=4, R=2, T=8192, cpr=1)
    E, k = wl.cfg["E"], wl.cfg["k"]
    run = harness.Runner(wl, n_streams=2, record_routing=True, use_fetch=False)
    run.run(policy=cep.CEP_WAIT_ALL)
    a = _out(run)
    m = cep.cep_get_batch_routing(run.ctx, 0, E, k)
    assert m["align"] == 256
    m_tiles = int(sum((c + 255) // 256 for c in m["cnt"]))
    assert m_tiles > 16 * 8 and m_tiles % 8, m["cnt"]
    mx, rel = U.check(wl, a)
    run.out.zero_()
    run.run(policy=cep.CEP_PER_CHUNK, n_streams=2)
    b = _out(run)
    run.close()
    assert np.array_equal(a, b)
    print(f"fp8 whole groups per XCD: pairs={wl.n_pairs} M tiles={m_tiles} rel={rel:.3e}")


def test_fp8_large_tile_all_rows_and_small_tile_bitwise():
    # The e4m3 8-wave 256-row tile (the large-batch tile of the e4m3
    # workload) over every row against the oracle: four experts of 1757 to
    # 4229 rows, each over several 256-row tiles ending in a partial one, one
    # of them fetched.  Per-chunk batches (at most 370 pairs) run the 4-wave
    # 128-row tile: each wave computes the same 128 x 64 block with the same
    # K order and promotion, so the same bits.
    wl = W.generate("fp8_fetch_d6144", 7, d=1024, I=512, E=4, Eg=16, R=4, T=2048, cpr=8)
    E, k = wl.cfg["E"], wl.cfg["k"]
    run = harness.Runner(wl, n_streams=2, record_routing=True, use_fetch=True)
    run.run(policy=cep.CEP_WAIT_ALL)
    a = _out(run)
    m = cep.cep_get_batch_routing(run.ctx, 0, E, k)
    assert m["align"] == 256
    assert (m["cnt"] > 1024).sum() >= 2 and (m["cnt"] % 256 != 0).all(), m["cnt"]
    mx, rel = U.check(wl, a)
    run.out.zero_()
    run.run(policy=cep.CEP_PER_CHUNK, n_streams=2)
    b = _out(run)
    aligns = {cep.cep_get_batch_routing(run.ctx, i, E, k)["align"]
              for i in range(cep.cep_get_batch_count(run.ctx))}
    run.close()
    assert aligns == {128}
    assert np.array_equal(a, b)
    print(f"fp8 256-row tile all rows: pairs={wl.n_pairs} max_abs={mx:.3e} rel={rel:.3e}")
