"""Weight fetch modes and the fallback (Section 3.3; Appendix C, "One-shot
weight fetching" and "FFN reassignment commit and fallback").

A fetched expert's work gives the same bits whether its weights were copied
into the fetch buffer (their GEMMs run after the copy), read in
place from the donor region, or read in place after a copy that failed to
start; and the same bits as a context holding every expert resident.  An
expert without weights keeps its chunks pending until a fetch brings them.
"""
import numpy as np
import pytest
import torch

from paper_2609_33252_amd import cep, harness, workload as W

from . import _util as U

pytestmark = pytest.mark.gpu

CASES = {
    "fp8": ("fp8_fetch_d6144", dict(T=256, cpr=2)),
    "bf16": ("zipf_stream_d7168", dict(d=1024, I=512, E=8, Eg=32, T=512, cpr=4, fetch_frac=0.25)),
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


@pytest.mark.parametrize("case", sorted(CASES))
def test_fetch_modes_equal_resident_bitwise(case):
    name, kw = CASES[case]
    wl = W.generate(name, 0, **kw)
    assert wl.fetched
    base = harness.Runner(wl, n_streams=1, use_fetch=False)
    base.run(policy=cep.CEP_WAIT_ALL)
    ref = _out(base)
    base.close()
    U.check(wl, ref)
    run = harness.Runner(wl, n_streams=2, use_fetch=True)
    theta = max(1, wl.n_pairs // 3)
    for mode in (cep.CEP_FETCH_COPY, cep.CEP_FETCH_IN_PLACE, cep.CEP_FETCH_FAIL_COPY,
                 cep.CEP_FETCH_COPY):
        run.out.zero_()
        run.run(policy=cep.CEP_THRESHOLD, theta=theta, n_streams=2, fetch_mode=mode)
        got = _out(run)
        assert np.array_equal(got, ref), mode
        st = run.stats()
        f = st["fetch"]
        assert f["experts"] == len(wl.fetched)
        if mode == cep.CEP_FETCH_COPY:
            assert not f["in_place"] and not f["fallback"]
            assert f["bytes"] == len(wl.fetched) * run.blob_bytes
            assert run.fetch_ready is not None
            assert all(b["fetched"] for b in st["batches"])
        else:
            # no copy gates the work: fetched experts' tiles still run after
            # the resident ones, reading the donor region
            assert f["in_place"] and f["bytes"] == 0
            assert f["fallback"] == (mode == cep.CEP_FETCH_FAIL_COPY)
            assert run.fetch_ready is None
            assert all(b["fetched"] for b in st["batches"])
    run.close()


def test_unfetched_expert_keeps_its_chunks_pending():
    name, kw = CASES["bf16"]
    wl = W.generate(name, 0, **kw)
    base = harness.Runner(wl, n_streams=1, use_fetch=False)
    base.run(policy=cep.CEP_WAIT_ALL)
    ref = _out(base)
    base.close()
    run = harness.Runner(wl, n_streams=2, use_fetch=True)
    ctx = run.ctx
    cep.cep_set_policy(ctx, cep.CEP_WAIT_ALL, 1, 2)
    run.gen += 1
    cep.cep_begin_layer(ctx, run.gen, run.chunks_per_replica, run.out)
    for ch in run.chunks[:-1]:
        cep.cep_submit_chunk(ctx, run.gen, ch.replica, ch.n_rows, ch.n_pairs, ch.token_idx,
                             ch.x, ch.ids, ch.w)
    ch = run.chunks[-1]
    # the last chunk triggers the wait-all launch, which needs the weights
    # of the experts that are not resident: refused, the chunk stays pending
    with pytest.raises(cep.CepError) as e:
        cep.cep_submit_chunk(ctx, run.gen, ch.replica, ch.n_rows, ch.n_pairs, ch.token_idx,
                             ch.x, ch.ids, ch.w)
    assert e.value.status == cep.CEP_ESTATE
    assert cep.cep_get_batch_count(ctx) == 0
    with pytest.raises(cep.CepError):
        cep.cep_flush(ctx)
    cep.cep_weight_fetch(ctx, list(wl.fetched),
                         [run.donor.data_ptr() + i * run.blob_bytes
                          for i in range(len(wl.fetched))], run.side)
    cep.cep_flush(ctx)
    assert cep.cep_get_batch_count(ctx) == 1
    cep.cep_combine(ctx)
    got = _out(run)
    run.close()
    assert np.array_equal(got, ref)


def test_fetch_buffer_reused_across_layers():
    # consecutive layers each fetch into the same buffer, one with no batch
    # after its fetch (an unconsumed copy); every layer's output is right
    name, kw = CASES["fp8"]
    wl = W.generate(name, 0, **kw)
    base = harness.Runner(wl, n_streams=1, use_fetch=False)
    base.run(policy=cep.CEP_WAIT_ALL)
    ref = _out(base)
    base.close()
    run = harness.Runner(wl, n_streams=3, use_fetch=True)
    for i in range(4):
        run.out.zero_()
        run.run(policy=cep.CEP_THRESHOLD, theta=200 + 300 * i, n_streams=1 + i % 3)
        assert np.array_equal(_out(run), ref), i
    run.close()


@pytest.mark.parametrize("name", ["fp8_fetch_d6144", "mxfp4_dsv4flash_d4096",
                                  "zipf_stream_d7168"])
def test_every_expert_fetched_large_tiles(name):
    # Every local expert fetched, batches of 256-row tiles: the resident
    # experts' launches have no tile (the persistent workgroups leave at
    # once) and the fetched experts' launches do all the work.  Every row
    # against the oracle, and bitwise equal to the all-resident layer.
    wl = W.generate(name, 31, d=512, I=256, E=4, Eg=8, k=4, R=2, T=4096, cpr=1, fetch_frac=1.0)
    assert len(wl.fetched) == wl.cfg["E"]
    E, k = wl.cfg["E"], wl.cfg["k"]
    print(f"case {name} pairs={wl.n_pairs}", flush=True)
    a = harness.Runner(wl, n_streams=1, record_routing=True, use_fetch=True)
    a.run(policy=cep.CEP_WAIT_ALL)
    ga = _out(a)
    assert cep.cep_get_batch_routing(a.ctx, 0, E, k)["align"] == 256
    assert all(b["fetched"] for b in a.stats()["batches"])
    a.close()
    b = harness.Runner(wl, n_streams=1, use_fetch=False)
    b.run(policy=cep.CEP_WAIT_ALL)
    gb = _out(b)
    b.close()
    assert np.array_equal(ga, gb)
    U.check(wl, ga)
