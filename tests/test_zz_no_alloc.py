"""The allocation-free entry point (cep_ffn_noalloc) against the existing
path it is a variant of: a one-chunk wait-all layer through cep_begin_layer,
cep_submit_chunk and cep_combine.  Two calls in a row, the second with a
smaller chunk (the shared scratch keeps the first call's contents), each
bitwise equal to the existing path and within the target tolerance of the
oracle; a chunk beyond the scratch is refused before any work."""
import numpy as np
import pytest
import torch

from paper_2609_33252_amd import cep, harness, workload as W

from . import _util as U

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cep.lib()
    torch.cuda.set_device(0)


def _existing(run, i):
    run.out.zero_()
    run.run_subset([i])
    torch.cuda.synchronize()
    cep.cep_get_status(run.ctx)
    return run.out.cpu().numpy()


def _noalloc(run, i):
    ch = run.chunks[i]
    out = torch.zeros_like(run.out)
    cep.cep_ffn_noalloc(run.ctx, ch.replica, ch.n_rows, ch.n_pairs, ch.token_idx, ch.x, ch.ids,
                        ch.w, out, torch.cuda.current_stream())
    torch.cuda.synchronize()
    cep.cep_get_status(run.ctx)
    return out.cpu().numpy()


CASES = {
    # bf16 weights and rows (rows read in place), 64-row and 256-row tiles
    "bf16": ("zipf_stream_d7168", dict(d=1024, I=512, Eg=16, R=2, T=2048, cpr=2, zipf=None)),
    # e4m3 weights (rows quantised into the scratch), 256-row then 128-row tiles
    "fp8": ("fp8_fetch_d6144", dict(d=1024, I=512, E=4, Eg=16, R=2, T=2048, cpr=2,
                                    fetch_frac=0.0)),
    # float32 rows packed to bf16
    "f32": ("tiny", dict(R=2, T=512, cpr=2)),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_noalloc_equals_existing_entry_point(case):
    name, kw = CASES[case]
    wl = W.generate(name, 0, **kw)
    run = harness.Runner(wl, n_streams=1)
    pairs = [ch.n_pairs for ch in run.chunks]
    big = int(np.argmax(pairs))
    # a second, smaller chunk: half the rows of another chunk
    other = next(i for i in range(len(run.chunks)) if i != big and pairs[i] > 0)
    ch = run.chunks[other]
    half = ch.n_rows // 2
    small = harness.DeviceChunk()
    small.replica, small.n_rows = ch.replica, half
    small.token_idx, small.x = ch.token_idx[:half], ch.x[:half]
    small.ids, small.w = ch.ids[:half], ch.w[:half]
    small.n_pairs = int((small.ids >= 0).sum().item())
    small.arrival_ms = ch.arrival_ms
    run.chunks.append(small)
    run.chunks_per_replica[small.replica] += 1
    s_idx = len(run.chunks) - 1
    assert 0 < small.n_pairs < pairs[big]
    for i in (big, s_idx):
        got = _noalloc(run, i)
        want = _existing(run, i)
        assert np.array_equal(got, want), (case, i)
        c = run.chunks[i]
        tok = np.stack([np.full(c.n_rows, c.replica), c.token_idx.cpu().numpy()], axis=1)
        U.check(wl, got[tok[:, 0], tok[:, 1]], tokens=tok)
        # rows of tokens not in the chunk are untouched
        mask = np.ones(got.shape[:2], bool)
        mask[tok[:, 0], tok[:, 1]] = False
        assert not got[mask].any()
    run.close()


def test_noalloc_refuses_a_chunk_beyond_its_scratch():
    # every slot local: 2048 rows x 8 slots = 16384 pairs need about 84 MB
    wl = W.generate("sync_d4096", 0, d=1024, I=512, E=8, Eg=8, k=8, R=1, T=2048, cpr=1)
    run = harness.Runner(wl, n_streams=1)
    ch = run.chunks[0]
    assert ch.n_pairs == 2048 * 8
    out = torch.full_like(run.out, 5.0)
    with pytest.raises(cep.CepError) as e:
        cep.cep_ffn_noalloc(run.ctx, ch.replica, ch.n_rows, ch.n_pairs, ch.token_idx, ch.x,
                            ch.ids, ch.w, out)
    assert e.value.status == cep.CEP_ENOMEM and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert torch.all(out == 5.0)
    run.close()
