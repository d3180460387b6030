"""GPU parity over a fixed set of small mixed shapes (through the C ABI).

Each case draws a seeded workload of its own width, expert count, top-k,
routing skew and weight format, runs one layer under its launch policy and
stream count, and checks
* every row against the oracle (the target tolerance of its format), and
* the output bitwise against a wait-all layer on one stream (the batch
  composition, tile shapes and streams do not change any result).

The shapes cross the tile regimes: weight-streaming batches (64-row tiles
listed by rows), mid-size batches (128-row tiles with 64-row halves), large
batches (256-row tiles with 64-row remainders for bf16, the persistent
8-wave tiles for e4m3, 8-wave tiles for MXFP4), with fetched experts for
some.
"""
import numpy as np
import pytest
import torch

from paper_2609_33252_amd import cep, harness, workload as W

from . import _util as U

pytestmark = pytest.mark.gpu

POL = {"wait_all": cep.CEP_WAIT_ALL, "per_chunk": cep.CEP_PER_CHUNK,
       "threshold": cep.CEP_THRESHOLD}

# (preset, seed, overrides, policy, theta as a fraction of the layer's pairs, streams)
CASES = [
    ("tiny", 21, dict(d=512, I=256, E=6, Eg=12, k=3, R=3, T=300, cpr=3), "per_chunk", 0, 3),
    ("sync_d4096", 22, dict(d=768, I=384, E=5, Eg=20, k=4, R=4, T=1024, cpr=4),
     "threshold", 0.3, 2),
    ("sync_d4096", 23, dict(d=512, I=256, E=4, Eg=8, k=4, R=2, T=2048, cpr=2),
     "per_chunk", 0, 2),
    ("zipf_imbalanced_d7168", 24, dict(d=1024, I=512, E=8, Eg=32, R=4, T=1024, cpr=8),
     "threshold", 0.25, 4),
    ("zipf_imbalanced_d7168", 25, dict(d=768, I=256, E=8, Eg=64, R=8, T=512, cpr=4,
                                       fetch_frac=0.25), "per_chunk", 0, 2),
    ("fp8_fetch_d6144", 26, dict(d=768, I=384, E=6, Eg=24, R=4, T=1024, cpr=2),
     "threshold", 0.4, 2),
    ("fp8_fetch_d6144", 27, dict(d=512, I=256, E=4, Eg=8, k=4, R=2, T=4096, cpr=4),
     "per_chunk", 0, 3),
    ("mxfp4_dsv4flash_d4096", 28, dict(d=768, I=512, E=6, Eg=24, R=4, T=1024, cpr=4,
                                       fetch_frac=0.2), "threshold", 0.3, 2),
    ("mxfp4_dsv4flash_d4096", 29, dict(d=512, I=256, E=4, Eg=8, k=4, R=2, T=4096, cpr=2),
     "per_chunk", 0, 2),
    # top-1: every token has one pair (the e4m3 and MXFP4 GEMM2 write every
    # output row themselves)
    ("sync_d4096", 41, dict(d=512, I=256, E=4, Eg=8, k=1, R=2, T=8192, cpr=2), "threshold",
     0.5, 2),
    ("fp8_fetch_d6144", 41, dict(d=512, I=256, E=4, Eg=8, k=1, R=2, T=8192, cpr=2),
     "threshold", 0.5, 2),
    ("mxfp4_dsv4flash_d4096", 41, dict(d=512, I=256, E=4, Eg=8, k=1, R=2, T=8192, cpr=2),
     "threshold", 0.5, 2),
]


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


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-{c[1]}" for c in CASES])
def test_mixed_shape_matches_oracle_and_wait_all(case):
    name, seed, over, pol, frac, streams = case
    wl = W.generate(name, seed, **over)
    E, k = wl.cfg["E"], wl.cfg["k"]
    print(f"case {name} seed={seed} pairs={wl.n_pairs} policy={pol} streams={streams}",
          flush=True)
    run = harness.Runner(wl, n_streams=streams, record_routing=True)
    run.run(policy=cep.CEP_WAIT_ALL)
    a = _out(run)
    run.out.zero_()
    theta = max(1, int(frac * wl.n_pairs))
    run.run(policy=POL[pol], theta=theta, n_streams=streams)
    b = _out(run)
    aligns = sorted({cep.cep_get_batch_routing(run.ctx, i, E, k)["align"]
                     for i in range(cep.cep_get_batch_count(run.ctx))})
    run.close()
    assert np.array_equal(a, b)
    mx, rel = U.check(wl, b)
    assert not b[~wl.delivered].any()
    print(f"  aligns={aligns} max_abs={mx:.3e} rel={rel:.3e}")
