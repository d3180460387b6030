"""GPU parity at the library's size limits (through the C ABI): the most local
experts and routing slots, the widest d_model and d_ff, for bf16, e4m3 and
MXFP4 weights.  Token counts are small so the oracle covers every row."""
import numpy as np
import pytest
import torch

from oracle import routing as orout
from paper_2609_33252_amd import cep, harness, workload as W

from . import _util as U

pytestmark = pytest.mark.gpu

MAX_E, MAX_K, MAX_DIM = 64, 16, 32768


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cep.lib()
    torch.cuda.set_device(0)


def _run(wl, **kw):
    run = harness.Runner(wl, n_streams=2, **kw)
    run.run(policy=cep.CEP_THRESHOLD, theta=max(1, wl.n_pairs // 2), n_streams=2)
    torch.cuda.synchronize()
    cep.cep_get_status(run.ctx)
    return run


def test_most_experts_and_slots():
    # 64 local experts, 16 slots per token: routing bit-exact, outputs in tolerance
    wl = W.generate("sync_d4096", 0, d=256, I=128, E=MAX_E, Eg=MAX_E, k=MAX_K, R=2, T=256,
                    cpr=2)
    run = _run(wl, record_routing=True)
    for b in range(cep.cep_get_batch_count(run.ctx)):
        m = cep.cep_get_batch_routing(run.ctx, b, MAX_E, MAX_K)
        ids = [wl.topk_local[wl.chunks[c].replica][wl.chunks[c].token_idx] for c in m["chunks"]]
        ref = orout.batch_routing(ids, MAX_E, m["align"])
        for key in ("cnt", "off", "off_pad", "perm_src", "pos_of"):
            assert np.array_equal(m[key], ref[key]), (b, key)
    got = run.out.cpu().numpy()
    run.close()
    U.check(wl, got)


@pytest.mark.parametrize("d,I", [(MAX_DIM, 128), (256, MAX_DIM)])
def test_widest_dims_bf16(d, I):
    wl = W.generate("sync_d4096", 1, d=d, I=I, E=2, Eg=4, k=2, R=1, T=64, cpr=2)
    run = _run(wl)
    got = run.out.cpu().numpy()
    run.close()
    mx, rel = U.check(wl, got)
    print(f"bf16 d={d} I={I}: pairs={wl.n_pairs} max_abs={mx:.3e} rel={rel:.3e}")


@pytest.mark.parametrize("d,I", [(MAX_DIM, 128), (256, MAX_DIM)])
def test_widest_dims_fp8_with_fetch(d, I):
    # the e4m3 GEMM keeps K/128 weight scales per row in LDS: K = 32768 is
    # its largest case; one of the two experts is fetched
    wl = W.generate("fp8_fetch_d6144", 2, d=d, I=I, E=2, Eg=4, k=2, R=1, T=64, cpr=1,
                    fetch_frac=0.5)
    assert len(wl.fetched) == 1
    run = _run(wl, use_fetch=True)
    got = run.out.cpu().numpy()
    run.close()
    mx, rel = U.check(wl, got)
    print(f"e4m3 d={d} I={I}: pairs={wl.n_pairs} max_abs={mx:.3e} rel={rel:.3e}")


@pytest.mark.parametrize("d,I", [(MAX_DIM, 128), (256, MAX_DIM)])
def test_widest_dims_mxfp4(d, I):
    wl = W.generate("mxfp4_dsv4flash_d4096", 3, d=d, I=I, E=2, Eg=4, k=2, R=1, T=64, cpr=2)
    run = _run(wl)
    got = run.out.cpu().numpy()
    run.close()
    mx, rel = U.check(wl, got)
    print(f"mxfp4 d={d} I={I}: pairs={wl.n_pairs} max_abs={mx:.3e} rel={rel:.3e}")
