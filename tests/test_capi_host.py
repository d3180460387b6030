"""C ABI checks that need no GPU: the library loads, exports every entry point
declared in include/cep.h, and rejects bad arguments before touching HIP."""
import ctypes
import os
import re

import pytest

from paper_2609_33252_amd import cep

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cep.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(cep.LIB_PATH):
        from paper_2609_33252_amd import build
        build.build()
    return cep.lib()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cep_[a-z_]+)\s*\(", text)))


def test_header_declares_the_binding_names():
    assert _declared() == sorted(cep.EXPORTED)


def test_every_declared_symbol_is_exported(L):
    for name in _declared():
        assert hasattr(L, name), name
    # nothing but the cep_* API is visible
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", cep.LIB_PATH], capture_output=True,
                         text=True).stdout
    text_syms = [l.split()[-1] for l in out.splitlines() if " T " in l]
    assert sorted(text_syms) == _declared()


def _cfg(**kw):
    base = dict(d_model=256, d_ff=128, n_local_experts=8, top_k=2, max_replicas=2,
                max_tokens_per_replica=256, w_dtype=cep.CEP_BF16, x_dtype=cep.CEP_BF16,
                n_streams=1)
    base.update(kw)
    return cep.make_config(**base)


def test_packed_bytes_and_validation(L):
    # bf16: W1 [2I][d] + W2 [d][I], 2 bytes each
    assert cep.cep_packed_expert_bytes(_cfg()) == 3 * 256 * 128 * 2
    # fp8: 1-byte codes plus float32 scales per 32-row group / 128 block
    fp8 = _cfg(w_dtype=cep.CEP_FP8_E4M3_B128)
    b = cep.cep_packed_expert_bytes(fp8)
    assert b >= 3 * 256 * 128 and b % 256 == 0
    # MXFP4: half-byte codes plus one E8M0 byte per 32 along K, no padding
    # at these sizes
    mx = _cfg(w_dtype=cep.CEP_MXFP4)
    assert cep.cep_packed_expert_bytes(mx) == 3 * 256 * 128 // 2 + 3 * 256 * 128 // 32
    assert cep.cep_packed_expert_bytes(_cfg(w_dtype=cep.CEP_MXFP4, x_dtype=cep.CEP_F32)) == 0
    assert cep.cep_packed_expert_bytes(_cfg(w_dtype=4)) == 0
    for bad in (dict(d_model=100), dict(d_ff=96), dict(n_local_experts=0),
                dict(n_local_experts=65), dict(top_k=0), dict(top_k=17), dict(n_streams=9),
                dict(x_dtype=cep.CEP_FP8_E4M3_B128), dict(max_replicas=0),
                dict(w_dtype=cep.CEP_FP8_E4M3_B128, x_dtype=cep.CEP_F32),
                dict(w_dtype=cep.CEP_FP8_E4M3_B128, d_model=384)):
        assert cep.cep_packed_expert_bytes(_cfg(**bad)) == 0, bad


def test_null_and_invalid_arguments_fail_cleanly(L):
    h = ctypes.c_void_p()
    w = cep.cep_weights()
    assert L.cep_init_experts(None, ctypes.byref(_cfg()), ctypes.byref(w), None, None) == cep.CEP_EINVAL
    assert L.cep_init_experts(ctypes.byref(h), ctypes.byref(_cfg(d_model=100)), ctypes.byref(w),
                              None, None) == cep.CEP_EINVAL
    assert L.cep_init_experts(ctypes.byref(h), ctypes.byref(_cfg()), ctypes.byref(w), None,
                              None) == cep.CEP_EINVAL  # NULL weight pointers
    # MXFP4 weights without their E8M0 scales
    wx = cep.cep_weights(1 << 20, 1 << 20, 1 << 20, None, None, None)
    assert L.cep_init_experts(ctypes.byref(h), ctypes.byref(_cfg(w_dtype=cep.CEP_MXFP4)),
                              ctypes.byref(wx), None, None) == cep.CEP_EINVAL
    assert b"scale" in L.cep_last_error(None)
    assert L.cep_pack_experts(ctypes.byref(_cfg()), ctypes.byref(w), 0, 1, None, None) == cep.CEP_EINVAL
    for fn, args in (("cep_set_policy", (0, 1, 1)), ("cep_flush", ()), ("cep_get_status", ()),
                     ("cep_combine", (None, None))):
        assert getattr(L, fn)(None, *args) == cep.CEP_EINVAL, fn
    assert L.cep_destroy(None) == cep.CEP_OK
    # the last failure without a context keeps its message
    assert L.cep_last_error(None) == b"cep_pack_experts: bad weights, dst or expert range"
    assert L.cep_get_batch_count(None) == 0
