"""ctypes binding of libcep (include/cep.h): same entry-point names, argument
marshalling only.  Torch tensors are passed as device pointers and torch
streams/events as HIP handles; every step of the path runs in libcep's HIP
kernels.  Importing this module does not load the library; the first call
does, and raises if libcep.so has not been built.
"""
from __future__ import annotations

import ctypes
import json
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcep.so")

CEP_OK, CEP_EINVAL, CEP_ENOMEM, CEP_EHIP, CEP_ESTATE, CEP_EBUSY = 0, -1, -2, -3, -4, -5
CEP_F32, CEP_BF16, CEP_FP8_E4M3_B128, CEP_MXFP4 = 0, 1, 2, 3
CEP_WAIT_ALL, CEP_PER_CHUNK, CEP_THRESHOLD = 0, 1, 2
CEP_FETCH_COPY, CEP_FETCH_IN_PLACE, CEP_FETCH_FAIL_COPY = 0, 1, 2
STATUS_NAMES = {0: "CEP_OK", -1: "CEP_EINVAL", -2: "CEP_ENOMEM", -3: "CEP_EHIP",
                -4: "CEP_ESTATE", -5: "CEP_EBUSY"}

EXPORTED = ["cep_packed_expert_bytes", "cep_pack_experts", "cep_init_experts", "cep_set_policy",
            "cep_begin_layer", "cep_submit_chunk", "cep_flush", "cep_weight_fetch",
            "cep_combine", "cep_get_batch_routing", "cep_get_batch_count", "cep_get_stats",
            "cep_get_status", "cep_last_error", "cep_destroy", "cep_set_phase_timing",
            "cep_set_fetch_mode", "cep_ffn_noalloc",
            "cep_profile_create",
            "cep_profile_peak", "cep_profile_theta", "cep_profile_eta", "cep_profile_latency",
            "cep_profile_destroy", "cep_oewf_create", "cep_oewf_begin_layer", "cep_oewf_set_rank",
            "cep_oewf_completion", "cep_oewf_makespan", "cep_oewf_select", "cep_oewf_evaluate",
            "cep_oewf_commit", "cep_oewf_destroy"]

OEWF_MAX_EXPERTS = 64


class cep_config(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int), ("d_ff", ctypes.c_int),
                ("n_local_experts", ctypes.c_int), ("top_k", ctypes.c_int),
                ("max_replicas", ctypes.c_int), ("max_tokens_per_replica", ctypes.c_int),
                ("w_dtype", ctypes.c_int), ("x_dtype", ctypes.c_int),
                ("n_streams", ctypes.c_int), ("max_pairs_per_batch", ctypes.c_int),
                ("fetch_buffer_bytes", ctypes.c_size_t), ("record_routing", ctypes.c_int)]


class cep_weights(ctypes.Structure):
    _fields_ = [("w_gate", ctypes.c_void_p), ("w_up", ctypes.c_void_p),
                ("w_down", ctypes.c_void_p), ("s_gate", ctypes.c_void_p),
                ("s_up", ctypes.c_void_p), ("s_down", ctypes.c_void_p)]


class cep_oewf_fetch(ctypes.Structure):
    _fields_ = [("helper", ctypes.c_int), ("donor", ctypes.c_int), ("n_experts", ctypes.c_int),
                ("experts", ctypes.c_int * OEWF_MAX_EXPERTS),
                ("tokens", ctypes.c_int64 * OEWF_MAX_EXPERTS), ("bytes", ctypes.c_int64),
                ("plan_id", ctypes.c_int64)]


class cep_oewf_decision(ctypes.Structure):
    _fields_ = [("admit", ctypes.c_int), ("Td", ctypes.c_double), ("Th", ctypes.c_double),
                ("Td2", ctypes.c_double), ("Th2", ctypes.c_double), ("alpha", ctypes.c_double),
                ("plan_id", ctypes.c_int64), ("n_trans", ctypes.c_int64),
                ("donor_version", ctypes.c_uint64), ("helper_version", ctypes.c_uint64)]


class CepError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def lib():
    """The loaded libcep.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_33252_amd.build` (needs hipcc)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        P = ctypes.POINTER
        L.cep_packed_expert_bytes.argtypes = [P(cep_config)]
        L.cep_packed_expert_bytes.restype = sz
        L.cep_pack_experts.argtypes = [P(cep_config), P(cep_weights), i32, i32, vp, vp]
        L.cep_init_experts.argtypes = [P(vp), P(cep_config), P(cep_weights), vp, vp]
        L.cep_set_policy.argtypes = [vp, i32, i32, i32]
        L.cep_begin_layer.argtypes = [vp, ctypes.c_uint32, i32, P(i32), vp]
        L.cep_submit_chunk.argtypes = [vp, ctypes.c_uint32, i32, i32, i32, vp, vp, vp, vp, vp,
                                       P(ctypes.c_int64)]
        L.cep_flush.argtypes = [vp]
        L.cep_weight_fetch.argtypes = [vp, P(i32), i32, P(vp), vp, P(vp)]
        L.cep_combine.argtypes = [vp, vp, P(vp)]
        L.cep_get_batch_routing.argtypes = [vp, i32, P(i32), P(i32), P(i32), vp, vp, vp, vp, vp,
                                            vp, P(i32)]
        L.cep_get_batch_count.argtypes = [vp]
        L.cep_get_stats.argtypes = [vp, ctypes.c_char_p, sz]
        L.cep_get_status.argtypes = [vp]
        L.cep_last_error.argtypes = [vp]
        L.cep_last_error.restype = ctypes.c_char_p
        L.cep_destroy.argtypes = [vp]
        L.cep_set_phase_timing.argtypes = [vp, i32]
        L.cep_set_fetch_mode.argtypes = [vp, i32]
        L.cep_ffn_noalloc.argtypes = [vp, i32, i32, i32, vp, vp, vp, vp, vp, vp]
        i64, f64 = ctypes.c_int64, ctypes.c_double
        L.cep_profile_create.argtypes = [P(i64), P(f64), i32, P(vp)]
        L.cep_profile_peak.argtypes = [vp]
        L.cep_profile_peak.restype = f64
        L.cep_profile_theta.argtypes = [vp, f64, P(i64)]
        L.cep_profile_eta.argtypes = [vp, i64, P(f64)]
        L.cep_profile_latency.argtypes = [vp, i64, P(f64)]
        L.cep_profile_destroy.argtypes = [vp]
        L.cep_profile_destroy.restype = None
        L.cep_oewf_create.argtypes = [i32, vp, P(vp)]
        L.cep_oewf_begin_layer.argtypes = [vp]
        L.cep_oewf_set_rank.argtypes = [vp, i32, i32, f64, f64, i64, f64]
        L.cep_oewf_completion.argtypes = [vp, i32, P(f64)]
        L.cep_oewf_makespan.argtypes = [vp, P(f64)]
        L.cep_oewf_select.argtypes = [vp, i32, i32, P(i64), P(i64), i64, P(cep_oewf_fetch)]
        L.cep_oewf_evaluate.argtypes = [vp, P(cep_oewf_fetch), i64, f64, P(cep_oewf_decision)]
        L.cep_oewf_commit.argtypes = [vp, P(cep_oewf_decision), i32, P(i32)]
        L.cep_oewf_destroy.argtypes = [vp]
        L.cep_oewf_destroy.restype = None
        for name in EXPORTED:
            if name not in ("cep_packed_expert_bytes", "cep_last_error", "cep_profile_peak",
                            "cep_profile_destroy", "cep_oewf_destroy"):
                getattr(L, name).restype = i32
        _lib = L
    return _lib


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(s):
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _event(e):
    if e is None:
        return None
    if isinstance(e, int):
        return e
    return e.cuda_event


def _check(ctx, rc):
    if rc != CEP_OK:
        raise CepError(rc, lib().cep_last_error(ctx).decode())
    return rc


def make_config(**kw) -> cep_config:
    c = cep_config()
    c.n_streams = 1
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def make_weights(w_gate, w_up, w_down, s_gate=None, s_up=None, s_down=None) -> cep_weights:
    return cep_weights(_ptr(w_gate), _ptr(w_up), _ptr(w_down), _ptr(s_gate), _ptr(s_up),
                       _ptr(s_down))


# ---------------------------------------------------------------- calls

def cep_packed_expert_bytes(cfg: cep_config) -> int:
    return int(lib().cep_packed_expert_bytes(ctypes.byref(cfg)))


def cep_pack_experts(cfg, weights, first, n, dst, stream=None):
    _check(None, lib().cep_pack_experts(ctypes.byref(cfg), ctypes.byref(weights), first, n,
                                        _ptr(dst), _stream(stream)))


def cep_init_experts(cfg, weights, resident=None, stream=None):
    """Returns the context handle (int)."""
    h = ctypes.c_void_p()
    res = None
    if resident is not None:
        res = (ctypes.c_uint8 * len(resident))(*[1 if r else 0 for r in resident])
    rc = lib().cep_init_experts(ctypes.byref(h), ctypes.byref(cfg), ctypes.byref(weights),
                                res, _stream(stream))
    _check(None, rc)
    return h.value


def cep_set_policy(ctx, policy, threshold_pairs=1, n_streams=1):
    _check(ctx, lib().cep_set_policy(ctx, policy, threshold_pairs, n_streams))


def cep_begin_layer(ctx, generation, chunks_per_replica, out):
    arr = (ctypes.c_int * len(chunks_per_replica))(*chunks_per_replica)
    _check(ctx, lib().cep_begin_layer(ctx, generation, len(chunks_per_replica), arr, _ptr(out)))


def cep_submit_chunk(ctx, generation, replica, n_rows, n_pairs, token_idx, x, topk_id, topk_w,
                     arrival=None):
    cid = ctypes.c_int64(-1)
    _check(ctx, lib().cep_submit_chunk(ctx, generation, replica, n_rows, n_pairs, _ptr(token_idx),
                                       _ptr(x), _ptr(topk_id), _ptr(topk_w), _event(arrival),
                                       ctypes.byref(cid)))
    return cid.value


def cep_flush(ctx):
    _check(ctx, lib().cep_flush(ctx))


def cep_weight_fetch(ctx, ids, src_blobs, side=None):
    """ids: list of local expert ids; src_blobs: device pointers (ints or
    tensors).  Returns the library-owned ready event handle (int or None)."""
    n = len(ids)
    a = (ctypes.c_int * max(n, 1))(*ids)
    b = (ctypes.c_void_p * max(n, 1))(*[_ptr(p) for p in src_blobs])
    ev = ctypes.c_void_p()
    _check(ctx, lib().cep_weight_fetch(ctx, a, n, b, _stream(side), ctypes.byref(ev)))
    return ev.value


def cep_combine(ctx, stream=None):
    ev = ctypes.c_void_p()
    _check(ctx, lib().cep_combine(ctx, _stream(stream), ctypes.byref(ev)))
    return ev.value


def cep_get_batch_count(ctx) -> int:
    return int(lib().cep_get_batch_count(ctx))


def cep_get_batch_routing(ctx, batch, n_experts, top_k):
    """Routing metadata of one batch as numpy arrays (needs record_routing)."""
    import numpy as np
    L = lib()
    align, npairs, nrows, nch = ctypes.c_int(), ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _check(ctx, L.cep_get_batch_routing(ctx, batch, ctypes.byref(align), ctypes.byref(npairs),
                                        ctypes.byref(nrows), None, None, None, None, None, None,
                                        ctypes.byref(nch)))
    cnt = np.zeros(n_experts, np.int32)
    off = np.zeros(n_experts + 1, np.int32)
    off_pad = np.zeros(n_experts + 1, np.int32)
    perm = np.zeros(max(npairs.value, 1), np.int32)
    chunks = np.zeros(max(nch.value, 1), np.int64)
    pos = np.full(max(nrows.value * top_k, 1), -7, np.int32)
    _check(ctx, L.cep_get_batch_routing(ctx, batch, None, None, None,
                                        cnt.ctypes.data, off.ctypes.data, off_pad.ctypes.data,
                                        perm.ctypes.data, pos.ctypes.data, chunks.ctypes.data,
                                        None))
    return dict(align=align.value, n_pairs=npairs.value, n_rows=nrows.value, cnt=cnt, off=off,
                off_pad=off_pad, perm_src=perm[:npairs.value], pos_of=pos[:nrows.value * top_k],
                chunks=chunks[:nch.value])


def cep_get_stats(ctx) -> dict:
    cap = 1 << 16
    while True:
        buf = ctypes.create_string_buffer(cap)
        rc = lib().cep_get_stats(ctx, buf, cap)
        if rc == CEP_ENOMEM:
            cap *= 4
            continue
        _check(ctx, rc)
        return json.loads(buf.value.decode())


def cep_set_phase_timing(ctx, on=True):
    _check(ctx, lib().cep_set_phase_timing(ctx, 1 if on else 0))


def cep_set_fetch_mode(ctx, mode):
    _check(ctx, lib().cep_set_fetch_mode(ctx, mode))


def cep_ffn_noalloc(ctx, replica, n_rows, n_pairs, token_idx, x, topk_id, topk_w, out,
                    stream=None):
    _check(ctx, lib().cep_ffn_noalloc(ctx, replica, n_rows, n_pairs, _ptr(token_idx), _ptr(x),
                                      _ptr(topk_id), _ptr(topk_w), _ptr(out), _stream(stream)))


def cep_get_status(ctx):
    _check(ctx, lib().cep_get_status(ctx))


def cep_last_error(ctx) -> str:
    return lib().cep_last_error(ctx).decode()


def cep_destroy(ctx):
    _check(None, lib().cep_destroy(ctx))


# ------------------------------------------------------------ FFN profile
class FfnProfile:
    """Owns a cep_ffn_profile: launch threshold theta(rho) and F(N)."""

    def __init__(self, counts, tput):
        n = list(counts)
        if len(n) != len(tput):
            raise ValueError("counts and throughputs differ in length")
        a = (ctypes.c_int64 * max(len(n), 1))(*n)
        b = (ctypes.c_double * max(len(n), 1))(*[float(x) for x in tput])
        h = ctypes.c_void_p()
        _check(None, lib().cep_profile_create(a, b, len(n), ctypes.byref(h)))
        self.handle = h.value

    @property
    def peak(self) -> float:
        return lib().cep_profile_peak(self.handle)

    def theta(self, rho: float) -> int:
        out = ctypes.c_int64()
        _check(None, lib().cep_profile_theta(self.handle, rho, ctypes.byref(out)))
        return out.value

    def eta(self, n: int) -> float:
        out = ctypes.c_double()
        _check(None, lib().cep_profile_eta(self.handle, n, ctypes.byref(out)))
        return out.value

    def latency(self, n: int) -> float:
        out = ctypes.c_double()
        _check(None, lib().cep_profile_latency(self.handle, n, ctypes.byref(out)))
        return out.value

    def close(self):
        if getattr(self, "handle", None):
            lib().cep_profile_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ------------------------------------------------------ OEWF coordinator
class Coordinator:
    """Owns a cep_oewf: the joint plan of one MoE layer over n_ranks ranks."""

    def __init__(self, n_ranks: int, profile: FfnProfile):
        h = ctypes.c_void_p()
        _check(None, lib().cep_oewf_create(n_ranks, profile.handle, ctypes.byref(h)))
        self.handle = h.value
        self.n_ranks = n_ranks

    def begin_layer(self):
        _check(None, lib().cep_oewf_begin_layer(self.handle))

    def set_rank(self, r, in_attention, A, D, N, T):
        _check(None, lib().cep_oewf_set_rank(self.handle, r, 1 if in_attention else 0, float(A),
                                             float(D), int(N), float(T)))

    def completion(self, r) -> float:
        out = ctypes.c_double()
        _check(None, lib().cep_oewf_completion(self.handle, r, ctypes.byref(out)))
        return out.value

    def makespan(self) -> float:
        out = ctypes.c_double()
        _check(None, lib().cep_oewf_makespan(self.handle, ctypes.byref(out)))
        return out.value

    def select(self, helper, tokens, expert_bytes, budget) -> cep_oewf_fetch:
        """tokens: [n_ranks][n_experts] ints; expert_bytes: [n_experts]."""
        n_e = len(expert_bytes)
        flat = [int(v) for row in tokens for v in row]
        if len(flat) != self.n_ranks * n_e:
            raise ValueError("tokens must be n_ranks x n_experts")
        a = (ctypes.c_int64 * len(flat))(*flat)
        b = (ctypes.c_int64 * n_e)(*[int(v) for v in expert_bytes])
        plan = cep_oewf_fetch()
        _check(None, lib().cep_oewf_select(self.handle, helper, n_e, a, b, int(budget),
                                           ctypes.byref(plan)))
        return plan

    def evaluate(self, plan, n_trans, s_h) -> cep_oewf_decision:
        dec = cep_oewf_decision()
        _check(None, lib().cep_oewf_evaluate(self.handle, ctypes.byref(plan), int(n_trans),
                                             float(s_h), ctypes.byref(dec)))
        return dec

    def commit(self, dec, donor_submitted=False) -> bool:
        out = ctypes.c_int()
        _check(None, lib().cep_oewf_commit(self.handle, ctypes.byref(dec),
                                           1 if donor_submitted else 0, ctypes.byref(out)))
        return bool(out.value)

    def close(self):
        if getattr(self, "handle", None):
            lib().cep_oewf_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
