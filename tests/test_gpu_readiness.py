"""Chunk readiness on each chunk's own signal (Section 3.2; Appendix C,
"Asynchronous dispatch": a lane's inputs become eligible when its own
completion signal fires, without waiting for other replicas).

The chunk buffers start out poisoned (NaN rows and coefficients, expert ids
and token slots out of range).  A dispatch stream writes each chunk's real
data after a bounded device-side delay and records that chunk's arrival
event; the host submits every chunk at once, before any of them has
arrived, each with its own event.  The library must read every chunk only
after its event: the output then equals the run on resident inputs, bit for
bit, under every policy and stream count.
"""
import ctypes
import json
import os
import subprocess
import sys

import numpy as np
import pytest
import torch

from paper_2609_33252_amd import cep, harness, workload as W

from . import _util as U

pytestmark = pytest.mark.gpu

# spin of the delay kernel before each delivery (clock64 ticks: well under a
# millisecond to tens of milliseconds, whatever the counter's rate)
DELAY = 1_000_000


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


class Late:
    """Real chunk data kept aside; poison and late delivery of the buffers
    the library reads."""

    def __init__(self, run):
        self.run = run
        self.src = [(ch.token_idx.clone(), ch.ids.clone(), ch.w.clone()) for ch in run.chunks]
        self.x_src = run.recv.clone()
        self.dispatch = torch.cuda.Stream()

    def poison(self):
        E = self.run.wl.cfg["E"]
        self.run.recv.fill_(float("nan"))
        for ch in self.run.chunks:
            ch.token_idx.fill_(-5)
            ch.ids.fill_(E + 5)
            ch.w.fill_(float("nan"))
        torch.cuda.synchronize()

    def deliver(self, order, delay=DELAY):
        """On the dispatch stream, in `order`: a delay, then the chunk's real
        rows, ids, coefficients and token slots, then its arrival event.
        Returns the events indexed by chunk."""
        run = self.run
        events = [None] * len(run.chunks)
        r0s = np.cumsum([0] + [ch.n_rows for ch in run.chunks])
        with torch.cuda.stream(self.dispatch):
            for i in order:
                ch = run.chunks[i]
                if delay:
                    torch.cuda._sleep(delay)
                t, ids, w = self.src[i]
                run.recv[r0s[i]:r0s[i + 1]].copy_(self.x_src[r0s[i]:r0s[i + 1]])
                ch.token_idx.copy_(t)
                ch.ids.copy_(ids)
                ch.w.copy_(w)
                ev = torch.cuda.Event(enable_timing=True)
                ev.record(self.dispatch)
                events[i] = ev
        return events


def _layer(run, events, policy, theta, streams):
    """One layer whose chunks are all submitted at once, chunk i behind
    events[i] (None: no event)."""
    ctx = run.ctx
    cep.cep_set_policy(ctx, policy, theta, streams)
    run.gen += 1
    cep.cep_begin_layer(ctx, run.gen, run.chunks_per_replica, run.out)
    for i, ch in enumerate(run.chunks):
        cep.cep_submit_chunk(ctx, run.gen, ch.replica, ch.n_rows, ch.n_pairs, ch.token_idx,
                             ch.x, ch.ids, ch.w, events[i])
    cep.cep_combine(ctx)


def _workload():
    return W.generate("zipf_stream_d7168", 5, d=1024, I=512, R=8, T=512, cpr=4)


def test_each_chunk_waits_for_its_own_arrival():
    wl = _workload()
    run = harness.Runner(wl, n_streams=4)
    run.run(policy=cep.CEP_WAIT_ALL)
    ref = _out(run)
    U.check(wl, ref)
    late = Late(run)
    n = len(run.chunks)
    # deliveries in reverse submission order: the first chunk submitted is
    # the last to arrive
    order = list(range(n))[::-1]
    for pol, theta, ns in ((cep.CEP_WAIT_ALL, 1, 1), (cep.CEP_PER_CHUNK, 1, 1),
                           (cep.CEP_PER_CHUNK, 1, 4), (cep.CEP_THRESHOLD, 300, 2),
                           (cep.CEP_THRESHOLD, 900, 3), (cep.CEP_THRESHOLD, 300, 4)):
        late.poison()
        run.out.zero_()
        events = late.deliver(order)
        _layer(run, events, pol, theta, ns)
        got = _out(run)
        assert np.array_equal(got, ref), (pol, theta, ns)
        st = run.stats()
        # every batch ended after the arrival of each of its chunks
        arr = [c["arrival_ms"] for c in st["chunks"]]
        for b in st["batches"]:
            last = max(arr[b["first_chunk"]:b["first_chunk"] + b["n_chunks"]])
            assert b["end_ms"] >= last, (pol, theta, ns, b)
    run.close()


def test_missing_waits_would_read_poison():
    # the same late delivery submitted without events reads the poison: the
    # check above is sensitive to a wait the library left out
    wl = _workload()
    run = harness.Runner(wl, n_streams=2)
    run.run(policy=cep.CEP_WAIT_ALL)
    ref = _out(run)
    late = Late(run)
    late.poison()
    run.out.zero_()
    late.deliver(range(len(run.chunks)))
    _layer(run, [None] * len(run.chunks), cep.CEP_PER_CHUNK, 1, 2)
    torch.cuda.synchronize()
    failed = False
    try:
        cep.cep_get_status(run.ctx)
    except cep.CepError:
        failed = True
    got = run.out.cpu().numpy()
    run.close()
    assert failed or not np.array_equal(got, ref)


def _own_stream():
    """A stream on a hardware queue of its own.  HIP runs a process's
    streams on a bounded set of hardware queues, and streams that share one
    run its packets in order: a long kernel on a torch pool stream may hold
    back a library stream on the same queue.  A stream with a CU mask (here
    every CU) gets a queue that no other stream shares."""
    hip = ctypes.CDLL("libamdhip64.so.7")  # the runtime torch already loaded
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    words = (n_cu + 31) // 32
    mask = (ctypes.c_uint32 * words)(*([0xFFFFFFFF] * words))
    h = ctypes.c_void_p()
    assert hip.hipExtStreamCreateWithCUMask(ctypes.byref(h), words, mask) == 0
    return hip, h, torch.cuda.ExternalStream(h.value)


def _late_chunk_scenario():
    """Chunk 0 arrives long after all others; per-chunk batches on two
    stream slots.  Returns (output equals the resident run, chunk 0's
    arrival ms, [(slot, first chunk, start ms, end ms)] per batch)."""
    wl = _workload()
    run = harness.Runner(wl, n_streams=2)
    run.run(policy=cep.CEP_WAIT_ALL)
    ref = _out(run)
    late = Late(run)
    late.poison()
    run.out.zero_()
    n = len(run.chunks)
    hip, h, slow = _own_stream()
    events = late.deliver(range(1, n), delay=0)
    with torch.cuda.stream(slow):
        torch.cuda._sleep(20 * DELAY)
    late.dispatch, keep = slow, late.dispatch
    events[0] = late.deliver([0], delay=0)[0]
    late.dispatch = keep
    _layer(run, events, cep.CEP_PER_CHUNK, 1, 2)
    got = _out(run)
    st = run.stats()
    timeline = [(b["slot"], b["first_chunk"], b["start_ms"], b["end_ms"]) for b in st["batches"]]
    result = (bool(np.array_equal(got, ref)), st["chunks"][0]["arrival_ms"], timeline)
    run.close()
    torch.cuda.synchronize()
    assert hip.hipStreamDestroy(h) == 0
    return result


def _late_chunk_child():
    torch.cuda.set_device(0)
    cep.lib()
    print(json.dumps(_late_chunk_scenario()), flush=True)


def test_late_chunk_blocks_only_its_own_batch():
    # batch 0 (chunk 0) waits on stream slot 0; the batches on slot 1 run as
    # soon as their own chunks are in, so they end before chunk 0 arrives (no
    # head-of-line blocking behind another replica's lane).  HIP runs a
    # process's streams on a bounded set of hardware queues, and which
    # streams share a queue depends on every stream the process has created
    # (torch's stream pool, earlier contexts); streams on one queue run its
    # packets in order.  The scenario therefore runs in a fresh child process,
    # whose few streams get distinct queues.
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c",
                        "from tests.test_gpu_readiness import _late_chunk_child; "
                        "_late_chunk_child()"],
                       cwd=root, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-3000:]
    equal, a0, timeline = json.loads(r.stdout.strip().splitlines()[-1])
    assert equal
    assert a0 > 0
    assert timeline[0][0] == 0 and timeline[0][1] == 0
    early = [b for b in timeline if b[0] == 1]
    assert early, "per-chunk batches on the second stream slot"
    for b in early:
        assert b[3] < a0, (a0, timeline)

