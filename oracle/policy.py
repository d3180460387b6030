"""streamFFN batch composition.  Test infrastructure only (see package docstring).

Section 3.2, "Launch threshold": ready expert tokens accumulate until their
count reaches the launch threshold theta; once all tokens have arrived the
threshold is bypassed and the remainder runs.  Section 4.3 ("Ablation study")
defines the two baselines: Sync starts the FFN only after every replica has
dispatched (here: theta = infinity), Async runs each source's ready inputs as
its own FFN invocation without a threshold (here: one batch per non-empty
chunk).  Appendix C ("Asynchronous dispatch") adds that readiness alone does
not launch anything: the threshold and final-flush rule decide.

Readings where the paper is silent:

* theta counts valid local (token, slot) pairs pending on this GPU, summed
  over all local experts; "reaches" means pending >= theta;
* a launch takes all pending chunks, whole, in FIFO order;
* "all tokens have arrived" means the last expected chunk of the layer has
  been submitted (or the caller flushes explicitly);
* a chunk with no valid pair carries no rows: it counts toward "all arrived"
  and never joins a batch;
* an optional per-batch pair capacity: a chunk that would push the pending
  count above it first launches what is pending.
"""
from __future__ import annotations

WAIT_ALL, PER_CHUNK, THRESHOLD = 0, 1, 2
INF = float("inf")


def batches(events, policy: int, theta: float = INF, cap: float = INF, n_expected=None):
    """Batch list for a submission sequence.

    events: sequence of ints (pairs in each submitted chunk, in submission
    order) or the string "flush" for an explicit flush.  Chunks are numbered
    0, 1, ... in submission order (flushes are not numbered).
    n_expected: chunks expected in the layer; after the n_expected-th chunk
    the final flush applies (default: the number of chunks in ``events``).
    Returns a list of batches, each a list of chunk numbers.
    """
    chunk_pairs = [e for e in events if e != "flush"]
    if n_expected is None:
        n_expected = len(chunk_pairs)
    if policy == WAIT_ALL:
        theta = INF
    elif policy == PER_CHUNK:
        theta = 1
    out, pending, pend_pairs, seen = [], [], 0, 0
    for ev in events:
        if ev == "flush":
            if pending:
                out.append(pending)
                pending, pend_pairs = [], 0
            continue
        n = int(ev)
        cid = seen
        seen += 1
        if n > cap:
            raise ValueError("chunk larger than the batch capacity")
        if n > 0:
            if pending and pend_pairs + n > cap:
                out.append(pending)
                pending, pend_pairs = [], 0
            pending.append(cid)
            pend_pairs += n
            if pend_pairs >= theta:
                out.append(pending)
                pending, pend_pairs = [], 0
        if seen == n_expected and pending:          # final flush
            out.append(pending)
            pending, pend_pairs = [], 0
    return out
