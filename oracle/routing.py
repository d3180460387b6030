"""Routing metadata of one grouped FFN invocation (one batch).
Test infrastructure only (see package docstring).

Follows Appendix C, "Grouped FFN invocations": the layout transform gathers
the selected rows of the ready source lanes into contiguous groups by expert,
derives per-expert row offsets from the per-expert counts, aligns every group
to the GEMM tile size, and keeps an inverse map from each grouped row back to
its source replica, token index and routing slot.

Readings where the paper is silent:

* canonical pair order inside a batch is (chunk position in the batch, row in
  the chunk, routing slot); a pair is valid when its local expert id >= 0;
* rows of one expert keep canonical order (a stable counting sort);
* a pair is identified by its flat index  row_in_batch * k + slot, where
  row_in_batch counts rows over the batch's chunks in order;
* the tile alignment A is a parameter of the implementation; padded offsets
  are  off_pad[e] = sum over e' < e of ceil(cnt[e'] / A) * A.
"""
from __future__ import annotations

import numpy as np


def batch_routing(chunk_ids, n_experts: int, align: int):
    """Counting-sort routing of one batch.

    chunk_ids: list of int arrays [n_i][k] with local expert ids (or -1), in
    the batch's chunk order.
    Returns dict with
      cnt      int32 [E]      pairs per expert
      off      int32 [E+1]    exclusive prefix sum of cnt (unpadded)
      off_pad  int32 [E+1]    exclusive prefix sum of tile-aligned counts
      perm_src int32 [P]      flat pair index at each unpadded grouped row
      pos_of   int32 [R*k]    padded grouped row of each flat pair, -1 if invalid
    """
    ids = (np.concatenate([np.asarray(c, np.int64).reshape(len(c), -1) for c in chunk_ids])
           if len(chunk_ids) else np.zeros((0, 1), np.int64))
    flat = ids.reshape(-1)
    cnt = np.zeros(n_experts, np.int64)
    for e in flat:                       # histogram
        if e >= 0:
            cnt[e] += 1
    off = np.zeros(n_experts + 1, np.int64)
    off_pad = np.zeros(n_experts + 1, np.int64)
    for e in range(n_experts):           # exclusive scans
        off[e + 1] = off[e] + cnt[e]
        off_pad[e + 1] = off_pad[e] + (cnt[e] + align - 1) // align * align
    fill = np.zeros(n_experts, np.int64)
    perm_src = np.zeros(int(off[-1]), np.int64)
    pos_of = np.full(flat.shape[0], -1, np.int64)
    for p, e in enumerate(flat):         # stable scatter in canonical order
        if e < 0:
            continue
        q = fill[e]
        perm_src[off[e] + q] = p
        pos_of[p] = off_pad[e] + q
        fill[e] += 1
    return dict(cnt=cnt.astype(np.int32), off=off.astype(np.int32),
                off_pad=off_pad.astype(np.int32), perm_src=perm_src.astype(np.int32),
                pos_of=pos_of.astype(np.int32))


def brute_force_routing(chunk_ids, n_experts: int, align: int):
    """Same metadata from Python's stable ``sorted`` on (expert, pair) keys."""
    ids = [int(e) for c in chunk_ids for e in np.asarray(c).reshape(-1)]
    pairs = [(e, p) for p, e in enumerate(ids) if e >= 0]
    order = sorted(pairs, key=lambda t: t[0])          # stable in p
    cnt = [sum(1 for e, _ in pairs if e == x) for x in range(n_experts)]
    off = [sum(cnt[:e]) for e in range(n_experts + 1)]
    pad = [-(-c // align) * align for c in cnt]
    off_pad = [sum(pad[:e]) for e in range(n_experts + 1)]
    perm_src = [p for _, p in order]
    pos_of = [-1] * len(ids)
    for i, (e, p) in enumerate(order):
        pos_of[p] = off_pad[e] + (i - off[e])
    return dict(cnt=np.array(cnt, np.int32), off=np.array(off, np.int32),
                off_pad=np.array(off_pad, np.int32), perm_src=np.array(perm_src, np.int32),
                pos_of=np.array(pos_of, np.int32))
