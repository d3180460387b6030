"""Discrete-event model of one MoE layer under OEWF (host side).

Ranks finish attention at their own times, dispatch, and run their FFN with
latency F(N).  Each rank, once its dispatch completes, is a helper: it asks
the coordinator for one fetch (Algorithm 1), the copy takes bytes / bw, and
when the weights are ready the coordinator decides whether the helper takes
over the fetched experts' tokens (admission test, versioned commit;
Section 3.3, Appendix C).  Execution follows the same completion-time model
the coordinator predicts with (the accurate-model assumption of Appendix E),
so every accepted update must not increase the layer's FFN completion time
and the final layer time must not exceed the no-fetch time.

The coordinator is anything with begin_layer / set_rank / select / evaluate /
commit, such as ``cep.Coordinator``.
"""
from __future__ import annotations

import numpy as np

def plan_tokens(plan):
    """Selected token total of a plan from either implementation (0 if none)."""
    if plan is None:
        return 0
    if hasattr(plan, "n_experts"):
        return int(sum(plan.tokens[i] for i in range(plan.n_experts)))
    return int(sum(plan.tokens))


def plan_bytes(plan):
    return 0 if plan is None else int(plan.bytes)


def random_layer(rng, R, E, dispatch_tput=4000.0):
    """Attention end times (skewed, as in imbalanced prefill), tokens each
    rank dispatches to every expert of every rank, and expert bytes."""
    attn = rng.lognormal(mean=1.0, sigma=0.6, size=R) * 2.0
    tok = rng.integers(0, 300, size=(R, R, E)) * (rng.random((R, R, E)) < 0.6)
    sent = tok.sum(axis=(1, 2))
    disp = sent / dispatch_tput
    b = rng.integers(20, 120, size=E).astype(np.int64)
    return attn, disp, tok, b


def simulate(coord, F, attn, disp, tok, expert_bytes, budget, bw, rng, s_mode="random"):
    """Runs one layer; returns (no-fetch makespan, final makespan, commits,
    list of makespans after each accepted commit)."""
    R = len(attn)
    N = tok.sum(axis=(0, 2)).astype(np.int64)   # tokens each rank receives
    start = attn + disp                          # dispatch complete = FFN may start
    done = start + np.array([F(int(n)) for n in N])
    base = float(done.max())
    coord.begin_layer()
    commits, trail = 0, []

    def refresh(t):
        # the plan relative to time t: donors still in attention carry the
        # model, everyone else its predicted completion
        for r in range(R):
            if attn[r] > t:
                coord.set_rank(r, True, attn[r] - t, disp[r], int(N[r]), 0.0)
            else:
                coord.set_rank(r, False, 0.0, 0.0, int(N[r]), max(0.0, done[r] - t))

    for h in np.argsort(start, kind="stable"):
        t = float(start[h])
        refresh(t)
        plan = coord.select(int(h), tok[h].tolist(), expert_bytes.tolist(), budget)
        ntr = plan_tokens(plan)
        if ntr == 0:
            continue
        d = int(plan.donor)
        t_ready = t + plan_bytes(plan) / bw
        # the donor's tokens are unstarted while it still computes attention
        if attn[d] <= t_ready or ntr > N[d]:
            continue
        refresh(t_ready)
        Th = max(0.0, done[h] - t_ready)
        s_h = {"random": float(rng.uniform(0.0, Th)), "zero": 0.0, "serial": Th}[s_mode]
        dec = coord.evaluate(plan, ntr, s_h)
        if coord.commit(dec):
            commits += 1
            N[d] -= ntr
            done[d] = start[d] + F(int(N[d]))
            done[h] = t_ready + dec.Th2
            trail.append(float(done.max()))
    return base, float(done.max()), commits, trail
