"""Opportunistic expert weight fetching (OEWF) coordinator (oracle).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

Section 3.3, "Coordinated greedy expert-weight selection" and "Cost-based
FFN reassignment"; Algorithm 1 (SelectWeights); Appendix C, "One-shot weight
fetching" and "FFN reassignment commit and fallback"; Appendix E
(non-degradation of OEWF).

A joint plan S of one MoE layer holds, per rank r:
  * in_attention -- r is still computing attention (a candidate donor);
  * A_r, D_r     -- remaining attention time and dispatch latency
                    (Eq. attention-remaining; the dispatch latency is the
                    dispatched-token count over the profiled dispatch
                    throughput, computed by the caller);
  * N_r          -- expert tokens r will receive (its FFN work);
  * T_r          -- completion time of a helper's own FFN work under S
                    (given by its stream schedule);
all on one clock measured from the decision instant.  A donor's predicted
completion is T_d(S) = A_d + D_d + F(N_d) (Eq. donor-completion) with F the
FFN latency model (Eq. ffn-throughput-latency, ``oracle.calibration``).

Readings (the paper leaves them open):
  * CandidateDonors(S, h) = every rank other than h still in attention;
  * ties in argmax_d T_d(S) go to the lowest rank; experts with equal
    |T_hde| / b_e keep ascending expert order;
  * the helper's completion after a reassignment is
    max{T_h(S), s_h + F(N_trans)} (Appendix E), i.e. alpha_h is derived from
    the planned launch time s_h of the reassigned kernel;
  * a commit applies only if the plan entries of the donor and the helper
    still carry the versions the decision read, the tokens are unclaimed and
    the donor has not submitted them; otherwise execution stays with the
    donor (fallback).
"""
from __future__ import annotations

from dataclasses import dataclass, field

from oracle import calibration as C


@dataclass
class Rank:
    in_attention: bool = False
    A: float = 0.0
    D: float = 0.0
    N: int = 0
    T: float = 0.0          # helper's own FFN completion (used when not a donor)
    version: int = 0
    fetched: bool = False   # one fetch decision per rank per layer


@dataclass
class FetchPlan:
    helper: int
    donor: int
    experts: list           # selected expert ids of the donor, in selection order
    tokens: list            # |T_h,d*,e| for each selected expert
    bytes: int
    committed: bool = False  # its tokens were reassigned to the helper


@dataclass
class Decision:
    """Outcome of the admission test, with the plan versions it read."""
    plan: FetchPlan
    n_trans: int
    admit: bool
    Td: float
    Th: float
    Td2: float
    Th2: float
    alpha: float
    donor_version: int
    helper_version: int


@dataclass
class Plan:
    """Joint plan S of one layer; F given as a throughput profile."""
    n_ranks: int
    prof_n: list
    prof_tput: list
    ranks: list = field(default_factory=list)

    def __post_init__(self):
        self.ranks = [Rank() for _ in range(self.n_ranks)]

    def F(self, N: int) -> float:
        return C.latency(self.prof_n, self.prof_tput, N)

    def set_rank(self, r, in_attention, A, D, N, T):
        k = self.ranks[r]
        k.in_attention, k.A, k.D, k.N, k.T = bool(in_attention), A, D, int(N), T
        k.version += 1

    def donor_completion(self, d) -> float:
        """T_d(S) = A_d + D_d + F(N_d)."""
        k = self.ranks[d]
        return k.A + k.D + self.F(k.N)

    def completion(self, r) -> float:
        """Predicted completion of rank r under S: the donor model while r is
        in attention, its own schedule's T otherwise."""
        k = self.ranks[r]
        return self.donor_completion(r) if k.in_attention else k.T

    def makespan(self) -> float:
        return max(self.completion(r) for r in range(self.n_ranks))

    # ------------------------------------------------------- Algorithm 1
    def select_weights(self, h, tokens, expert_bytes, budget):
        """SelectWeights(h).  tokens[d][e] = |T_h,d,e| (tokens helper h
        dispatched to expert e of rank d); expert_bytes[e] = b_e; budget =
        B_h.  Returns a FetchPlan or None (no candidate, or nothing fits).
        A helper decides once per layer (a second call raises)."""
        k = self.ranks[h]
        if k.fetched:
            raise RuntimeError("one fetch decision per rank per layer")
        k.fetched = True
        donors = [d for d in range(self.n_ranks) if d != h and self.ranks[d].in_attention]
        if not donors:
            return None
        # d* = argmax T_d(S); the first maximum (lowest rank) on ties
        best = donors[0]
        for d in donors[1:]:
            if self.donor_completion(d) > self.donor_completion(best):
                best = d
        eligible = [e for e in range(len(expert_bytes)) if tokens[best][e] > 0]
        # descending |T_hde| / b_e; Python's sort is stable, so equal ratios
        # keep ascending expert order
        order = sorted(eligible, key=lambda e: -(tokens[best][e] / expert_bytes[e]))
        chosen, left = [], budget
        for e in order:
            if expert_bytes[e] <= left:
                chosen.append(e)
                left -= expert_bytes[e]
            else:
                break
        if not chosen:
            return None
        return FetchPlan(helper=h, donor=best, experts=chosen,
                         tokens=[int(tokens[best][e]) for e in chosen],
                         bytes=sum(int(expert_bytes[e]) for e in chosen))

    # -------------------------------------------------- reassignment test
    def evaluate(self, p: FetchPlan, n_trans: int, s_h: float) -> Decision:
        """Eqs. swf-completion-times and swf-admission on the latest plan for
        moving n_trans of the fetch plan's unstarted tokens to the helper,
        launched s_h after the decision, s_h in [0, T_h(S)] (Appendix E)."""
        d, h = self.ranks[p.donor], self.ranks[p.helper]
        if not (0 <= n_trans <= min(sum(p.tokens), d.N)):
            raise ValueError("n_trans outside [0, min(plan tokens, N_d)]")
        if not (0.0 <= s_h <= h.T):
            raise ValueError("s_h must lie in [0, T_h(S)]")
        Td = d.A + d.D + self.F(d.N)
        Th = h.T
        if n_trans == 0:  # nothing moves: the plan is unchanged
            return Decision(p, 0, False, Td, Th, Td, Th, 0.0, d.version, h.version)
        ft = self.F(n_trans)
        Td2 = d.A + d.D + self.F(d.N - n_trans)
        Th2 = max(Th, s_h + ft)
        alpha = max(0.0, s_h + ft - Th) / ft
        admit = max(Td2, Th2) <= max(Td, Th)
        return Decision(p, n_trans, admit, Td, Th, Td2, Th2, alpha, d.version, h.version)

    def commit(self, dec: Decision, donor_submitted: bool = False) -> bool:
        """Version-checked commit of an admitted decision: applies only if the
        donor's and the helper's entries are unchanged since the evaluation,
        the plan's tokens are unclaimed and the donor has not submitted them.
        On success the donor's residual count and the helper's completion
        change together; otherwise execution stays with the donor."""
        p = dec.plan
        d, h = self.ranks[p.donor], self.ranks[p.helper]
        ok = (dec.admit and not p.committed and not donor_submitted
              and d.version == dec.donor_version and h.version == dec.helper_version)
        if ok:
            d.N -= dec.n_trans
            h.T = dec.Th2
            d.version += 1
            h.version += 1
            p.committed = True
        return ok
