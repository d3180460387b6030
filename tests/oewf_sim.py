"""Test-side pieces of the OEWF layer simulation: the oracle coordinator
behind the library's call shapes, and the shared model from the package."""
from __future__ import annotations

from paper_2609_33252_amd.layer_sim import plan_bytes, plan_tokens, random_layer, simulate  # noqa: F401


class OracleAdapter:
    """Gives oracle.oewf.Plan the library's call shapes."""

    def __init__(self, plan):
        self.p = plan

    def begin_layer(self):
        for k in self.p.ranks:
            k.fetched = False
            k.version += 1

    def set_rank(self, r, in_attention, A, D, N, T):
        self.p.set_rank(r, in_attention, A, D, N, T)

    def makespan(self):
        return self.p.makespan()

    def select(self, h, tokens, expert_bytes, budget):
        return self.p.select_weights(h, tokens, expert_bytes, budget)

    def evaluate(self, plan, n_trans, s_h):
        return self.p.evaluate(plan, n_trans, s_h)

    def commit(self, dec, donor_submitted=False):
        return self.p.commit(dec, donor_submitted)
