// Opportunistic expert weight fetching: the coordinator's joint plan of one
// MoE layer (Section 3.3; Algorithm 1; Appendix C, "One-shot weight
// fetching" and "FFN reassignment commit and fallback"; Appendix E).  Host
// code only: it decides which donor experts a helper fetches (the copy itself
// is cep_weight_fetch) and whether the helper takes over their tokens.
//
// Per rank the plan holds whether it still computes attention (a candidate
// donor), its remaining attention time A and dispatch latency D, the expert
// tokens N it receives, and, once out of attention, the completion time T of
// its own FFN work.  A donor's predicted completion is
// T_d(S) = A_d + D_d + F(N_d) (Eq. donor-completion).  All times share one
// clock measured from the decision instant.
//
// Readings: candidate donors are the other ranks still in attention; ties in
// the donor argmax go to the lowest rank and equal |T_hde| / b_e keep
// ascending expert order; the helper's completion after a reassignment is
// max{T_h(S), s_h + F(N_trans)} with s_h in [0, T_h(S)] the planned launch
// time of the reassigned invocation (Appendix E), which fixes alpha_h.
#include "cep.h"
#include "common.h"
#include "profile.h"

#include <algorithm>
#include <mutex>
#include <new>
#include <vector>

namespace {

struct RankEntry {
  bool in_attention = false;
  double A = 0, D = 0, T = 0;
  int64_t N = 0;
  uint64_t version = 0;
  bool decided = false;  // one fetch decision per rank per layer
};

struct PlanRec {
  int helper, donor;
  int64_t tokens;
  bool committed;
};

}  // namespace

struct cep_oewf {
  cep_ffn_profile F;
  std::vector<RankEntry> ranks;
  std::vector<PlanRec> plans;
  std::mutex mu;  // select / evaluate / commit are atomic with respect to each other

  double donor_completion(int d) const {
    const RankEntry &k = ranks[d];
    return k.A + k.D + cep::profile_latency(F, k.N);
  }
  double completion(int r) const {
    return ranks[r].in_attention ? donor_completion(r) : ranks[r].T;
  }
};

namespace {
int bad(const char *m) { return cep::set_global_error(CEP_EINVAL, m); }
}  // namespace

CEP_API int cep_oewf_create(int n_ranks, const cep_ffn_profile *F, cep_oewf **out) {
  if (!out) return bad("cep_oewf_create: out is NULL");
  *out = nullptr;
  if (n_ranks < 1 || n_ranks > 4096 || !F) return bad("cep_oewf_create: bad rank count or profile");
  cep_oewf *o = new (std::nothrow) cep_oewf();
  if (!o) return cep::set_global_error(CEP_ENOMEM, "cep_oewf_create: out of host memory");
  o->F = *F;
  o->ranks.resize(n_ranks);
  *out = o;
  return CEP_OK;
}

CEP_API int cep_oewf_begin_layer(cep_oewf *o) {
  if (!o) return bad("cep_oewf_begin_layer: NULL coordinator");
  std::lock_guard<std::mutex> g(o->mu);
  for (RankEntry &k : o->ranks) {
    k.decided = false;
    ++k.version;
  }
  o->plans.clear();
  return CEP_OK;
}

CEP_API int cep_oewf_set_rank(cep_oewf *o, int r, int in_attention, double A, double D,
                              int64_t N, double T) {
  if (!o) return bad("cep_oewf_set_rank: NULL coordinator");
  if (r < 0 || r >= (int)o->ranks.size()) return bad("cep_oewf_set_rank: rank out of range");
  if (!(A >= 0) || !(D >= 0) || !(T >= 0) || N < 0)
    return bad("cep_oewf_set_rank: times and counts must be >= 0");
  std::lock_guard<std::mutex> g(o->mu);
  RankEntry &k = o->ranks[r];
  k.in_attention = in_attention != 0;
  k.A = A;
  k.D = D;
  k.N = N;
  k.T = T;
  ++k.version;
  return CEP_OK;
}

CEP_API int cep_oewf_completion(cep_oewf *o, int r, double *t) {
  if (!o || !t) return bad("cep_oewf_completion: NULL argument");
  if (r < 0 || r >= (int)o->ranks.size()) return bad("cep_oewf_completion: rank out of range");
  std::lock_guard<std::mutex> g(o->mu);
  *t = o->completion(r);
  return CEP_OK;
}

CEP_API int cep_oewf_makespan(cep_oewf *o, double *t) {
  if (!o || !t) return bad("cep_oewf_makespan: NULL argument");
  std::lock_guard<std::mutex> g(o->mu);
  double m = 0;
  for (int r = 0; r < (int)o->ranks.size(); ++r) m = std::max(m, o->completion(r));
  *t = m;
  return CEP_OK;
}

CEP_API int cep_oewf_select(cep_oewf *o, int helper, int n_experts, const int64_t *tokens,
                            const int64_t *expert_bytes, int64_t budget, cep_oewf_fetch *plan) {
  if (!o || !plan) return bad("cep_oewf_select: NULL argument");
  const int R = (int)o->ranks.size();
  if (helper < 0 || helper >= R) return bad("cep_oewf_select: helper out of range");
  if (n_experts < 1 || n_experts > CEP_OEWF_MAX_EXPERTS || !tokens || !expert_bytes || budget < 0)
    return bad("cep_oewf_select: bad expert arrays or budget");
  for (int e = 0; e < n_experts; ++e)
    if (expert_bytes[e] <= 0) return bad("cep_oewf_select: expert bytes must be > 0");
  for (long long i = 0; i < (long long)R * n_experts; ++i)
    if (tokens[i] < 0) return bad("cep_oewf_select: negative token count");
  std::lock_guard<std::mutex> g(o->mu);
  RankEntry &hk = o->ranks[helper];
  if (hk.decided)
    return cep::set_global_error(CEP_EBUSY, "cep_oewf_select: one decision per rank per layer");
  hk.decided = true;
  *plan = cep_oewf_fetch{};
  plan->helper = helper;
  plan->donor = -1;
  plan->plan_id = -1;
  // d* = argmax_{d in D} T_d(S), D = other ranks still in attention
  int best = -1;
  double best_t = 0;
  for (int d = 0; d < R; ++d) {
    if (d == helper || !o->ranks[d].in_attention) continue;
    const double t = o->donor_completion(d);
    if (best < 0 || t > best_t) {
      best = d;
      best_t = t;
    }
  }
  if (best < 0) return CEP_OK;  // no candidate donor: empty selection
  const int64_t *tk = tokens + (size_t)best * n_experts;
  // experts of d* with tokens from h, by descending |T_hde| / b_e (stable)
  std::vector<int> order;
  for (int e = 0; e < n_experts; ++e)
    if (tk[e] > 0) order.push_back(e);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
    return (double)tk[a] / (double)expert_bytes[a] > (double)tk[b] / (double)expert_bytes[b];
  });
  int64_t left = budget, ntok = 0;
  plan->donor = best;
  for (int e : order) {
    if (expert_bytes[e] > left) break;
    plan->experts[plan->n_experts] = e;
    plan->tokens[plan->n_experts] = tk[e];
    ++plan->n_experts;
    left -= expert_bytes[e];
    plan->bytes += expert_bytes[e];
    ntok += tk[e];
  }
  if (plan->n_experts == 0) return CEP_OK;  // nothing fits the budget
  plan->plan_id = (int64_t)o->plans.size();
  o->plans.push_back(PlanRec{helper, best, ntok, false});
  return CEP_OK;
}

namespace {

// admission test on the current plan; caller holds the lock
int evaluate_locked(cep_oewf *o, const cep_oewf_fetch *plan, int64_t n_trans, double s_h,
                    cep_oewf_decision *dec) {
  if (plan->plan_id < 0 || plan->plan_id >= (int64_t)o->plans.size())
    return bad("cep_oewf_evaluate: unknown fetch plan");
  const PlanRec &pr = o->plans[plan->plan_id];
  if (pr.helper != plan->helper || pr.donor != plan->donor)
    return bad("cep_oewf_evaluate: fetch plan does not match the coordinator's record");
  const RankEntry &d = o->ranks[pr.donor];
  const RankEntry &h = o->ranks[pr.helper];
  if (n_trans < 0 || n_trans > std::min(pr.tokens, d.N))
    return bad("cep_oewf_evaluate: n_trans outside [0, min(plan tokens, N_d)]");
  if (!(s_h >= 0.0 && s_h <= h.T)) return bad("cep_oewf_evaluate: s_h outside [0, T_h(S)]");
  cep_oewf_decision r{};
  r.plan_id = plan->plan_id;
  r.n_trans = n_trans;
  r.donor_version = d.version;
  r.helper_version = h.version;
  r.Td = d.A + d.D + cep::profile_latency(o->F, d.N);
  r.Th = h.T;
  if (n_trans == 0) {  // nothing moves: the plan is unchanged
    r.admit = 0;
    r.Td2 = r.Td;
    r.Th2 = r.Th;
    r.alpha = 0;
  } else {
    const double ft = cep::profile_latency(o->F, n_trans);
    r.Td2 = d.A + d.D + cep::profile_latency(o->F, d.N - n_trans);
    r.Th2 = std::max(r.Th, s_h + ft);
    r.alpha = std::max(0.0, s_h + ft - r.Th) / ft;
    r.admit = std::max(r.Td2, r.Th2) <= std::max(r.Td, r.Th) ? 1 : 0;
  }
  *dec = r;
  return CEP_OK;
}

int commit_locked(cep_oewf *o, const cep_oewf_decision *dec, int donor_submitted, int *committed) {
  *committed = 0;
  // a decision of an earlier layer names a plan that no longer exists (or,
  // by index, a newer one whose entries carry later versions): fallback
  if (dec->plan_id < 0 || dec->plan_id >= (int64_t)o->plans.size()) return CEP_OK;
  PlanRec &pr = o->plans[dec->plan_id];
  RankEntry &d = o->ranks[pr.donor];
  RankEntry &h = o->ranks[pr.helper];
  if (!dec->admit || pr.committed || donor_submitted || d.version != dec->donor_version ||
      h.version != dec->helper_version || dec->n_trans > d.N)
    return CEP_OK;  // fallback: execution stays with the donor
  d.N -= dec->n_trans;
  h.T = dec->Th2;
  ++d.version;
  ++h.version;
  pr.committed = true;
  *committed = 1;
  return CEP_OK;
}

}  // namespace

CEP_API int cep_oewf_evaluate(cep_oewf *o, const cep_oewf_fetch *plan, int64_t n_trans,
                              double s_h, cep_oewf_decision *dec) {
  if (!o || !plan || !dec) return bad("cep_oewf_evaluate: NULL argument");
  std::lock_guard<std::mutex> g(o->mu);
  return evaluate_locked(o, plan, n_trans, s_h, dec);
}

CEP_API int cep_oewf_commit(cep_oewf *o, const cep_oewf_decision *dec, int donor_submitted,
                            int *committed) {
  if (!o || !dec || !committed) return bad("cep_oewf_commit: NULL argument");
  std::lock_guard<std::mutex> g(o->mu);
  return commit_locked(o, dec, donor_submitted, committed);
}

CEP_API void cep_oewf_destroy(cep_oewf *o) { delete o; }
