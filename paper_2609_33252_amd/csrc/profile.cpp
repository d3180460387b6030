// FFN throughput profile: the streamFFN launch threshold (Section 3.2,
// "Launch threshold") and the FFN latency model F(N) = N / (eta(N) P_peak)
// (Section 3.3, Eq. ffn-throughput-latency).  Host code only.
//
// Between profiled counts eta is linear in N; below the smallest profiled
// count the latency is that count's latency (eta scales with N); above the
// largest, eta keeps its last value.
#include "cep.h"
#include "common.h"
#include "profile.h"

#include <cmath>
#include <new>

namespace cep {

double profile_eta(const cep_ffn_profile &p, int64_t N) {
  const std::vector<int64_t> &n = p.n;
  const size_t last = n.size() - 1;
  if (N <= n[0]) return p.eta[0] * (double)N / (double)n[0];
  if (N >= n[last]) return p.eta[last];
  size_t i = 0;
  while (n[i + 1] < N) ++i;  // n[i] < N <= n[i+1]
  const double f = (double)(N - n[i]) / (double)(n[i + 1] - n[i]);
  return p.eta[i] + f * (p.eta[i + 1] - p.eta[i]);
}

double profile_latency(const cep_ffn_profile &p, int64_t N) {
  return N == 0 ? 0.0 : (double)N / (profile_eta(p, N) * p.peak);
}

}  // namespace cep

CEP_API int cep_profile_create(const int64_t *n, const double *tput, int count,
                               cep_ffn_profile **out) {
  if (!out) return cep::set_global_error(CEP_EINVAL, "cep_profile_create: out is NULL");
  *out = nullptr;
  if (count < 1 || !n || !tput)
    return cep::set_global_error(CEP_EINVAL, "cep_profile_create: empty profile");
  double peak = 0;
  for (int i = 0; i < count; ++i) {
    if (n[i] <= 0 || (i > 0 && n[i] <= n[i - 1]))
      return cep::set_global_error(CEP_EINVAL,
                                   "cep_profile_create: counts must be positive and increasing");
    if (!(tput[i] > 0) || !std::isfinite(tput[i]))
      return cep::set_global_error(CEP_EINVAL,
                                   "cep_profile_create: throughputs must be positive and finite");
    peak = std::max(peak, tput[i]);
  }
  cep_ffn_profile *p = new (std::nothrow) cep_ffn_profile();
  if (!p) return cep::set_global_error(CEP_ENOMEM, "cep_profile_create: out of host memory");
  p->n.assign(n, n + count);
  p->eta.resize(count);
  for (int i = 0; i < count; ++i) p->eta[i] = tput[i] / peak;
  p->peak = peak;
  *out = p;
  return CEP_OK;
}

CEP_API double cep_profile_peak(const cep_ffn_profile *p) { return p ? p->peak : 0.0; }

CEP_API int cep_profile_theta(const cep_ffn_profile *p, double rho, int64_t *theta) {
  if (!p || !theta) return cep::set_global_error(CEP_EINVAL, "cep_profile_theta: NULL argument");
  if (!(rho > 0.0 && rho <= 1.0))
    return cep::set_global_error(CEP_EINVAL, "cep_profile_theta: rho must lie in (0, 1]");
  for (size_t i = 0; i < p->n.size(); ++i)
    if (p->eta[i] >= rho) {
      *theta = p->n[i];
      return CEP_OK;
    }
  return cep::set_global_error(CEP_EINVAL, "cep_profile_theta: no profiled count reaches rho");
}

CEP_API int cep_profile_eta(const cep_ffn_profile *p, int64_t N, double *eta) {
  if (!p || !eta) return cep::set_global_error(CEP_EINVAL, "cep_profile_eta: NULL argument");
  if (N < 1) return cep::set_global_error(CEP_EINVAL, "cep_profile_eta: N must be >= 1");
  *eta = cep::profile_eta(*p, N);
  return CEP_OK;
}

CEP_API int cep_profile_latency(const cep_ffn_profile *p, int64_t N, double *latency) {
  if (!p || !latency)
    return cep::set_global_error(CEP_EINVAL, "cep_profile_latency: NULL argument");
  if (N < 0) return cep::set_global_error(CEP_EINVAL, "cep_profile_latency: N must be >= 0");
  *latency = cep::profile_latency(*p, N);
  return CEP_OK;
}

CEP_API void cep_profile_destroy(cep_ffn_profile *p) { delete p; }
