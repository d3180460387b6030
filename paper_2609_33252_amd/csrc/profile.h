// FFN throughput profile shared by the profile entry points and the OEWF
// coordinator.  Internal to libcep.
#pragma once

#include <cstdint>
#include <vector>

struct cep_ffn_profile {
  std::vector<int64_t> n;   // profiled expert-token counts, ascending
  std::vector<double> eta;  // throughput / peak at those counts
  double peak = 0;          // observed peak throughput
};

namespace cep {
// eta(N) for N >= 1 and F(N) = N / (eta(N) P_peak) for N >= 0 (F(0) = 0)
double profile_eta(const cep_ffn_profile &p, int64_t N);
double profile_latency(const cep_ffn_profile &p, int64_t N);
int set_global_error(int code, const char *msg);
}  // namespace cep
