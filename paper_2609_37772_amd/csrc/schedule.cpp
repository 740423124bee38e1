// Host-only helpers of the C ABI: the per-token step tables built from integer
// budgets (Sec. 4.2, Eqs. 4-5) and the availability-latency controller
// (App. B timing model, App. C.3 measurement).
#include <cstdint>
#include <string>

#include "uad_internal.h"

namespace uad {

bool build_schedule_host(const int32_t *budgets, int batch, int chunk, int max_steps, int32_t *n_steps, float *t,
                         float *dt, uint8_t *mask, std::string *err) {
  if (!budgets || !n_steps || !t || !dt || !mask) {
    *err = "null pointer";
    return false;
  }
  if (batch < 1 || chunk < 1 || max_steps < 1) {
    *err = "sizes must be >= 1";
    return false;
  }
  const long M = (long)batch * chunk;
  int n = 0;
  for (long i = 0; i < M; ++i) {
    if (budgets[i] < 1 || budgets[i] > max_steps) {
      *err = "budget outside 1..max_steps";
      return false;
    }
    if (budgets[i] > n) n = budgets[i];
  }
  *n_steps = n;
  for (int k = 0; k < n; ++k)
    for (long i = 0; i < M; ++i) {
      const int N = budgets[i];
      const int left = k < N ? N - k : 0;  // steps this token still has to take
      // t = (N - min(k,N)) / N, one correctly rounded fp32 division of integers
      t[k * M + i] = (float)left / (float)N;
      dt[k * M + i] = k < N ? -(1.0f / (float)N) : 0.0f;
      mask[k * M + i] = k < N ? 0 : 1;
    }
  return true;
}

}  // namespace uad

extern "C" uad_status uad_aal(const double *release, int32_t n, double t_act, double *aal_out) {
  if (!release || !aal_out || n < 1) return UAD_E_INVALID;
  double clock = 0.0, wait = 0.0;
  for (int j = 0; j < n; ++j) {
    if (release[j] > clock) {
      wait += release[j] - clock;
      clock = release[j];
    }
    clock += t_act;  // action j executes for t_act
  }
  *aal_out = wait / n;
  return UAD_OK;
}
