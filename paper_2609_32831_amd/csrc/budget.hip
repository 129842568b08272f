// budget.hip -- budget decisions on the device (Sec. 3.3 Eq. 1-3 and the
// Sec. 3.4 translation) and the calibration policy rule (Sec. 3.2,
// App. B): single-workgroup kernels over a few dozen values, so a chunk
// boundary's decision needs no host round trip.
#include "budget_rules.h"
#include "uc_common.h"

namespace uc {
namespace {

#pragma clang fp contract(off)

__global__ void budget_step_kernel(uc_budget_params p, const float* __restrict__ mass,
                                   int n_steps, uc_budget_state* __restrict__ st) {
  if (threadIdx.x != 0) return;
  const int cand[2] = {p.ev, p.qt};
  const int eb = dtype_bytes(p.dtype);
  // Eq. 1: per step, the Mean over (query head, query row) is the raw sum
  // over the KV heads divided by Hq * M; the chunk mass is the mean over steps
  double m[2] = {0.0, 0.0};
  for (int t = 0; t < n_steps; ++t)
    for (int c = 0; c < 2; ++c) {
      double s = 0.0;
      for (int h = 0; h < p.Hkv; ++h)
        s += (double)mass[((size_t)t * p.Hkv + h) * p.n_segs + cand[c]];
      m[c] += s / ((double)p.Hq * p.M);
    }
  for (int c = 0; c < 2; ++c) m[c] /= n_steps;
  const double S[2] = {(double)p.Hkv * 2.0 * p.n_ev * p.D * eb,
                       (double)p.Hkv * 2.0 * p.n_qt * p.D * eb};
  const bool first = st->n_boundaries == 0;
  double rho, b_prev[2];
  int k_prev, cfg_prev;
  if (first) {
    st->M0 = m[0] + m[1];
    rho = p.rho_init;
    b_prev[0] = S[0];
    b_prev[1] = S[1];
    k_prev = p.n_ev;
    cfg_prev = -1;
  } else {
    rho = rules::retention_next(st->rho, p.rho_init, p.rho_min, m[0] + m[1], st->M0);
    b_prev[0] = st->b[0];
    b_prev[1] = st->b[1];
    k_prev = st->k;
    cfg_prev = st->cfg;
  }
  const double B = rho * (S[0] + S[1]);
  double b[2];
  rules::type_budget(2, m, b_prev, B, b);
  const int64_t kb = rules::evict_rows(b[0] / p.Hkv, 0.0, p.n_ev, p.D, eb);
  const int k = kb < k_prev ? (int)kb : k_prev;
  int bits = 0, group = 0;
  const int cfg = rules::quant_config(b[1], p.n_qt, p.D, eb, p.Hkv, cfg_prev < 0 ? 0 : cfg_prev,
                                      &bits, &group);
  st->rho = rho;
  st->B = B;
  st->m[0] = m[0];
  st->m[1] = m[1];
  st->b[0] = b[0];
  st->b[1] = b[1];
  st->k_prev = k_prev;
  st->cfg_prev = cfg_prev;
  st->k = k;
  st->cfg = cfg;
  st->bits = bits;
  st->group = group;
  st->n_boundaries += 1;
}

__global__ void calibrate_policy_kernel(const float* __restrict__ frac, int rows, int n_types,
                                        double threshold, double* __restrict__ conc,
                                        int32_t* __restrict__ evict) {
  const int a = threadIdx.x;
  if (a >= n_types) return;
  double s = 0.0;
  for (int r = 0; r < rows; ++r) s += (double)frac[(size_t)r * n_types + a];
  const double c = s / rows;
  conc[a] = c;
  evict[a] = c >= threshold ? 1 : 0;
}

}  // namespace

hipError_t launch_budget_step(const uc_budget_params& p, const float* mass, int n_steps,
                              uc_budget_state* state, hipStream_t st) {
  hipLaunchKernelGGL(budget_step_kernel, dim3(1), dim3(64), 0, st, p, mass, n_steps, state);
  return hipGetLastError();
}

hipError_t launch_calibrate_policy(const float* frac, int rows, int n_types, double threshold,
                                   double* conc, int32_t* evict, hipStream_t st) {
  hipLaunchKernelGGL(calibrate_policy_kernel, dim3(1), dim3(64), 0, st, frac, rows, n_types,
                     threshold, conc, evict);
  return hipGetLastError();
}

}  // namespace uc
