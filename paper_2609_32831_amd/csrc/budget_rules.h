// budget_rules.h -- storage accounting and the budget rules of Sec. 3.3
// (Eq. 2, Eq. 3) and Sec. 3.4 (budget -> rows kept / precision and grouping),
// written once for the host helpers of the C ABI and for the device kernels
// that take the same decisions without a host round trip.  Double precision
// with contraction off, so host and device give identical results.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace uc {
namespace rules {

#pragma clang fp contract(off)

// Bytes of one (b, h_kv) of a packed segment: codes of K and V, float scale
// and minimum per key group and channel and per value row and channel group,
// and the residual tail rows at eb bytes per element.  -1 if invalid.
__host__ __device__ inline int64_t packed_bytes(int64_t N, int D, int G, int bits, int eb) {
  if (N < 0 || D < 1 || G < 1 || D % G || !(bits == 2 || bits == 4 || bits == 8)) return -1;
  const int64_t nf = (int64_t)G * (N / G);
  const int64_t codes = 2 * nf * D * bits / 8;
  const int64_t kmeta = (nf / G) * D * 2 * (int64_t)sizeof(float);
  const int64_t vmeta = nf * (D / G) * 2 * (int64_t)sizeof(float);
  return codes + kmeta + vmeta + (N - nf) * 2 * (int64_t)D * eb;
}

// Kept rows plus one int32 logical index per row.
__host__ __device__ inline int64_t evicted_bytes(int64_t rows, int D, int eb) {
  return rows * (2 * (int64_t)D * eb + (int64_t)sizeof(int32_t));
}

// Largest k with fixed + evicted_bytes(k) <= budget, clamped to [0, N].
__host__ __device__ inline int64_t evict_rows(double budget, double fixed, int64_t N, int D,
                                              int eb) {
  const double per = (double)evicted_bytes(1, D, eb);
  const double k = floor((budget - fixed) / per);
  if (!(k > 0.0)) return 0;
  return k >= (double)N ? N : (int64_t)k;
}

// Number of (bits, group) configurations for head dim D (groups 32 .. D).
__host__ __device__ inline int quant_groups(int D) {
  int ng = 0;
  for (int g = 32; g <= D; g *= 2) ++ng;
  return ng;
}

// Sec. 3.4: the first configuration at or after `first` (decreasing
// fidelity: bits 8, 4, 2; groups 32 .. D within one width) whose n_heads
// packed segments of N rows fit the budget, else the last one.
__host__ __device__ inline int quant_config(double budget, int64_t N, int D, int eb, int n_heads,
                                            int first, int* bits, int* group) {
  const int ng = quant_groups(D);
  const int n_cfg = 3 * ng;
  int pick = n_cfg - 1;
  for (int i = first; i < n_cfg; ++i) {
    const int64_t per_head = packed_bytes(N, D, 32 << (i % ng), 8 >> (i / ng), eb);
    if ((double)n_heads * (double)per_head <= budget) {
      pick = i;
      break;
    }
  }
  if (bits) *bits = 8 >> (pick / ng);
  if (group) *group = 32 << (pick % ng);
  return pick;
}

// Sec. 3.3 Eq. 2 with the redistribution rule stated under it: a type whose
// proportional share reaches its previous allocation keeps that allocation;
// the rest of the total is shared again in proportion to mass among the
// uncapped types with positive mass, until no type is capped; zero mass gets
// nothing.  n <= 64.
__host__ __device__ inline void type_budget(int n, const double* mass, const double* b_prev,
                                            double B_total, double* b_next) {
  bool active[64];
  for (int a = 0; a < n; ++a) {
    b_next[a] = 0.0;
    active[a] = mass[a] > 0.0;
  }
  double remaining = B_total;
  for (;;) {
    double msum = 0.0;
    int n_active = 0;
    for (int a = 0; a < n; ++a)
      if (active[a]) {
        msum += mass[a];
        ++n_active;
      }
    if (n_active == 0) return;
    bool capped[64];
    bool capped_any = false;
    for (int a = 0; a < n; ++a) {
      capped[a] = active[a] && mass[a] / msum * remaining >= b_prev[a];
      capped_any = capped_any || capped[a];
    }
    if (!capped_any) {
      for (int a = 0; a < n; ++a)
        if (active[a]) b_next[a] = mass[a] / msum * remaining;
      return;
    }
    for (int a = 0; a < n; ++a)
      if (capped[a]) {
        b_next[a] = b_prev[a];
        remaining -= b_prev[a];
        active[a] = false;
      }
  }
}

// Sec. 3.3 Eq. 3.  NaN for parameters outside 0 < rho_min <= rho_init <= 1,
// M_0 > 0.
__host__ __device__ inline double retention_next(double rho, double rho_init, double rho_min,
                                                 double M_c, double M_0) {
  if (!(rho_min > 0.0 && rho_min <= rho_init && rho_init <= 1.0 && M_0 > 0.0)) return NAN;
  const double r = rho_init * M_c / M_0;
  const double lo = r > rho_min ? r : rho_min;
  return rho < lo ? rho : lo;
}

}  // namespace rules
}  // namespace uc
