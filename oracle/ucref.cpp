/*
 * ucref.cpp -- CPU oracle for mixed-policy KV attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Used by the test suite, the smoke check and the
 * benchmark's CPU-baseline leg; never by the product path.  Shares no code
 * with the GPU library.
 *
 * Every function states the passage of the UniCache paper it follows.  Where
 * the paper is silent the reading taken is stated next to the code (and
 * listed with the others in the design notes).
 *
 * Build: g++ -O2 -fopenmp -ffp-contract=off (no fast-math): the quantizer's
 * codes are defined by IEEE binary32 arithmetic with one rounding per
 * operation, which this guarantees on x86-64.
 */
#include "ucref.h"

#include <omp.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <vector>

/* ---- element types ------------------------------------------------------ */

static double widen_one(const void* x, int dtype, int64_t i) {
  if (dtype == 0) return (double)((const float*)x)[i];
  uint16_t h = ((const uint16_t*)x)[i];
  if (dtype == 2) {  // bf16: the upper half of a binary32
    uint32_t u = (uint32_t)h << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return (double)f;
  }
  // fp16: 1 sign, 5 exponent (bias 15), 10 fraction bits
  int sign = (h >> 15) & 1, e = (h >> 10) & 31, m = h & 1023;
  double v;
  if (e == 0) v = std::ldexp((double)m, -24);
  else if (e == 31) v = m ? std::numeric_limits<double>::quiet_NaN()
                          : std::numeric_limits<double>::infinity();
  else v = std::ldexp((double)(1024 + m), e - 25);
  return sign ? -v : v;
}

void ucref_widen(const void* x, int dtype, int64_t n, double* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = widen_one(x, dtype, i);
}

/* Round a binary32 value to bf16 (8 significant bits, binary32 exponent
 * range) or fp16 (11 significant bits, normal range from 2^-14, subnormal
 * quantum 2^-24, overflow at 65520), nearest-even, returned exactly as a
 * double.  The quantum of x is a power of two, so x / quantum and the product
 * back are exact in double and nearbyint (default mode: nearest-even) is the
 * only rounding. */
static double round_value(float xf, int dtype) {
  double x = (double)xf;
  if (dtype == 0 || x == 0.0 || !std::isfinite(x)) return x;
  int p = dtype == 2 ? 8 : 11;         // significant bits
  int emin = dtype == 2 ? -126 : -14;  // exponent of the smallest normal
  int ex;
  std::frexp(std::fabs(x), &ex);       // |x| = f * 2^ex, f in [0.5, 1)
  int e = std::max(ex - 1, emin);      // floor(log2 |x|), clamped to normals
  double quantum = std::ldexp(1.0, e - (p - 1));
  double r = std::nearbyint(x / quantum) * quantum;
  double maxfinite = dtype == 2 ? std::ldexp(255.0, 120) /* (2-2^-7)*2^127 */
                                : 65504.0;
  if (std::fabs(r) > maxfinite) return std::copysign(std::numeric_limits<double>::infinity(), x);
  return r;
}

void ucref_round_value(const float* x, int dtype, int64_t n, double* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = round_value(x[i], dtype);
}

static size_t elem_size(int dtype) { return dtype == 0 ? 4 : 2; }

/* ---- quantization ----------------------------------------------------------
 * App. E "Physical, type-aware KV storage": quantised segments keep packed
 * low-bit codes with scales and minima plus a short residual tail.  The
 * quantizer is the asymmetric min/max group quantizer of the quantization
 * baseline the paper treats as representative (App. A, KIVI): keys per
 * channel, values per token.
 *   group (keys):   channel c over rows gG .. gG+G-1
 *   group (values): channels gG .. gG+G-1 of one row
 *   mn = min, mx = max, s = (mx - mn) / (2^b - 1)               (binary32)
 *   code = s > 0 ? clamp(rint((x - mn) / s), 0, 2^b - 1) : 0    (binary32)
 *   value of a code = fmaf(code, s, mn) rounded to the segment's dtype.
 * Rows past n_full = G*floor(N/G) form the residual tail, kept as stored.
 * Packing: channel c of a row lives in byte c*b/8 at bit (c % (8/b))*b. */

static inline int quant_code(float x, float mn, float s, int qmax) {
  if (!(s > 0.0f)) return 0;
  float t = (x - mn) / s;
  int c = (int)std::rint(t);
  return std::min(std::max(c, 0), qmax);
}

static inline void put_code(uint8_t* row, int c, int b, int code) {
  int per_byte = 8 / b;
  int byte = c / per_byte;
  int shift = (c % per_byte) * b;
  row[byte] = (uint8_t)(row[byte] | (code << shift));
}

static inline int get_code(const uint8_t* row, int c, int b) {
  int per_byte = 8 / b;
  return (row[c / per_byte] >> ((c % per_byte) * b)) & ((1 << b) - 1);
}

static bool quant_args_ok(int N, int D, int G, const int32_t* bits, int BH) {
  if (N < 0 || D <= 0 || G <= 0 || D % G != 0) return false;
  for (int i = 0; i < BH; ++i)
    if (bits[i] != 2 && bits[i] != 4 && bits[i] != 8) return false;
  return true;
}

int ucref_quantize(int BH, int N, int D, int G, const int32_t* bits, int dtype,
                   const void* k, const void* v, uint8_t* codes_k,
                   uint8_t* codes_v, const int64_t* code_off, float* scale_k,
                   float* min_k, float* scale_v, float* min_v, void* tail_k,
                   void* tail_v) {
  if (!quant_args_ok(N, D, G, bits, BH)) return -1;
  const int n_full = G * (N / G), n_tail = N - n_full, ngk = n_full / G,
            ngv = D / G;
  const size_t es = elem_size(dtype);
  for (int bh = 0; bh < BH; ++bh) {
    const int b = bits[bh], qmax = (1 << b) - 1, row_bytes = D * b / 8;
    const float denom = (float)qmax;
    uint8_t* ck = codes_k + code_off[bh];
    uint8_t* cv = codes_v + code_off[bh];
    std::memset(ck, 0, (size_t)n_full * row_bytes);
    std::memset(cv, 0, (size_t)n_full * row_bytes);
    auto X = [&](const void* t, int r, int c) {
      return (float)widen_one(t, dtype, ((int64_t)bh * N + r) * D + c);
    };
    // keys: one channel over G consecutive rows
    for (int g = 0; g < ngk; ++g) {
      for (int c = 0; c < D; ++c) {
        float mn = X(k, g * G, c), mx = mn;
        for (int r = g * G; r < g * G + G; ++r) {
          float x = X(k, r, c);
          mn = std::min(mn, x);
          mx = std::max(mx, x);
        }
        float s = (mx - mn) / denom;
        scale_k[((int64_t)bh * ngk + g) * D + c] = s;
        min_k[((int64_t)bh * ngk + g) * D + c] = mn;
        for (int r = g * G; r < g * G + G; ++r)
          put_code(ck + (int64_t)r * row_bytes, c, b, quant_code(X(k, r, c), mn, s, qmax));
      }
    }
    // values: G consecutive channels of one row
    for (int r = 0; r < n_full; ++r) {
      for (int g = 0; g < ngv; ++g) {
        float mn = X(v, r, g * G), mx = mn;
        for (int c = g * G; c < g * G + G; ++c) {
          float x = X(v, r, c);
          mn = std::min(mn, x);
          mx = std::max(mx, x);
        }
        float s = (mx - mn) / denom;
        scale_v[((int64_t)bh * n_full + r) * ngv + g] = s;
        min_v[((int64_t)bh * n_full + r) * ngv + g] = mn;
        for (int c = g * G; c < g * G + G; ++c)
          put_code(cv + (int64_t)r * row_bytes, c, b, quant_code(X(v, r, c), mn, s, qmax));
      }
    }
    // residual tail: the stored bytes, unchanged
    if (n_tail > 0) {
      const size_t row = (size_t)D * es;
      std::memcpy((char*)tail_k + (size_t)bh * n_tail * row,
                  (const char*)k + ((size_t)bh * N + n_full) * row, n_tail * row);
      std::memcpy((char*)tail_v + (size_t)bh * n_tail * row,
                  (const char*)v + ((size_t)bh * N + n_full) * row, n_tail * row);
    }
  }
  return 0;
}

int ucref_dequant(int BH, int N, int D, int G, const int32_t* bits, int dtype,
                  const uint8_t* codes_k, const uint8_t* codes_v,
                  const int64_t* code_off, const float* scale_k,
                  const float* min_k, const float* scale_v, const float* min_v,
                  const void* tail_k, const void* tail_v, double* khat,
                  double* vhat) {
  if (!quant_args_ok(N, D, G, bits, BH)) return -1;
  const int n_full = G * (N / G), n_tail = N - n_full, ngk = n_full / G,
            ngv = D / G;
  for (int bh = 0; bh < BH; ++bh) {
    const int b = bits[bh], row_bytes = D * b / 8;
    const uint8_t* ck = codes_k + code_off[bh];
    const uint8_t* cv = codes_v + code_off[bh];
    for (int r = 0; r < N; ++r) {
      for (int c = 0; c < D; ++c) {
        int64_t o = ((int64_t)bh * N + r) * D + c;
        if (r < n_full) {
          int64_t ik = ((int64_t)bh * ngk + r / G) * D + c;
          int64_t iv = ((int64_t)bh * n_full + r) * ngv + c / G;
          float xk = std::fmaf((float)get_code(ck + (int64_t)r * row_bytes, c, b),
                               scale_k[ik], min_k[ik]);
          float xv = std::fmaf((float)get_code(cv + (int64_t)r * row_bytes, c, b),
                               scale_v[iv], min_v[iv]);
          khat[o] = round_value(xk, dtype);
          vhat[o] = round_value(xv, dtype);
        } else {
          int64_t t = ((int64_t)bh * n_tail + (r - n_full)) * D + c;
          khat[o] = widen_one(tail_k, dtype, t);
          vhat[o] = widen_one(tail_v, dtype, t);
        }
      }
    }
  }
  return 0;
}

/* ---- importance scores ------------------------------------------------------
 * Sec. 3.3 (Eq. 1 and the probabilities P_{h,q,k} it sums) and App. E
 * ("Batched GQA token selection": scores aggregated over the query heads that
 * share a KV head).  For each (b, h_kv) and each observation row (g, w):
 *   s_j = sm_scale * <q, k_j> over every row j of the whole context,
 *   P_j = exp(s_j - max s) / sum_i exp(s_i - max s),
 *   score[j] += P_j,   mass[seg(j)] += P_j.
 * Readings: P is normalised over all segments; the group and window are
 * combined by summation. */
void ucref_score(int B, int Hq, int Hkv, int D, int W, int64_t N,
                 const double* q, const double* k, const int32_t* seg_of_row,
                 int n_segs, double sm_scale, double* score, double* mass) {
  const int G = Hq / Hkv;
#pragma omp parallel for schedule(dynamic)
  for (int bh = 0; bh < B * Hkv; ++bh) {
    const int b = bh / Hkv, h = bh % Hkv;
    const double* K = k + (int64_t)bh * N * D;
    double* sc = score + (int64_t)bh * N;
    double* ms = mass + (int64_t)bh * n_segs;
    for (int64_t j = 0; j < N; ++j) sc[j] = 0.0;
    for (int a = 0; a < n_segs; ++a) ms[a] = 0.0;
    std::vector<double> s(N);
    for (int g = 0; g < G; ++g) {
      for (int w = 0; w < W; ++w) {
        const double* qr = q + (((int64_t)b * Hq + h * G + g) * W + w) * D;
        double mx = -std::numeric_limits<double>::infinity();
        for (int64_t j = 0; j < N; ++j) {
          double dot = 0.0;
          for (int c = 0; c < D; ++c) dot += qr[c] * K[j * D + c];
          s[j] = dot * sm_scale;
          mx = std::max(mx, s[j]);
        }
        double Z = 0.0;
        for (int64_t j = 0; j < N; ++j) Z += std::exp(s[j] - mx);
        for (int64_t j = 0; j < N; ++j) {
          double P = std::exp(s[j] - mx) / Z;
          sc[j] += P;
          ms[seg_of_row[j]] += P;
        }
      }
    }
  }
}

/* ---- selection --------------------------------------------------------------
 * App. E ("heavy-hitter and recent-token selection independently for each KV
 * head"; "store only retained KV entries and their logical token indices").
 * The last n_recent positions are always kept; of the rest, the k - n_recent
 * positions first in the order (score descending, index ascending) are kept.
 * Output in ascending position (Sec. 3.4: segments are reassembled in their
 * original token order). */
int ucref_select(int BH, int N, const float* scores, int k, int n_recent,
                 int32_t* keep_idx) {
  if (k < 0 || k > N || n_recent < 0 || n_recent > k) return -1;
  for (int bh = 0; bh < BH; ++bh) {
    const float* s = scores + (int64_t)bh * N;
    std::vector<int32_t> order(N - n_recent);
    for (int i = 0; i < N - n_recent; ++i) order[i] = i;
    std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
      if (s[a] != s[b]) return s[a] > s[b];
      return a < b;
    });
    std::vector<int32_t> kept(order.begin(), order.begin() + (k - n_recent));
    for (int i = N - n_recent; i < N; ++i) kept.push_back(i);
    std::sort(kept.begin(), kept.end());
    if (k > 0) std::memcpy(keep_idx + (int64_t)bh * k, kept.data(), sizeof(int32_t) * k);
  }
  return 0;
}

/* ---- calibration statistic -------------------------------------------------
 * Sec. 3.2 and App. B ("Calibration Setting"): attention concentration of a
 * type = the fraction of its attention mass captured by its top 10 % of
 * tokens.  For every row: the k largest scores (sorted copy) summed in
 * double, divided by the double sum of all scores (0 if that sum is 0). */
int ucref_topk_mass(int BH, int N, const float* scores, int k, double* frac) {
  if (k < 0 || k > N) return -1;
  for (int r = 0; r < BH; ++r) {
    std::vector<float> s(scores + (int64_t)r * N, scores + (int64_t)(r + 1) * N);
    std::sort(s.begin(), s.end(), [](float a, float b) { return a > b; });
    double top = 0.0, all = 0.0;
    for (int i = 0; i < N; ++i) {
      all += s[i];
      if (i < k) top += s[i];
    }
    frac[r] = all > 0.0 ? top / all : 0.0;
  }
  return 0;
}

/* ---- attention --------------------------------------------------------------
 * App. E ("Attention over heterogeneous cache segments": one softmax shared by
 * all segments; the reference implementation evaluates compression with
 * attention masks and fake quantization).  For each (b, h_q, m):
 *   s_j = sm_scale * <q, k_j> for the present rows j (present = not evicted),
 *   o = sum_j exp(s_j - mx) v_j / Z,  Z = sum_j exp(s_j - mx),
 *   lse = mx + ln Z,  seg_lse[a] = mx + ln sum_{j in a} exp(s_j - mx),
 *   seg_mass[a] = sum_{j in a} P_j  (the bracket of Sec. 3.3 Eq. 1 for one
 *   head and query).
 * No causal mask (observation, decode and latent queries see every cached
 * row). */
void ucref_attend(int B, int Hq, int Hkv, int D, int M, int64_t N,
                  const double* q, const double* k, const double* v,
                  const uint8_t* present, const int32_t* seg_of_row,
                  int n_segs, double sm_scale, double* o, double* lse,
                  double* seg_lse, double* seg_mass) {
  const int G = Hq / Hkv;
  const double NEG_INF = -std::numeric_limits<double>::infinity();
#pragma omp parallel for schedule(dynamic) collapse(2)
  for (int bq = 0; bq < B * Hq; ++bq) {
    for (int m = 0; m < M; ++m) {
      const int b = bq / Hq, hq = bq % Hq, bh = b * Hkv + hq / G;
      const double* K = k + (int64_t)bh * N * D;
      const double* V = v + (int64_t)bh * N * D;
      const uint8_t* pr = present ? present + (int64_t)bh * N : nullptr;
      const double* qr = q + ((int64_t)bq * M + m) * D;
      std::vector<double> s(N);
      double mx = NEG_INF;
      for (int64_t j = 0; j < N; ++j) {
        if (pr && !pr[j]) continue;
        double dot = 0.0;
        for (int c = 0; c < D; ++c) dot += qr[c] * K[j * D + c];
        s[j] = dot * sm_scale;
        mx = std::max(mx, s[j]);
      }
      std::vector<double> acc(D, 0.0), zs(n_segs, 0.0);
      double Z = 0.0;
      for (int64_t j = 0; j < N; ++j) {
        if (pr && !pr[j]) continue;
        double e = std::exp(s[j] - mx);
        Z += e;
        zs[seg_of_row[j]] += e;
        for (int c = 0; c < D; ++c) acc[c] += e * V[j * D + c];
      }
      double* orow = o + ((int64_t)bq * M + m) * D;
      for (int c = 0; c < D; ++c) orow[c] = acc[c] / Z;
      if (lse) lse[(int64_t)bq * M + m] = mx + std::log(Z);
      for (int a = 0; a < n_segs; ++a) {
        int64_t i = ((int64_t)bq * M + m) * n_segs + a;
        if (seg_lse) seg_lse[i] = zs[a] > 0.0 ? mx + std::log(zs[a]) : NEG_INF;
        if (seg_mass) seg_mass[i] = zs[a] / Z;
      }
    }
  }
}

/* ---- storage accounting and budgets -----------------------------------------
 * Sec. 3.3: S_a is a type's original storage cost and the shared budget is
 * B = rho * sum_a S_a; Sec. 3.4: an eviction policy's budget fixes how many
 * tokens it keeps, a quantization policy's its precision and grouping.
 * Reading: a budget counts every stored byte of one (b, h_kv) -- kept rows,
 * the int32 logical index of each evicted-segment survivor, codes, float
 * scales and minima, and the residual tail. */
int64_t ucref_dense_bytes(int64_t rows, int D, int dtype) {
  return rows * 2 * D * (int64_t)elem_size(dtype);
}

int64_t ucref_evicted_bytes(int64_t rows, int D, int dtype) {
  return rows * (2 * D * (int64_t)elem_size(dtype) + 4);
}

int64_t ucref_packed_bytes(int64_t N, int D, int G, int bits, int dtype) {
  if (N < 0 || D <= 0 || G <= 0 || D % G || (bits != 2 && bits != 4 && bits != 8)) return -1;
  int64_t n_full = G * (N / G), tail = N - n_full;
  int64_t codes = 2 * n_full * D * bits / 8;
  int64_t k_meta = (n_full / G) * D * 2 * 4;  // float scale + float min per channel and row group
  int64_t v_meta = n_full * (D / G) * 2 * 4;  // float scale + float min per row and channel group
  return codes + k_meta + v_meta + ucref_dense_bytes(tail, D, dtype);
}

int64_t ucref_evict_rows(double budget, double fixed, int64_t N, int D, int dtype) {
  double per_row = (double)ucref_evicted_bytes(1, D, dtype);
  double k = std::floor((budget - fixed) / per_row);
  if (!(k > 0)) return 0;
  return k > (double)N ? N : (int64_t)k;
}

/* Per-head code widths under a budget: all heads at 2 bits, then heads move
 * to 4 bits in descending mass (equal mass: lower head first) while the total
 * stays within the budget. */
int ucref_assign_bits(int n_heads, const double* mass, int64_t N, int D, int G,
                      int dtype, double budget, double fixed, int32_t* bits) {
  int64_t b2 = ucref_packed_bytes(N, D, G, 2, dtype), b4 = ucref_packed_bytes(N, D, G, 4, dtype);
  if (b2 < 0 || n_heads <= 0) return -1;
  std::vector<int> order(n_heads);
  for (int i = 0; i < n_heads; ++i) { order[i] = i; bits[i] = 2; }
  std::sort(order.begin(), order.end(), [&](int a, int b) {
    if (mass[a] != mass[b]) return mass[a] > mass[b];
    return a < b;
  });
  double total = fixed + (double)b2 * n_heads;
  for (int i = 0; i < n_heads; ++i) {
    if (total + (double)(b4 - b2) > budget) break;
    total += (double)(b4 - b2);
    bits[order[i]] = 4;
  }
  return 0;
}

/* Sec. 3.4: a quantization policy's budget fixes its precision and its
 * grouping.  Configurations are numbered in decreasing fidelity: widths 8, 4,
 * 2 bits and, for one width, groups 32, 64, ..., D (finer first), so
 * configuration i has bits = 8 >> (i / ng) and group = 32 << (i % ng) with ng
 * the number of groups.  Returns the first configuration at or after `first`
 * (a type never regains fidelity it gave up) whose n_heads packed segments
 * fit the budget, or the last one if none fits; -1 for invalid arguments. */
int ucref_quant_config(double budget, int64_t N, int D, int dtype, int n_heads, int first) {
  if (D < 32 || (D & (D - 1)) || N < 0 || n_heads <= 0) return -1;
  int ng = 0;
  for (int g = 32; g <= D; g *= 2) ++ng;
  const int n_cfg = 3 * ng;
  if (first < 0 || first >= n_cfg) return -1;
  for (int i = first; i < n_cfg; ++i) {
    const int bits = 8 >> (i / ng), group = 32 << (i % ng);
    if ((double)n_heads * (double)ucref_packed_bytes(N, D, group, bits, dtype) <= budget) return i;
  }
  return n_cfg - 1;
}

/* Sec. 3.3 Eq. 2 with the redistribution stated under it: each type gets
 * its mass share of B_total, capped at its previous allocation; what capped
 * types cannot take is shared again, in proportion to mass, among the
 * uncapped types with positive mass; if every such type is capped the rest is
 * left unused.  Types with zero mass get zero. */
int ucref_type_budget(int n, const double* mass, const double* b_prev,
                      double B_total, double* b_next) {
  if (n <= 0) return -1;
  std::vector<int> active;
  for (int a = 0; a < n; ++a) {
    b_next[a] = 0.0;
    if (mass[a] > 0.0) active.push_back(a);
  }
  double remaining = B_total;
  while (!active.empty()) {
    double msum = 0.0;
    for (int a : active) msum += mass[a];
    std::vector<int> capped, uncapped;
    for (int a : active) {
      if (mass[a] / msum * remaining >= b_prev[a]) capped.push_back(a);
      else uncapped.push_back(a);
    }
    if (capped.empty()) {
      for (int a : active) b_next[a] = mass[a] / msum * remaining;
      break;
    }
    for (int a : capped) {
      b_next[a] = b_prev[a];
      remaining -= b_prev[a];
    }
    active = uncapped;
  }
  return 0;
}

/* Sec. 3.3 Eq. 3. */
double ucref_retention_next(double rho, double rho_init, double rho_min,
                            double M_c, double M_0) {
  if (!(rho_min > 0.0 && rho_min <= rho_init && rho_init <= 1.0 && M_0 > 0.0))
    return std::numeric_limits<double>::quiet_NaN();
  return std::min(rho, std::max(rho_min, rho_init * M_c / M_0));
}

int ucref_set_threads(int n) {
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
}
