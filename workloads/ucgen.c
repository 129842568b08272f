/*
 * ucgen.c -- seeded synthetic inputs for the mixed-policy KV attention
 * workloads.  Shared by the CPU oracle and the GPU library's tests and
 * benchmark; it holds none of the method's arithmetic, only input recipes.
 *
 * Random numbers: counter-based SplitMix64.  Output n of a stream with seed s
 * is mix64(s + (n + 1) * 0x9E3779B97F4A7C15) (Steele, Lea, Flood, "Fast
 * splittable pseudorandom number generators", OOPSLA 2014).  A uniform is the
 * top 53 bits scaled by 2^-53.  Standard normals use the Box-Muller transform
 * on the pair (2p, 2p+1) of uniforms: element 2p takes the cosine branch,
 * element 2p+1 the sine branch, so element i of a stream depends only on
 * (seed, i) and any sub-range can be produced independently.
 *
 * Rounding to a storage type: fp64 -> binary32 (round to nearest even) ->
 * bf16 / fp16 (round to nearest even).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t ucgen_raw(uint64_t seed, uint64_t n) { return mix64(seed + (n + 1) * GOLDEN); }

double ucgen_uniform(uint64_t seed, uint64_t n) {
  return (double)(ucgen_raw(seed, n) >> 11) * 0x1.0p-53;
}

/* Stream seed from a base seed and a list of ids (config, tensor, segment,
 * b, h, step, ...). */
uint64_t ucgen_stream(uint64_t base, const uint64_t* ids, int n_ids) {
  uint64_t s = mix64(base + GOLDEN);
  for (int i = 0; i < n_ids; ++i) s = mix64(s ^ (ids[i] + GOLDEN));
  return s;
}

double ucgen_normal_at(uint64_t seed, uint64_t i) {
  const double two_pi = 6.283185307179586476925286766559;
  uint64_t p = i >> 1;
  double u1 = ucgen_uniform(seed, 2 * p);
  double u2 = ucgen_uniform(seed, 2 * p + 1);
  double r = sqrt(-2.0 * log1p(-u1)); /* 1 - u1 lies in (0, 1] */
  double a = two_pi * u2;
  return (i & 1) ? r * sin(a) : r * cos(a);
}

void ucgen_normal(uint64_t seed, uint64_t start, int64_t n, double* out) {
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < n; ++k) out[k] = ucgen_normal_at(seed, start + (uint64_t)k);
}

void ucgen_uniform_fill(uint64_t seed, uint64_t start, int64_t n, double* out) {
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < n; ++k) out[k] = ucgen_uniform(seed, start + (uint64_t)k);
}

/* ---- storage rounding ---------------------------------------------------- */
static inline uint32_t f32_bits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

static inline uint16_t f32_to_bf16(float f) {
  uint32_t u = f32_bits(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

/* binary32 -> binary16, round to nearest even, with subnormals and overflow
 * to infinity. */
static inline uint16_t f32_to_f16(float f) {
  uint32_t u = f32_bits(f);
  uint32_t sign = (u >> 16) & 0x8000u;
  uint32_t a = u & 0x7FFFFFFFu;
  if (a >= 0x7F800000u) return (uint16_t)(sign | 0x7C00u | (a > 0x7F800000u ? 0x200u : 0u));
  if (a >= 0x477FF000u) return (uint16_t)(sign | 0x7C00u); /* rounds to >= 65520 */
  if (a < 0x38800000u) {                                 /* result subnormal or 0 */
    if (a < 0x33000000u) return (uint16_t)sign;           /* < 2^-25: rounds to 0 */
    uint32_t e = a >> 23;
    uint32_t m = (a & 0x7FFFFFu) | 0x800000u;
    uint32_t shift = 126 - e; /* 14..24: value = m * 2^(e-150); unit 2^-24 */
    uint32_t q = m >> shift;
    uint32_t rem = m & ((1u << shift) - 1u);
    uint32_t half = 1u << (shift - 1);
    if (rem > half || (rem == half && (q & 1u))) ++q;
    return (uint16_t)(sign | q);
  }
  uint32_t e = (a >> 23) - 112; /* rebias 127 -> 15 */
  uint32_t m = a & 0x7FFFFFu;
  uint32_t q = (e << 10) | (m >> 13);
  uint32_t rem = m & 0x1FFFu;
  if (rem > 0x1000u || (rem == 0x1000u && (q & 1u))) ++q;
  return (uint16_t)(sign | q);
}

/* dtype codes: 0 = fp32, 1 = fp16, 2 = bf16 */
static inline void store(void* out, int64_t k, double x, int dtype) {
  float f = (float)x;
  if (dtype == 0) ((float*)out)[k] = f;
  else if (dtype == 1) ((uint16_t*)out)[k] = f32_to_f16(f);
  else ((uint16_t*)out)[k] = f32_to_bf16(f);
}

void ucgen_round(const double* x, int64_t n, int dtype, void* out) {
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < n; ++k) store(out, k, x[k], dtype);
}

/*
 * Rows of one tensor [BH, N, D]: for row-block bh the stream is
 * ucgen_stream(base, {bh0 + bh}) and element (r, d) is normal number
 * (row0 + r) * D + d of it, so a tensor generated in pieces along r equals the
 * tensor generated whole.
 *   x = z * chan_scale[bh, d]                 (chan_scale NULL: 1)
 *     + row_coef[bh, r] * add_dir[bh, d]      (row_coef NULL: 1; add_dir NULL: 0)
 * then rounded to dtype.  When master is non-NULL the fp64 values are also
 * written there.
 */
void ucgen_rows(uint64_t base, int64_t bh0, int BH, int64_t N, int D, int64_t row0,
                const double* chan_scale, const double* add_dir,
                const double* row_coef, int dtype, void* out, double* master) {
  int64_t total = (int64_t)BH * N;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < total; ++t) {
    int64_t bh = t / N, r = t % N;
    uint64_t id = (uint64_t)(bh0 + bh);
    uint64_t seed = ucgen_stream(base, &id, 1);
    double coef = row_coef ? row_coef[t] : 1.0;
    for (int d = 0; d < D; ++d) {
      double z = ucgen_normal_at(seed, (uint64_t)(row0 + r) * (uint64_t)D + (uint64_t)d);
      double x = z * (chan_scale ? chan_scale[bh * D + d] : 1.0);
      if (add_dir) x += coef * add_dir[bh * D + d];
      int64_t k = t * D + d;
      if (master) master[k] = x;
      store(out, k, x, dtype);
    }
  }
}

/* Random-walk drift of an fp64 master copy: x += sigma * z, then the rounded
 * copy is stored.  master[k] is element start + k of the whole tensor and z
 * is element start + k of the stream ucgen_stream(base, {step}), so any slice
 * of a tensor drifts exactly as it does inside the whole. */
void ucgen_drift(uint64_t base, uint64_t step, double sigma, int64_t start, int64_t n,
                 double* master, int dtype, void* out) {
  uint64_t seed = ucgen_stream(base, &step, 1);
#pragma omp parallel for schedule(static)
  for (int64_t k = 0; k < n; ++k) {
    master[k] += sigma * ucgen_normal_at(seed, (uint64_t)(start + k));
    store(out, k, master[k], dtype);
  }
}
