// attend_generic.hip -- shared-softmax attention over heterogeneous segments
// for any element type (fp32 / fp16 / bf16 rows and queries), plus the
// log-sum-exp merge of chunk results (App. E, "Attention over heterogeneous
// cache segments": one softmax normalisation across all segments; results of
// separately evaluated chunks merged with log-sum-exp statistics).
//
// Work split: every segment's rows are cut into chunks (ChunkPlan); one
// workgroup handles one (chunk, query head, query row).  Its four waves take
// interleaved rows of the chunk; a lane owns D/64 dimensions, so a logit is a
// lane-partial dot product reduced with wave shuffles.  Each chunk leaves an
// unnormalised partial (running max m, sum l, accumulator o) in the
// workspace, in base-2 units (logits pre-multiplied by log2(e)); the combine
// kernel merges them into o, lse and the per-segment lse.
//
// This path runs on VALU only.  It serves queries and rows that are not bf16
// (the bf16 path uses matrix cores) and cross-checks the fast kernels.
#include <math.h>

#include "uc_common.h"

namespace uc {
namespace {

template <int D>
struct RowLoader {
  static constexpr int PER = D / 64;
  // K and V values of row r for dims lane + 64*i
  __device__ static inline void load(const KSeg& s, int bh, int r, int lane, int bits, int64_t off,
                                     float (&kv)[PER], float (&vv)[PER]) {
    if (s.kind == UC_SEG_DENSE) {
      const int64_t base = ((int64_t)bh * s.row_stride + r) * D + lane;
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        kv[i] = load_elem(s.k, s.dtype, base + 64 * i);
        vv[i] = load_elem(s.v, s.dtype, base + 64 * i);
      }
    } else if (r < s.n_full) {
      const int rb = D * bits / 8, G = s.group;
      const uint8_t* ck = s.codes_k + off + (int64_t)r * rb;
      const uint8_t* cv = s.codes_v + off + (int64_t)r * rb;
      const int mask = (1 << bits) - 1, per_byte = 8 / bits;
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int d = lane + 64 * i;
        const int sh = (d % per_byte) * bits, by = d / per_byte;
        const int qk = (ck[by] >> sh) & mask, qv = (cv[by] >> sh) & mask;
        const int64_t ik = ((int64_t)bh * s.kgroups + r / G) * D + d;
        const int64_t iv = ((int64_t)bh * s.cap_full + r) * (D / G) + d / G;
        kv[i] = round_to(fmaf((float)qk, s.scale_k[ik], s.min_k[ik]), s.dtype);
        vv[i] = round_to(fmaf((float)qv, s.scale_v[iv], s.min_v[iv]), s.dtype);
      }
    } else {
      const int64_t base = ((int64_t)bh * s.tail_stride + (r - s.n_full)) * D + lane;
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        kv[i] = load_elem(s.tail_k, s.dtype, base + 64 * i);
        vv[i] = load_elem(s.tail_v, s.dtype, base + 64 * i);
      }
    }
  }
};

__device__ inline int chunk_segment(const ChunkPlan& plan, int nseg, int c) {
  int si = 0;
  while (si + 1 < nseg && c >= plan.first[si + 1]) ++si;
  return si;
}

template <int D>
__global__ __launch_bounds__(256) void attend_generic_kernel(KSegs segs, ChunkPlan plan,
                                                             const void* __restrict__ q, int q_dt,
                                                             int Hq, int Hkv, int M,
                                                             float scale_log2, float* partial,
                                                             int want_o, int ps) {
  constexpr int PER = D / 64;
  __shared__ float red_m[4], red_l[4];
  __shared__ float red_o[4][D];
  const int c = blockIdx.x, bq = blockIdx.y, m = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int si = chunk_segment(plan, segs.n, c);
  const KSeg& s = segs.s[si];
  const int r0 = (c - plan.first[si]) * plan.rows[si];
  const int r1 = min(r0 + plan.rows[si], s.n_rows);
  const int G = Hq / Hkv, b = bq / Hq, hq = bq % Hq, bh = b * Hkv + hq / G;

  int bits = 0;
  int64_t off = 0;
  const bool ok = s.kind == UC_SEG_DENSE || head_codes(s, bh, D, bits, off);

  float qv[PER];
  const int64_t qbase = ((int64_t)bq * M + m) * D + lane;
#pragma unroll
  for (int i = 0; i < PER; ++i) qv[i] = load_elem(q, q_dt, qbase + 64 * i) * scale_log2;

  float mx = -INFINITY, l = 0.0f, acc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) acc[i] = 0.0f;
  if (ok) {
    for (int r = r0 + wave; r < r1; r += 4) {
      float kv[PER], vv[PER];
      RowLoader<D>::load(s, bh, r, lane, bits, off, kv, vv);
      float d = 0.0f;
#pragma unroll
      for (int i = 0; i < PER; ++i) d = fmaf(qv[i], kv[i], d);
      d = wave_sum(d);
      const float mn = fmaxf(mx, d);
      const float alpha = exp2f(mx - mn), p = exp2f(d - mn);
      l = l * alpha + p;
      if (want_o) {
#pragma unroll
        for (int i = 0; i < PER; ++i) acc[i] = fmaf(p, vv[i], acc[i] * alpha);
      }
      mx = mn;
    }
  }
  if (lane == 0) {
    red_m[wave] = mx;
    red_l[wave] = l;
  }
#pragma unroll
  for (int i = 0; i < PER; ++i) red_o[wave][lane + 64 * i] = acc[i];
  __syncthreads();
  if (wave != 0) return;
  float M_ = fmaxf(fmaxf(red_m[0], red_m[1]), fmaxf(red_m[2], red_m[3]));
  float w[4], L = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    w[j] = red_m[j] == -INFINITY ? 0.0f : exp2f(red_m[j] - M_);
    L += w[j] * red_l[j];
  }
  const int C = plan.n_chunks;
  float* out = partial + (((int64_t)bq * M + m) * C + c) * ps;
  if (lane == 0) {
    out[0] = ok ? M_ : 0.0f;
    out[1] = ok ? L : __builtin_nanf("");
  }
  if (want_o) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int d = lane + 64 * i;
      out[2 + d] = w[0] * red_o[0][d] + w[1] * red_o[1][d] + w[2] * red_o[2][d] + w[3] * red_o[3][d];
    }
  }
}

// One wave per query row: merge the chunk partials (m, l, o) of that row by
// log-sum-exp in a single pass.  Lane = (record group rg = lane / 16, dims
// (lane % 16) * D/16 ...): each record group merges every fourth record
// online (independent loads, running maximum), then the four groups are
// merged with cross-lane exchanges.  Records with m = -inf hold no rows
// (their other fields are loaded but never used).  Per-segment log-sum-exps
// take one more pass over m and l only.
template <int D>
__global__ __launch_bounds__(64) void attend_combine_kernel(ChunkPlan plan, int nseg, int ps,
                                                            const float* __restrict__ partial,
                                                            float* o, float* lse, float* seg_lse) {
  constexpr int PD = D / 16;  // dims per lane
  const int64_t qi = blockIdx.x;
  const int lane = threadIdx.x;
  const int C = plan.n_chunks;
  const float* P = partial + qi * C * ps;
  const int rg = lane >> 4, d0 = (lane & 15) * PD;
  float m = -INFINITY, l = 0.0f, acc[PD];
#pragma unroll
  for (int i = 0; i < PD; ++i) acc[i] = 0.0f;
  // two records per pass, every load issued before any value is used (one
  // memory latency per pass, not one per field); an empty record's other
  // fields are not defined, so it is dropped by selects after loading
  for (int c0 = rg; c0 < C; c0 += 8) {
    const bool two = c0 + 4 < C;
    const float* pr[2] = {P + (int64_t)c0 * ps, P + (int64_t)(two ? c0 + 4 : c0) * ps};
    float mc[2], lc[2], oc[2][PD];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      mc[r] = pr[r][0];
      lc[r] = pr[r][1];
      if (o) {
#pragma unroll
        for (int i = 0; i < PD; ++i) oc[r][i] = pr[r][2 + d0 + i];
      }
    }
    if (!two) mc[1] = -INFINITY;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const bool live = mc[r] != -INFINITY;
      const float mn = fmaxf(m, mc[r]);
      const float a = exp2f(m - mn), b = exp2f(mc[r] - mn);
      l = live ? fmaf(l, a, lc[r] * b) : l;
      if (o) {
#pragma unroll
        for (int i = 0; i < PD; ++i) acc[i] = live ? fmaf(acc[i], a, oc[r][i] * b) : acc[i];
      }
      m = live ? mn : m;
    }
  }
  float M = fmaxf(m, __shfl_xor(m, 16, 64));
  M = fmaxf(M, __shfl_xor(M, 32, 64));
  const float sc = m == -INFINITY ? 0.0f : exp2f(m - M);
  l *= sc;
  l += __shfl_xor(l, 16, 64);
  l += __shfl_xor(l, 32, 64);
  if (lse && lane == 0) lse[qi] = (M + log2f(l)) * kLn2;
  if (o) {
    const float inv = 1.0f / l;
#pragma unroll
    for (int i = 0; i < PD; ++i) {
      float v = acc[i] * sc;
      v += __shfl_xor(v, 16, 64);
      v += __shfl_xor(v, 32, 64);
      acc[i] = v * inv;
    }
    if (rg == 0) {
#pragma unroll
      for (int i = 0; i < PD; ++i) o[qi * D + d0 + i] = acc[i];
    }
  }
  if (seg_lse) {
    for (int a = 0; a < nseg; ++a) {
      float ma = -INFINITY, la = 0.0f;
      for (int c = plan.first[a] + lane; c < plan.first[a + 1]; c += 64) {
        const float* pc = P + (int64_t)c * ps;
        const float mc = pc[0];
        if (mc == -INFINITY) continue;
        const float mn = fmaxf(ma, mc);
        la = fmaf(la, exp2f(ma - mn), pc[1] * exp2f(mc - mn));
        ma = mn;
      }
      const float mw = wave_max(ma);
      la = wave_sum(ma == -INFINITY ? 0.0f : la * exp2f(ma - mw));
      if (lane == 0) seg_lse[qi * nseg + a] = la > 0.0f ? (mw + log2f(la)) * kLn2 : -INFINITY;
    }
  }
}

// Importance scores, second pass: one thread per key row.  For every
// observation row (g, w) of the KV head, p = exp(s - lse) with lse from the
// first pass; the column sums run in double.  Per-chunk segment masses go to
// mass_partial[bh, chunk].
struct ScorePtrs {
  float* p[kMaxSeg];
};

template <int D>
__global__ __launch_bounds__(256) void score_colsum_kernel(KSegs segs, ChunkPlan plan,
                                                           const void* __restrict__ q, int q_dt,
                                                           int Hq, int Hkv, int W, int q_ld,
                                                           float scale_log2,
                                                           const float* __restrict__ lse,
                                                           ScorePtrs scores,
                                                           double* mass_partial) {
  constexpr int QB = 16;  // query rows staged per round
  __shared__ float qs[QB][D];
  __shared__ float ls[QB];
  __shared__ double red[4];
  const int c = blockIdx.x, bh = blockIdx.y;
  const int si = chunk_segment(plan, segs.n, c);
  const KSeg& s = segs.s[si];
  const int r = (c - plan.first[si]) * plan.rows[si] + threadIdx.x;
  const int r_end = min((c - plan.first[si] + 1) * plan.rows[si], s.n_rows);
  const bool live = r < r_end;
  const int G = Hq / Hkv, b = bh / Hkv, hkv = bh % Hkv;
  int bits = 0;
  int64_t off = 0;
  const bool ok = s.kind == UC_SEG_DENSE || head_codes(s, bh, D, bits, off);

  // the key row, dequantised, in registers
  float kr[D];
  if (live && ok) {
    if (s.kind == UC_SEG_DENSE) {
      const int64_t base = ((int64_t)bh * s.row_stride + r) * D;
#pragma unroll
      for (int d = 0; d < D; ++d) kr[d] = load_elem(s.k, s.dtype, base + d);
    } else if (r < s.n_full) {
      const int rb = D * bits / 8, Gq = s.group;
      const uint8_t* ck = s.codes_k + off + (int64_t)r * rb;
      const int mask = (1 << bits) - 1, per_byte = 8 / bits;
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int qk = (ck[d / per_byte] >> ((d % per_byte) * bits)) & mask;
        const int64_t ik = ((int64_t)bh * s.kgroups + r / Gq) * D + d;
        kr[d] = round_to(fmaf((float)qk, s.scale_k[ik], s.min_k[ik]), s.dtype);
      }
    } else {
      const int64_t base = ((int64_t)bh * s.tail_stride + (r - s.n_full)) * D;
#pragma unroll
      for (int d = 0; d < D; ++d) kr[d] = load_elem(s.tail_k, s.dtype, base + d);
    }
  } else {
#pragma unroll
    for (int d = 0; d < D; ++d) kr[d] = 0.0f;
  }

  double acc = 0.0;
  const int nq = G * W;
  for (int q0 = 0; q0 < nq; q0 += QB) {
    __syncthreads();
    for (int e = threadIdx.x; e < QB * D; e += blockDim.x) {
      const int j = e / D, d = e % D, qr = q0 + j;
      float val = 0.0f;
      if (qr < nq) {
        const int g = qr / W, w = qr % W;
        val = load_elem(q, q_dt, (((int64_t)b * Hq + hkv * G + g) * q_ld + w) * D + d) * scale_log2;
      }
      qs[j][d] = val;
    }
    if (threadIdx.x < QB) {
      const int qr = q0 + threadIdx.x;
      float lv = 0.0f;
      if (qr < nq) {
        const int g = qr / W, w = qr % W;
        lv = lse[((int64_t)b * Hq + hkv * G + g) * W + w] * kLog2e;
      }
      ls[threadIdx.x] = lv;
    }
    __syncthreads();
    const int jn = min(QB, nq - q0);
    for (int j = 0; j < jn; ++j) {
      float d = 0.0f;
#pragma unroll
      for (int e = 0; e < D; ++e) d = fmaf(qs[j][e], kr[e], d);
      acc += (double)exp2f(d - ls[j]);
    }
  }
  if (!ok) acc = __builtin_nan("");
  if (live) {
    float* sp = scores.p[si];
    if (sp) sp[(int64_t)bh * s.n_rows + r] = (float)acc;
  }
  // chunk mass (fixed-order reduction: deterministic)
  double part = live ? acc : 0.0;
  part = wave_sum_d(part);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = part;
  __syncthreads();
  if (threadIdx.x == 0 && mass_partial)
    mass_partial[(int64_t)bh * plan.n_chunks + c] = red[0] + red[1] + red[2] + red[3];
}

__global__ void mass_finalize_kernel(ChunkPlan plan, int nseg, const double* __restrict__ part,
                                     float* mass) {
  const int bh = blockIdx.x, a = threadIdx.x;
  if (a >= nseg) return;
  double s = 0.0;
  for (int c = plan.first[a]; c < plan.first[a + 1]; ++c) s += part[(int64_t)bh * plan.n_chunks + c];
  mass[(int64_t)bh * nseg + a] = (float)s;
}

// Eq. 1 bracket from attention statistics: sum over the query heads of a KV
// head and the query rows of P mass per segment = exp(seg_lse - lse).  One
// 1024-thread workgroup per (b, h_kv); each term is exp of the exact
// double-precision difference evaluated in binary32 (relative error below
// 1e-6), and the terms are summed in double.  A thread takes rows tid,
// tid + 1024, ... and issues the loads of kMassRows of them before summing,
// so the row loop waits on memory once per kMassRows rows instead of once
// per row.
constexpr int kMassRows = 8;
__global__ __launch_bounds__(1024) void segment_mass_kernel(int Hq, int Hkv, int M, int nseg,
                                                            const float* __restrict__ lse,
                                                            const float* __restrict__ seg_lse,
                                                            float* mass) {
  __shared__ double red[16][kMaxSeg];
  const int bh = blockIdx.x, b = bh / Hkv, hkv = bh % Hkv, G = Hq / Hkv;
  double acc[kMaxSeg];
  for (int a = 0; a < kMaxSeg; ++a) acc[a] = 0.0;
  const int n = G * M;
  // the G*M rows of one KV head are contiguous in lse / seg_lse
  const int64_t q0 = ((int64_t)b * Hq + hkv * G) * M;
  for (int i0 = threadIdx.x; i0 < n; i0 += kMassRows * blockDim.x) {
    float L[kMassRows], sl[kMassRows][kMaxSeg];
#pragma unroll
    for (int u = 0; u < kMassRows; ++u) {
      const int i = i0 + u * blockDim.x;
      L[u] = i < n ? lse[q0 + i] : 0.0f;
#pragma unroll
      for (int a = 0; a < kMaxSeg; ++a)
        sl[u][a] = i < n && a < nseg ? seg_lse[(q0 + i) * nseg + a] : -INFINITY;
    }
#pragma unroll
    for (int u = 0; u < kMassRows; ++u)
#pragma unroll
      for (int a = 0; a < kMaxSeg; ++a)
        if (sl[u][a] != -INFINITY) acc[a] += (double)expf((float)((double)sl[u][a] - (double)L[u]));
  }
  for (int a = 0; a < nseg; ++a) {
    double v = wave_sum_d(acc[a]);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6][a] = v;
  }
  __syncthreads();
  if (threadIdx.x < nseg) {
    const int a = threadIdx.x;
    double t = 0.0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) t += red[w][a];
    mass[(int64_t)bh * nseg + a] = (float)t;
  }
}

// Row log-sum-exps of the observation rows taken from a caller's array with
// a leading dimension: dst[r * W + w] = src[r * ld + w] for r = b * Hq + h.
__global__ void lse_rows_kernel(const float* __restrict__ src, int64_t ld, int W,
                                float* __restrict__ dst) {
  const int64_t r = blockIdx.x;
  for (int w = threadIdx.x; w < W; w += blockDim.x) dst[r * W + w] = src[r * ld + w];
}

}  // namespace

hipError_t launch_attend_generic(const uc_shape& sh, const KSegs& segs, const ChunkPlan& plan,
                                 const void* q, int q_dt, int M, float sm_scale, float* partial,
                                 bool want_o, hipStream_t st) {
  dim3 grid(plan.n_chunks, sh.B * sh.Hq, M);
  const float sl2 = sm_scale * kLog2e;
  const int ps = want_o ? sh.D + 2 : 2;
  if (sh.D == 64)
    hipLaunchKernelGGL(attend_generic_kernel<64>, grid, dim3(256), 0, st, segs, plan, q, q_dt,
                       sh.Hq, sh.Hkv, M, sl2, partial, (int)want_o, ps);
  else
    hipLaunchKernelGGL(attend_generic_kernel<128>, grid, dim3(256), 0, st, segs, plan, q, q_dt,
                       sh.Hq, sh.Hkv, M, sl2, partial, (int)want_o, ps);
  return hipGetLastError();
}

hipError_t launch_attend_combine(const uc_shape& sh, const KSegs& segs, const ChunkPlan& plan,
                                 int M, const float* partial, float* o, float* lse, float* seg_lse,
                                 hipStream_t st) {
  const int64_t Q = (int64_t)sh.B * sh.Hq * M;
  const int ps = o ? sh.D + 2 : 2;
  if (sh.D == 64)
    hipLaunchKernelGGL(attend_combine_kernel<64>, dim3((unsigned)Q), dim3(64), 0, st, plan, segs.n,
                       ps, partial, o, lse, seg_lse);
  else
    hipLaunchKernelGGL(attend_combine_kernel<128>, dim3((unsigned)Q), dim3(64), 0, st, plan,
                       segs.n, ps, partial, o, lse, seg_lse);
  return hipGetLastError();
}

hipError_t launch_score_colsum(const uc_shape& sh, const KSegs& segs, const ChunkPlan& plan,
                               const void* q, int q_dt, int W, int q_ld, float sm_scale,
                               const float* lse,
                               float* const* scores, double* mass_partial, hipStream_t st) {
  ScorePtrs sp{};
  for (int i = 0; i < segs.n; ++i) sp.p[i] = scores ? scores[i] : nullptr;
  dim3 grid(plan.n_chunks, sh.B * sh.Hkv);
  const float sl2 = sm_scale * kLog2e;
  if (sh.D == 64)
    hipLaunchKernelGGL(score_colsum_kernel<64>, grid, dim3(256), 0, st, segs, plan, q, q_dt, sh.Hq,
                       sh.Hkv, W, q_ld, sl2, lse, sp, mass_partial);
  else
    hipLaunchKernelGGL(score_colsum_kernel<128>, grid, dim3(256), 0, st, segs, plan, q, q_dt,
                       sh.Hq, sh.Hkv, W, q_ld, sl2, lse, sp, mass_partial);
  return hipGetLastError();
}

hipError_t launch_mass_finalize(const ChunkPlan& plan, int BH, int n_segs,
                                const double* mass_partial, float* mass, hipStream_t st) {
  hipLaunchKernelGGL(mass_finalize_kernel, dim3(BH), dim3(64), 0, st, plan, n_segs, mass_partial,
                     mass);
  return hipGetLastError();
}

hipError_t launch_lse_rows(const float* src, int64_t ld, int W, int rows, float* dst,
                          hipStream_t st) {
  hipLaunchKernelGGL(lse_rows_kernel, dim3(rows), dim3(256), 0, st, src, ld, W, dst);
  return hipGetLastError();
}

hipError_t launch_segment_mass(const uc_shape& sh, int M, int n_segs, const float* lse,
                               const float* seg_lse, float* mass, hipStream_t st) {
  hipLaunchKernelGGL(segment_mass_kernel, dim3(sh.B * sh.Hkv), dim3(1024), 0, st, sh.Hq, sh.Hkv,
                     M, n_segs, lse, seg_lse, mass);
  return hipGetLastError();
}

}  // namespace uc
