// quantize.hip -- group-wise asymmetric min/max quantization of one segment
// into packed low-bit codes, float scales/minima and a residual tail
// (App. E, "Physical, type-aware KV storage").
//
//   keys:   one channel over G consecutive rows     (per-channel groups)
//   values: G consecutive channels of one row       (per-token groups)
//   mn = min, mx = max, s = (mx - mn) / (2^b - 1)
//   code = s > 0 ? clamp(rint((x - mn) / s), 0, 2^b - 1) : 0
// All in IEEE binary32 with correctly rounded division and no contraction, so
// codes and scales are reproducible bit for bit.
//
// Layout of the output (see unicache.h): row r of a head's codes occupies
// D*b/8 bytes; channel c sits in byte c*b/8 at bit (c % (8/b))*b.  One lane
// owns one channel; lanes of one 32-bit word (32/b consecutive channels)
// OR their shifted codes together with cross-lane shuffles and the first lane
// of the word stores it, so each row's codes leave as coalesced 32-bit stores.
#pragma clang fp contract(off)

#include "uc_common.h"

namespace uc {
namespace {

__device__ inline int quant_code(float x, float mn, float s, int qmax) {
  if (!(s > 0.0f)) return 0;
  float t = __fdiv_rn(x - mn, s);
  int c = (int)rintf(t);
  return min(max(c, 0), qmax);
}

// OR-combine the shifted codes of the 32/b lanes that share a word; returns
// the word in every lane of the group.
__device__ inline uint32_t pack_word(int code, int c, int b) {
  const int cpw = 32 / b;
  uint32_t w = (uint32_t)code << ((c % cpw) * b);
  for (int o = 1; o < cpw; o <<= 1) w |= (uint32_t)__shfl_xor((int)w, o, 64);
  return w;
}

// Keys: block = D threads (one per channel), one block per (row group, bh).
__global__ void quantize_k_kernel(KSeg seg, const void* __restrict__ k, int dt, int N, int D) {
  const int g = blockIdx.x, bh = blockIdx.y, c = threadIdx.x;
  const int G = seg.group;
  int b;
  int64_t off;
  float* scale = const_cast<float*>(seg.scale_k) + ((int64_t)bh * seg.kgroups + g) * D + c;
  float* mnp = const_cast<float*>(seg.min_k) + ((int64_t)bh * seg.kgroups + g) * D + c;
  if (!head_codes(seg, bh, D, b, off) || (off & 15)) {
    *scale = __builtin_nanf("");
    return;
  }
  const int qmax = (1 << b) - 1;
  const int64_t base = ((int64_t)bh * N + (int64_t)g * G) * D + c;
  float mn = load_elem(k, dt, base), mx = mn;
  for (int r = 1; r < G; ++r) {
    float x = load_elem(k, dt, base + (int64_t)r * D);
    mn = fminf(mn, x);
    mx = fmaxf(mx, x);
  }
  const float s = __fdiv_rn(mx - mn, (float)qmax);
  *scale = s;
  *mnp = mn;
  const int row_bytes = D * b / 8;
  uint8_t* codes = const_cast<uint8_t*>(seg.codes_k) + off + (int64_t)g * G * row_bytes;
  const int cpw = 32 / b;
  for (int r = 0; r < G; ++r) {
    int code = quant_code(load_elem(k, dt, base + (int64_t)r * D), mn, s, qmax);
    uint32_t w = pack_word(code, c, b);
    if (c % cpw == 0) *reinterpret_cast<uint32_t*>(codes + (int64_t)r * row_bytes + c * b / 8) = w;
  }
}

// Values: block = 256 threads = (256 / D) rows x D channels; group min/max
// through LDS.
__global__ void quantize_v_kernel(KSeg seg, const void* __restrict__ v, int dt, int N, int D) {
  __shared__ float xs[256];
  __shared__ float ss[256], ms[256];
  const int rows_per_block = 256 / D;
  const int lr = threadIdx.x / D, c = threadIdx.x % D;
  const int r = blockIdx.x * rows_per_block + lr, bh = blockIdx.y;
  const int G = seg.group, ngv = D / G;
  int b;
  int64_t off;
  const bool ok = head_codes(seg, bh, D, b, off) && !(off & 15);
  const bool live = r < seg.n_full;
  float x = live ? load_elem(v, dt, ((int64_t)bh * N + r) * D + c) : 0.0f;
  xs[threadIdx.x] = x;
  __syncthreads();
  if (live && c % G == 0) {
    float mn = xs[threadIdx.x], mx = mn;
    for (int i = 1; i < G; ++i) {
      float y = xs[threadIdx.x + i];
      mn = fminf(mn, y);
      mx = fmaxf(mx, y);
    }
    const float s = ok ? __fdiv_rn(mx - mn, (float)((1 << b) - 1)) : __builtin_nanf("");
    ss[threadIdx.x] = s;
    ms[threadIdx.x] = mn;
    const int64_t mi = ((int64_t)bh * seg.cap_full + r) * ngv + c / G;
    const_cast<float*>(seg.scale_v)[mi] = s;
    const_cast<float*>(seg.min_v)[mi] = mn;
  }
  __syncthreads();
  if (!ok) return;  // uniform over the block: bh is per block
  const int gl = threadIdx.x - (c % G);
  const int code = live ? quant_code(x, ms[gl], ss[gl], (1 << b) - 1) : 0;
  const uint32_t w = pack_word(code, c, b);
  const int cpw = 32 / b;
  if (live && c % cpw == 0) {
    const int row_bytes = D * b / 8;
    uint8_t* codes = const_cast<uint8_t*>(seg.codes_v) + off + (int64_t)r * row_bytes;
    *reinterpret_cast<uint32_t*>(codes + c * b / 8) = w;
  }
}

// ---- vectorised forms for 2-byte dtypes and head dims 64 / 128: a lane
// holds 8 consecutive channels of a row (one 16-byte load) and writes their
// 8 codes as one 16-, 32- or 64-bit store.  Min and max are exact and the
// scale, division and rounding are those of quant_code, so the results are
// the same bits as the per-element forms above.

// 8 channels starting at element e (16-byte aligned) as floats
__device__ inline void load8(const void* p, int dt, int64_t e, float (&x)[8]) {
  const uint4 w = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(p) + e);
  const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint16_t lo = (uint16_t)(u[j] & 0xFFFFu), hi = (uint16_t)(u[j] >> 16);
    x[2 * j] = dt == UC_BF16 ? bf16_to_f32(lo) : f16_to_f32(lo);
    x[2 * j + 1] = dt == UC_BF16 ? bf16_to_f32(hi) : f16_to_f32(hi);
  }
}

// the b-bit codes of 8 consecutive channels (channel e at bit b*e) stored at p
__device__ inline void store_codes8(uint8_t* p, const int (&code)[8], int b) {
  uint64_t w = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) w |= (uint64_t)code[e] << (b * e);
  if (b == 2) *reinterpret_cast<uint16_t*>(p) = (uint16_t)w;
  else if (b == 4) *reinterpret_cast<uint32_t*>(p) = (uint32_t)w;
  else *reinterpret_cast<uint64_t*>(p) = w;
}

// Values, group G >= 8: a group is G/8 neighbouring lanes of one row; its
// min and max combine by shuffles.  Block = 256 lanes = 256/(D/8) rows.
__global__ __launch_bounds__(256) void quantize_v_vec_kernel(KSeg seg, const void* __restrict__ v,
                                                             int dt, int N, int D) {
  const int cpr = D / 8;  // lanes per row
  const int c8 = threadIdx.x % cpr;
  const int r = blockIdx.x * (256 / cpr) + threadIdx.x / cpr, bh = blockIdx.y;
  const int G = seg.group, lpg = G / 8;
  int b;
  int64_t off;
  const bool ok = head_codes(seg, bh, D, b, off) && !(off & 15);
  const bool live = r < seg.n_full;
  float x[8];
  if (live) {
    load8(v, dt, ((int64_t)bh * N + r) * D + c8 * 8, x);
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = 0.0f;
  }
  float mn = x[0], mx = x[0];
#pragma unroll
  for (int e = 1; e < 8; ++e) {
    mn = fminf(mn, x[e]);
    mx = fmaxf(mx, x[e]);
  }
  // the lanes of a group are aligned and lie in one row, so rows past n_full
  // only combine among themselves
  for (int o = 1; o < lpg; o <<= 1) {
    mn = fminf(mn, __shfl_xor(mn, o, 64));
    mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  }
  const int qmax = ok ? (1 << b) - 1 : 1;
  const float s = ok ? __fdiv_rn(mx - mn, (float)qmax) : __builtin_nanf("");
  if (!live) return;
  if (c8 % lpg == 0) {
    const int64_t mi = ((int64_t)bh * seg.cap_full + r) * (D / G) + c8 / lpg;
    const_cast<float*>(seg.scale_v)[mi] = s;
    const_cast<float*>(seg.min_v)[mi] = mn;
  }
  if (!ok) return;
  int code[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) code[e] = quant_code(x[e], mn, s, qmax);
  store_codes8(const_cast<uint8_t*>(seg.codes_v) + off + (int64_t)r * (D * b / 8) + c8 * b, code,
               b);
}

// Keys: one block of 256 lanes per (row group, bh); a lane holds 8 channels
// of rows rr, rr + RB, ... of the group (RB = 256/(D/8) rows per pass, at
// most 8 rows per lane since G <= D); per-channel min and max combine over
// the lanes of a wave by shuffles, then over the four waves through LDS.
__global__ __launch_bounds__(256) void quantize_k_vec_kernel(KSeg seg, const void* __restrict__ k,
                                                             int dt, int N, int D) {
  __shared__ float red[2][4][128];
  const int cpr = D / 8, RB = 256 / cpr;
  const int c8 = threadIdx.x % cpr, rr = threadIdx.x / cpr;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = blockIdx.x, bh = blockIdx.y, G = seg.group;
  int b;
  int64_t off;
  float* scale = const_cast<float*>(seg.scale_k) + ((int64_t)bh * seg.kgroups + g) * D + c8 * 8;
  float* mnp = const_cast<float*>(seg.min_k) + ((int64_t)bh * seg.kgroups + g) * D + c8 * 8;
  if (!head_codes(seg, bh, D, b, off) || (off & 15)) {  // uniform over the block
    if (rr == 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) scale[e] = __builtin_nanf("");
    }
    return;
  }
  const int qmax = (1 << b) - 1;
  const int64_t base = ((int64_t)bh * N + (int64_t)g * G) * D + c8 * 8;
  uint4 raw[8];
  float mn[8], mx[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    mn[e] = INFINITY;
    mx[e] = -INFINITY;
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = rr + i * RB;
    if (r < G) {
      raw[i] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(k) + base +
                                               (int64_t)r * D);
      float x[8];
      load8(k, dt, base + (int64_t)r * D, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        mn[e] = fminf(mn[e], x[e]);
        mx[e] = fmaxf(mx[e], x[e]);
      }
    }
  }
  for (int o = cpr; o < 64; o <<= 1) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      mn[e] = fminf(mn[e], __shfl_xor(mn[e], o, 64));
      mx[e] = fmaxf(mx[e], __shfl_xor(mx[e], o, 64));
    }
  }
  if (lane < cpr) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      red[0][wave][c8 * 8 + e] = mn[e];
      red[1][wave][c8 * 8 + e] = mx[e];
    }
  }
  __syncthreads();
  float s[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float a = red[0][0][c8 * 8 + e], z = red[1][0][c8 * 8 + e];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      a = fminf(a, red[0][w][c8 * 8 + e]);
      z = fmaxf(z, red[1][w][c8 * 8 + e]);
    }
    mn[e] = a;
    s[e] = __fdiv_rn(z - a, (float)qmax);
  }
  if (rr == 0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      scale[e] = s[e];
      mnp[e] = mn[e];
    }
  }
  const int row_bytes = D * b / 8;
  uint8_t* codes = const_cast<uint8_t*>(seg.codes_k) + off + (int64_t)g * G * row_bytes + c8 * b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int r = rr + i * RB;
    if (r < G) {
      const uint32_t u[4] = {raw[i].x, raw[i].y, raw[i].z, raw[i].w};
      int code[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint16_t lo = (uint16_t)(u[j] & 0xFFFFu), hi = (uint16_t)(u[j] >> 16);
        const float x0 = dt == UC_BF16 ? bf16_to_f32(lo) : f16_to_f32(lo);
        const float x1 = dt == UC_BF16 ? bf16_to_f32(hi) : f16_to_f32(hi);
        code[2 * j] = quant_code(x0, mn[2 * j], s[2 * j], qmax);
        code[2 * j + 1] = quant_code(x1, mn[2 * j + 1], s[2 * j + 1], qmax);
      }
      store_codes8(codes + (int64_t)r * row_bytes, code, b);
    }
  }
}

// Residual tail: rows n_full..N-1 copied unchanged (16 bytes per lane).
__global__ void copy_tail_kernel(KSeg seg, const void* __restrict__ k, const void* __restrict__ v,
                                 int N, int row_bytes) {
  const int bh = blockIdx.y;
  const int64_t tail_bytes = (int64_t)seg.tail_len * row_bytes;
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 16;
  if (i >= tail_bytes) return;
  const int64_t src = ((int64_t)bh * N + seg.n_full) * row_bytes + i;
  const int64_t dst = (int64_t)bh * seg.tail_stride * row_bytes + i;
  *reinterpret_cast<uint4*>((char*)seg.tail_k + dst) =
      *reinterpret_cast<const uint4*>((const char*)k + src);
  *reinterpret_cast<uint4*>((char*)seg.tail_v + dst) =
      *reinterpret_cast<const uint4*>((const char*)v + src);
}

// Dequantisation of a whole packed segment into dense rows of its dtype:
// one thread per (row, channel) element of one (b, h_kv) (blockIdx.y);
// rows < n_full decode their code, tail rows are copied.
__global__ void dequantize_kernel(KSeg s, void* __restrict__ kout, void* __restrict__ vout,
                                  int D) {
  const int bh = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int N = s.n_rows;
  if (e >= (int64_t)N * D) return;
  const int r = (int)(e / D), c = (int)(e % D);
  const int64_t o = (int64_t)bh * N * D + e;
  float xk, xv;
  if (r >= s.n_full) {
    const int64_t t = ((int64_t)bh * s.tail_stride + (r - s.n_full)) * D + c;
    xk = load_elem(s.tail_k, s.dtype, t);
    xv = load_elem(s.tail_v, s.dtype, t);
  } else {
    int b;
    int64_t off;
    if (!head_codes(s, bh, D, b, off)) {
      xk = xv = __builtin_nanf("");
    } else {
      const int G = s.group, ngv = D / G;
      const int64_t byte = off + (int64_t)r * (D * b / 8) + c * b / 8;
      const int shift = (c % (8 / b)) * b, mask = (1 << b) - 1;
      const int ck = (s.codes_k[byte] >> shift) & mask;
      const int cv = (s.codes_v[byte] >> shift) & mask;
      const int64_t ki = ((int64_t)bh * s.kgroups + r / G) * D + c;
      const int64_t vi = ((int64_t)bh * s.cap_full + r) * ngv + c / G;
      xk = round_to(__builtin_fmaf((float)ck, s.scale_k[ki], s.min_k[ki]), s.dtype);
      xv = round_to(__builtin_fmaf((float)cv, s.scale_v[vi], s.min_v[vi]), s.dtype);
    }
  }
  if (s.dtype == UC_F32) {
    static_cast<float*>(kout)[o] = xk;
    static_cast<float*>(vout)[o] = xv;
  } else if (s.dtype == UC_BF16) {
    static_cast<uint16_t*>(kout)[o] = f32_to_bf16_bits(xk);
    static_cast<uint16_t*>(vout)[o] = f32_to_bf16_bits(xv);
  } else {
    static_cast<uint16_t*>(kout)[o] = f32_to_f16_bits(xk);
    static_cast<uint16_t*>(vout)[o] = f32_to_f16_bits(xv);
  }
}

// Streaming append: rows j0 .. j0+n-1 of each head's new rows (n_new per
// head) go to tail rows pos .. pos+n-1 (16 bytes per lane).
__global__ void stream_copy_kernel(const char* __restrict__ knew, const char* __restrict__ vnew,
                                   int n_new, int j0, int n, char* tk, char* tv, int tail_stride,
                                   int pos, int row_bytes) {
  const int bh = blockIdx.y;
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 16;
  if (i >= (int64_t)n * row_bytes) return;
  const int64_t src = ((int64_t)bh * n_new + j0) * row_bytes + i;
  const int64_t dst = ((int64_t)bh * tail_stride + pos) * row_bytes + i;
  *reinterpret_cast<uint4*>(tk + dst) = *reinterpret_cast<const uint4*>(knew + src);
  *reinterpret_cast<uint4*>(tv + dst) = *reinterpret_cast<const uint4*>(vnew + src);
}

}  // namespace

// Rows enter the tail; whenever it holds G rows they are quantised in place
// as the next row group of the codes and scales (a view of the segment whose
// storage starts at that group; the strides stay the segment's) and the tail
// empties.
hipError_t launch_stream_append(const uc_shape& sh, const KSeg& seg, const void* knew,
                                const void* vnew, int n_new, hipStream_t st) {
  const int G = seg.group, D = sh.D, BH = sh.B * sh.Hkv;
  const int row_bytes = D * dtype_bytes(seg.dtype), code_row = D * seg.bits / 8;
  int n_full = seg.n_full, tail = seg.tail_len;
  for (int j = 0; j < n_new;) {
    const int take = min(G - tail, n_new - j);
    const int64_t lanes = (int64_t)take * row_bytes / 16;
    hipLaunchKernelGGL(stream_copy_kernel, dim3((unsigned)((lanes + 255) / 256), BH), dim3(256), 0,
                       st, (const char*)knew, (const char*)vnew, n_new, j, take,
                       (char*)seg.tail_k, (char*)seg.tail_v, seg.tail_stride, tail, row_bytes);
    j += take;
    tail += take;
    if (tail == G) {
      KSeg v = seg;
      v.n_rows = v.n_full = G;
      v.tail_len = 0;
      v.codes_k = seg.codes_k + (int64_t)n_full * code_row;
      v.codes_v = seg.codes_v + (int64_t)n_full * code_row;
      v.codes_bytes = seg.codes_bytes - (uint64_t)n_full * code_row;
      v.scale_k = seg.scale_k + (int64_t)(n_full / G) * D;
      v.min_k = seg.min_k + (int64_t)(n_full / G) * D;
      v.scale_v = seg.scale_v + (int64_t)n_full * (D / G);
      v.min_v = seg.min_v + (int64_t)n_full * (D / G);
      hipError_t e = launch_quantize(sh, seg.tail_k, seg.tail_v, seg.dtype, G, v, st);
      if (e != hipSuccess) return e;
      n_full += G;
      tail = 0;
    }
  }
  return hipGetLastError();
}

hipError_t launch_dequantize(const uc_shape& sh, const KSeg& seg, void* kout, void* vout,
                             hipStream_t st) {
  const int64_t n = (int64_t)seg.n_rows * sh.D;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(dequantize_kernel, dim3((unsigned)((n + 255) / 256), sh.B * sh.Hkv),
                     dim3(256), 0, st, seg, kout, vout, sh.D);
  return hipGetLastError();
}

hipError_t launch_quantize(const uc_shape& sh, const void* k, const void* v, int dt, int N,
                           const KSeg& out, hipStream_t st) {
  const int BH = sh.B * sh.Hkv, D = sh.D;
  if (out.n_full > 0) {
    // vectorised forms: 2-byte dtypes, head dim 64 or 128, 16-byte aligned
    // rows (values also need groups of at least 8 channels)
    const bool vec = dt != UC_F32 && (D == 64 || D == 128) && !((uintptr_t)k & 15) &&
                     !((uintptr_t)v & 15);
    if (vec)
      hipLaunchKernelGGL(quantize_k_vec_kernel, dim3(out.n_full / out.group, BH), dim3(256), 0, st,
                         out, k, dt, N, D);
    else
      hipLaunchKernelGGL(quantize_k_kernel, dim3(out.n_full / out.group, BH), dim3(D), 0, st, out,
                         k, dt, N, D);
    if (vec && out.group >= 8) {
      const int rpb = 256 / (D / 8);
      hipLaunchKernelGGL(quantize_v_vec_kernel, dim3((out.n_full + rpb - 1) / rpb, BH), dim3(256),
                         0, st, out, v, dt, N, D);
    } else {
      const int rpb = 256 / D;
      hipLaunchKernelGGL(quantize_v_kernel, dim3((out.n_full + rpb - 1) / rpb, BH), dim3(256), 0,
                         st, out, v, dt, N, D);
    }
  }
  if (out.tail_len > 0) {
    const int row_bytes = D * dtype_bytes(dt);
    const int64_t lanes = ((int64_t)out.tail_len * row_bytes + 15) / 16;
    hipLaunchKernelGGL(copy_tail_kernel, dim3((unsigned)((lanes + 255) / 256), BH), dim3(256), 0,
                       st, out, k, v, N, row_bytes);
  }
  return hipGetLastError();
}

}  // namespace uc
