// select.hip -- per-KV-head top-k token selection, ordered compaction and
// row gather (App. E, "Batched GQA token selection" and "Physical, type-aware
// KV storage": heavy-hitter plus recent-token selection per KV head; only the
// retained rows and their logical indices are stored, in token order).
//
// One 1024-thread workgroup per (b, h_kv) row of scores:
//  1. radix select, 8 bits per pass over order-preserving 32-bit keys of the
//     float scores, finds the exact k'-th largest key tau (k' = k - n_recent)
//     and how many rows equal to tau must be taken;
//  2. ordered compaction: each thread owns a contiguous run of positions,
//     counts rows above tau and rows equal to tau, a block-wide exclusive scan
//     gives every run its output offset, and ties are taken lowest position
//     first -- the result is the unique set of the (score, -index) order,
//     written in ascending position;
//  3. the last n_recent positions follow unconditionally.
// The gather kernel then copies the kept K/V rows with 16-byte lanes.
#include <algorithm>
#include <cstring>

#include "uc_common.h"

namespace uc {
namespace {

constexpr int kSelThreads = 1024;

__device__ inline uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;  // -0 ranks as +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kSelWaves = kSelThreads / 64;

// Exclusive prefix over the block's waves of one value per wave (lane 0's
// x); returns it in every lane of the wave.  wave_tot holds kSelWaves words.
__device__ inline uint32_t wave_exclusive(uint32_t x, uint32_t* wave_tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) wave_tot[wave] = x;
  __syncthreads();
  uint32_t r = 0;
  for (int w = 0; w < wave; ++w) r += wave_tot[w];
  __syncthreads();
  return r;
}

// Radix select finds tau (the k'-th largest order key) 8 bits at a time:
// each wave counts the keys that match the prefix found so far in a
// histogram of its own (so hot bins, where scores share an exponent, are
// contended by 64 lanes only), the 16 histograms are summed, and one wave
// locates the digit with a scan over the bins from the top.  Compaction:
// wave w takes the w-th contiguous run of positions, reading 64 consecutive
// keys at a time; a kept key's output slot is the number of kept keys before
// it: (keys above tau before it) + min(keys equal to tau before it, need),
// from ballots within the wave and exclusive sums over the waves.
// With k_dev the row count is read from device memory (k = max(*k_dev, 0));
// k >= N then writes nothing.  Output row stride: keep_ld.
__global__ __launch_bounds__(kSelThreads) void select_kernel(const float* __restrict__ scores, int N,
                                                             int k, int n_recent,
                                                             int32_t* __restrict__ keep,
                                                             const int32_t* __restrict__ k_dev,
                                                             int64_t keep_ld) {
  __shared__ uint32_t whist[kSelWaves][256];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t wave_tot[kSelWaves];
  __shared__ uint32_t sh_digit, sh_need;
  const int bh = blockIdx.x, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  if (k_dev) {
    k = max(*k_dev, 0);
    if (k >= N) return;  // nothing evicted: the caller keeps its rows
  }
  const float* s = scores + (int64_t)bh * N;
  int32_t* out = keep + (int64_t)bh * keep_ld;
  const int Nc = N - n_recent, kc = k - n_recent;

  uint32_t prefix = 0, need = (uint32_t)kc;
  if (kc > 0) {
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      const uint32_t hi_mask = pass == 0 ? 0u : (0xFFFFFFFFu << (32 - 8 * pass));
      for (int t = lane; t < 256; t += 64) whist[wave][t] = 0u;
      __syncthreads();
      for (int i = tid; i < Nc; i += kSelThreads) {
        const uint32_t key = order_key(s[i]);
        if ((key & hi_mask) == prefix) atomicAdd(&whist[wave][(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (tid < 256) {
        uint32_t h = 0;
#pragma unroll
        for (int w = 0; w < kSelWaves; ++w) h += whist[w][tid];
        hist[tid] = h;
      }
      __syncthreads();
      if (wave == 0) {
        // lane l owns bins 255-4l .. 252-4l, taken from the top
        uint32_t c[4], tot = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          c[j] = hist[255 - 4 * lane - j];
          tot += c[j];
        }
        uint32_t inc = tot;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t y = __shfl_up(inc, o, 64);
          if (lane >= o) inc += y;
        }
        uint32_t before = inc - tot;  // keys in higher bins than this lane's
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (before < need && before + c[j] >= need) {
            sh_digit = (uint32_t)(255 - 4 * lane - j);
            sh_need = need - before;
          }
          before += c[j];
        }
      }
      __syncthreads();
      prefix |= sh_digit << shift;
      need = sh_need;
      __syncthreads();
    }
  }
  // prefix is the k'-th largest key; `need` rows equal to it are kept
  if (kc > 0) {
    const int per = (Nc + kSelWaves - 1) / kSelWaves;
    const int i0 = min(wave * per, Nc), i1 = min(i0 + per, Nc);
    uint32_t cgt = 0, ceq = 0;
    for (int b0 = i0; b0 < i1; b0 += 64) {
      const int i = b0 + lane;
      const uint32_t key = i < i1 ? order_key(s[i]) : 0u;
      cgt += (uint32_t)__popcll(__ballot(i < i1 && key > prefix));
      ceq += (uint32_t)__popcll(__ballot(i < i1 && key == prefix));
    }
    uint32_t gt = wave_exclusive(cgt, wave_tot);
    uint32_t eq = wave_exclusive(ceq, wave_tot);
    const uint64_t below = (1ull << lane) - 1ull;  // lanes before this one
    for (int b0 = i0; b0 < i1; b0 += 64) {
      const int i = b0 + lane;
      const uint32_t key = i < i1 ? order_key(s[i]) : 0u;
      const uint64_t bg = __ballot(i < i1 && key > prefix);
      const uint64_t be = __ballot(i < i1 && key == prefix);
      const uint32_t g_rank = gt + (uint32_t)__popcll(bg & below);
      const uint32_t e_rank = eq + (uint32_t)__popcll(be & below);
      if (i < i1) {
        if (key > prefix) out[g_rank + min(e_rank, need)] = i;
        else if (key == prefix && e_rank < need) out[g_rank + e_rank] = i;
      }
      gt += (uint32_t)__popcll(bg);
      eq += (uint32_t)__popcll(be);
    }
  }
  for (int j = tid; j < n_recent; j += kSelThreads) out[kc + j] = Nc + j;
}

// Copy kept rows: 16 bytes per lane; grid.y = (b, h_kv).  Row strides:
// keep_ld (indices), src_ld and dst_ld (rows); with k_dev as in select_kernel.
__global__ void gather_kernel(const int32_t* __restrict__ keep, int N, int k, const char* ksrc,
                              const char* vsrc, char* kdst, char* vdst, int row_bytes,
                              const int32_t* __restrict__ k_dev, int64_t keep_ld, int64_t src_ld,
                              int64_t dst_ld) {
  const int bh = blockIdx.y;
  if (k_dev) {
    k = max(*k_dev, 0);
    if (k >= N) return;
  }
  const int lanes_per_row = row_bytes / 16;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)k * lanes_per_row) return;
  const int j = (int)(e / lanes_per_row), piece = (int)(e % lanes_per_row);
  const int src_row = keep[(int64_t)bh * keep_ld + j];
  if (src_row < 0 || src_row >= N) return;
  const int64_t so = ((int64_t)bh * src_ld + src_row) * row_bytes + piece * 16;
  const int64_t dof = ((int64_t)bh * dst_ld + j) * row_bytes + piece * 16;
  *reinterpret_cast<uint4*>(kdst + dof) = *reinterpret_cast<const uint4*>(ksrc + so);
  *reinterpret_cast<uint4*>(vdst + dof) = *reinterpret_cast<const uint4*>(vsrc + so);
}

// Fraction of a row's score mass on its k selected positions (double sums).
__global__ void topk_fraction_kernel(const float* __restrict__ scores,
                                     const int32_t* __restrict__ keep, int N, int k,
                                     float* __restrict__ frac) {
  __shared__ double red[2][4];
  const int r = blockIdx.x;
  const float* s = scores + (int64_t)r * N;
  double top = 0.0, all = 0.0;
  for (int j = threadIdx.x; j < k; j += blockDim.x) top += s[keep[(int64_t)r * k + j]];
  for (int i = threadIdx.x; i < N; i += blockDim.x) all += s[i];
  top = wave_sum_d(top);
  all = wave_sum_d(all);
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = top;
    red[1][threadIdx.x >> 6] = all;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const double t = red[0][0] + red[0][1] + red[0][2] + red[0][3];
    const double a = red[1][0] + red[1][1] + red[1][2] + red[1][3];
    frac[r] = a > 0.0 ? (float)(t / a) : 0.0f;
  }
}

// Host bytes carried in the kernel arguments and stored to device memory:
// small descriptor tables reach the GPU in stream order with no staging copy
// or host synchronisation.
constexpr int kBlobWords = 760;
struct Blob {
  uint32_t w[kBlobWords];
};
__global__ void blob_store_kernel(Blob b, int n, uint32_t* __restrict__ dst) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) dst[i] = b.w[i];
}

// out[bh, j] = outer[bh, inner[bh, j]] (-1 for an inner value out of range);
// rows of outer, inner and out are outer_ld, inner_ld and out_ld apart.  An
// element is read before it is written, so out may be inner (in place).
// outer NULL: out = inner (the inner indices are already logical).  With
// k_dev as in select_kernel (n_outer playing N).
__global__ void compose_index_kernel(const int32_t* outer, int n_outer, const int32_t* inner,
                                     int k, int32_t* out, const int32_t* __restrict__ k_dev,
                                     int64_t outer_ld, int64_t inner_ld, int64_t out_ld) {
  const int bh = blockIdx.y;
  if (k_dev) {
    k = max(*k_dev, 0);
    if (k >= n_outer) return;
  }
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= k) return;
  const int i = inner[(int64_t)bh * inner_ld + j];
  const int r = !outer ? i : (i >= 0 && i < n_outer) ? outer[(int64_t)bh * outer_ld + i] : -1;
  out[(int64_t)bh * out_ld + j] = r;
}

// Decode append: rows pos..pos+n_new-1 of a dense segment.
__global__ void append_kernel(const char* knew, const char* vnew, int n_new, char* kd, char* vd,
                              int row_stride, int pos, int row_bytes) {
  const int bh = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per_bh = (int64_t)n_new * row_bytes / 16;
  if (e >= per_bh) return;
  const int64_t src = (int64_t)bh * n_new * row_bytes + e * 16;
  const int64_t dst = ((int64_t)bh * row_stride + pos) * row_bytes + e * 16;
  *reinterpret_cast<uint4*>(kd + dst) = *reinterpret_cast<const uint4*>(knew + src);
  *reinterpret_cast<uint4*>(vd + dst) = *reinterpret_cast<const uint4*>(vnew + src);
}

}  // namespace

hipError_t launch_select(const float* scores, int BH, int N, int k, int n_recent, int32_t* keep,
                         hipStream_t st) {
  hipLaunchKernelGGL(select_kernel, dim3(BH), dim3(kSelThreads), 0, st, scores, N, k, n_recent,
                     keep, nullptr, (int64_t)k);
  return hipGetLastError();
}

hipError_t launch_gather(const int32_t* keep, int BH, int N, int k, const void* ksrc,
                         const void* vsrc, void* kdst, void* vdst, int elem_bytes, int D,
                         hipStream_t st) {
  const int row_bytes = D * elem_bytes;
  const int64_t lanes = (int64_t)k * (row_bytes / 16);
  if (lanes == 0) return hipSuccess;
  hipLaunchKernelGGL(gather_kernel, dim3((unsigned)((lanes + 255) / 256), BH), dim3(256), 0, st,
                     keep, N, k, (const char*)ksrc, (const char*)vsrc, (char*)kdst, (char*)vdst,
                     row_bytes, nullptr, (int64_t)k, (int64_t)N, (int64_t)k);
  return hipGetLastError();
}

hipError_t launch_topk_mass(const float* scores, int BH, int N, int k, float* frac,
                            int32_t* keep, hipStream_t st) {
  if (k > 0) {
    hipError_t e = launch_select(scores, BH, N, k, 0, keep, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(topk_fraction_kernel, dim3(BH), dim3(256), 0, st, scores, keep, N, k, frac);
  return hipGetLastError();
}

hipError_t launch_blob_upload(const void* host, size_t bytes, void* dev, hipStream_t st) {
  // bytes is a multiple of 4 (descriptor tables of ints and pointers)
  const uint32_t* src = (const uint32_t*)host;
  const size_t words = bytes / 4;
  for (size_t i = 0; i < words; i += kBlobWords) {
    const int n = (int)std::min<size_t>(kBlobWords, words - i);
    Blob b;
    memcpy(b.w, src + i, (size_t)n * 4);
    hipLaunchKernelGGL(blob_store_kernel, dim3(1), dim3(256), 0, st, b, n, (uint32_t*)dev + i);
  }
  return hipGetLastError();
}

hipError_t launch_compose_index(const int32_t* outer, int n_outer, const int32_t* inner, int BH,
                                int k, int32_t* out, hipStream_t st) {
  if (k == 0 || BH == 0) return hipSuccess;
  hipLaunchKernelGGL(compose_index_kernel, dim3((k + 255) / 256, BH), dim3(256), 0, st, outer,
                     n_outer, inner, k, out, nullptr, (int64_t)n_outer, (int64_t)k, (int64_t)k);
  return hipGetLastError();
}

hipError_t launch_evict_step(int BH, int N, const float* scores, const int32_t* k_dev,
                             const void* ksrc, const void* vsrc, int64_t src_ld,
                             const int32_t* idx_src, void* kdst, void* vdst, int32_t* idx_dst,
                             int64_t dst_ld, int row_bytes, hipStream_t st) {
  if (N == 0) return hipSuccess;  // k >= N whatever k is
  hipLaunchKernelGGL(select_kernel, dim3(BH), dim3(kSelThreads), 0, st, scores, N, 0, 0, idx_dst,
                     k_dev, dst_ld);
  const int64_t lanes = (int64_t)N * (row_bytes / 16);  // grid for k = N - 1 at most
  hipLaunchKernelGGL(gather_kernel, dim3((unsigned)((lanes + 255) / 256), BH), dim3(256), 0, st,
                     (const int32_t*)idx_dst, N, 0, (const char*)ksrc, (const char*)vsrc,
                     (char*)kdst, (char*)vdst, row_bytes, k_dev, dst_ld, src_ld, dst_ld);
  // local positions -> logical indices, in place
  hipLaunchKernelGGL(compose_index_kernel, dim3((N + 255) / 256, BH), dim3(256), 0, st, idx_src, N,
                     (const int32_t*)idx_dst, 0, idx_dst, k_dev, src_ld, dst_ld, dst_ld);
  return hipGetLastError();
}

hipError_t launch_append(const uc_shape& sh, const void* knew, const void* vnew, int n_new,
                         const KSeg& seg, int pos, hipStream_t st) {
  const int row_bytes = sh.D * dtype_bytes(seg.dtype);
  const int64_t lanes = (int64_t)n_new * row_bytes / 16;
  if (lanes == 0) return hipSuccess;
  hipLaunchKernelGGL(append_kernel, dim3((unsigned)((lanes + 255) / 256), sh.B * sh.Hkv), dim3(256),
                     0, st, (const char*)knew, (const char*)vnew, n_new, (char*)seg.k,
                     (char*)seg.v, seg.row_stride, pos, row_bytes);
  return hipGetLastError();
}

}  // namespace uc
