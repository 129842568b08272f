// uc_common.h -- internal definitions shared by the library's kernels and its
// host-side entry points (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "unicache.h"

namespace uc {

constexpr int kMaxSeg = UC_MAX_SEGMENTS;
// bytes that hold the prepared views of one multi-query attention call
constexpr size_t kPrefillViewBytes = 1024;

// compute units of the current device (cached after the first call)
int device_cus();

// Kernel-side copy of one segment descriptor, passed by value in kernel
// arguments.  Derived fields (n_full, tail_len, row_stride) are resolved on
// the host.
struct KSeg {
  int kind, dtype, n_rows, row_stride;
  int group, bits, n_full, tail_len;
  // packed strides per (b, h_kv): rows of code / value-scale storage, key
  // scale groups, tail rows (n_full, n_full/G, tail_len without a capacity)
  int cap_full, kgroups, tail_stride;
  const void* k;
  const void* v;
  const uint8_t* head_bits;
  const int64_t* code_off;
  uint64_t codes_bytes;
  const uint8_t* codes_k;
  const uint8_t* codes_v;
  const float* scale_k;
  const float* min_k;
  const float* scale_v;
  const float* min_v;
  const void* tail_k;
  const void* tail_v;
};

struct KSegs {
  KSeg s[kMaxSeg];
  int n;
};

// Decode append fused into the decode kernel: rows pos .. pos+n_new-1 of
// every (b, h_kv) of a dense segment receive k_new / v_new [BH, n_new, row]
// (the first workgroup of each (b, h_kv) copies them); n_new = 0: none.
struct AppendOp {
  const char* kn;
  const char* vn;
  char* kd;
  char* vd;
  int n_new, row_stride, pos, row_bytes;
};

// Batched requests: request r's segments are flat[first .. first + n - 1]
// (one-request layouts); table, grid entries and flat live in the workspace.
struct BatchDesc {
  int first, n;
  int W;      // the request's workgroups per KV head (by its share of the bytes)
  int split;  // segment taken around the others (staggered packed phases), or -1
};

// A run of the one-dimensional grid: workgroups start .. start + Hkv*nw - 1
// are workgroups w0 .. w0 + nw - 1 of every KV head of request req.  With
// two runs per request the first holds its early half (dispatched in the
// launch's first half), the second its late half.
struct BatchGrid {
  int start, req, w0, nw;
};

// A batch of at most kArgReq requests and kArgSeg segments in all travels
// in the attention kernel's arguments (11.8 KB) instead of being stored
// into the workspace by separate launches first.
constexpr int kArgReq = 32, kArgSeg = 64;
struct BatchArgs {
  BatchDesc table[kArgReq];
  BatchGrid grid[2 * kArgReq];
  KSeg flat[kArgSeg];
};

// Split of every segment's rows into chunks (work items of the split-K
// attention and of the scoring passes); chunks never straddle segments.
struct ChunkPlan {
  int n_chunks;
  int first[kMaxSeg + 1];  // first chunk of segment s; first[n] = n_chunks
  int rows[kMaxSeg];       // rows per chunk of segment s
};

__host__ __device__ inline int dtype_bytes(int dt) { return dt == UC_F32 ? 4 : 2; }

// ---- element conversions --------------------------------------------------
__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ inline float f16_to_f32(uint16_t h) {
  _Float16 f;
  __builtin_memcpy(&f, &h, 2);
  return (float)f;
}

// binary32 -> bf16 bits, round to nearest even (NaN stays NaN)
__device__ inline uint16_t f32_to_bf16_bits(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ inline uint16_t f32_to_f16_bits(float x) {
  _Float16 f = (_Float16)x;  // v_cvt_f16_f32: round to nearest even
  uint16_t h;
  __builtin_memcpy(&h, &f, 2);
  return h;
}

__device__ inline float load_elem(const void* p, int dt, int64_t i) {
  if (dt == UC_F32) return static_cast<const float*>(p)[i];
  uint16_t h = static_cast<const uint16_t*>(p)[i];
  return dt == UC_BF16 ? bf16_to_f32(h) : f16_to_f32(h);
}

// value of x after rounding to dtype dt
__device__ inline float round_to(float x, int dt) {
  if (dt == UC_F32) return x;
  if (dt == UC_BF16) return bf16_to_f32(f32_to_bf16_bits(x));
  return f16_to_f32(f32_to_f16_bits(x));
}

// Resolve where one (b, h_kv)'s codes live; false if the device-side values
// are outside the segment's capacities (the head is then skipped).
__device__ inline bool head_codes(const KSeg& s, int bh, int D, int& bits, int64_t& off) {
  if (s.head_bits) {
    bits = s.head_bits[bh];
    off = s.code_off[bh];
  } else {
    bits = s.bits;
    off = s.code_off ? s.code_off[bh] : (int64_t)bh * s.cap_full * D * s.bits / 8;
  }
  // per-head widths are bounded by the segment's bits (kernels are chosen by it)
  if (bits != 2 && bits != 4 && bits != 8) return false;
  if (s.head_bits && bits > s.bits) return false;
  int64_t need = (int64_t)s.n_full * D * bits / 8;
  return off >= 0 && (uint64_t)(off + need) <= s.codes_bytes;
}

// ---- wave helpers (64 lanes) ------------------------------------------------
__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ inline float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ inline double wave_sum_d(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

}  // namespace uc

// ---- launchers implemented in the kernel translation units -------------------
namespace uc {
// Events bracketing the attention kernel of the current uc_attend_mixed call
// (null when timing was not requested); the launchers call these around the
// kernel that reads the segments.
hipError_t kernel_timer_begin(hipStream_t st);
hipError_t kernel_timer_end(hipStream_t st);

hipError_t launch_quantize(const uc_shape& sh, const void* k, const void* v, int dt, int N,
                           const KSeg& out, hipStream_t st);
hipError_t launch_dequantize(const uc_shape& sh, const KSeg& seg, void* kout, void* vout,
                             hipStream_t st);
hipError_t launch_stream_append(const uc_shape& sh, const KSeg& seg, const void* knew,
                                const void* vnew, int n_new, hipStream_t st);
hipError_t launch_topk_mass(const float* scores, int BH, int N, int k, float* frac,
                            int32_t* keep, hipStream_t st);
hipError_t launch_blob_upload(const void* host, size_t bytes, void* dev, hipStream_t st);
hipError_t launch_compose_index(const int32_t* outer, int n_outer, const int32_t* inner, int BH,
                                int k, int32_t* out, hipStream_t st);
hipError_t launch_attend_generic(const uc_shape& sh, const KSegs& segs, const ChunkPlan& plan,
                                 const void* q, int q_dt, int M, float sm_scale, float* partial,
                                 bool want_o, hipStream_t st);
hipError_t launch_attend_combine(const uc_shape& sh, const KSegs& segs, const ChunkPlan& plan,
                                 int M, const float* partial, float* o, float* lse, float* seg_lse,
                                 hipStream_t st);
hipError_t launch_score_colsum(const uc_shape& sh, const KSegs& segs, const ChunkPlan& plan,
                               const void* q, int q_dt, int W, int q_ld, float sm_scale,
                               const float* lse,
                               float* const* scores, double* mass_partial, hipStream_t st);
hipError_t launch_mass_finalize(const ChunkPlan& plan, int BH, int n_segs,
                                const double* mass_partial, float* mass, hipStream_t st);
hipError_t launch_select(const float* scores, int BH, int N, int k, int n_recent, int32_t* keep,
                         hipStream_t st);
hipError_t launch_gather(const int32_t* keep, int BH, int N, int k, const void* ksrc,
                         const void* vsrc, void* kdst, void* vdst, int elem_bytes, int D,
                         hipStream_t st);
hipError_t launch_append(const uc_shape& sh, const void* knew, const void* vnew, int n_new,
                         const KSeg& seg, int pos, hipStream_t st);
hipError_t launch_budget_step(const uc_budget_params& p, const float* mass, int n_steps,
                              uc_budget_state* state, hipStream_t st);
hipError_t launch_calibrate_policy(const float* frac, int rows, int n_types, double threshold,
                                   double* conc, int32_t* evict, hipStream_t st);
hipError_t launch_evict_step(int BH, int N, const float* scores, const int32_t* k_dev,
                             const void* ksrc, const void* vsrc, int64_t src_ld,
                             const int32_t* idx_src, void* kdst, void* vdst, int32_t* idx_dst,
                             int64_t dst_ld, int row_bytes, hipStream_t st);
hipError_t launch_lse_rows(const float* src, int64_t ld, int W, int rows, float* dst,
                          hipStream_t st);
hipError_t launch_segment_mass(const uc_shape& sh, int M, int n_segs, const float* lse,
                               const float* seg_lse, float* mass, hipStream_t st);
}  // namespace uc
