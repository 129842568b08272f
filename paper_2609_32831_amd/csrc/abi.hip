// abi.hip -- the C ABI entry points of libunicache: argument validation,
// work planning, workspace carving and kernel dispatch, plus the host-only
// storage-accounting and budget helpers.  Every check runs before any launch,
// so a failing call writes nothing and enqueues nothing.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <new>
#include <vector>

#include "budget_rules.h"
#include "uc_common.h"

using namespace uc;

namespace uc {
bool decode_mfma_eligible(const uc_shape& sh, const KSegs& segs, int q_dt, int M);
bool score_mfma_eligible(const uc_shape& sh, const KSegs& segs, int q_dt);
bool prefill_mfma_eligible(const uc_shape& sh, const KSegs& segs, int q_dt, int M);
size_t prefill_mfma_workspace(const uc_shape& sh, const KSegs& segs);
hipError_t launch_prefill_mfma(const uc_shape& sh, const KSegs& segs, const void* q, int M,
                               float sm_scale, float* o, float* lse, float* seg_lse, void* ws,
                               hipStream_t st);
hipError_t launch_prefill_prepare(const uc_shape& sh, const KSegs& segs, void* ws, hipStream_t st,
                                  void* views_out);
hipError_t launch_prefill_run(const uc_shape& sh, int n_segs, const void* views, const void* q,
                              int M, float sm_scale, float* o, float* lse, float* seg_lse,
                              void* ws, hipStream_t st);
int score_mfma_chunk_rows();
hipError_t launch_score_lse_mfma(const uc_shape& sh, const KSegs& segs, const ChunkPlan& plan,
                                 const void* q, int W, float sm_scale, float* partial,
                                 hipStream_t st);
hipError_t launch_score_col_mfma(const uc_shape& sh, const KSegs& segs, const ChunkPlan& plan,
                                 const void* q, int W, int q_ld, float sm_scale, const float* lse,
                                 float* const* scores, double* mass_partial, double* colpart,
                                 hipStream_t st);
int score_mfma_qblocks(int nq);
size_t decode_mfma_workspace(const uc_shape& sh, const KSegs& segs, int M);
hipError_t launch_decode_mfma(const uc_shape& sh, const KSegs& segs, const void* q, int M,
                              float sm_scale, float* o, float* lse, float* seg_lse, void* ws,
                              hipStream_t st, const AppendOp* ap = nullptr);
int decode_batch_wgs(const uc_shape& sh);
size_t decode_batch_desc_bytes(int n_req, int n_segs_total);
size_t decode_batch_workspace(const uc_shape& sh, int M, int n_segs_total);
int decode_split_segment(const KSegs& segs);
size_t decode_batch_table_bytes(int n_req);
size_t decode_batch_grid_bytes(int n_req);
hipError_t launch_decode_batch(const uc_shape& sh, int n_segs_total, int W_max, int n_wgs,
                               int n_grid, int skew, const BatchArgs* args, const void* q, int M,
                               float sm_scale, float* o, float* lse, void* ws, hipStream_t st);
int read_probe_wgs();
hipError_t launch_read_probe(const void* buf, size_t bytes, int pattern, void* sink,
                             hipStream_t st);
}  // namespace uc

namespace {

thread_local char g_err[512] = "";
thread_local const char* g_last_kernel = "";
std::atomic<int> g_path{UC_PATH_AUTO};

// timing events: pending (set by uc_set_kernel_events) and active (taken by
// one attention call for its duration; an entry point that calls another
// keeps them for the inner call's attention kernel)
thread_local hipEvent_t g_ev_pending[2] = {nullptr, nullptr};
thread_local hipEvent_t g_ev_active[2] = {nullptr, nullptr};
thread_local int g_ev_depth = 0;

struct TimerScope {
  TimerScope() {
    if (g_ev_depth++ == 0) {
      g_ev_active[0] = g_ev_pending[0];
      g_ev_active[1] = g_ev_pending[1];
      g_ev_pending[0] = g_ev_pending[1] = nullptr;
    }
  }
  ~TimerScope() {
    if (--g_ev_depth == 0) g_ev_active[0] = g_ev_active[1] = nullptr;
  }
};

uc_status fail(uc_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

uc_status ok() {
  g_err[0] = 0;
  return UC_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
bool dtype_ok(int dt) { return dt == UC_F32 || dt == UC_F16 || dt == UC_BF16; }
bool pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

uc_status check_shape(const uc_shape* sh) {
  if (!sh) return fail(UC_E_INVALID, "shape is NULL");
  if (sh->B < 1 || sh->Hq < 1 || sh->Hkv < 1)
    return fail(UC_E_INVALID, "B, Hq, Hkv must be >= 1 (got %d, %d, %d)", sh->B, sh->Hq, sh->Hkv);
  if (sh->Hq % sh->Hkv) return fail(UC_E_INVALID, "Hq %% Hkv != 0 (%d, %d)", sh->Hq, sh->Hkv);
  if (sh->D != 64 && sh->D != 128) return fail(UC_E_INVALID, "D must be 64 or 128 (got %d)", sh->D);
  return UC_OK;
}

int64_t n_full_of(int N, int G) { return (int64_t)G * (N / G); }

// Validate one segment descriptor against the shape; fill the kernel copy.
uc_status check_segment(const uc_shape& sh, const uc_segment& s, int idx, KSeg& ks,
                        bool require_packed_buffers) {
  memset(&ks, 0, sizeof ks);
  if (s.kind != UC_SEG_DENSE && s.kind != UC_SEG_PACKED)
    return fail(UC_E_INVALID, "segment %d: bad kind %d", idx, s.kind);
  if (!dtype_ok(s.dtype)) return fail(UC_E_INVALID, "segment %d: bad dtype %d", idx, s.dtype);
  if (s.n_rows < 0) return fail(UC_E_INVALID, "segment %d: n_rows < 0", idx);
  ks.kind = s.kind;
  ks.dtype = s.dtype;
  ks.n_rows = s.n_rows;
  const int64_t BH = (int64_t)sh.B * sh.Hkv;
  if (s.kind == UC_SEG_DENSE) {
    ks.row_stride = s.row_stride ? s.row_stride : s.n_rows;
    if (ks.row_stride < s.n_rows)
      return fail(UC_E_INVALID, "segment %d: row_stride %d < n_rows %d", idx, ks.row_stride, s.n_rows);
    if (s.n_rows > 0 && (!s.k || !s.v)) return fail(UC_E_INVALID, "segment %d: k/v NULL", idx);
    if (!aligned16(s.k) || !aligned16(s.v))
      return fail(UC_E_INVALID, "segment %d: k/v not 16-byte aligned", idx);
    ks.k = s.k;
    ks.v = s.v;
    return UC_OK;
  }
  const int G = s.group;
  if (!pow2(G) || G < 8 || G > 128 || sh.D % G)
    return fail(UC_E_INVALID, "segment %d: group %d must be a power of two in [8,128] dividing D", idx, G);
  if (s.bits != 2 && s.bits != 4 && s.bits != 8)
    return fail(UC_E_INVALID, "segment %d: bits %d not in {2,4,8}", idx, s.bits);
  if (s.head_bits && !s.code_off)
    return fail(UC_E_INVALID, "segment %d: head_bits given without code_off", idx);
  ks.group = G;
  ks.bits = s.bits;
  ks.n_full = (int)n_full_of(s.n_rows, G);
  ks.tail_len = s.n_rows - ks.n_full;
  if (s.row_stride < 0 || (s.row_stride > 0 && s.row_stride < s.n_rows))
    return fail(UC_E_INVALID, "segment %d: row_stride %d < n_rows %d", idx, s.row_stride, s.n_rows);
  ks.row_stride = s.row_stride;
  ks.cap_full = s.row_stride ? (int)n_full_of(s.row_stride, G) : ks.n_full;
  ks.kgroups = ks.cap_full / G;
  ks.tail_stride = s.row_stride ? G : ks.tail_len;
  ks.head_bits = s.head_bits;
  ks.code_off = s.code_off;
  ks.codes_bytes = s.codes_bytes;
  if (!s.head_bits && !s.code_off) {
    const uint64_t need = (uint64_t)BH * ks.cap_full * sh.D * s.bits / 8;
    if (s.codes_bytes < need)
      return fail(UC_E_INVALID, "segment %d: codes_bytes %llu < %llu needed", idx,
                  (unsigned long long)s.codes_bytes, (unsigned long long)need);
  }
  if (ks.n_full > 0 || require_packed_buffers) {
    if (!s.codes_k || !s.codes_v || !s.scale_k || !s.min_k || !s.scale_v || !s.min_v)
      return fail(UC_E_INVALID, "segment %d: packed buffer NULL", idx);
  }
  if ((ks.tail_len > 0 || s.row_stride > 0) && (!s.tail_k || !s.tail_v))
    return fail(UC_E_INVALID, "segment %d: tail of %d rows but tail_k/tail_v NULL", idx, ks.tail_len);
  const void* ptrs[] = {s.codes_k, s.codes_v, s.scale_k, s.min_k, s.scale_v, s.min_v, s.tail_k, s.tail_v};
  for (const void* p : ptrs)
    if (!aligned16(p)) return fail(UC_E_INVALID, "segment %d: packed pointer not 16-byte aligned", idx);
  ks.codes_k = s.codes_k;
  ks.codes_v = s.codes_v;
  ks.scale_k = s.scale_k;
  ks.min_k = s.min_k;
  ks.scale_v = s.scale_v;
  ks.min_v = s.min_v;
  ks.tail_k = s.tail_k;
  ks.tail_v = s.tail_v;
  return UC_OK;
}

uc_status check_segments(const uc_shape* sh, const uc_segment* segs, int n, KSegs& ks) {
  uc_status st = check_shape(sh);
  if (st) return st;
  if (!segs) return fail(UC_E_INVALID, "segs is NULL");
  if (n < 1 || n > kMaxSeg) return fail(UC_E_INVALID, "n_segs %d not in [1,%d]", n, kMaxSeg);
  memset(&ks, 0, sizeof ks);
  ks.n = n;
  int64_t total = 0;
  for (int i = 0; i < n; ++i) {
    st = check_segment(*sh, segs[i], i, ks.s[i], false);
    if (st) return st;
    total += segs[i].n_rows;
  }
  if (total <= 0) return fail(UC_E_INVALID, "all segments are empty");
  if (total > INT32_MAX) return fail(UC_E_UNSUPPORTED, "more than 2^31-1 rows");
  return UC_OK;
}

// Chunk plan: rows per chunk for every segment (empty segments get no chunk).
ChunkPlan make_plan(const KSegs& ks, int rows_min, int max_chunks_per_seg) {
  ChunkPlan p{};
  int c = 0;
  for (int i = 0; i < ks.n; ++i) {
    const int n = ks.s[i].n_rows;
    int rows = std::max(rows_min, (n + max_chunks_per_seg - 1) / max_chunks_per_seg);
    p.first[i] = c;
    p.rows[i] = rows;
    c += n > 0 ? (n + rows - 1) / rows : 0;
  }
  for (int i = ks.n; i <= kMaxSeg; ++i) p.first[i] = c;
  p.n_chunks = c;
  return p;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Generic attention partials: one (m, l[, o]) per (query row, chunk).  The
// size is a bound on the chunks of any plan for these segments or for
// segments with fewer rows (min(max_chunks, ceil(n / rows_min)) per segment),
// so a workspace sized at the largest row counts serves smaller ones.
constexpr int kAttRows = 256, kAttMaxChunks = 64, kLseRows = 512, kLseMaxChunks = 32;

size_t generic_ws(const uc_shape& sh, const KSegs& ks, int rows_min, int max_chunks, int M,
                  bool want_o) {
  size_t chunks = 0;
  for (int i = 0; i < ks.n; ++i)
    chunks += std::min<size_t>(max_chunks, (ks.s[i].n_rows + rows_min - 1) / rows_min);
  const size_t stride = want_o ? (size_t)sh.D + 2 : 2;
  return align256((size_t)sh.B * sh.Hq * M * chunks * stride * sizeof(float));
}

ChunkPlan attend_plan(const KSegs& ks) { return make_plan(ks, kAttRows, kAttMaxChunks); }
ChunkPlan score_lse_plan(const KSegs& ks) { return make_plan(ks, kLseRows, kLseMaxChunks); }
ChunkPlan score_col_plan(const KSegs& ks) { return make_plan(ks, 256, 1 << 20); }

uc_status launched(hipError_t e) {
  if (e != hipSuccess) return fail(UC_E_DEVICE, "HIP launch error: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

namespace uc {
hipError_t kernel_timer_begin(hipStream_t st) {
  return g_ev_active[0] ? hipEventRecord(g_ev_active[0], st) : hipSuccess;
}
hipError_t kernel_timer_end(hipStream_t st) {
  return g_ev_active[1] ? hipEventRecord(g_ev_active[1], st) : hipSuccess;
}
}  // namespace uc

extern "C" {

uc_status uc_set_kernel_events(void* start, void* stop) {
  g_ev_pending[0] = (hipEvent_t)start;
  g_ev_pending[1] = (hipEvent_t)stop;
  return ok();
}

const char* uc_status_string(uc_status s) {
  switch (s) {
    case UC_OK: return "UC_OK";
    case UC_E_INVALID: return "UC_E_INVALID: invalid argument";
    case UC_E_UNSUPPORTED: return "UC_E_UNSUPPORTED: unsupported combination";
    case UC_E_WORKSPACE: return "UC_E_WORKSPACE: workspace too small";
    case UC_E_DEVICE: return "UC_E_DEVICE: HIP error";
  }
  return "unknown uc_status";
}

const char* uc_last_error(void) { return g_err; }

const char* uc_last_kernel(void) { return g_last_kernel; }

int uc_set_path(int path) {
  if (path != UC_PATH_AUTO && path != UC_PATH_VALU) return -1;
  return g_path.exchange(path);
}

// ---------------------------------------------------------------- attention
size_t uc_attend_workspace_size(const uc_shape* shape, const uc_segment* segs, int n_segs,
                                uc_dtype q_dt, int M) {
  KSegs ks;
  if (check_segments(shape, segs, n_segs, ks) || M < 1 || !dtype_ok(q_dt)) return 0;
  if (g_path.load() == UC_PATH_AUTO && decode_mfma_eligible(*shape, ks, q_dt, M))
    return decode_mfma_workspace(*shape, ks, M);
  if (g_path.load() == UC_PATH_AUTO && prefill_mfma_eligible(*shape, ks, q_dt, M))
    return prefill_mfma_workspace(*shape, ks);
  return generic_ws(*shape, ks, kAttRows, kAttMaxChunks, M, true);
}

uc_status uc_attend_mixed(const uc_shape* shape, const uc_segment* segs, int n_segs,
                          const void* q, uc_dtype q_dt, int M, float sm_scale, float* o,
                          float* lse, float* seg_lse, void* ws, size_t ws_bytes, void* stream) {
  TimerScope timer;
  KSegs ks;
  uc_status st = check_segments(shape, segs, n_segs, ks);
  if (st) return st;
  if (!q || !o) return fail(UC_E_INVALID, "q or o is NULL");
  if (!dtype_ok(q_dt)) return fail(UC_E_INVALID, "bad q dtype %d", q_dt);
  if (M < 1) return fail(UC_E_INVALID, "M must be >= 1 (got %d)", M);
  if (!(sm_scale > 0.0f) || !isfinite(sm_scale)) return fail(UC_E_INVALID, "sm_scale must be finite and > 0");
  if ((int64_t)shape->B * shape->Hq * M > INT32_MAX) return fail(UC_E_UNSUPPORTED, "too many query rows");
  hipStream_t s = (hipStream_t)stream;
  if (g_path.load() == UC_PATH_AUTO && decode_mfma_eligible(*shape, ks, q_dt, M)) {
    const size_t need = decode_mfma_workspace(*shape, ks, M);
    if (ws_bytes < need || (need && !ws))
      return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
    g_last_kernel = "decode_mfma";
    return launched(launch_decode_mfma(*shape, ks, q, M, sm_scale, o, lse, seg_lse, ws, s));
  }
  if (g_path.load() == UC_PATH_AUTO && prefill_mfma_eligible(*shape, ks, q_dt, M)) {
    const size_t need = prefill_mfma_workspace(*shape, ks);
    if (ws_bytes < need || (need && !ws))
      return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
    g_last_kernel = "prefill_mfma";
    return launched(launch_prefill_mfma(*shape, ks, q, M, sm_scale, o, lse, seg_lse, ws, s));
  }
  const ChunkPlan p = attend_plan(ks);
  const size_t need = generic_ws(*shape, ks, kAttRows, kAttMaxChunks, M, true);
  if (ws_bytes < need || !ws) return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  float* partial = (float*)ws;
  g_last_kernel = "attend_valu";
  hipError_t e = kernel_timer_begin(s);
  if (e == hipSuccess) e = launch_attend_generic(*shape, ks, p, q, q_dt, M, sm_scale, partial, true, s);
  if (e == hipSuccess) e = kernel_timer_end(s);
  if (e == hipSuccess) e = launch_attend_combine(*shape, ks, p, M, partial, o, lse, seg_lse, s);
  return launched(e);
}

// ---------------------------------------------------------------- allocation-free attention
// One file-scope scratch array per GPU, in place of the caller's workspace.
// The host takes its device address once per device with that device current
// and uses only that address afterwards (the array's name is a host-side
// stand-in in host code).
static __device__ __align__(256) unsigned char scratch[UC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

uc_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(UC_E_DEVICE, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(UC_E_UNSUPPORTED, "device %d >= %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(UC_E_DEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return UC_OK;
}
}  // namespace

extern "C" uc_status uc_attend_mixed_noalloc(const uc_shape* shape, const uc_segment* segs,
                                             int n_segs, const void* q, uc_dtype q_dt, int M,
                                             float sm_scale, float* o, float* lse,
                                             float* seg_lse, void* stream) {
  KSegs ks;
  uc_status st = check_segments(shape, segs, n_segs, ks);
  if (st) return st;
  if (M < 1 || !dtype_ok(q_dt)) return fail(UC_E_INVALID, "bad M (%d) or q dtype (%d)", M, q_dt);
  const size_t need = uc_attend_workspace_size(shape, segs, n_segs, q_dt, M);
  if (need > UC_SCRATCH_BYTES)
    return fail(UC_E_UNSUPPORTED,
                "this call needs %zu bytes of scratch, above the %u-byte static array; use "
                "uc_attend_mixed with a workspace", need, (unsigned)UC_SCRATCH_BYTES);
  void* ws = nullptr;
  st = scratch_address(&ws);
  if (st) return st;
  return uc_attend_mixed(shape, segs, n_segs, q, q_dt, M, sm_scale, o, lse, seg_lse, ws,
                         UC_SCRATCH_BYTES, stream);
}

// ---------------------------------------------------------------- decode step, append fused
uc_status uc_attend_append(const uc_shape* shape, const uc_segment* segs, int n_segs, int tail,
                           const void* k_new, const void* v_new, int n_new, const void* q,
                           uc_dtype q_dt, int M, float sm_scale, float* o, float* lse,
                           float* seg_lse, void* ws, size_t ws_bytes, void* stream) {
  TimerScope timer;
  if (!segs) return fail(UC_E_INVALID, "segs is NULL");
  if (n_segs < 1 || n_segs > kMaxSeg) return fail(UC_E_INVALID, "n_segs %d not in [1,%d]", n_segs, kMaxSeg);
  if (tail < 0 || tail >= n_segs) return fail(UC_E_INVALID, "tail %d not in [0,%d)", tail, n_segs);
  if (segs[tail].kind != UC_SEG_DENSE) return fail(UC_E_INVALID, "segment %d (tail) is not dense", tail);
  if (n_new < 0) return fail(UC_E_INVALID, "n_new must be >= 0 (got %d)", n_new);
  // the segments as they stand after the append: validates capacity and rows
  uc_segment after[kMaxSeg];
  memcpy(after, segs, (size_t)n_segs * sizeof(uc_segment));
  const int pos = segs[tail].n_rows;
  if (pos < 0) return fail(UC_E_INVALID, "segment %d: n_rows < 0", tail);
  if (n_new > 0) {
    if (!segs[tail].row_stride || (int64_t)pos + n_new > segs[tail].row_stride)
      return fail(UC_E_INVALID, "tail rows %lld after the append exceed row_stride %d",
                  (long long)pos + n_new, segs[tail].row_stride);
    if (!k_new || !v_new) return fail(UC_E_INVALID, "k_new or v_new is NULL");
    if (!aligned16(k_new) || !aligned16(v_new))
      return fail(UC_E_INVALID, "k_new/v_new not 16-byte aligned");
  }
  after[tail].n_rows = pos + n_new;
  KSegs ks;
  uc_status st = check_segments(shape, after, n_segs, ks);
  if (st) return st;
  if (!q || !o) return fail(UC_E_INVALID, "q or o is NULL");
  if (!dtype_ok(q_dt)) return fail(UC_E_INVALID, "bad q dtype %d", q_dt);
  if (M < 1) return fail(UC_E_INVALID, "M must be >= 1 (got %d)", M);
  if (!(sm_scale > 0.0f) || !isfinite(sm_scale)) return fail(UC_E_INVALID, "sm_scale must be finite and > 0");
  if ((int64_t)shape->B * shape->Hq * M > INT32_MAX) return fail(UC_E_UNSUPPORTED, "too many query rows");
  hipStream_t s = (hipStream_t)stream;
  const bool fused = n_new > 0 && !seg_lse && n_segs < kMaxSeg && g_path.load() == UC_PATH_AUTO &&
                     decode_mfma_eligible(*shape, ks, q_dt, M);
  if (!fused) {
    // the two calls this one stands for, checked before either is enqueued
    const size_t need = uc_attend_workspace_size(shape, after, n_segs, q_dt, M);
    if (ws_bytes < need || (need && !ws)) return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
    if (n_new > 0) {
      KSeg t = ks.s[tail];
      hipError_t e = launch_append(*shape, k_new, v_new, n_new, t, pos, s);
      if (e != hipSuccess) return launched(e);
    }
    return uc_attend_mixed(shape, after, n_segs, q, q_dt, M, sm_scale, o, lse, seg_lse, ws,
                           ws_bytes, stream);
  }
  // the tail as it stood, plus the new rows as a dense segment of their own
  // read from k_new / v_new (softmax does not depend on the rows' order);
  // without per-segment outputs every record belongs to one softmax
  const size_t need = decode_mfma_workspace(*shape, ks, M);
  if (ws_bytes < need || (need && !ws)) return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  ks.s[tail].n_rows = pos;
  KSeg& nk = ks.s[ks.n++];
  memset(&nk, 0, sizeof nk);
  nk.kind = UC_SEG_DENSE;
  nk.dtype = ks.s[tail].dtype;
  nk.n_rows = n_new;
  nk.row_stride = n_new;
  nk.k = k_new;
  nk.v = v_new;
  AppendOp ap{(const char*)k_new, (const char*)v_new, (char*)ks.s[tail].k, (char*)ks.s[tail].v,
              n_new, ks.s[tail].row_stride, pos, shape->D * dtype_bytes(nk.dtype)};
  g_last_kernel = "decode_mfma_append";
  return launched(launch_decode_mfma(*shape, ks, q, M, sm_scale, o, lse, nullptr, ws, s, &ap));
}

// ---------------------------------------------------------------- execution plans
}  // extern "C"

struct uc_plan_s {
  uc_shape shape;
  uc_segment segs[kMaxSeg];  // the frozen layout; segs[tail].n_rows advances
  KSegs ks;                  // its derived device layout, kept in step
  int n_segs, tail, M;
  uc_dtype q_dt;
  float sm_scale;
  size_t ws_need;            // enough for every call up to the tail's capacity
  // multi-query attention: the workspace prepared by the last call (packed
  // rows dequantised, V converted) and the views over it, reused while the
  // segments stay as they are
  void* prepared_ws;
  alignas(16) char views[kPrefillViewBytes];
};

extern "C" {

uc_status uc_plan_create(const uc_shape* shape, const uc_segment* segs, int n_segs, int tail,
                         uc_dtype q_dt, int M, float sm_scale, uc_plan* out) {
  if (!out) return fail(UC_E_INVALID, "out is NULL");
  *out = nullptr;
  KSegs ks;
  uc_status st = check_segments(shape, segs, n_segs, ks);
  if (st) return st;
  if (tail < -1 || tail >= n_segs) return fail(UC_E_INVALID, "tail %d not in [-1,%d)", tail, n_segs);
  if (tail >= 0 && (segs[tail].kind != UC_SEG_DENSE || segs[tail].row_stride < 1))
    return fail(UC_E_INVALID, "segment %d (tail) is not a dense segment with a row capacity", tail);
  if (n_segs >= kMaxSeg)
    return fail(UC_E_UNSUPPORTED, "a plan takes at most %d segments", kMaxSeg - 1);
  if (!dtype_ok(q_dt)) return fail(UC_E_INVALID, "bad q dtype %d", q_dt);
  if (M < 1) return fail(UC_E_INVALID, "M must be >= 1 (got %d)", M);
  if (!(sm_scale > 0.0f) || !isfinite(sm_scale)) return fail(UC_E_INVALID, "sm_scale must be finite and > 0");
  if ((int64_t)shape->B * shape->Hq * M > INT32_MAX) return fail(UC_E_UNSUPPORTED, "too many query rows");
  uc_plan p = new (std::nothrow) uc_plan_s;
  if (!p) return fail(UC_E_INVALID, "out of host memory");
  p->shape = *shape;
  memcpy(p->segs, segs, (size_t)n_segs * sizeof(uc_segment));
  p->ks = ks;
  p->n_segs = n_segs;
  p->tail = tail;
  p->M = M;
  p->q_dt = q_dt;
  p->sm_scale = sm_scale;
  p->prepared_ws = nullptr;
  // workspace: the path selected now (uc_set_path), at the tail's capacity
  // (the sizes only grow with the row counts).  A call after the path was
  // switched goes through uc_attend_mixed / uc_attend_append, which check
  // the workspace against that path's own need.
  uc_segment full[kMaxSeg];
  memcpy(full, segs, (size_t)n_segs * sizeof(uc_segment));
  if (tail >= 0) full[tail].n_rows = full[tail].row_stride;
  KSegs kf;
  check_segments(shape, full, n_segs, kf);
  size_t need;
  if (g_path.load() == UC_PATH_AUTO && prefill_mfma_eligible(*shape, kf, q_dt, M)) {
    need = prefill_mfma_workspace(*shape, kf);
  } else {
    need = generic_ws(*shape, kf, kAttRows, kAttMaxChunks, M, true);
    if (g_path.load() == UC_PATH_AUTO && decode_mfma_eligible(*shape, kf, q_dt, M))
      need = std::max(need, decode_mfma_workspace(*shape, kf, M));
  }
  p->ws_need = need;
  *out = p;
  return ok();
}

size_t uc_plan_workspace_size(uc_plan plan) { return plan ? plan->ws_need : 0; }

int uc_plan_tail_rows(uc_plan plan) {
  return plan && plan->tail >= 0 ? plan->segs[plan->tail].n_rows : -1;
}

uc_status uc_plan_invalidate(uc_plan plan) {
  if (!plan) return fail(UC_E_INVALID, "plan is NULL");
  plan->prepared_ws = nullptr;
  return ok();
}

uc_status uc_plan_attend(uc_plan plan, const void* q, float* o, float* lse, float* seg_lse,
                         void* ws, size_t ws_bytes, void* stream) {
  TimerScope timer;
  if (!plan) return fail(UC_E_INVALID, "plan is NULL");
  if (!q || !o) return fail(UC_E_INVALID, "q or o is NULL");
  if (ws_bytes < plan->ws_need || (plan->ws_need && !ws))
    return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, plan->ws_need);
  const uc_shape& sh = plan->shape;
  if (g_path.load() != UC_PATH_AUTO || !prefill_mfma_eligible(sh, plan->ks, plan->q_dt, plan->M)) {
    plan->prepared_ws = nullptr;
    return uc_attend_mixed(&sh, plan->segs, plan->n_segs, q, plan->q_dt, plan->M, plan->sm_scale,
                           o, lse, seg_lse, ws, ws_bytes, stream);
  }
  hipStream_t s = (hipStream_t)stream;
  if (plan->prepared_ws != ws) {
    const hipError_t e = launch_prefill_prepare(sh, plan->ks, ws, s, plan->views);
    if (e != hipSuccess) return launched(e);
    plan->prepared_ws = ws;
  }
  g_last_kernel = "prefill_mfma";
  return launched(launch_prefill_run(sh, plan->n_segs, plan->views, q, plan->M, plan->sm_scale, o,
                                     lse, seg_lse, ws, s));
}

uc_status uc_plan_attend_append(uc_plan plan, const void* k_new, const void* v_new, int n_new,
                                const void* q, float* o, float* lse, void* ws, size_t ws_bytes,
                                void* stream) {
  TimerScope timer;
  if (!plan) return fail(UC_E_INVALID, "plan is NULL");
  if (plan->tail < 0) return fail(UC_E_INVALID, "the plan has no tail segment to append to");
  const int tail = plan->tail, pos = plan->segs[tail].n_rows;
  if (n_new < 0) return fail(UC_E_INVALID, "n_new must be >= 0 (got %d)", n_new);
  if (n_new > 0) {
    if ((int64_t)pos + n_new > plan->segs[tail].row_stride)
      return fail(UC_E_INVALID, "tail rows %lld after the append exceed row_stride %d",
                  (long long)pos + n_new, plan->segs[tail].row_stride);
    if (!k_new || !v_new) return fail(UC_E_INVALID, "k_new or v_new is NULL");
    if (!aligned16(k_new) || !aligned16(v_new))
      return fail(UC_E_INVALID, "k_new/v_new not 16-byte aligned");
  }
  if (!q || !o) return fail(UC_E_INVALID, "q or o is NULL");
  if (ws_bytes < plan->ws_need || (plan->ws_need && !ws))
    return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, plan->ws_need);
  const uc_shape& sh = plan->shape;
  uc_status st;
  if (n_new > 0 && g_path.load() == UC_PATH_AUTO && decode_mfma_eligible(sh, plan->ks, plan->q_dt, plan->M)) {
    // the fused step of uc_attend_append, on the layout derived at creation
    KSegs ks = plan->ks;
    KSeg& nk = ks.s[ks.n++];
    memset(&nk, 0, sizeof nk);
    nk.kind = UC_SEG_DENSE;
    nk.dtype = ks.s[tail].dtype;
    nk.n_rows = n_new;
    nk.row_stride = n_new;
    nk.k = k_new;
    nk.v = v_new;
    AppendOp ap{(const char*)k_new, (const char*)v_new, (char*)ks.s[tail].k, (char*)ks.s[tail].v,
                n_new, ks.s[tail].row_stride, pos, sh.D * dtype_bytes(nk.dtype)};
    g_last_kernel = "decode_mfma_append";
    st = launched(launch_decode_mfma(sh, ks, q, plan->M, plan->sm_scale, o, lse, nullptr, ws,
                                     (hipStream_t)stream, &ap));
  } else {
    st = uc_attend_append(&sh, plan->segs, plan->n_segs, tail, k_new, v_new, n_new, q,
                          plan->q_dt, plan->M, plan->sm_scale, o, lse, nullptr, ws, ws_bytes, stream);
  }
  if (st == UC_OK && n_new > 0) {
    plan->segs[tail].n_rows += n_new;
    plan->ks.s[tail].n_rows += n_new;
    plan->prepared_ws = nullptr;  // the tail's rows changed
  }
  return st;
}

uc_status uc_plan_destroy(uc_plan plan) {
  delete plan;
  return ok();
}

// ---------------------------------------------------------------- batched requests
// Time of a packed row relative to a dense one in the batched decode kernel
// (a third of the bytes, more vector-ALU work), for sharing rows among
// workgroups.  Measured on one MI355X with 16 requests of int4 text and
// dense rows: 0.33 (bytes) 63.1 us, 0.6 60.0 us, 1.0 (rows) 61.7 us.
constexpr double kPackedRowCost = 0.6;


// Validates every request against a one-request shape; true if all of them
// can run in the batched decode kernel.
static uc_status batch_check(const uc_shape* shape, const uc_segment* const* segs,
                             const int* n_segs, uc_dtype q_dt, int M, std::vector<KSegs>& ks,
                             bool& batched) {
  uc_status st = check_shape(shape);
  if (st) return st;
  if (!segs || !n_segs) return fail(UC_E_INVALID, "segs or n_segs is NULL");
  if (!dtype_ok(q_dt)) return fail(UC_E_INVALID, "bad q dtype %d", q_dt);
  if (M < 1) return fail(UC_E_INVALID, "M must be >= 1 (got %d)", M);
  const uc_shape one{1, shape->Hq, shape->Hkv, shape->D};
  ks.resize(shape->B);
  batched = g_path.load() == UC_PATH_AUTO;
  for (int r = 0; r < shape->B; ++r) {
    st = check_segments(&one, segs[r], n_segs[r], ks[r]);
    if (st) {
      char why[sizeof g_err];
      snprintf(why, sizeof why, "%s", g_err);
      return fail(st, "request %d: %s", r, why);
    }
    batched = batched && decode_mfma_eligible(one, ks[r], q_dt, M);
  }
  return UC_OK;
}

size_t uc_attend_batch_workspace_size(const uc_shape* shape, const uc_segment* const* segs,
                                      const int* n_segs, uc_dtype q_dt, int M) {
  std::vector<KSegs> ks;
  bool batched = false;
  if (batch_check(shape, segs, n_segs, q_dt, M, ks, batched)) return 0;
  int total = 0;
  for (int r = 0; r < shape->B; ++r) total += n_segs[r];
  if (batched) return decode_batch_workspace(*shape, M, total);
  const uc_shape one{1, shape->Hq, shape->Hkv, shape->D};
  size_t need = 0;
  for (int r = 0; r < shape->B; ++r)
    need = std::max(need, uc_attend_workspace_size(&one, segs[r], n_segs[r], q_dt, M));
  return need;
}

uc_status uc_attend_batch(const uc_shape* shape, const uc_segment* const* segs, const int* n_segs,
                          const void* q, uc_dtype q_dt, int M, float sm_scale, float* o,
                          float* lse, void* ws, size_t ws_bytes, void* stream) {
  TimerScope timer;
  std::vector<KSegs> ks;
  bool batched = false;
  uc_status st = batch_check(shape, segs, n_segs, q_dt, M, ks, batched);
  if (st) return st;
  if (!q || !o) return fail(UC_E_INVALID, "q or o is NULL");
  if (!(sm_scale > 0.0f) || !isfinite(sm_scale)) return fail(UC_E_INVALID, "sm_scale must be finite and > 0");
  if ((int64_t)shape->B * shape->Hq * M > INT32_MAX) return fail(UC_E_UNSUPPORTED, "too many query rows");
  hipStream_t s = (hipStream_t)stream;
  if (batched) {
    int total = 0;
    for (int r = 0; r < shape->B; ++r) total += n_segs[r];
    const size_t need = decode_batch_workspace(*shape, M, total);
    if (ws_bytes < need || !ws) return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
    // request table, grid runs and flat descriptors, in the workspace's
    // layout; a small batch passes them in the attention kernel's arguments,
    // a larger one sends them to the workspace inside small kernels'
    // arguments first (no staging, no host wait)
    const int B = shape->B, Hkv = shape->Hkv;
    const size_t tbytes = decode_batch_table_bytes(B), gbytes = decode_batch_grid_bytes(B);
    std::vector<char> desc(decode_batch_desc_bytes(B, total), 0);
    BatchDesc* table = (BatchDesc*)desc.data();
    BatchGrid* grid = (BatchGrid*)(desc.data() + tbytes);
    KSeg* flat = (KSeg*)(desc.data() + tbytes + gbytes);
    // workgroups per KV head: one unit each, then a unit at a time to the
    // request with the most weighted rows per workgroup until the budget (a
    // round of resident workgroups) is spent, which minimises the largest
    // share (packed rows weighted by kPackedRowCost).
    // Workgroups go in pairs when the budget gives every request one (an
    // early and a late workgroup per pair, so the launch's two halves hold
    // the same number and every CU pairs one of each).
    const int budget = decode_batch_wgs(*shape);
    const int unit = budget >= 2 * B ? 2 : 1;
    std::vector<double> rows(B, 0.0);
    for (int r = 0; r < B; ++r)
      for (int i = 0; i < n_segs[r]; ++i)
        rows[r] += ks[r].s[i].n_rows * (ks[r].s[i].kind == UC_SEG_PACKED ? kPackedRowCost : 1.0);
    std::vector<int> W(B, unit);
    for (int left = budget - unit * B; left >= unit; left -= unit) {
      int best = 0;
      for (int r = 1; r < B; ++r)
        if (rows[r] * W[best] > rows[best] * W[r]) best = r;  // rows/W largest, lower r on ties
      W[best] += unit;
    }
    int pos = 0, W_max = 1, n_wgs = 0, n_grid = 0;
    for (int r = 0; r < B; ++r) {
      W_max = std::max(W_max, W[r]);
      table[r] = BatchDesc{pos, n_segs[r], W[r], decode_split_segment(ks[r])};
      for (int i = 0; i < n_segs[r]; ++i) flat[pos++] = ks[r].s[i];
    }
    // grid runs: workgroups 0 .. W/2 - 1 of every request (the early ones,
    // dispatched in the launch's first half), then the others
    for (int half = 0; half < 2; ++half)
      for (int r = 0; r < B; ++r) {
        const int w0 = half ? W[r] / 2 : 0, nw = half ? W[r] - W[r] / 2 : W[r] / 2;
        if (nw == 0) continue;
        grid[n_grid++] = BatchGrid{n_wgs, r, w0, nw};
        n_wgs += nw * Hkv;
      }
    // early workgroups take the larger share when the grid is two per CU
    const int skew = n_wgs == 2 * device_cus() ? 600 : 0;
    g_last_kernel = "decode_batch";
    hipError_t e = hipSuccess;
    if (B <= kArgReq && total <= kArgSeg) {
      static thread_local BatchArgs args;  // 11.8 KB: not on the stack
      memset(&args, 0, sizeof args);
      memcpy(args.table, table, sizeof(BatchDesc) * B);
      memcpy(args.grid, grid, sizeof(BatchGrid) * n_grid);
      memcpy(args.flat, flat, sizeof(KSeg) * total);
      e = launch_decode_batch(*shape, total, W_max, n_wgs, n_grid, skew, &args, q, M, sm_scale, o,
                              lse, ws, s);
    } else {
      e = launch_blob_upload(desc.data(), desc.size(), ws, s);
      if (e == hipSuccess)
        e = launch_decode_batch(*shape, total, W_max, n_wgs, n_grid, skew, nullptr, q, M,
                                sm_scale, o, lse, ws, s);
    }
    return launched(e);
  }
  // one call per request (the timing hook is not applied here)
  g_ev_active[0] = g_ev_active[1] = nullptr;
  const uc_shape one{1, shape->Hq, shape->Hkv, shape->D};
  const size_t qrow = (size_t)shape->Hq * M * shape->D * (q_dt == UC_F32 ? 4 : 2);
  for (int r = 0; r < shape->B; ++r) {
    st = uc_attend_mixed(&one, segs[r], n_segs[r], (const char*)q + r * qrow, q_dt, M, sm_scale,
                         o + (size_t)r * shape->Hq * M * shape->D,
                         lse ? lse + (size_t)r * shape->Hq * M : nullptr, nullptr, ws, ws_bytes,
                         stream);
    if (st) {
      char why[sizeof g_err];
      snprintf(why, sizeof why, "%s", g_err);
      return fail(st, "request %d: %s", r, why);
    }
  }
  return ok();
}

// ---------------------------------------------------------------- scoring
static bool score_fast(const uc_shape& sh, const KSegs& ks, int q_dt) {
  return g_path.load() == UC_PATH_AUTO && score_mfma_eligible(sh, ks, q_dt);
}

// matrix-core scoring: both passes use one plan of score_mfma_chunk_rows()
// keys per chunk
static ChunkPlan score_mfma_plan(const KSegs& ks) {
  return make_plan(ks, score_mfma_chunk_rows(), 1 << 30);
}

// workspace parts: pass-1 records, row log-sum-exps, chunk masses (fp64),
// and (matrix-core path) the column pass's per-group column sums (fp64);
// every part grows monotonically with the row counts
static void score_ws_parts(const uc_shape& sh, const KSegs& ks, int W, bool fast, size_t& part1,
                           size_t& lse_b, size_t& mass_b, size_t& col_b) {
  lse_b = align256((size_t)sh.B * sh.Hq * W * sizeof(float));
  col_b = 0;
  if (fast) {
    const ChunkPlan p = score_mfma_plan(ks);
    const int C = p.n_chunks;
    part1 = align256((size_t)sh.B * sh.Hq * W * C * 2 * sizeof(float));
    mass_b = align256((size_t)sh.B * sh.Hkv * C * sizeof(double));
    // groups x chunks x heads is at most min(query blocks, 512 / (chunks x
    // heads) + 1) x chunks x heads: sized by that bound, which (unlike the
    // group count itself) never shrinks as rows are added
    const size_t base = (size_t)sh.B * sh.Hkv * C;
    const size_t qb = (size_t)score_mfma_qblocks((sh.Hq / sh.Hkv) * W);
    if (qb > 1)
      col_b = align256(std::min(qb * base, 512 + base) * score_mfma_chunk_rows() * sizeof(double));
    return;
  }
  part1 = generic_ws(sh, ks, kLseRows, kLseMaxChunks, W, false);
  mass_b = align256((size_t)sh.B * sh.Hkv * score_col_plan(ks).n_chunks * sizeof(double));
}

size_t uc_score_workspace_size(const uc_shape* shape, const uc_segment* segs, int n_segs, int W) {
  KSegs ks;
  if (check_segments(shape, segs, n_segs, ks) || W < 1) return 0;
  // the larger of the two paths' needs, so the size does not depend on the
  // query dtype or the selected path
  size_t a, b, c, d, a2, b2, c2, d2;
  score_ws_parts(*shape, ks, W, false, a, b, c, d);
  score_ws_parts(*shape, ks, W, true, a2, b2, c2, d2);
  return std::max(a + b + c + d, a2 + b2 + c2 + d2);
}

uc_status uc_score_importance(const uc_shape* shape, const uc_segment* segs, int n_segs,
                              const void* q_obs, uc_dtype q_dt, int W, float sm_scale,
                              float* const* scores_out, float* mass_out, void* ws,
                              size_t ws_bytes, void* stream) {
  KSegs ks;
  uc_status st = check_segments(shape, segs, n_segs, ks);
  if (st) return st;
  if (!q_obs) return fail(UC_E_INVALID, "q_obs is NULL");
  if (!dtype_ok(q_dt)) return fail(UC_E_INVALID, "bad q dtype %d", q_dt);
  if (W < 1) return fail(UC_E_INVALID, "W must be >= 1 (got %d)", W);
  if (!(sm_scale > 0.0f) || !isfinite(sm_scale)) return fail(UC_E_INVALID, "sm_scale must be finite and > 0");
  if ((int64_t)shape->B * shape->Hq * W > INT32_MAX) return fail(UC_E_UNSUPPORTED, "too many query rows");
  const bool fast = score_fast(*shape, ks, q_dt);
  size_t a, b, c, d;
  score_ws_parts(*shape, ks, W, fast, a, b, c, d);
  if (!ws || ws_bytes < a + b + c + d)
    return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, a + b + c + d);
  hipStream_t s = (hipStream_t)stream;
  float* partial = (float*)ws;
  float* lse = (float*)((char*)ws + a);
  double* mpart = (double*)((char*)ws + a + b);
  double* colpart = d ? (double*)((char*)ws + a + b + c) : nullptr;
  float* sp[kMaxSeg] = {};
  if (scores_out)
    for (int i = 0; i < n_segs; ++i) sp[i] = scores_out[i];
  hipError_t e;
  ChunkPlan p2;
  g_last_kernel = fast ? "score_mfma" : "score_valu";
  if (fast) {
    const ChunkPlan p = score_mfma_plan(ks);
    e = launch_score_lse_mfma(*shape, ks, p, q_obs, W, sm_scale, partial, s);
    if (e == hipSuccess) e = launch_attend_combine(*shape, ks, p, W, partial, nullptr, lse, nullptr, s);
    if (e == hipSuccess)
      e = launch_score_col_mfma(*shape, ks, p, q_obs, W, W, sm_scale, lse, sp, mpart, colpart, s);
    p2 = p;
  } else {
    const ChunkPlan p1 = score_lse_plan(ks);
    p2 = score_col_plan(ks);
    e = launch_attend_generic(*shape, ks, p1, q_obs, q_dt, W, sm_scale, partial, false, s);
    if (e == hipSuccess) e = launch_attend_combine(*shape, ks, p1, W, partial, nullptr, lse, nullptr, s);
    if (e == hipSuccess)
      e = launch_score_colsum(*shape, ks, p2, q_obs, q_dt, W, W, sm_scale, lse, sp, mpart, s);
  }
  if (e == hipSuccess && mass_out)
    e = launch_mass_finalize(p2, shape->B * shape->Hkv, n_segs, mpart, mass_out, s);
  return launched(e);
}

uc_status uc_score_columns(const uc_shape* shape, const uc_segment* segs, int n_segs,
                           const void* q_obs, int64_t q_ld, uc_dtype q_dt, int W, float sm_scale,
                           const float* row_lse, int64_t lse_ld, float* const* scores_out,
                           float* mass_out, void* ws, size_t ws_bytes, void* stream) {
  KSegs ks;
  uc_status st = check_segments(shape, segs, n_segs, ks);
  if (st) return st;
  if (!q_obs) return fail(UC_E_INVALID, "q_obs is NULL");
  if (!dtype_ok(q_dt)) return fail(UC_E_INVALID, "bad q dtype %d", q_dt);
  if (W < 1) return fail(UC_E_INVALID, "W must be >= 1 (got %d)", W);
  if (!(sm_scale > 0.0f) || !isfinite(sm_scale)) return fail(UC_E_INVALID, "sm_scale must be finite and > 0");
  if ((int64_t)shape->B * shape->Hq * W > INT32_MAX) return fail(UC_E_UNSUPPORTED, "too many query rows");
  if (!row_lse) return fail(UC_E_INVALID, "row_lse is NULL");
  if (lse_ld < W) return fail(UC_E_INVALID, "lse_ld=%lld < W=%d", (long long)lse_ld, W);
  if (q_ld < W || q_ld > INT32_MAX) return fail(UC_E_INVALID, "q_ld=%lld < W=%d", (long long)q_ld, W);
  const bool fast = score_fast(*shape, ks, q_dt);
  size_t a, b, c, d;
  score_ws_parts(*shape, ks, W, fast, a, b, c, d);
  if (!ws || ws_bytes < a + b + c + d)
    return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, a + b + c + d);
  float* sp[kMaxSeg] = {};
  bool any = false;
  if (scores_out)
    for (int i = 0; i < n_segs; ++i) {
      sp[i] = scores_out[i];
      any = any || sp[i] != nullptr;
    }
  g_last_kernel = fast ? "score_mfma" : "score_valu";
  if (!any && !mass_out) return ok();
  // without masses, the chunks of segments whose scores are not wanted are
  // left out of the plan (the kernels read the row counts from ks)
  KSegs kp = ks;
  if (!mass_out)
    for (int i = 0; i < n_segs; ++i)
      if (!sp[i]) kp.s[i].n_rows = 0;
  hipStream_t s = (hipStream_t)stream;
  float* lse = (float*)((char*)ws + a);
  double* mpart = mass_out ? (double*)((char*)ws + a + b) : nullptr;
  double* colpart = d ? (double*)((char*)ws + a + b + c) : nullptr;
  const ChunkPlan p2 = fast ? score_mfma_plan(kp) : score_col_plan(kp);
  hipError_t e = hipSuccess;
  if (p2.n_chunks > 0) {
    e = launch_lse_rows(row_lse, lse_ld, W, shape->B * shape->Hq, lse, s);
    if (e == hipSuccess)
      e = fast ? launch_score_col_mfma(*shape, ks, p2, q_obs, W, (int)q_ld, sm_scale, lse, sp,
                                       mpart, colpart, s)
               : launch_score_colsum(*shape, ks, p2, q_obs, q_dt, W, (int)q_ld, sm_scale, lse, sp,
                                     mpart, s);
  }
  if (e == hipSuccess && mass_out)
    e = launch_mass_finalize(p2, shape->B * shape->Hkv, n_segs, mpart, mass_out, s);
  return launched(e);
}

uc_status uc_segment_mass(const uc_shape* shape, int M, int n_segs, const float* lse,
                          const float* seg_lse, float* mass_out, void* stream) {
  uc_status st = check_shape(shape);
  if (st) return st;
  if (M < 1 || n_segs < 1 || n_segs > kMaxSeg) return fail(UC_E_INVALID, "bad M or n_segs");
  if (!lse || !seg_lse || !mass_out) return fail(UC_E_INVALID, "NULL pointer");
  return launched(launch_segment_mass(*shape, M, n_segs, lse, seg_lse, mass_out, (hipStream_t)stream));
}

// ---------------------------------------------------------------- selection
size_t uc_select_workspace_size(int BH, int N) {
  (void)BH;
  (void)N;
  return 0;
}

uc_status uc_select_keep(const float* scores, int BH, int N, int k, int n_recent,
                         int32_t* keep_idx, const void* k_src, const void* v_src, void* k_dst,
                         void* v_dst, uc_dtype dt, int D, void* ws, size_t ws_bytes,
                         void* stream) {
  (void)ws;
  (void)ws_bytes;
  if (BH < 1 || N < 0) return fail(UC_E_INVALID, "BH must be >= 1 and N >= 0");
  if (k < 0 || k > N) return fail(UC_E_INVALID, "k=%d not in [0, N=%d]", k, N);
  if (n_recent < 0 || n_recent > k) return fail(UC_E_INVALID, "n_recent=%d not in [0, k=%d]", n_recent, k);
  if (k > 0 && !keep_idx) return fail(UC_E_INVALID, "keep_idx is NULL");
  if (N > 0 && k > n_recent && !scores) return fail(UC_E_INVALID, "scores is NULL");
  if (k_src) {
    if (!v_src || !k_dst || !v_dst) return fail(UC_E_INVALID, "gather buffers NULL");
    if (!dtype_ok(dt)) return fail(UC_E_INVALID, "bad dtype %d", dt);
    if (D != 64 && D != 128) return fail(UC_E_INVALID, "D must be 64 or 128");
    if (!aligned16(k_src) || !aligned16(v_src) || !aligned16(k_dst) || !aligned16(v_dst))
      return fail(UC_E_INVALID, "gather pointers not 16-byte aligned");
  }
  if (k == 0) return ok();
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = launch_select(scores, BH, N, k, n_recent, keep_idx, s);
  if (e == hipSuccess && k_src)
    e = launch_gather(keep_idx, BH, N, k, k_src, v_src, k_dst, v_dst, dtype_bytes(dt), D, s);
  return launched(e);
}

// ---------------------------------------------------------------- device-sized eviction
uc_status uc_evict_step(const uc_shape* shape, const float* scores, const uc_segment* cur,
                        const int32_t* k_dev, const uc_segment* out, void* stream) {
  uc_status st = check_shape(shape);
  if (st) return st;
  if (!cur || !out) return fail(UC_E_INVALID, "cur or out is NULL");
  if (cur->kind != UC_SEG_DENSE || out->kind != UC_SEG_DENSE)
    return fail(UC_E_INVALID, "cur and out must be dense segments");
  KSeg kc, ko;
  st = check_segment(*shape, *cur, 0, kc, false);
  if (st) return st;
  uc_segment o = *out;
  o.n_rows = 0;  // not read
  st = check_segment(*shape, o, 1, ko, false);
  if (st) return st;
  if (cur->dtype != out->dtype) return fail(UC_E_INVALID, "cur and out differ in dtype");
  const int N = kc.n_rows;
  if (ko.row_stride < N)
    return fail(UC_E_INVALID, "out row_stride %d < cur n_rows %d", ko.row_stride, N);
  if (N == 0) return ok();
  if (!scores || !k_dev) return fail(UC_E_INVALID, "scores or k_dev is NULL");
  if (!out->k || !out->v || !out->idx) return fail(UC_E_INVALID, "out k/v/idx NULL");
  const int64_t BH = (int64_t)shape->B * shape->Hkv;
  const size_t row_bytes = (size_t)shape->D * dtype_bytes(cur->dtype);
  auto overlap = [&](const void* a, size_t na, const void* b, size_t nb) {
    const char* x = (const char*)a;
    const char* y = (const char*)b;
    return x < y + nb && y < x + na;
  };
  const size_t cur_rows = (size_t)BH * kc.row_stride * row_bytes;
  const size_t out_rows = (size_t)BH * ko.row_stride * row_bytes;
  if (overlap(out->k, out_rows, cur->k, cur_rows) || overlap(out->k, out_rows, cur->v, cur_rows) ||
      overlap(out->v, out_rows, cur->k, cur_rows) || overlap(out->v, out_rows, cur->v, cur_rows) ||
      overlap(out->k, out_rows, out->v, out_rows))
    return fail(UC_E_INVALID, "out rows overlap cur rows or each other");
  if (cur->idx &&
      overlap(out->idx, (size_t)BH * ko.row_stride * 4, cur->idx, (size_t)BH * kc.row_stride * 4))
    return fail(UC_E_INVALID, "out idx overlaps cur idx");
  return launched(launch_evict_step((int)BH, N, scores, k_dev, cur->k, cur->v, kc.row_stride,
                                    (const int32_t*)cur->idx, out->k, out->v, (int32_t*)out->idx,
                                    ko.row_stride, (int)row_bytes, (hipStream_t)stream));
}

// ---------------------------------------------------------------- quantize
uc_status uc_quantize_segment(const uc_shape* shape, const void* k, const void* v, uc_dtype dt,
                              int N, const uc_segment* out, void* stream) {
  uc_status st = check_shape(shape);
  if (st) return st;
  if (!out) return fail(UC_E_INVALID, "out is NULL");
  if (!dtype_ok(dt)) return fail(UC_E_INVALID, "bad dtype %d", dt);
  if (N < 0) return fail(UC_E_INVALID, "N < 0");
  if (out->kind != UC_SEG_PACKED) return fail(UC_E_INVALID, "out must be a packed segment");
  if (out->n_rows != N) return fail(UC_E_INVALID, "out->n_rows %d != N %d", out->n_rows, N);
  if (out->dtype != dt) return fail(UC_E_INVALID, "out->dtype != dt");
  KSeg ks;
  st = check_segment(*shape, *out, 0, ks, false);
  if (st) return st;
  if (N > 0 && (!k || !v)) return fail(UC_E_INVALID, "k or v is NULL");
  if (!aligned16(k) || !aligned16(v)) return fail(UC_E_INVALID, "k/v not 16-byte aligned");
  if (N == 0) return ok();
  return launched(launch_quantize(*shape, k, v, dt, N, ks, (hipStream_t)stream));
}

uc_status uc_dequantize_segment(const uc_shape* shape, const uc_segment* seg, void* k_out,
                                void* v_out, void* stream) {
  uc_status st = check_shape(shape);
  if (st) return st;
  if (!seg || seg->kind != UC_SEG_PACKED) return fail(UC_E_INVALID, "seg must be a packed segment");
  KSeg ks;
  st = check_segment(*shape, *seg, 0, ks, false);
  if (st) return st;
  if (seg->n_rows == 0) return ok();
  if (!k_out || !v_out) return fail(UC_E_INVALID, "k_out or v_out is NULL");
  if (!aligned16(k_out) || !aligned16(v_out)) return fail(UC_E_INVALID, "k_out/v_out not 16-byte aligned");
  return launched(launch_dequantize(*shape, ks, k_out, v_out, (hipStream_t)stream));
}

uc_status uc_stream_append(const uc_shape* shape, const uc_segment* seg, const void* k_new,
                           const void* v_new, int n_new, void* stream) {
  uc_status st = check_shape(shape);
  if (st) return st;
  if (!seg || seg->kind != UC_SEG_PACKED) return fail(UC_E_INVALID, "seg must be a packed segment");
  if (seg->row_stride <= 0) return fail(UC_E_INVALID, "seg needs a row capacity (row_stride > 0)");
  if (seg->head_bits || seg->code_off)
    return fail(UC_E_UNSUPPORTED, "streaming needs the uniform code layout (no head_bits/code_off)");
  KSeg ks;
  st = check_segment(*shape, *seg, 0, ks, true);
  if (st) return st;
  if (n_new < 0) return fail(UC_E_INVALID, "n_new < 0");
  if ((int64_t)seg->n_rows + n_new > seg->row_stride)
    return fail(UC_E_INVALID, "n_rows + n_new = %lld > row_stride %d",
                (long long)seg->n_rows + n_new, seg->row_stride);
  if (n_new == 0) return ok();
  if (!k_new || !v_new) return fail(UC_E_INVALID, "k_new or v_new is NULL");
  if (!aligned16(k_new) || !aligned16(v_new)) return fail(UC_E_INVALID, "k_new/v_new not 16-byte aligned");
  return launched(launch_stream_append(*shape, ks, k_new, v_new, n_new, (hipStream_t)stream));
}

size_t uc_topk_mass_workspace_size(int BH, int k) {
  if (BH < 1 || k < 0) return 0;
  return (((size_t)BH * k * sizeof(int32_t)) + 255) & ~(size_t)255;
}

uc_status uc_topk_mass(const float* scores, int BH, int N, int k, float* frac_out, void* ws,
                       size_t ws_bytes, void* stream) {
  if (BH < 1 || N < 0) return fail(UC_E_INVALID, "BH must be >= 1 and N >= 0");
  if (k < 0 || k > N) return fail(UC_E_INVALID, "k = %d outside [0, N = %d]", k, N);
  if (!frac_out || (N > 0 && !scores)) return fail(UC_E_INVALID, "NULL pointer");
  const size_t need = uc_topk_mass_workspace_size(BH, k);
  if (k > 0 && (ws_bytes < need || !ws)) return fail(UC_E_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  return launched(launch_topk_mass(scores, BH, N, k, frac_out, (int32_t*)ws, (hipStream_t)stream));
}

uc_status uc_compose_index(const int32_t* outer, int n_outer, const int32_t* inner, int BH, int k,
                           int32_t* out, void* stream) {
  if (BH < 0 || k < 0 || n_outer < 0) return fail(UC_E_INVALID, "BH, k and n_outer must be >= 0");
  if ((int64_t)BH * k == 0) return ok();
  if (!outer || !inner || !out) return fail(UC_E_INVALID, "NULL pointer");
  const char* o0 = (const char*)out;
  const char* o1 = o0 + (size_t)BH * k * sizeof(int32_t);
  auto overlaps = [&](const int32_t* p, size_t n) {
    const char* a = (const char*)p;
    return a < o1 && o0 < a + n * sizeof(int32_t);
  };
  if (overlaps(outer, (size_t)BH * n_outer) || overlaps(inner, (size_t)BH * k))
    return fail(UC_E_INVALID, "out overlaps outer or inner");
  return launched(launch_compose_index(outer, n_outer, inner, BH, k, out, (hipStream_t)stream));
}

// ---------------------------------------------------------------- append
uc_status uc_append_rows(const uc_shape* shape, const void* k_new, const void* v_new, int n_new,
                         const uc_segment* seg, int pos, void* stream) {
  uc_status st = check_shape(shape);
  if (st) return st;
  if (!seg || seg->kind != UC_SEG_DENSE) return fail(UC_E_INVALID, "seg must be a dense segment");
  KSeg ks;
  st = check_segment(*shape, *seg, 0, ks, false);
  if (st) return st;
  if (n_new < 0 || pos < 0) return fail(UC_E_INVALID, "n_new and pos must be >= 0");
  if ((int64_t)pos + n_new > ks.row_stride)
    return fail(UC_E_INVALID, "pos + n_new = %lld > row_stride %d", (long long)pos + n_new, ks.row_stride);
  if (n_new == 0) return ok();
  if (!k_new || !v_new || !seg->k || !seg->v) return fail(UC_E_INVALID, "NULL pointer");
  if (!aligned16(k_new) || !aligned16(v_new)) return fail(UC_E_INVALID, "k_new/v_new not 16-byte aligned");
  ks.k = seg->k;
  ks.v = seg->v;
  return launched(launch_append(*shape, k_new, v_new, n_new, ks, pos, (hipStream_t)stream));
}

// ---------------------------------------------------------------- host helpers
int64_t uc_dense_bytes(int64_t rows, int D, uc_dtype dt) {
  return rows * 2 * (int64_t)D * dtype_bytes(dt);
}

int64_t uc_evicted_bytes(int64_t rows, int D, uc_dtype dt) {
  return rules::evicted_bytes(rows, D, dtype_bytes(dt));
}

int64_t uc_packed_bytes(int64_t N, int D, int G, int bits, uc_dtype dt) {
  if (!dtype_ok(dt)) return -1;
  return rules::packed_bytes(N, D, G, bits, dtype_bytes(dt));
}

int64_t uc_evict_rows_for_budget(double budget_bytes, double fixed_bytes, int64_t N, int D,
                                 uc_dtype dt) {
  return rules::evict_rows(budget_bytes, fixed_bytes, N, D, dtype_bytes(dt));
}

int uc_quant_config(double budget_bytes, int64_t N, int D, uc_dtype dt, int n_heads, int first,
                    int* bits, int* group) {
  if (D < 32 || !pow2(D) || N < 0 || n_heads < 1 || !dtype_ok(dt)) return -1;
  if (first < 0 || first >= 3 * rules::quant_groups(D)) return -1;
  return rules::quant_config(budget_bytes, N, D, dtype_bytes(dt), n_heads, first, bits, group);
}

uc_status uc_assign_bits(int n_heads, const float* mass, int64_t N, int D, int G, uc_dtype dt,
                         double budget_bytes, double fixed_bytes, uint8_t* bits_out) {
  if (n_heads < 1 || !mass || !bits_out) return fail(UC_E_INVALID, "bad arguments");
  const int64_t b2 = uc_packed_bytes(N, D, G, 2, dt), b4 = uc_packed_bytes(N, D, G, 4, dt);
  if (b2 < 0) return fail(UC_E_INVALID, "bad packed geometry");
  std::vector<int> order(n_heads);
  for (int i = 0; i < n_heads; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return mass[a] > mass[b]; });
  double total = fixed_bytes + (double)b2 * n_heads;
  for (int i = 0; i < n_heads; ++i) bits_out[i] = 2;
  for (int i = 0; i < n_heads; ++i) {
    if (total + (double)(b4 - b2) > budget_bytes) break;
    total += (double)(b4 - b2);
    bits_out[order[i]] = 4;
  }
  return ok();
}

uc_status uc_type_budget(int n_types, const double* mass, const double* b_prev, double B_total,
                         double* b_next) {
  if (n_types < 1 || n_types > 64 || !mass || !b_prev || !b_next)
    return fail(UC_E_INVALID, "bad arguments");
  rules::type_budget(n_types, mass, b_prev, B_total, b_next);
  return ok();
}

double uc_retention_next(double rho, double rho_init, double rho_min, double M_c, double M_0) {
  return rules::retention_next(rho, rho_init, rho_min, M_c, M_0);
}

// ---------------------------------------------------------------- budget decisions on the device
uc_status uc_budget_step(const uc_budget_params* p, const float* mass, int n_steps,
                         uc_budget_state* state, void* stream) {
  if (!p || !mass || !state) return fail(UC_E_INVALID, "NULL pointer");
  if (p->Hq < 1 || p->Hkv < 1 || p->Hq % p->Hkv || p->M < 1 || p->D < 32 || !pow2(p->D))
    return fail(UC_E_INVALID, "bad Hq / Hkv / M / D (%d, %d, %d, %d)", p->Hq, p->Hkv, p->M, p->D);
  if (p->n_segs < 1 || p->n_segs > kMaxSeg) return fail(UC_E_INVALID, "n_segs %d", p->n_segs);
  if (p->ev < 0 || p->ev >= p->n_segs || p->qt < 0 || p->qt >= p->n_segs || p->ev == p->qt)
    return fail(UC_E_INVALID, "ev (%d) and qt (%d) must be distinct segments", p->ev, p->qt);
  if (p->n_ev < 0 || p->n_qt < 0 || !dtype_ok(p->dtype)) return fail(UC_E_INVALID, "bad rows or dtype");
  if (!(p->rho_min > 0.0 && p->rho_min <= p->rho_init && p->rho_init <= 1.0))
    return fail(UC_E_INVALID, "need 0 < rho_min <= rho_init <= 1");
  if (n_steps < 1) return fail(UC_E_INVALID, "n_steps must be >= 1");
  if (((uintptr_t)state & 7u) || ((uintptr_t)mass & 3u)) return fail(UC_E_INVALID, "misaligned pointer");
  return launched(launch_budget_step(*p, mass, n_steps, state, (hipStream_t)stream));
}

uc_status uc_calibrate_policy(const float* frac, int rows, int n_types, double threshold,
                              double* conc_out, int32_t* evict_out, void* stream) {
  if (rows < 1 || n_types < 1 || n_types > kMaxSeg) return fail(UC_E_INVALID, "bad rows or n_types");
  if (!frac || !conc_out || !evict_out) return fail(UC_E_INVALID, "NULL pointer");
  if (!isfinite(threshold)) return fail(UC_E_INVALID, "threshold must be finite");
  return launched(launch_calibrate_policy(frac, rows, n_types, threshold, conc_out, evict_out,
                                          (hipStream_t)stream));
}

}  // extern "C"

// ---------------------------------------------------------------- read probe
size_t uc_read_probe_unit(void) { return (size_t)4096 * read_probe_wgs(); }
size_t uc_read_probe_sink_bytes(void) { return (size_t)16 * 4 * read_probe_wgs(); }

uc_status uc_read_probe(const void* buf, size_t bytes, int pattern, void* sink, void* stream) {
  if (!buf || !sink) return fail(UC_E_INVALID, "buf or sink is NULL");
  if (pattern != UC_PROBE_LINES && pattern != UC_PROBE_OPERAND)
    return fail(UC_E_INVALID, "unknown probe pattern %d", pattern);
  const size_t unit = uc_read_probe_unit();
  if (bytes == 0 || bytes % unit)
    return fail(UC_E_INVALID, "bytes %zu is not a positive multiple of %zu", bytes, unit);
  return launched(launch_read_probe(buf, bytes, pattern, sink, (hipStream_t)stream));
}
