/*
 * unicache.h -- C ABI of the mixed-policy KV-cache attention library for
 * AMD Instinct MI355X (gfx950).
 *
 * The library implements the data-parallel hot path of UniCache
 * ("UniCache: Task- and Type-Aware KV Cache Compression for Unified
 * Multimodal Models"): attention over a KV cache split into typed segments,
 * each segment stored under its own compression policy (Sec. 3.1, Sec. 3.4,
 * App. E "Physical, type-aware KV storage").
 *
 *   uc_score_importance  attention-probability importance per cached token and
 *                        attention mass per segment (Sec. 3.3, Eq. 1;
 *                        App. E "Efficient attention-guided allocation")
 *   uc_score_columns     the same scores from the row normalisers of an
 *                        attention pass already run (its second pass only)
 *   uc_select_keep       per-KV-head top-k token eviction with compaction
 *   uc_evict_step        the same with the row count read on the device
 *                        (App. E "Batched GQA token selection")
 *   uc_quantize_segment  group-wise asymmetric low-bit quantization
 *                        (App. E "Physical, type-aware KV storage")
 *   uc_attend_mixed      one shared-softmax attention pass over dense,
 *                        compacted and packed segments
 *                        (App. E "Attention over heterogeneous cache segments")
 *   uc_append_rows       decode-time write of new K/V rows into a protected
 *                        dense segment (Sec. 3.1, protected objects)
 *   uc_attend_append     one decode step: the append and the attention in
 *                        one launch (Sec. 3.1 and App. E)
 *   uc_plan_*            decode steps on a frozen, validated layout
 *                        (App. E "Cached metadata and execution plans")
 *   host helpers         byte accounting and budget -> policy configuration
 *                        (Sec. 3.3 Eq. 2 and Eq. 3, Sec. 3.4)
 *
 * Conventions shared by every call
 * --------------------------------
 * - Tensors are row-major with the innermost dimension last.
 * - Query head h attends through KV head h / (Hq / Hkv) (grouped-query
 *   attention; the query heads of one KV head form its "group").
 * - Device pointers are plain HIP device addresses; `stream` is a
 *   hipStream_t passed as void* (NULL = the default stream).
 * - Ownership: the caller allocates every input, output and workspace
 *   buffer.  The library never allocates or frees device memory, never
 *   synchronises the stream, and only enqueues work on `stream`.  Buffers
 *   must stay valid until that work completes.
 * - Errors: every argument check happens on the host before any launch; on
 *   error nothing is written and no work is enqueued.  UC_E_INVALID covers
 *   bad sizes, null required pointers and misaligned pointers,
 *   UC_E_UNSUPPORTED a legal but unimplemented combination, UC_E_WORKSPACE
 *   a workspace smaller than the matching *_workspace_size helper reports,
 *   UC_E_DEVICE a HIP error reported at launch.  uc_last_error() returns a
 *   thread-local text describing the last failure of the calling thread.
 * - Values stored in device memory (codes, per-head bit widths, offsets)
 *   are not inspected on the host.  Kernels bound every access by the
 *   capacities given in the descriptors; a head whose device-side offsets
 *   would leave those capacities is skipped and its outputs are set to NaN.
 *   NaN or Inf inside K, V, Q or scores gives undefined (but in-bounds)
 *   results.
 */
#ifndef UNICACHE_H
#define UNICACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Every enum below also names the ends of the 32-bit range, so that any
 * int32 a caller passes is a value of the type (out-of-range values are then
 * rejected by the checks, not undefined); these two are never valid
 * arguments. */
#define UC_ENUM_RANGE(p) p##_RANGE_MIN_ = -2147483647 - 1, p##_RANGE_MAX_ = 2147483647

typedef enum {
  UC_OK = 0,
  UC_E_INVALID = 1,
  UC_E_UNSUPPORTED = 2,
  UC_E_WORKSPACE = 3,
  UC_E_DEVICE = 4,
  UC_ENUM_RANGE(UC_STATUS)
} uc_status;

/* Element type of dense rows, residual-tail rows, queries and of the value a
 * dequantised code is rounded to (round-to-nearest-even). */
typedef enum { UC_F32 = 0, UC_F16 = 1, UC_BF16 = 2, UC_ENUM_RANGE(UC_DTYPE) } uc_dtype;

/* Storage kind of one segment (App. E "Physical, type-aware KV storage"):
 * UC_SEG_DENSE  rows kept in their original representation -- protected
 *               segments, segments kept at full precision, and the compacted
 *               survivors of an eviction policy (ascending token order);
 * UC_SEG_PACKED low-bit codes with per-group scales and minima plus a short
 *               residual tail of rows held in `dtype`. */
typedef enum { UC_SEG_DENSE = 0, UC_SEG_PACKED = 1, UC_ENUM_RANGE(UC_SEG_KIND) } uc_seg_kind;

/* Batch B, query heads Hq, KV heads Hkv (Hq % Hkv == 0), head dim D. */
typedef struct {
  int32_t B, Hq, Hkv, D;
} uc_shape;

#define UC_MAX_SEGMENTS 8

/* One segment of the logical KV sequence.  Segments are passed as an array in
 * logical token order; attention treats their rows as one sequence under one
 * softmax (Sec. 3.4: compressed candidates and protected segments are
 * reassembled in their original order).
 *
 * Dense segment (kind = UC_SEG_DENSE):
 *   k, v      [B, Hkv, row_stride, D] elements of `dtype`; rows 0..n_rows-1 of
 *             each (b, h_kv) are live.  row_stride = 0 means n_rows.
 *   idx       optional int32 [B, Hkv, n_rows] logical positions of the rows
 *             (an eviction policy's survivors); carried for the caller, never
 *             read by attention (softmax is invariant to row order).
 *
 * Packed segment (kind = UC_SEG_PACKED), N = n_rows, G = group,
 * n_full = G * floor(N / G), tail_len = N - n_full, and the per-head strides
 * C_full = n_full, T = tail_len when row_stride = 0; with a row capacity
 * R = row_stride >= N (a segment that grows, see uc_stream_append)
 * C_full = G * floor(R / G) and T = G, so rows never move as N grows:
 *   bits      code width in {2, 4, 8}: the uniform width when head_bits is
 *             NULL, else an upper bound on the per-head widths (the library
 *             picks kernels from it).
 *   head_bits optional device uint8 [B*Hkv]: per-(b, h_kv) code width in
 *             {2, 4, 8}, at most bits; then code_off is required.  Heads
 *             whose entry breaks this get NaN attention outputs.
 *   code_off  device int64 [B*Hkv]: byte offset of each (b, h_kv)'s codes in
 *             codes_k / codes_v, a multiple of 16.  NULL (with head_bits NULL)
 *             means (b*Hkv + h) * C_full * D * bits / 8.
 *   codes_bytes  capacity in bytes of each of codes_k and codes_v.
 *   codes_k, codes_v  row r of a head occupies D*bits/8 bytes at
 *             offset + r*D*bits/8; channel c sits in byte c*bits/8 at bit
 *             (c % (8/bits)) * bits (least significant bits first).
 *   scale_k, min_k  float [B, Hkv, C_full/G, D] (the first n_full/G groups
 *             of each head live): keys are quantised per channel over groups
 *             of G consecutive rows.
 *   scale_v, min_v  float [B, Hkv, C_full, D/G] (the first n_full rows of
 *             each head live): values are quantised per row over groups of G
 *             consecutive channels.
 *   tail_k, tail_v  [B, Hkv, T, D] of `dtype`: rows 0..tail_len-1 of each
 *             head hold the last N - n_full rows, unquantised.  May be NULL
 *             when tail_len == 0 and row_stride == 0.
 *   A code q of a group with scale s and minimum m stands for the value
 *   round_to(dtype, fmaf((float)q, s, m)).
 *
 * All pointers of a packed segment must be 16-byte aligned; dense k/v must be
 * 16-byte aligned and D * sizeof(dtype) is a multiple of 16 by construction
 * (D in {64, 128}). */
typedef struct {
  int32_t kind;       /* uc_seg_kind */
  int32_t dtype;      /* uc_dtype */
  int32_t n_rows;     /* logical rows per (b, h_kv); may be 0 */
  int32_t row_stride; /* allocated rows per (b, h_kv) (capacity); 0 = n_rows */
  void* k;
  void* v;
  const int32_t* idx;
  int32_t group;
  int32_t bits;
  const uint8_t* head_bits;
  const int64_t* code_off;
  uint64_t codes_bytes;
  uint8_t* codes_k;
  uint8_t* codes_v;
  float* scale_k;
  float* min_k;
  float* scale_v;
  float* min_v;
  void* tail_k;
  void* tail_v;
} uc_segment;

/* ------------------------------------------------------------------------ */
/* Importance scoring (Sec. 3.3 Eq. 1 and its attention probabilities P;
 * App. E "Batched GQA token selection": scores are aggregated over the query
 * heads that share a KV head).
 *
 * For every (b, h_kv) let Q be the G*W observation rows (g, w) -- query head
 * h_kv*G + g, window position w -- of q_obs [B, Hq, W, D] (q_dt).  Each row's
 * logits s_j = sm_scale * <q, k_j> run over every row j of every segment in
 * logical order (packed rows dequantised), P = softmax over all of them, and
 *   scores_out[s][b, h_kv, j] = sum over the G*W rows of P_j   (j in segment s)
 *   mass_out[b, h_kv, s]       = sum over the G*W rows and j in s of P_j
 * Sums are accumulated in double and rounded once to float.
 * scores_out is a host array of n_segs device pointers; an entry (or the whole
 * array) may be NULL to skip that segment's scores.  mass_out is device float
 * [B, Hkv, n_segs] or NULL.  Dense segments may be fp32/fp16/bf16; a packed
 * segment's dequantised rows are rounded to its dtype.  ws must hold
 * uc_score_workspace_size(...) bytes. */
uc_status uc_score_importance(const uc_shape* shape, const uc_segment* segs,
                              int n_segs, const void* q_obs, uc_dtype q_dt,
                              int W, float sm_scale, float* const* scores_out,
                              float* mass_out, void* ws, size_t ws_bytes,
                              void* stream);

size_t uc_score_workspace_size(const uc_shape* shape, const uc_segment* segs,
                               int n_segs, int W);

/* Importance scores from the row log-sum-exps of an attention pass already
 * run over the same segments (Sec. 3.3 Eq. 1: P is the softmax whose
 * normaliser that pass computed; App. E "Efficient attention-guided
 * allocation": attention statistics gathered next to attention).  The result
 * is that of uc_score_importance with its first pass (each row's
 * log-sum-exp over every segment) replaced by the caller's values:
 *   q_obs, q_ld  observation row (b, h, w) at q_obs + ((b*Hq + h)*q_ld + w)*D
 *                (q_ld >= W; q_ld = W is the contiguous [B, Hq, W, D] block,
 *                and the last W rows of a [B, Hq, M, D] query block are
 *                q + (M - W)*D with q_ld = M);
 *   row_lse      device float; observation row (b, h, w) has its natural-log
 *                normaliser at row_lse[(b*Hq + h)*lse_ld + w], e.g. the lse
 *                output of uc_attend_mixed for the same query rows over the
 *                same segments (pass lse + (M - W) with lse_ld = M to score
 *                the last W of its M rows);
 *   lse_ld       >= W.
 * Every other argument, the outputs and the workspace
 * (uc_score_workspace_size) are as for uc_score_importance.  With mass_out
 * NULL only the segments whose scores_out entry is set are read; with
 * neither, nothing is enqueued.  The probabilities are exp(s - lse) with the
 * caller's lse: a normaliser that is not the log-sum-exp of the row gives
 * scores scaled by the ratio (rows of one head need not sum to G*W). */
uc_status uc_score_columns(const uc_shape* shape, const uc_segment* segs,
                           int n_segs, const void* q_obs, int64_t q_ld,
                           uc_dtype q_dt, int W, float sm_scale,
                           const float* row_lse, int64_t lse_ld,
                           float* const* scores_out, float* mass_out, void* ws,
                           size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Top-k token selection and physical compaction for one eviction-managed
 * segment (App. E "Batched GQA token selection" and "Physical, type-aware KV
 * storage": heavy-hitter plus recent-token selection per KV head, then only
 * the retained rows and their logical indices are stored).
 *
 * scores [BH, N] float (BH = B*Hkv rows).  For each row the last n_recent
 * positions are always kept; of the other N - n_recent positions the
 * k - n_recent with the largest (score, -index) are kept (equal scores: the
 * lower index wins).  keep_idx [BH, k] int32 receives the kept positions in
 * ascending order.  When k_src is non-NULL the kept rows of k_src/v_src
 * [BH, N, D] (dtype dt) are gathered, in the same order, into k_dst/v_dst
 * [BH, k, D].  0 <= n_recent <= k <= N.  ws must hold
 * uc_select_workspace_size(BH, N) bytes. */
uc_status uc_select_keep(const float* scores, int BH, int N, int k,
                         int n_recent, int32_t* keep_idx, const void* k_src,
                         const void* v_src, void* k_dst, void* v_dst,
                         uc_dtype dt, int D, void* ws, size_t ws_bytes,
                         void* stream);

size_t uc_select_workspace_size(int BH, int N);

/* One eviction step whose row count is decided on the device (Sec. 3.3
 * dynamic budget with the Sec. 3.4 translation: an eviction-managed type
 * keeps k rows per KV head; App. E "Batched GQA token selection" and
 * "Physical, type-aware KV storage").  With N = cur->n_rows and
 * k = max(*k_dev, 0), read by the kernels:
 *   k >= N  nothing is written (the caller keeps cur);
 *   k <  N  for each (b, h_kv) the rows of uc_select_keep(scores, BH, N, k,
 *           0, ...) -- the k largest (score, -index), ascending -- are
 *           copied to rows 0..k-1 of out, and out->idx[bh, j] receives
 *           cur->idx[bh, i] for the j-th kept row i (i itself when cur->idx
 *           is NULL, i.e. cur holds the segment's original rows).
 *   scores  device float [B*Hkv, N] (uc_score_importance / uc_score_columns
 *           output for cur);
 *   cur     dense segment; idx, when given, int32 with the rows' row_stride
 *           ([B, Hkv, row_stride]);
 *   out     dense segment of cur's dtype with row_stride >= N and k, v, idx
 *           non-NULL (idx int32 [B, Hkv, row_stride]); its n_rows is not
 *           read: after the call it holds k rows.  out must not overlap cur;
 *   k_dev   device int32, e.g. the k field of a uc_budget_state that
 *           uc_budget_step writes earlier on the same stream.
 * The host does not learn k from this call: it reads the decision back to
 * size the calls that follow.  Three launches; no workspace. */
uc_status uc_evict_step(const uc_shape* shape, const float* scores,
                        const uc_segment* cur, const int32_t* k_dev,
                        const uc_segment* out, void* stream);

/* ------------------------------------------------------------------------ */
/* Group-wise asymmetric min/max quantization of one segment (App. E
 * "Physical, type-aware KV storage": packed low-bit codes, scales, minima and
 * a short residual tail).
 *
 * k, v [B, Hkv, N, D] of dtype dt are read; `out` (kind UC_SEG_PACKED,
 * n_rows = N, dtype = dt) names the destination buffers, its bit widths and
 * its group G.  For a group x_1..x_G (keys: one channel over G consecutive
 * rows; values: G consecutive channels of one row), in IEEE binary32:
 *   mn = min x,  mx = max x,  s = (mx - mn) / (2^bits - 1),
 *   code = s > 0 ? clamp(rint((x - mn) / s), 0, 2^bits - 1) : 0
 * (rint rounds half to even).  Rows n_full..N-1 are copied unchanged to the
 * tail.  G must be a power of two in [8, 128] dividing D. */
uc_status uc_quantize_segment(const uc_shape* shape, const void* k,
                              const void* v, uc_dtype dt, int N,
                              const uc_segment* out, void* stream);

/* ------------------------------------------------------------------------ */
/* Attention over the mixed segments under one shared softmax (App. E
 * "Attention over heterogeneous cache segments"; chunk outputs merged with
 * log-sum-exp statistics).
 *
 * q [B, Hq, M, D] (q_dt) -> o float [B, Hq, M, D]:
 *   o = sum_j softmax_j(sm_scale * <q, k_j>) v_j
 * over every row j of every segment in logical order (packed rows
 * dequantised as described for uc_segment).  No causal mask.
 * lse     optional float [B, Hq, M]: natural-log log-sum-exp of the logits.
 * seg_lse optional float [B, Hq, M, n_segs]: the same restricted to one
 *         segment; -inf for a segment with no rows.
 * M = 1 is decode; M > 1 is a query block (prefill / denoising step).  The
 * sequence (sum of n_rows) must be non-empty.  ws must hold
 * uc_attend_workspace_size(...) bytes. */
uc_status uc_attend_mixed(const uc_shape* shape, const uc_segment* segs,
                          int n_segs, const void* q, uc_dtype q_dt, int M,
                          float sm_scale, float* o, float* lse, float* seg_lse,
                          void* ws, size_t ws_bytes, void* stream);

/* uc_attend_mixed for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same computation, kernels and results, with the workspace taken from
 * a static device array of UC_SCRATCH_BYTES bytes that the library holds on
 * every GPU it runs on until the process ends.  The call allocates nothing
 * (no hipMalloc, no allocating library routine); the caller still passes q,
 * o and the optional lse / seg_lse.  A call whose uc_attend_workspace_size
 * exceeds UC_SCRATCH_BYTES (large prefill blocks over packed segments) fails
 * with UC_E_UNSUPPORTED before any launch.  Every call on one GPU shares
 * that GPU's array: calls that may overlap on one GPU (different streams
 * without ordering between them) race and must not be issued; calls ordered
 * on one stream are safe.  The array's contents are not preserved between
 * calls and need no initialisation. */
#define UC_SCRATCH_BYTES (16u << 20)
uc_status uc_attend_mixed_noalloc(const uc_shape* shape, const uc_segment* segs,
                                  int n_segs, const void* q, uc_dtype q_dt, int M,
                                  float sm_scale, float* o, float* lse, float* seg_lse,
                                  void* stream);

/* Workspace bytes for uc_attend_mixed.  The value never decreases when a
 * segment gains rows, so a workspace sized for the largest row counts (say a
 * decode tail at full capacity) serves every call with fewer rows. */
size_t uc_attend_workspace_size(const uc_shape* shape, const uc_segment* segs,
                                int n_segs, uc_dtype q_dt, int M);

/* Per-segment attention mass from attention statistics (Sec. 3.3 Eq. 1: the
 * bracket summed over the query heads of one KV head and the query rows).
 * lse [B, Hq, M] and seg_lse [B, Hq, M, n_segs] as written by uc_attend_mixed;
 * mass_out [B, Hkv, n_segs] float receives
 *   sum over (g, m) of exp(seg_lse[b, h_kv*G + g, m, a] - lse[b, h_kv*G + g, m])
 * with each term the binary32 exponential of the exact double difference
 * (relative error below 1e-6), accumulated in double.  Dividing by G*M gives the Mean over heads and
 * queries of Eq. 1 for one layer and step. */
uc_status uc_segment_mass(const uc_shape* shape, int M, int n_segs,
                          const float* lse, const float* seg_lse,
                          float* mass_out, void* stream);

/* ------------------------------------------------------------------------ */
/* Decode append (Sec. 3.1: newly produced K/V belong to a protected segment
 * kept in its original representation).  Copies n_new rows of k_new / v_new
 * [B, Hkv, n_new, D] (dtype of seg) into rows pos..pos+n_new-1 of every
 * (b, h_kv) of the dense segment `seg`; requires pos + n_new <= row_stride.
 * The caller then raises seg->n_rows itself. */
uc_status uc_append_rows(const uc_shape* shape, const void* k_new,
                         const void* v_new, int n_new, const uc_segment* seg,
                         int pos, void* stream);

/* One decode step with the append fused in (Sec. 3.1 protected segment and
 * Sec. 3.4 attention over the reassembled sequence).  The result is that of
 *   uc_append_rows(shape, k_new, v_new, n_new, &segs[tail], segs[tail].n_rows)
 * followed by uc_attend_mixed over segs with segs[tail].n_rows raised by
 * n_new, up to the order of floating-point summation.
 *   segs[tail]   a dense segment with row_stride >= n_rows + n_new; its n_rows
 *                is the row count BEFORE this call, and the caller raises it
 *                by n_new afterwards (segs is read, never written).
 *   k_new, v_new [B, Hkv, n_new, D] device, dtype of segs[tail], 16-byte
 *                aligned; n_new = 0 is a plain uc_attend_mixed.
 *   q .. stream  as for uc_attend_mixed; ws needs uc_attend_workspace_size of
 *                the segments as they stand after the append.
 * With the decode matrix-core kernel (bf16, D = 128, (Hq/Hkv)*M <= 16, no
 * seg_lse, fewer than UC_MAX_SEGMENTS segments) one launch attends the new
 * rows straight from k_new / v_new and also stores them into segs[tail];
 * otherwise the library runs the two calls above (every check, the workspace
 * size included, comes before either launch, so an error stores nothing). */
uc_status uc_attend_append(const uc_shape* shape, const uc_segment* segs,
                           int n_segs, int tail, const void* k_new,
                           const void* v_new, int n_new, const void* q,
                           uc_dtype q_dt, int M, float sm_scale, float* o,
                           float* lse, float* seg_lse, void* ws,
                           size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Execution plans (App. E, "Cached metadata and execution plans": once a
 * physical layout is frozen, attention reuses its segment boundaries and type
 * identifiers instead of matching segments and preparing operators again).
 * A plan holds a copy of the segment descriptors and the device layout
 * derived from them, validated once; its calls then check only their own
 * pointers.  The layout is frozen except for segs[tail] (tail >= 0), a dense
 * segment with a row capacity whose row count the plan advances by every
 * decode step's n_new (the caller's descriptors are not written;
 * uc_plan_tail_rows reports the count); tail = -1 freezes every segment.
 * Host memory only; a plan is used by one thread at a time, and the segment
 * buffers it points into must outlive it.
 *   uc_plan_create   validates as uc_attend_append would (shape, segments,
 *                    q_dt, M, sm_scale; segs[tail] dense with row_stride >=
 *                    1 unless tail = -1; at most UC_MAX_SEGMENTS - 1
 *                    segments) and writes the new plan to *out (NULL on
 *                    error). */
typedef struct uc_plan_s* uc_plan;
uc_status uc_plan_create(const uc_shape* shape, const uc_segment* segs,
                         int n_segs, int tail, uc_dtype q_dt, int M,
                         float sm_scale, uc_plan* out);
/* Workspace bytes that serve every step of the plan up to the tail's
 * capacity on the kernel path selected when the plan was created
 * (uc_set_path); a call made after the path was switched needs that path's
 * uc_attend_workspace_size and fails with UC_E_WORKSPACE without it (0 for
 * a NULL plan). */
size_t uc_plan_workspace_size(uc_plan plan);
/* The tail's current row count (-1 for a NULL plan or one without a tail). */
int uc_plan_tail_rows(uc_plan plan);
/* Attention over the plan's segments as they stand: the result of
 * uc_attend_mixed(shape, segs, n_segs, q, q_dt, M, sm_scale, o, lse, seg_lse,
 * ws, ws_bytes, stream).  On the multi-query matrix-core path ((Hq/Hkv)*M >
 * 16) the first call with a given ws also prepares it -- packed rows
 * dequantised, V converted to fp16, the range flag -- and later calls with
 * the same ws reuse that preparation (App. E: packed KV dequantised into a
 * reusable workspace), so between them the segments' contents and ws must
 * not change: after writing to a segment (re-quantisation, appended rows
 * outside the plan) or using ws for other calls, call uc_plan_invalidate.
 * ws: at least uc_plan_workspace_size bytes. */
uc_status uc_plan_attend(uc_plan plan, const void* q, float* o, float* lse,
                         float* seg_lse, void* ws, size_t ws_bytes,
                         void* stream);
/* Drops the plan's prepared workspace; the next uc_plan_attend prepares it
 * again. */
uc_status uc_plan_invalidate(uc_plan plan);
/* One decode step on the plan: exactly uc_attend_append(shape, segs, n_segs,
 * tail, k_new, v_new, n_new, q, q_dt, M, sm_scale, o, lse, NULL, ws,
 * ws_bytes, stream) with the plan's arguments and the tail at its current row
 * count, which then advances by n_new (and a prepared workspace is dropped).
 * ws: at least uc_plan_workspace_size bytes.  A plan without a tail refuses
 * it.  On error nothing is enqueued and the row count stays. */
uc_status uc_plan_attend_append(uc_plan plan, const void* k_new,
                                const void* v_new, int n_new, const void* q,
                                float* o, float* lse, void* ws,
                                size_t ws_bytes, void* stream);
/* Frees the plan (NULL is allowed). */
uc_status uc_plan_destroy(uc_plan plan);

/* ------------------------------------------------------------------------ */
/* Host helpers: storage accounting and budget -> policy configuration
 * (Sec. 3.3 "S_a, the original storage cost"; Sec. 3.4: an eviction policy is
 * configured by how many tokens it keeps, a quantization policy by its
 * precision and grouping).  No device work. */

/* Bytes of one (b, h_kv) of a segment kept dense: rows * 2 * D * elem. */
int64_t uc_dense_bytes(int64_t rows, int D, uc_dtype dt);
/* Bytes of one (b, h_kv) of a compacted eviction segment: kept rows plus one
 * int32 logical index per row. */
int64_t uc_evicted_bytes(int64_t rows, int D, uc_dtype dt);
/* Bytes of one (b, h_kv) of a packed segment: codes, float scale/min of K and
 * V, and the residual tail in dt.  Returns -1 for invalid arguments. */
int64_t uc_packed_bytes(int64_t N, int D, int G, int bits, uc_dtype dt);
/* Largest k with fixed_bytes + uc_evicted_bytes(k) <= budget_bytes, clamped
 * to [0, N]. */
int64_t uc_evict_rows_for_budget(double budget_bytes, double fixed_bytes,
                                 int64_t N, int D, uc_dtype dt);
/* Per-head code widths of one batch element's quantised segment under a byte
 * budget: every head starts at 2 bits; heads are raised to 4 bits in
 * descending order of `mass` (equal mass: lower head first) while
 * fixed_bytes + the sum of packed bytes stays <= budget_bytes.
 * bits_out[n_heads]. */
uc_status uc_assign_bits(int n_heads, const float* mass, int64_t N, int D,
                         int G, uc_dtype dt, double budget_bytes,
                         double fixed_bytes, uint8_t* bits_out);

/* Sec. 3.3 Eq. 2: b_next[a] = min(b_prev[a], m[a] / sum_j m[j] * B_total),
 * with the budget a capped type cannot use redistributed proportionally to
 * mass over the uncapped types with positive mass until none is left or
 * every such type is capped.  n_types <= 64. */
uc_status uc_type_budget(int n_types, const double* mass, const double* b_prev,
                         double B_total, double* b_next);

/* Sec. 3.3 Eq. 3: rho_next = min(rho, max(rho_min, rho_init * M_c / M_0)),
 * requires 0 < rho_min <= rho_init <= 1 and M_0 > 0; returns NAN otherwise. */
double uc_retention_next(double rho, double rho_init, double rho_min,
                         double M_c, double M_0);

/* ------------------------------------------------------------------------ */
/* Dynamic storage budget of one request, decided on the device from the type
 * masses the attention passes produced (Sec. 3.3 Eq. 1-3; Sec. 3.4, a budget
 * becomes the rows an eviction-managed type keeps and the precision and
 * grouping of a quantisation-managed type; App. E "Efficient
 * attention-guided allocation": a small kernel determines the allocation for
 * the next chunk).  Two candidate types take part: segment `ev`
 * (eviction-managed) and segment `qt` (quantisation-managed); other segments
 * are kept and stay outside the budget. */
typedef struct {
  int32_t Hq, Hkv, D, M;   /* query heads, KV heads, head dim, query rows per timestep */
  int32_t n_segs;          /* segments per row of the mass array */
  int32_t ev, qt;          /* segment indices of the two candidate types */
  int32_t n_ev, n_qt;      /* their rows per KV head before any compression */
  int32_t dtype;           /* their element type (uc_dtype) */
  double rho_init, rho_min;
} uc_budget_params;

/* Device-resident state, 8-byte aligned; the caller zero-fills it before the
 * first boundary (n_boundaries = 0).  After each uc_budget_step:
 *   rho, B      retention ratio and total budget B = rho * (S_ev + S_qt),
 *               S_a = Hkv * dense bytes of type a's original rows
 *   M0          candidate mass of the first (full-KV) boundary
 *   m[0], m[1]  Eq. 1 chunk masses of ev and qt
 *   b[0], b[1]  Eq. 2 budgets of ev and qt in bytes (the b^(c-1) of the next)
 *   k           rows per KV head ev keeps: min(previous k, the rows whose
 *               bytes (2*D*elem + 4 per row) fit b[0] / Hkv)
 *   cfg, bits, group  qt's configuration (as uc_quant_config numbers them):
 *               the first at or after the previous one whose Hkv packed
 *               segments fit b[1]
 *   k_prev, cfg_prev  the values before this boundary (n_ev and -1 at the
 *               first): k < k_prev means re-selection, cfg != cfg_prev
 *               re-quantisation */
typedef struct {
  double rho, B, M0;
  double m[2];
  double b[2];
  int32_t k, cfg, bits, group;
  int32_t k_prev, cfg_prev;
  int32_t n_boundaries, reserved;
} uc_budget_state;

/* One chunk boundary.  mass: device float [n_steps, Hkv, n_segs], the raw
 * per-segment sums of the chunk's timesteps as uc_segment_mass writes them
 * (one request, B = 1).  Eq. 1: m_a = (1 / n_steps) sum over the steps of
 * (sum over KV heads of mass) / (Hq * M), summed in double.  At the first
 * boundary (the full-KV step, n_boundaries = 0): M0 = m_ev + m_qt,
 * rho = rho_init, b^(0) = S.  Later: rho = Eq. 3 with M_c = m_ev + m_qt.
 * Then B, Eq. 2 over (ev, qt) and the Sec. 3.4 translation; one workgroup,
 * enqueued on `stream`, no host synchronisation. */
uc_status uc_budget_step(const uc_budget_params* params, const float* mass, int n_steps,
                         uc_budget_state* state, void* stream);

/* Calibration-based policy assignment (Sec. 3.2; App. B "Calibration
 * Setting").  frac: device float [rows, n_types], one concentration per
 * (calibration example, KV head) and type, as uc_topk_mass writes them.
 * conc_out[a] (device double) = the mean over the rows of frac[., a], summed
 * in double in row order; evict_out[a] (device int32) = 1 if conc_out[a] >=
 * threshold (eviction), else 0 (quantisation).  n_types <= UC_MAX_SEGMENTS. */
uc_status uc_calibrate_policy(const float* frac, int rows, int n_types, double threshold,
                              double* conc_out, int32_t* evict_out, void* stream);

/* ------------------------------------------------------------------------ */
/* Kernel path selection for uc_attend_mixed (process-wide; for cross-checks):
 * UC_PATH_AUTO (default) uses the matrix-core kernels where the inputs allow
 * (bf16 rows and queries, D = 128, at most 16 query rows per KV head for
 * decode), UC_PATH_VALU forces the vector-ALU kernels for every input.
 * Returns the previous setting, or -1 for an unknown value. */
#define UC_PATH_AUTO 0
#define UC_PATH_VALU 1
int uc_set_path(int path);

/* ------------------------------------------------------------------------ */
/* Batched attention over requests of different segment layouts (App. E,
 * "Batched attention and CFG execution": compatible attention calls are
 * combined into one variable-length launch).  shape->B is the number of
 * requests; request r has its own segments segs[r][0 .. n_segs[r]-1], each
 * described with the layout of a single batch element (B = 1: k/v
 * [1, Hkv, row_stride, D], codes and scales of Hkv heads, ...), so row counts,
 * segment kinds and policies may differ between requests.  q [B, Hq, M, D]
 * and o [B, Hq, M, D], lse [B, Hq, M] (optional) are laid out as for B batch
 * elements.  Each request's o and lse equal those of uc_attend_mixed on its
 * own segments (up to the order of floating-point sums).  When every request
 * fits the matrix-core decode kernel (bf16, D = 128, G*M <= 16, packed groups
 * >= 32 and widths <= 4) all of them run in one launch (plus the merge of
 * partial results); otherwise the requests run one call each.  segs and
 * n_segs are host arrays; ws must hold uc_attend_batch_workspace_size(...)
 * bytes (descriptors and partial records).  No per-segment lse. */
uc_status uc_attend_batch(const uc_shape* shape, const uc_segment* const* segs,
                          const int* n_segs, const void* q, uc_dtype q_dt, int M,
                          float sm_scale, float* o, float* lse, void* ws,
                          size_t ws_bytes, void* stream);
size_t uc_attend_batch_workspace_size(const uc_shape* shape,
                                      const uc_segment* const* segs,
                                      const int* n_segs, uc_dtype q_dt, int M);

/* ------------------------------------------------------------------------ */
/* Dequantised rows of a packed segment (App. E storage; the stored-value
 * definition x_hat = round_to_dtype(fmaf(code, scale, min)) that attention
 * uses).  k_out and v_out [B, Hkv, seg->n_rows, D] in seg->dtype, device,
 * 16-byte aligned, receive rows 0 .. n_full-1 decoded and the residual tail
 * rows copied.  Used to re-quantise a segment at a lower width or coarser
 * grouping when its budget shrinks (Sec. 3.4; the loss is irreversible).
 * A head whose code offset or width lies outside the segment's capacities
 * gets NaN rows. */
uc_status uc_dequantize_segment(const uc_shape* shape, const uc_segment* seg,
                                void* k_out, void* v_out, void* stream);

/* Streaming residual tail (App. E storage: the N mod G most recent rows of a
 * quantised segment stay unquantised in its tail).  Appends n_new rows
 * k_new / v_new [B, Hkv, n_new, D] (seg->dtype, device, 16-byte aligned) to a
 * packed segment with a row capacity (row_stride > 0) and the uniform code
 * layout (head_bits and code_off NULL): the rows enter the tail, and every
 * time the tail holds G rows they are quantised as the segment's next row
 * group exactly as uc_quantize_segment quantises a group (key scale/min per
 * channel over the G rows, value scale/min per row and channel group), so the
 * segment always equals the quantisation of all its rows.  seg->n_rows is the
 * row count before the call; the caller adds n_new to it afterwards.
 * Requires n_rows + n_new <= row_stride; UC_E_UNSUPPORTED for per-head
 * widths.  Calls on one segment are ordered by the stream. */
uc_status uc_stream_append(const uc_shape* shape, const uc_segment* seg,
                           const void* k_new, const void* v_new, int n_new,
                           void* stream);

/* Attention concentration for calibration-based policy assignment (Sec. 3.2;
 * App. B, "Calibration Setting": the fraction of a type's attention mass that
 * its top 10 % of tokens capture; a type at 0.5 or above is assigned
 * eviction, otherwise quantisation).  For every row r < BH of scores [BH, N]
 * (non-negative, e.g. one segment's uc_score_importance output per
 * (b, h_kv)): frac_out[r] = (sum of the k largest scores) / (sum of all N
 * scores), summed in double; 0 when the sum is 0.  0 <= k <= N.  ws must hold
 * uc_topk_mass_workspace_size(BH, k) bytes. */
uc_status uc_topk_mass(const float* scores, int BH, int N, int k, float* frac_out,
                       void* ws, size_t ws_bytes, void* stream);
size_t uc_topk_mass_workspace_size(int BH, int k);

/* Logical indices after a second eviction inside already compacted rows
 * (App. E: retained entries keep their logical token indices; Sec. 3.3:
 * eviction is irreversible, so a smaller budget selects among the rows still
 * kept).  out[bh, j] = outer[bh, inner[bh, j]] for bh < BH and j < k, where
 * outer [BH, n_outer] holds the logical indices of the compacted rows and
 * inner [BH, k] the positions kept among them (as uc_select_keep returns
 * them); an inner value outside [0, n_outer) gives -1.  All int32, device;
 * out must not overlap outer or inner. */
uc_status uc_compose_index(const int32_t* outer, int n_outer, const int32_t* inner,
                           int BH, int k, int32_t* out, void* stream);

/* Sec. 3.4: a quantisation policy's budget sets its precision and grouping.
 * Configurations are numbered in decreasing fidelity: widths 8, 4, 2 bits
 * and, within one width, groups 32, 64, ..., D (finer first); configuration
 * i has bits = 8 >> (i / ng), group = 32 << (i % ng), ng = log2(D / 32) + 1.
 * Returns the first configuration at or after `first` (a type never regains
 * fidelity it gave up) whose n_heads packed segments of N rows fit
 * budget_bytes, or the last one if none fits, and writes its bits and group;
 * -1 for invalid arguments (D not a power of two >= 32, N < 0, n_heads < 1,
 * first out of range). */
int uc_quant_config(double budget_bytes, int64_t N, int D, uc_dtype dt, int n_heads,
                    int first, int* bits, int* group);

/* ------------------------------------------------------------------------ */
/* Timing hook (instrumentation, for measuring the attention kernel on its
 * own).  The next attention call (uc_attend_mixed, uc_attend_append or
 * uc_attend_batch) made on the calling thread records
 * `start` on its stream immediately before the kernel that reads the
 * segments and `stop` immediately after it, so the pair brackets that kernel
 * alone: the merge of partial results and the prefill path's dequantisation
 * pass fall outside it.  Both are hipEvent_t handles passed as void*,
 * created and owned by the caller; either may be NULL.  The setting is per
 * thread and applies to exactly one such call, which clears it
 * (also when that call fails validation, in which case nothing is recorded).
 * An event-record failure makes that call return UC_E_DEVICE. */
uc_status uc_set_kernel_events(void* start, void* stop);

/* Streaming-read probe (instrumentation: the rate at which a plain read of
 * HBM proceeds on this device, for the attention kernels' roofline fractions
 * to be read against).  Reads the device buffer buf[0 .. bytes) once with
 * non-temporal 16-byte loads in the decode kernel's launch shape: two
 * 256-thread workgroups per CU, workgroup g streaming the g-th of
 * 2*CUs equal contiguous regions, its four waves taking 4 KB pieces (16 rows
 * of 256 bytes) in turn.  UC_PROBE_LINES loads each piece as whole 128-byte
 * lines (four rows per load); UC_PROBE_OPERAND in the A-operand layout of a
 * 16x16x32 matrix instruction (16 rows x 64 bytes per load, half of each
 * line), the pattern of loading keys straight into operand registers.  Wave
 * w of workgroup g stores the XOR of the 16-byte words it read into
 * sink[(4g + w) * 16 .. +16) (uc_read_probe_sink_bytes() bytes in all, device
 * memory owned by the caller).  UC_E_INVALID for NULL pointers, an unknown
 * pattern, or bytes not a positive multiple of uc_read_probe_unit(). */
#define UC_PROBE_LINES 0
#define UC_PROBE_OPERAND 1
size_t uc_read_probe_unit(void);
size_t uc_read_probe_sink_bytes(void);
uc_status uc_read_probe(const void* buf, size_t bytes, int pattern, void* sink,
                        void* stream);

/* ------------------------------------------------------------------------ */
const char* uc_status_string(uc_status s);
/* Thread-local description of the calling thread's last error ("" if none). */
const char* uc_last_error(void);
/* Name of the main kernel the calling thread's last successful launch of
 * uc_attend_mixed, uc_attend_append, uc_attend_batch or uc_score_importance
 * ran ("decode_mfma", "decode_mfma_append", "prefill_mfma", "attend_valu",
 * "decode_batch", "score_mfma", "score_valu"; "" before any).  Lets tests
 * assert the path a case reaches; static storage, never freed. */
const char* uc_last_kernel(void);

#ifdef __cplusplus
}
#endif

#endif /* UNICACHE_H */
