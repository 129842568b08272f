// score_mfma.hip -- attention-guided importance scores on the CDNA4 matrix
// cores (Sec. 3.2, Eq. 1 and App. E, "Batched GQA token selection": the
// attention probability each cached token receives from the observation
// queries, summed over the query heads that share its KV head).
//
// For one KV head the observation block is the G*W query rows of its query
// heads (row g*W + w is head h_kv*G + g, position w; these rows are
// contiguous in q).  Softmax normalises each query row over every key of
// every segment, so the scores take two passes over the keys:
//   pass 1  per (key chunk, query block of <= 256 rows, b*h_kv): running
//           maximum and sum of exp2 per query row over the chunk's keys, one
//           (m, l) record per (row, chunk); the attention combine kernel
//           merges the records into the row log-sum-exps.
//   pass 2  per (key chunk, b*h_kv): p = exp2(s - lse) for every query row,
//           summed over the rows per key (column sums), for all query blocks
//           of the head; the per-key sums are written as the scores and
//           their total is the chunk's probability mass (Eq. 1 bracket).
// Both passes compute S^T = K Q^T with v_mfma_f32_16x16x32_bf16: a wave
// takes 32-key tiles of the chunk (keys straight from HBM into the A-operand
// layout; packed rows decoded in registers to their stored bf16 values) and
// runs them against every 16-row query tile of the block, whose B operands
// it reads from the block staged in LDS.  Logits are in base 2 (q.k times
// scale*log2(e)).
// Column sums: a lane sums its key's probabilities over the query tiles in
// fp32, the 16 query columns of a tile are added by a butterfly, and the
// query blocks are accumulated in fp64 in LDS; chunk masses are fp64.
#include <algorithm>

#include "mfma_util.h"
#include "uc_common.h"

namespace uc {
namespace {

using namespace mf;

constexpr int WAVES = 4;
constexpr int TPW = 4;               // key tiles per wave and sub-chunk
constexpr int SUB = WAVES * TPW * TILE;  // 512 keys per sub-chunk (K held in registers)
constexpr int CHUNK = 2 * SUB;       // keys per workgroup
constexpr int QB = 256;              // query rows per block (16 tiles)
constexpr int QT = QB / 16;
constexpr int QROW = D * 2 + 16;     // bytes of one staged query row (16 B padding)
constexpr float kLazy = 8.0f;

// A wave's TPW key tiles of a sub-chunk as A operands: k[i][blk*4 + t] =
// row (tile i) blk*16 + i16, dims t*32 + g4*8 .. +7.  Rows past the
// descriptor's end read as zeros.
struct KTiles {
  u4 k[TPW][8];
};

__device__ inline void k_issue(__amdgpu_buffer_rsrc_t rk, int row0, int lane, u4 (&k)[8]) {
  const int i16 = lane & 15, g4 = lane >> 4;
  const int ko = (row0 + i16) * ROWB + g4 * 16;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    k[t] = bload(rk, ko, t * 64);
    k[4 + t] = bload(rk, ko, 16 * ROWB + t * 64);
  }
}

// Where one (b, h_kv)'s key rows of a segment come from: dense rows, or
// (packed) code rows 0 .. n_full-1 decoded in registers and residual-tail
// rows n_full .. read as stored.  n_full is a multiple of the group G >= 32,
// so a 32-row tile is all codes or all tail, and a code tile lies inside one
// key group (one scale and minimum per channel).
struct KSrc {
  __amdgpu_buffer_rsrc_t rk;   // dense rows, or the tail rows of a packed segment
  __amdgpu_buffer_rsrc_t rc;   // packed: this head's code rows
  const float* sk;             // packed: this head's key scales [groups, D]
  const float* mk;             // packed: this head's key minima
  int n_full, bits, G;         // n_full = 0 for dense segments
  bool bad;                    // packed head whose device-side layout is invalid
};

__device__ inline KSrc k_source(const KSeg& ks, int bh, int r1) {
  KSrc src{};
  if (ks.kind == UC_SEG_DENSE) {
    const int64_t base = (int64_t)bh * ks.row_stride * D;
    src.rk = rsrc((const uint16_t*)ks.k + base, (uint32_t)r1 * ROWB);
    return src;
  }
  src.n_full = ks.n_full;
  src.G = ks.group;
  const int64_t tb = (int64_t)bh * ks.tail_stride * D;
  src.rk = rsrc((const uint16_t*)ks.tail_k + tb, (uint32_t)max(0, r1 - ks.n_full) * ROWB);
  int bits;
  int64_t off;
  src.bad = !head_codes(ks, bh, D, bits, off) || (off & 15);
  src.bits = bits;
  const uint32_t rb = (uint32_t)(D * bits / 8);
  src.rc = rsrc(ks.codes_k + (src.bad ? 0 : off), src.bad ? 0u : (uint32_t)ks.n_full * rb);
  src.sk = ks.scale_k + (int64_t)bh * ks.kgroups * D;
  src.mk = ks.min_k + (int64_t)bh * ks.kgroups * D;
  return src;
}

// 8 channels of one code word (BITS per channel, least significant first)
// as bf16 A-operand bits: round_to_bf16(fmaf(code, scale, min)), the stored
// value of each code
template <int BITS>
__device__ inline u4 k_decode8(uint64_t w, const float (&sc)[8], const float (&mn)[8]) {
  constexpr uint32_t mask = (1u << BITS) - 1;
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float a = fmaf((float)(uint32_t)((w >> (2 * j * BITS)) & mask), sc[2 * j], mn[2 * j]);
    const float b = fmaf((float)(uint32_t)((w >> ((2 * j + 1) * BITS)) & mask), sc[2 * j + 1],
                         mn[2 * j + 1]);
    o[j] = bf2(a, b);
  }
  return u4{o[0], o[1], o[2], o[3]};
}

// channels c0 .. c0+7 of code rows ra and ra + 16 (one key group: shared
// scales and minima)
template <int BITS>
__device__ inline void k_decode_pair(const KSrc& src, int ra, int c0, u4& ka, u4& kb) {
  const int rb = D * BITS / 8;
  uint64_t wa, wb;
  if (BITS == 4) {
    wa = bload32(src.rc, ra * rb + c0 / 2, 0);
    wb = bload32(src.rc, (ra + 16) * rb + c0 / 2, 0);
  } else if (BITS == 2) {
    wa = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(src.rc, ra * rb + c0 / 4, 0, 0);
    wb = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(src.rc, (ra + 16) * rb + c0 / 4, 0, 0);
  } else {
    wa = __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(src.rc, ra * rb + c0, 0, 0));
    wb = __builtin_bit_cast(uint64_t,
                            __builtin_amdgcn_raw_buffer_load_b64(src.rc, (ra + 16) * rb + c0, 0, 0));
  }
  const int64_t g = (int64_t)(ra / src.G) * D + c0;
  const f4 s0 = *reinterpret_cast<const f4*>(src.sk + g), s1 = *reinterpret_cast<const f4*>(src.sk + g + 4);
  const f4 m0 = *reinterpret_cast<const f4*>(src.mk + g), m1 = *reinterpret_cast<const f4*>(src.mk + g + 4);
  const float sc[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
  const float mn[8] = {m0[0], m0[1], m0[2], m0[3], m1[0], m1[1], m1[2], m1[3]};
  ka = k_decode8<BITS>(wa, sc, mn);
  kb = k_decode8<BITS>(wb, sc, mn);
}

// a wave's 32-row key tile at row0 as A operands (see KTiles); without
// PACKED every segment of the call is dense
template <bool PACKED>
__device__ inline void k_load(const KSrc& src, int row0, int lane, u4 (&k)[8]) {
  if (!PACKED || row0 >= src.n_full) {  // dense rows, or a packed segment's tail
    k_issue(src.rk, row0 - src.n_full, lane, k);
    return;
  }
  const int i16 = lane & 15, g4 = lane >> 4;
  if (src.bad) {
    const uint32_t nan2 = 0x7FC07FC0u;
#pragma unroll
    for (int t = 0; t < 8; ++t) k[t] = u4{nan2, nan2, nan2, nan2};
    return;
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int c0 = t * 32 + g4 * 8;
    if (src.bits == 4) k_decode_pair<4>(src, row0 + i16, c0, k[t], k[4 + t]);
    else if (src.bits == 2) k_decode_pair<2>(src, row0 + i16, c0, k[t], k[4 + t]);
    else k_decode_pair<8>(src, row0 + i16, c0, k[t], k[4 + t]);
  }
}

// B operands (Q^T) of query tile qt, four 32-dim steps, from the staged block
__device__ inline void q_tile(const char* qs, int qt, int lane, u4 (&qb)[4]) {
  const int i16 = lane & 15, g4 = lane >> 4;
  const char* qrow = qs + (qt * 16 + i16) * QROW + g4 * 16;
#pragma unroll
  for (int t = 0; t < 4; ++t) qb[t] = *reinterpret_cast<const u4*>(qrow + t * 64);
}

// S^T of a key tile against one query tile: s0 = keys 0..15, s1 = keys
// 16..31; lane (i16, g4) holds keys g4*4 + j (+16) of query column i16
__device__ inline void s_tile(const u4 (&k)[8], const u4 (&qb)[4], f4& s0, f4& s1) {
  s0 = f4{0.f, 0.f, 0.f, 0.f};
  s1 = s0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    s0 = mfma(k[t], qb[t], s0);
    s1 = mfma(k[4 + t], qb[t], s1);
  }
}

// stage query rows [q0, q0 + QB) of the head's observation block (rows past nq
// are zero) into LDS; row g*W + w of the block is window row w of the
// group's query head g, which starts ld rows after head g - 1
__device__ inline void stage_q(char* qs, const uint16_t* qh, int q0, int nq, int W, int ld) {
  for (int e = threadIdx.x; e < QB * (D / 8); e += blockDim.x) {
    const int r = e / (D / 8), c = e % (D / 8);
    u4 v = u4{0, 0, 0, 0};
    if (q0 + r < nq) {
      const int g = (q0 + r) / W, w = q0 + r - g * W;
      v = *reinterpret_cast<const u4*>(qh + ((int64_t)g * ld + w) * D + c * 8);
    }
    *reinterpret_cast<u4*>(qs + r * QROW + c * 16) = v;
  }
}

// chunk c of the plan -> segment and row range
__device__ inline int chunk_rows(const ChunkPlan& p, const KSegs& segs, int c, int& r0, int& r1) {
  int si = 0;
  while (si + 1 < segs.n && c >= p.first[si + 1]) ++si;
  r0 = (c - p.first[si]) * p.rows[si];
  r1 = min(r0 + p.rows[si], segs.s[si].n_rows);
  return si;
}

// raw logits of one lane for one key tile: 8 keys (tile rows g4*4 + j and
// 16 + g4*4 + j); with MASK, keys at or past r1 are -inf
template <bool MASK>
__device__ inline void logits(const f4& s0, const f4& s1, int row0, int r1, int g4, float* x) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    x[j] = !MASK || row0 + g4 * 4 + j < r1 ? s0[j] : -INFINITY;
    x[4 + j] = !MASK || row0 + 16 + g4 * 4 + j < r1 ? s1[j] : -INFINITY;
  }
}

// Pass 1 on two key tiles (16 keys of the lane's query column): the lane's
// running (m, l) over base-2 logits, re-referenced to the maximum so far, so
// every v_exp_f32 argument is <= 0 (probabilities below 2^-126 of the
// reference flush to zero).  A lane with no valid key yet keeps m = -inf and
// l = 0.
template <bool MASK>
__device__ inline void lse_half(const f4 (&s)[2][2], int row0a, int row0b, int r1, int g4,
                                float scale_log2, float& m, float& l) {
  float x[16];
  logits<MASK>(s[0][0], s[0][1], row0a, r1, g4, x);
  logits<MASK>(s[1][0], s[1][1], row0b, r1, g4, x + 8);
  float mx[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) mx[j] = fmaxf(fmaxf(x[j], x[4 + j]), fmaxf(x[8 + j], x[12 + j]));
  // the scale is positive: the maximum of the raw logits gives it
  const float mn = fmaxf(m, fmaxf(fmaxf(mx[0], mx[1]), fmaxf(mx[2], mx[3])) * scale_log2);
  const float ref = mn == -INFINITY ? 0.0f : mn;
  float e[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int j = 0; j < 16; ++j) e[j & 3] += __builtin_amdgcn_exp2f(fmaf(x[j], scale_log2, -ref));
  l = fmaf(l, __builtin_amdgcn_exp2f(m - ref), (e[0] + e[1]) + (e[2] + e[3]));
  m = mn;
}

// Pass 2 on two key tiles: p = exp2(s - lse) added to the lanes' column sums
// (p <= 1 since s <= lse; probabilities below 2^-126 flush to zero)
__device__ inline void col_half(const f4 (&s)[2][2], float lq, float scale_log2, float (&c0)[8],
                                float (&c1)[8]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    c0[j] += __builtin_amdgcn_exp2f(fmaf(s[0][0][j], scale_log2, -lq));
    c0[4 + j] += __builtin_amdgcn_exp2f(fmaf(s[0][1][j], scale_log2, -lq));
    c1[j] += __builtin_amdgcn_exp2f(fmaf(s[1][0][j], scale_log2, -lq));
    c1[4 + j] += __builtin_amdgcn_exp2f(fmaf(s[1][1][j], scale_log2, -lq));
  }
}

static_assert(TPW == 4, "the sub-chunk loops take a wave's key tiles in two pairs");

// One sub-chunk of pass 1 for one wave.  The loop over query tiles keeps the
// matrix cores and the vector ALUs busy together: while the exponentials of
// one pair of key tiles run, the scores of the next pair are computed (the
// pair (2, 3) of query tile t, then the pair (0, 1) of tile t + 1).  The
// loop body has no branch, so the compiler can interleave the two.  rm / rl
// hold the wave's (m, l) per query row; the four key-row lanes of a query
// column agree after the merge and all store it.
template <bool MASK>
__device__ inline void lse_sub(const KTiles& K, const char* qs, float* rm, float* rl, int nqt,
                               int sc, int r1, int wave, int lane, float scale_log2) {
  const int i16 = lane & 15, g4 = lane >> 4;
  int row[TPW];
#pragma unroll
  for (int i = 0; i < TPW; ++i) row[i] = sc + (wave + i * WAVES) * TILE;
  u4 qb[4];
  f4 sa[2][2], sb[2][2];
  q_tile(qs, 0, lane, qb);
  s_tile(K.k[0], qb, sa[0][0], sa[0][1]);
  s_tile(K.k[1], qb, sa[1][0], sa[1][1]);
  for (int t = 0; t < nqt; ++t) {
    // the wave's state so far enters through one of the four key-row lanes
    float m = rm[t * 16 + i16], l = rl[t * 16 + i16];
    m = g4 == 0 ? m : -INFINITY;
    l = g4 == 0 ? l : 0.0f;
    s_tile(K.k[2], qb, sb[0][0], sb[0][1]);
    s_tile(K.k[3], qb, sb[1][0], sb[1][1]);
    lse_half<MASK>(sa, row[0], row[1], r1, g4, scale_log2, m, l);
    q_tile(qs, t + 1 < nqt ? t + 1 : t, lane, qb);  // the last round's pair is unused
    s_tile(K.k[0], qb, sa[0][0], sa[0][1]);
    s_tile(K.k[1], qb, sa[1][0], sa[1][1]);
    lse_half<MASK>(sb, row[2], row[3], r1, g4, scale_log2, m, l);
    // merge the four key-row lanes (g4) of each query column
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float m2 = __shfl_xor(m, o, 64), l2 = __shfl_xor(l, o, 64);
      const float mn = fmaxf(m, m2);
      const float ref = mn == -INFINITY ? 0.0f : mn;
      l = fmaf(l, __builtin_amdgcn_exp2f(m - ref), l2 * __builtin_amdgcn_exp2f(m2 - ref));
      m = mn;
    }
    rm[t * 16 + i16] = m;
    rl[t * 16 + i16] = l;
  }
}

// One sub-chunk of pass 2 for one wave, pipelined like pass 1.  Tiles past
// r1 read zero rows; their sums land in column slots nobody reads.
__device__ inline void col_sub(const KTiles& K, const char* qs, const float* ls, int nqt,
                               int lane, float scale_log2, float (&cs)[TPW][8]) {
  const int i16 = lane & 15;
  u4 qb[4];
  f4 sa[2][2], sb[2][2];
  q_tile(qs, 0, lane, qb);
  s_tile(K.k[0], qb, sa[0][0], sa[0][1]);
  s_tile(K.k[1], qb, sa[1][0], sa[1][1]);
  for (int t = 0; t < nqt; ++t) {
    const float lq = ls[t * 16 + i16];
    s_tile(K.k[2], qb, sb[0][0], sb[0][1]);
    s_tile(K.k[3], qb, sb[1][0], sb[1][1]);
    col_half(sa, lq, scale_log2, cs[0], cs[1]);
    q_tile(qs, t + 1 < nqt ? t + 1 : t, lane, qb);  // the last round's pair is unused
    s_tile(K.k[0], qb, sa[0][0], sa[0][1]);
    s_tile(K.k[1], qb, sa[1][0], sa[1][1]);
    col_half(sb, lq, scale_log2, cs[2], cs[3]);
  }
}

// ---------------------------------------------------------------- pass 1
// grid (chunks, query blocks, b*h_kv); one (m, l) record per (row, chunk)
template <bool PACKED>
__global__ __launch_bounds__(256, 2) void score_lse_kernel(KSegs segs, ChunkPlan plan,
                                                           const uint16_t* __restrict__ q, int Hq,
                                                           int Hkv, int W, float scale_log2,
                                                           float* __restrict__ partial) {
  __shared__ __attribute__((aligned(16))) char qs[QB * QROW];
  __shared__ float red_m[WAVES][QB], red_l[WAVES][QB];
  const int c = blockIdx.x, qb = blockIdx.y, bh = blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int G = Hq / Hkv, nq = G * W, b = bh / Hkv, hkv = bh % Hkv;
  int r0, r1;
  const int si = chunk_rows(plan, segs, c, r0, r1);
  const KSeg& ks = segs.s[si];
  const uint16_t* qh = q + ((int64_t)b * Hq + hkv * G) * W * D;
  const int q0 = qb * QB;
  const int nqt = min(QT, (nq - q0 + 15) / 16);
  stage_q(qs, qh, q0, nq, W, W);
  for (int e = threadIdx.x; e < WAVES * QB; e += blockDim.x) {
    red_m[e / QB][e % QB] = -INFINITY;
    red_l[e / QB][e % QB] = 0.0f;
  }
  __syncthreads();

  const KSrc src = k_source(ks, bh, r1);
  for (int sc = r0; sc < r1; sc += SUB) {
    // the wave's tiles of this sub-chunk: rows sc + (wave + i*WAVES)*TILE
    KTiles K;
#pragma unroll
    for (int i = 0; i < TPW; ++i) k_load<PACKED>(src, sc + (wave + i * WAVES) * TILE, lane, K.k[i]);
    if (sc + SUB <= r1)
      lse_sub<false>(K, qs, red_m[wave], red_l[wave], nqt, sc, r1, wave, lane, scale_log2);
    else
      lse_sub<true>(K, qs, red_m[wave], red_l[wave], nqt, sc, r1, wave, lane, scale_log2);
  }
  __syncthreads();
  const int C = plan.n_chunks;
  for (int r = threadIdx.x; r < nqt * 16; r += blockDim.x) {
    if (q0 + r >= nq) continue;
    float mm = -INFINITY;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) mm = fmaxf(mm, red_m[w][r]);
    float ll = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w)
      if (red_m[w][r] != -INFINITY) ll += red_l[w][r] * exp2f(red_m[w][r] - mm);
    const int64_t qi = ((int64_t)b * Hq + hkv * G) * W + q0 + r;  // global query row
    partial[(qi * C + c) * 2] = mm;
    partial[(qi * C + c) * 2 + 1] = ll;
  }
}

// ---------------------------------------------------------------- pass 2
struct ScoreOut {
  float* p[kMaxSeg];
};

// grid (chunks, query-block groups, b*h_kv): the query blocks
// [s*qbs, (s+1)*qbs) of the head.  With one group the scores and chunk mass
// are written directly; with several, each group's column sums (double) go
// to colpart and score_col_reduce_kernel adds them in group order.
template <bool PACKED>
__global__ __launch_bounds__(256, 2) void score_col_kernel(KSegs segs, ChunkPlan plan,
                                                           const uint16_t* __restrict__ q, int Hq,
                                                           int Hkv, int W, int q_ld,
                                                           float scale_log2,
                                                           const float* __restrict__ lse,
                                                           ScoreOut out,
                                                           double* __restrict__ mass_partial,
                                                           int qbs, double* __restrict__ colpart) {
  __shared__ __attribute__((aligned(16))) char qs[QB * QROW];
  __shared__ float ls[QB];
  __shared__ double colsum[CHUNK];
  __shared__ double red[WAVES];
  // the first pass walks heads and chunks in grid order, so this one walks
  // them backwards: the keys it reads first are those the first pass read
  // last, which the last-level cache may still hold
  const int c = gridDim.x - 1 - blockIdx.x, sg = blockIdx.y, bh = gridDim.z - 1 - blockIdx.z;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int G = Hq / Hkv, nq = G * W, b = bh / Hkv, hkv = bh % Hkv;
  int r0, r1;
  const int si = chunk_rows(plan, segs, c, r0, r1);
  const KSeg& ks = segs.s[si];
  const uint16_t* qh = q + ((int64_t)b * Hq + hkv * G) * q_ld * D;
  const float* lh = lse + ((int64_t)b * Hq + hkv * G) * W;
  for (int e = threadIdx.x; e < CHUNK; e += blockDim.x) colsum[e] = 0.0;

  const KSrc src = k_source(ks, bh, r1);
  const int q_end = min(nq, (sg + 1) * qbs * QB);
  for (int q0 = sg * qbs * QB; q0 < q_end; q0 += QB) {
    const int nqt = min(QT, (nq - q0 + 15) / 16);
    __syncthreads();  // the previous block's readers are done
    stage_q(qs, qh, q0, nq, W, q_ld);
    for (int r = threadIdx.x; r < QB; r += blockDim.x)
      ls[r] = q0 + r < nq ? lh[q0 + r] * kLog2e : INFINITY;  // padded rows: p = 0
    __syncthreads();
    for (int sc = r0; sc < r1; sc += SUB) {
      KTiles K;
#pragma unroll
      for (int i = 0; i < TPW; ++i) k_load<PACKED>(src, sc + (wave + i * WAVES) * TILE, lane, K.k[i]);
      float cs[TPW][8];
#pragma unroll
      for (int i = 0; i < TPW; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) cs[i][j] = 0.0f;
      col_sub(K, qs, ls, nqt, lane, scale_log2, cs);
      // sum the 16 query columns (lanes i16), then add to the chunk's sums
#pragma unroll
      for (int i = 0; i < TPW; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          float v = cs[i][j];
          v += __shfl_xor(v, 1, 64);
          v += __shfl_xor(v, 2, 64);
          v += __shfl_xor(v, 4, 64);
          v += __shfl_xor(v, 8, 64);
          cs[i][j] = v;
        }
        if (i16 == 0) {
          const int kt = sc - r0 + (wave + i * WAVES) * TILE;  // tile offset in the chunk
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            colsum[kt + g4 * 4 + j] += (double)cs[i][j];
            colsum[kt + 16 + g4 * 4 + j] += (double)cs[i][4 + j];
          }
        }
      }
    }
  }
  __syncthreads();
  if (colpart) {  // one group of several: its column sums, reduced later
    double* cp = colpart + (((int64_t)sg * gridDim.z + bh) * plan.n_chunks + c) * CHUNK;
    for (int e = threadIdx.x; e < CHUNK; e += blockDim.x) cp[e] = colsum[e];
    return;
  }
  // scores (rows past r1 were masked by never being written) and the
  // chunk's mass (fixed-order reduction: deterministic)
  float* sp = out.p[si];
  double part = 0.0;
  for (int e = threadIdx.x; e < CHUNK; e += blockDim.x) {
    if (r0 + e < r1) {
      if (sp) sp[(int64_t)bh * ks.n_rows + r0 + e] = (float)colsum[e];
      part += colsum[e];
    }
  }
  part = wave_sum_d(part);
  if (lane == 0) red[wave] = part;
  __syncthreads();
  if (threadIdx.x == 0 && mass_partial)
    mass_partial[(int64_t)bh * plan.n_chunks + c] = red[0] + red[1] + red[2] + red[3];
}

// grid (chunks, b*h_kv): the groups' column sums added in group order, then
// the scores and the chunk's mass as the single-group kernel writes them
__global__ __launch_bounds__(256) void score_col_reduce_kernel(KSegs segs, ChunkPlan plan,
                                                               int n_groups,
                                                               const double* __restrict__ colpart,
                                                               ScoreOut out,
                                                               double* __restrict__ mass_partial) {
  __shared__ double red[4];
  const int c = blockIdx.x, bh = blockIdx.y, BH = gridDim.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int r0, r1;
  const int si = chunk_rows(plan, segs, c, r0, r1);
  const KSeg& ks = segs.s[si];
  float* sp = out.p[si];
  double part = 0.0;
  for (int e = threadIdx.x; e < CHUNK; e += blockDim.x) {
    if (r0 + e >= r1) continue;
    double v = 0.0;
    for (int g = 0; g < n_groups; ++g)
      v += colpart[(((int64_t)g * BH + bh) * plan.n_chunks + c) * CHUNK + e];
    if (sp) sp[(int64_t)bh * ks.n_rows + r0 + e] = (float)v;
    part += v;
  }
  part = wave_sum_d(part);
  if (lane == 0) red[wave] = part;
  __syncthreads();
  if (threadIdx.x == 0 && mass_partial)
    mass_partial[(int64_t)bh * plan.n_chunks + c] = red[0] + red[1] + red[2] + red[3];
}

}  // namespace

bool score_mfma_eligible(const uc_shape& sh, const KSegs& segs, int q_dt) {
  if (sh.D != D || q_dt != UC_BF16) return false;
  for (int i = 0; i < segs.n; ++i) {
    if (segs.s[i].dtype != UC_BF16) return false;
    // packed: key groups of >= 32 rows, so a 32-row tile shares one scale set
    if (segs.s[i].kind == UC_SEG_PACKED && segs.s[i].group < TILE) return false;
  }
  return true;
}

int score_mfma_chunk_rows() { return CHUNK; }

// a packed segment with code rows among the plan's chunks (the plan may
// leave segments out)
static bool has_packed(const KSegs& segs, const ChunkPlan& plan) {
  for (int i = 0; i < segs.n; ++i)
    if (segs.s[i].kind == UC_SEG_PACKED && segs.s[i].n_full > 0 && plan.first[i + 1] > plan.first[i])
      return true;
  return false;
}

int score_mfma_qblocks(int nq) { return (nq + QB - 1) / QB; }

// query-block groups of the column pass: enough workgroups to fill the chip
// (about 512) when chunks x heads alone do not
static int score_col_groups(const uc_shape& sh, const ChunkPlan& plan, int W) {
  const int qblocks = score_mfma_qblocks((sh.Hq / sh.Hkv) * W);
  const int base = plan.n_chunks * sh.B * sh.Hkv;
  const int want = (512 + base - 1) / base;
  return std::max(1, std::min(qblocks, want));
}

hipError_t launch_score_lse_mfma(const uc_shape& sh, const KSegs& segs, const ChunkPlan& plan,
                                 const void* q, int W, float sm_scale, float* partial,
                                 hipStream_t st) {
  const int nq = (sh.Hq / sh.Hkv) * W;
  dim3 grid(plan.n_chunks, score_mfma_qblocks(nq), sh.B * sh.Hkv);
  if (has_packed(segs, plan))
    hipLaunchKernelGGL(score_lse_kernel<true>, grid, dim3(256), 0, st, segs, plan,
                       (const uint16_t*)q, sh.Hq, sh.Hkv, W, sm_scale * kLog2e, partial);
  else
    hipLaunchKernelGGL(score_lse_kernel<false>, grid, dim3(256), 0, st, segs, plan,
                       (const uint16_t*)q, sh.Hq, sh.Hkv, W, sm_scale * kLog2e, partial);
  return hipGetLastError();
}

hipError_t launch_score_col_mfma(const uc_shape& sh, const KSegs& segs, const ChunkPlan& plan,
                                 const void* q, int W, int q_ld, float sm_scale, const float* lse,
                                 float* const* scores, double* mass_partial, double* colpart,
                                 hipStream_t st) {
  ScoreOut so{};
  for (int i = 0; i < segs.n; ++i) so.p[i] = scores ? scores[i] : nullptr;
  const int groups = score_col_groups(sh, plan, W);
  const int qblocks = score_mfma_qblocks((sh.Hq / sh.Hkv) * W);
  const int qbs = (qblocks + groups - 1) / groups;
  const int n_groups = (qblocks + qbs - 1) / qbs;
  dim3 grid(plan.n_chunks, n_groups, sh.B * sh.Hkv);
  if (has_packed(segs, plan))
    hipLaunchKernelGGL(score_col_kernel<true>, grid, dim3(256), 0, st, segs, plan,
                       (const uint16_t*)q, sh.Hq, sh.Hkv, W, q_ld, sm_scale * kLog2e, lse, so,
                       mass_partial, qbs, n_groups > 1 ? colpart : nullptr);
  else
    hipLaunchKernelGGL(score_col_kernel<false>, grid, dim3(256), 0, st, segs, plan,
                       (const uint16_t*)q, sh.Hq, sh.Hkv, W, q_ld, sm_scale * kLog2e, lse, so,
                       mass_partial, qbs, n_groups > 1 ? colpart : nullptr);
  if (n_groups > 1)
    hipLaunchKernelGGL(score_col_reduce_kernel, dim3(plan.n_chunks, sh.B * sh.Hkv), dim3(256), 0,
                       st, segs, plan, n_groups, (const double*)colpart, so, mass_partial);
  return hipGetLastError();
}

}  // namespace uc
