// attend_decode.hip -- decode attention (a query block of at most 16 rows per
// KV head: the grouped query heads times M) over bf16 segments on the CDNA4
// matrix cores (App. E, "Attention over heterogeneous cache segments": one
// softmax across all segments, chunk results merged by log-sum-exp).
//
// Work item: W workgroups per (b, h_kv) -- two per CU, one round -- each
// taking the same tile-aligned share of every segment.  Each of the four
// waves takes every fourth 32-row tile of its share with two register sets
// (A/B): while tile t is computed, the loads of tiles t+1 and t+2 are
// outstanding.  A tile is consumed in two halves so its registers are
// refilled as early as possible:
//   head: V (or dequantised K and V for packed rows) goes to the wave's LDS
//         tile; S^T = K Q^T runs on v_mfma_f32_16x16x32_bf16 with the 32 keys
//         as two 16-row A blocks and the query block (padded to 16 rows) as
//         the B operand.  Dense K is loaded straight into the A-operand
//         layout (lane = key row, 8 consecutive head dims per step), so it
//         never touches LDS.
//   tail: online softmax per query in base 2, then O^T += V^T P with V^T
//         read by ds_read_b64_tr_b16 and P split into bf16 hi + lo parts (16
//         significant bits of probability).
// Softmax rescaling is lazy: probabilities are taken against a reference
// maximum m that is only raised (with the usual rescale of l and O) when some
// logit of the wave exceeds m by more than 2^8 in base 2, detected with one
// wave-wide ballot; otherwise the tile skips the cross-lane maximum and the
// rescale.  l and O always share the same reference, so the result is the
// same softmax; probabilities stay below 2^8 before normalisation.
// All loads are raw buffer loads whose descriptor ends at the range's last
// row (reads past it return zeros), so they need no clamping or branches;
// only a range's last tile can be partial, and only the epilogue tiles of the
// loop mask rows past the end.  Packed segments: whole row groups are packed
// and the key row groups span whole tiles, so packed tiles are always full;
// the residual tail rows (stored at the segment dtype) take the dense path.
// LDS rows are padded by 32 bytes, which keeps the transposing reads free of
// bank conflicts and their addresses affine in the head dimension.  The four
// waves merge through LDS and the workgroup writes unnormalised partials
// (m, l, o) per query row; the combine kernel merges them.
#include "mfma_util.h"
#include "uc_common.h"

namespace uc {
namespace {

using namespace mf;

constexpr int WAVES = 4;
constexpr float kLazy = 8.0f;  // base-2 headroom before the reference max is raised

// running softmax state of the lane's query (i16) and its O^T accumulators
struct State {
  float m, l;
  f4 acc[8];
};

__device__ inline void state_init(State& st) {
  st.m = -INFINITY;
  st.l = 0.0f;
#pragma unroll
  for (int d = 0; d < 8; ++d) st.acc[d] = f4{0.f, 0.f, 0.f, 0.f};
}

// softmax over one tile's scores + O^T += V^T P (V from the wave's LDS tile).
// MASK: the tile may reach past r_end (only a chunk's last tile does).
template <bool MASK>
__device__ inline void softmax_pv(State& st, const f4& s0, const f4& s1, float scale_log2,
                                  int row0, int r_end, const char* lv, int i16, int g4) {
  float p[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    p[j] = s0[j];
    p[4 + j] = s1[j];
  }
  if (MASK) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (row0 + g4 * 4 + j >= r_end) p[j] = -INFINITY;
      if (row0 + 16 + g4 * 4 + j >= r_end) p[4 + j] = -INFINITY;
    }
  }
  // the scale is positive, so the maximum of the raw logits gives the maximum
  float mx = fmaxf(fmaxf(fmaxf(p[0], p[1]), fmaxf(p[2], p[3])),
                   fmaxf(fmaxf(p[4], p[5]), fmaxf(p[6], p[7]))) * scale_log2;
  if (__builtin_amdgcn_ballot_w64(mx > st.m + kLazy)) {  // rare: raise the reference max
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(st.m, mx);
    const float alpha = __builtin_amdgcn_exp2f(st.m - m_new);
    st.l *= alpha;
#pragma unroll
    for (int d = 0; d < 8; ++d) st.acc[d] *= alpha;
    st.m = m_new;
  }
  // exponents are at most kLazy, so v_exp_f32 needs no range reduction; tiny
  // probabilities may flush to zero
  float e[8], psum = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    e[j] = __builtin_amdgcn_exp2f(fmaf(p[j], scale_log2, -st.m));
    psum += e[j];
  }
  u4 phi, plo;
  split_p(e, phi, plo);
  st.l += psum;
#pragma unroll
  for (int d = 0; d < 8; ++d) {
    const u4 vt = vt_operand(lv, d, i16, g4);
    st.acc[d] = mfma(vt, phi, st.acc[d]);
    st.acc[d] = mfma(vt, plo, st.acc[d]);
  }
}

// The query block's B operands (Q^T, four 32-dim steps) live in LDS, shared
// by the workgroup's waves: reloading them per tile is cheaper than holding
// 16 more registers in the streaming loops.
constexpr int QOPB = 4 * 64 * 16;

__device__ inline u4 q_operand(const char* lq, int t, int lane) {
  return *reinterpret_cast<const u4*>(lq + (t * 64 + lane) * 16);
}

// ---------------------------------------------------------------- dense rows
// K and V rows are both loaded as whole lines: load i covers rows 4i .. 4i+3
// of the tile, 256 contiguous bytes each (lane = row lane/16, 16-byte chunk
// lane%16).  Loading K straight into the matrix-core operand layout instead
// (16 rows x 64 bytes per load, half of each 128-byte line) streams about 15 %
// slower on this chip, so K takes the way through the wave's LDS tile that
// dequantised packed rows take.
struct DenseSet {
  u4 k[8];  // k[i] = row lane/16 + 4*i, 16-byte chunk lane%16
  u4 v[8];  // likewise for V
};

__device__ inline void dense_issue(__amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv, int row0,
                                   int lane, DenseSet& S) {
  const int i16 = lane & 15, g4 = lane >> 4;
  const int o = (row0 + g4) * ROWB + i16 * 16;
#pragma unroll
  for (int i = 0; i < 8; ++i) S.k[i] = bload<kNT>(rk, o, i * 4 * ROWB);
#pragma unroll
  for (int i = 0; i < 8; ++i) S.v[i] = bload<kNT>(rv, o, i * 4 * ROWB);
}

__device__ inline void dense_head(const DenseSet& S, char* lk, char* lv, const char* lq, int lane,
                                  f4& s0, f4& s1) {
  const int i16 = lane & 15, g4 = lane >> 4;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    *reinterpret_cast<u4*>(lk + toff(g4 + 4 * i, i16)) = S.k[i];
    *reinterpret_cast<u4*>(lv + toff(g4 + 4 * i, i16)) = S.v[i];
  }
  s0 = f4{0.f, 0.f, 0.f, 0.f};
  s1 = s0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    // A operands: rows blk*16 + i16, dims t*32 + g4*8 .. +7
    const u4 k0 = *reinterpret_cast<const u4*>(lk + toff(i16, t * 4 + g4));
    const u4 k1 = *reinterpret_cast<const u4*>(lk + toff(16 + i16, t * 4 + g4));
    const u4 qb = q_operand(lq, t, lane);
    s0 = mfma(k0, qb, s0);
    s1 = mfma(k1, qb, s1);
  }
}

// Rows [r0, r1) of one head's dense rows at kb / vb (row-major, D per row).
// The wave takes tiles wave, wave + WAVES, ...; only the last tile of the
// range can be partial, and it is always one of the epilogue tiles.
__device__ __attribute__((always_inline)) inline void dense_loop(State& st, const uint16_t* kb, const uint16_t* vb, int r0, int r1,
                                  int wave, int lane, const char* lq, float scale_log2,
                                  char* lk, char* lv) {
  const int n_tiles = (r1 - r0 + TILE - 1) / TILE;
  const int n_mine = n_tiles > wave ? (n_tiles - wave + WAVES - 1) / WAVES : 0;
  if (n_mine == 0) return;
  const int i16 = lane & 15, g4 = lane >> 4;
  const __amdgpu_buffer_rsrc_t rk = rsrc(kb, (uint32_t)r1 * ROWB);
  const __amdgpu_buffer_rsrc_t rv = rsrc(vb, (uint32_t)r1 * ROWB);
  auto row_of = [&](int k) { return r0 + (wave + k * WAVES) * TILE; };
  DenseSet A, B;
  f4 s0, s1;
  // both sets are issued unconditionally (rows past r1 read as zeros without
  // touching memory), so the loop is entered with exactly the outstanding
  // loads of its back edge and the compiler's wait counts stay loose
  dense_issue(rk, rv, row_of(0), lane, A);
  dense_issue(rk, rv, row_of(1), lane, B);
  int k = 0;
  // steady state without branches, so the compiler's wait counts keep the
  // other set's loads in flight: consume A, refill A, consume B, refill B
  for (; k + 3 < n_mine; k += 2) {
    dense_head(A, lk, lv, lq, lane, s0, s1);
    dense_issue(rk, rv, row_of(k + 2), lane, A);
    softmax_pv<false>(st, s0, s1, scale_log2, row_of(k), r1, lv, i16, g4);
    dense_head(B, lk, lv, lq, lane, s0, s1);
    dense_issue(rk, rv, row_of(k + 3), lane, B);
    softmax_pv<false>(st, s0, s1, scale_log2, row_of(k + 1), r1, lv, i16, g4);
  }
  const int left = n_mine - k;  // 1..3 tiles; A holds tile k, B tile k+1
  dense_head(A, lk, lv, lq, lane, s0, s1);
  if (left == 3) dense_issue(rk, rv, row_of(k + 2), lane, A);
  softmax_pv<true>(st, s0, s1, scale_log2, row_of(k), r1, lv, i16, g4);
  if (left >= 2) {
    dense_head(B, lk, lv, lq, lane, s0, s1);
    softmax_pv<true>(st, s0, s1, scale_log2, row_of(k + 1), r1, lv, i16, g4);
  }
  if (left == 3) {
    dense_head(A, lk, lv, lq, lane, s0, s1);
    softmax_pv<true>(st, s0, s1, scale_log2, row_of(k + 2), r1, lv, i16, g4);
  }
}

// ---------------------------------------------------------------- packed rows
// Only whole row groups are packed and groups span whole 32-row tiles, so a
// packed tile is always full and lies in one key row group.  Lane (c8, g4)
// owns channels c8*8 .. c8*8+7 of rows g4 + 4*i (i < 8); the BITS-bit codes of
// those 8 channels fill BITS bytes.
template <int BITS>
struct PackedSet {
  // 128-bit groups throughout (element [i] is row g4 + 4*i): this keeps the
  // two register sets of the pipelined loop in whole register tuples
  u4 ck[2], cv[2];  // code words (the low 16 bits at 2 bits per code)
  u4 sv[2], mv[2];  // value scale/min bits of the lane's channel group, per row
  u4 sk[2], mk[2];  // key scale/min bits of the lane's 8 channels (the tile's row group)
};

struct PackedSeg {
  __amdgpu_buffer_rsrc_t ck, cv, sk, mk, sv, mv;  // one head's codes and scales
  int lgG, ngv;                                   // log2(group), value groups per row
};

// the 8 codes of a lane's channels as floats (channel e of the lane -> c[e]);
// the masks are opaque so each code is one v_cvt_f32_ubyteN
template <int BITS>
__device__ inline void codes8(uint32_t w0, float (&c)[8]) {
  if constexpr (BITS == 4) {
    const uint32_t m = opaque(0x0F0F0F0Fu);
    const uint32_t lo = w0 & m, hi = (w0 >> 4) & m;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      c[2 * b] = (float)((lo >> (8 * b)) & 0xFFu);
      c[2 * b + 1] = (float)((hi >> (8 * b)) & 0xFFu);
    }
  } else {  // channel e at bits 2e: masks pick channels e and e + 4 into bytes 0 and 1
    const uint32_t m = opaque(0x0303u);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t t = (w0 >> (2 * e)) & m;
      c[e] = (float)(t & 0xFFu);
      c[4 + e] = (float)((t >> 8) & 0xFFu);
    }
  }
}

template <int BITS>
__device__ inline void packed_issue(const PackedSeg& P, int row0, int lane, PackedSet<BITS>& S) {
  const int c8 = lane & 15, g4 = lane >> 4;
  constexpr int RB = D * BITS / 8;  // code bytes per row
  const int so = ((row0 >> P.lgG) * D + c8 * 8) * 4;
  S.sk[0] = bload(P.sk, so, 0);
  S.sk[1] = bload(P.sk, so, 16);
  S.mk[0] = bload(P.mk, so, 0);
  S.mk[1] = bload(P.mk, so, 16);
  const int co = (row0 + g4) * RB + c8 * BITS;
  const int vo = ((row0 + g4) * P.ngv + ((c8 * 8) >> P.lgG)) * 4;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    if constexpr (BITS == 4) {
      S.ck[i >> 2][i & 3] = bload32<kNT>(P.ck, co, i * 4 * RB);
      S.cv[i >> 2][i & 3] = bload32<kNT>(P.cv, co, i * 4 * RB);
    } else {
      S.ck[i >> 2][i & 3] = __builtin_amdgcn_raw_buffer_load_b16(P.ck, co, i * 4 * RB, kNT);
      S.cv[i >> 2][i & 3] = __builtin_amdgcn_raw_buffer_load_b16(P.cv, co, i * 4 * RB, kNT);
    }
    S.sv[i >> 2][i & 3] = bload32<kNT>(P.sv, vo, i * 16 * P.ngv);
    S.mv[i >> 2][i & 3] = bload32<kNT>(P.mv, vo, i * 16 * P.ngv);
  }
}

// dequantise one row's 8 channels of K and V into packed bf16 (4 x u32 each):
// round_to_bf16(fmaf(code, scale, min)), the stored-value definition
template <int BITS>
__device__ inline void dequant_row(const PackedSet<BITS>& S, int i, u4& kk, u4& vv) {
  float qk[8], qv[8];
  codes8<BITS>(S.ck[i >> 2][i & 3], qk);
  codes8<BITS>(S.cv[i >> 2][i & 3], qv);
  const float sv = __uint_as_float(S.sv[i >> 2][i & 3]), mv = __uint_as_float(S.mv[i >> 2][i & 3]);
  float xk[8], xv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    xk[e] = fmaf(qk[e], __uint_as_float(S.sk[e >> 2][e & 3]), __uint_as_float(S.mk[e >> 2][e & 3]));
    xv[e] = fmaf(qv[e], sv, mv);
  }
  kk = u4{bf2(xk[0], xk[1]), bf2(xk[2], xk[3]), bf2(xk[4], xk[5]), bf2(xk[6], xk[7])};
  vv = u4{bf2(xv[0], xv[1]), bf2(xv[2], xv[3]), bf2(xv[4], xv[5]), bf2(xv[6], xv[7])};
}

template <int BITS>
__device__ inline void packed_head(const PackedSet<BITS>& S, char* lk, char* lv,
                                   const char* lq, int lane, f4& s0, f4& s1) {
  const int c8 = lane & 15, g4 = lane >> 4;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int rr = g4 + 4 * i;
    u4 kk, vv;
    dequant_row<BITS>(S, i, kk, vv);
    *reinterpret_cast<u4*>(lk + toff(rr, c8)) = kk;
    *reinterpret_cast<u4*>(lv + toff(rr, c8)) = vv;
    __builtin_amdgcn_sched_barrier(0);  // one row's temporaries at a time
  }
  const int i16 = lane & 15;
  s0 = f4{0.f, 0.f, 0.f, 0.f};
  s1 = s0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const u4 k0 = *reinterpret_cast<const u4*>(lk + toff(i16, t * 4 + g4));
    const u4 k1 = *reinterpret_cast<const u4*>(lk + toff(16 + i16, t * 4 + g4));
    const u4 qb = q_operand(lq, t, lane);
    s0 = mfma(k0, qb, s0);
    s1 = mfma(k1, qb, s1);
  }
}

// Rows [r0, r1) of one head's packed rows; both ends are multiples of TILE.
template <int BITS>
__device__ __attribute__((always_inline)) inline void packed_loop(State& st, const PackedSeg& P, int r0, int r1, int wave,
                                   int lane, const char* lq, float scale_log2, char* lk,
                                   char* lv) {
  const int n_tiles = (r1 - r0) / TILE;
  const int n_mine = n_tiles > wave ? (n_tiles - wave + WAVES - 1) / WAVES : 0;
  if (n_mine == 0) return;
  const int i16 = lane & 15, g4 = lane >> 4;
  auto row_of = [&](int k) { return r0 + (wave + k * WAVES) * TILE; };
  PackedSet<BITS> A, B;
  f4 s0, s1;
  packed_issue<BITS>(P, row_of(0), lane, A);
  packed_issue<BITS>(P, row_of(1), lane, B);  // past the range: zeros, as above
  int k = 0;
  // the scheduling barriers keep the refill loads behind the dequantisation
  // that frees their registers (hoisting them would need a third set)
  for (; k + 3 < n_mine; k += 2) {
    packed_head<BITS>(A, lk, lv, lq, lane, s0, s1);
    __builtin_amdgcn_sched_barrier(0);
    packed_issue<BITS>(P, row_of(k + 2), lane, A);
    __builtin_amdgcn_sched_barrier(0);
    softmax_pv<false>(st, s0, s1, scale_log2, row_of(k), r1, lv, i16, g4);
    __builtin_amdgcn_sched_barrier(0);
    packed_head<BITS>(B, lk, lv, lq, lane, s0, s1);
    __builtin_amdgcn_sched_barrier(0);
    packed_issue<BITS>(P, row_of(k + 3), lane, B);
    __builtin_amdgcn_sched_barrier(0);
    softmax_pv<false>(st, s0, s1, scale_log2, row_of(k + 1), r1, lv, i16, g4);
    __builtin_amdgcn_sched_barrier(0);
  }
  const int left = n_mine - k;
  packed_head<BITS>(A, lk, lv, lq, lane, s0, s1);
  if (left == 3) packed_issue<BITS>(P, row_of(k + 2), lane, A);
  softmax_pv<false>(st, s0, s1, scale_log2, row_of(k), r1, lv, i16, g4);
  if (left >= 2) {
    packed_head<BITS>(B, lk, lv, lq, lane, s0, s1);
    softmax_pv<false>(st, s0, s1, scale_log2, row_of(k + 1), r1, lv, i16, g4);
  }
  if (left == 3) {
    packed_head<BITS>(A, lk, lv, lq, lane, s0, s1);
    softmax_pv<false>(st, s0, s1, scale_log2, row_of(k + 2), r1, lv, i16, g4);
  }
}

// ---------------------------------------------------------------- kernel
// Work split: W workgroups per (b, h_kv) (two per CU, one round).  Workgroup
// w takes the w-th of W equal tile-aligned shares of every segment.  With
// per-segment statistics requested, each workgroup writes one partial record
// (m, l, o) per segment for its query rows (slot s*W + w; m = -inf for an
// empty share); otherwise one running state spans all segments and one record
// per workgroup (slot w) is written.  The combine kernel merges the records.
// Packed tiles cost several times the vector-ALU work of dense tiles per
// byte; if every workgroup took its packed share first, the whole chip would
// be ALU-bound for that phase and HBM underused.  With a split segment (the
// largest dense one, chosen on the host when packed rows are present), each
// workgroup instead takes the first part of its share of that segment, then
// the other segments, then the rest; the part before is a fraction
// ((w + bh) mod W) / W of its tiles, so the packed phases of the workgroups
// are staggered over the launch.
struct DecodePlan {
  int W;        // workgroups per (b, h_kv)
  int n_seg;
  int per_seg;  // 1: one record per segment and workgroup
  int split;    // segment taken around the others (see above), or -1
  int skew;     // share weights of a head's early / late workgroups, see share_row_skewed
};

// tile-aligned share w of n rows among W workgroups
__device__ inline int share_row(int n, int w, int W) {
  const int64_t r = ((int64_t)n * w + W - 1) / W;
  const int64_t rt = (r + TILE - 1) / TILE * TILE;
  return (int)(rt < n ? rt : n);
}

// Share boundaries when the first W/2 workgroups of a head are dispatched in
// the launch's first half and the others in its second half: weights
// 1000 + skew for the first, 1000 - skew for the second (integer sums, so
// the last share ends exactly at n).  With two workgroups per CU the one
// dispatched first wins the issue arbitration: with equal shares it finished
// far ahead of its partner and the launch ended with one workgroup per CU.
__device__ inline int share_row_skewed(int n, int w, int W, int skew) {
  const int h = W / 2;
  auto cum = [&](int x) {
    return (int64_t)min(x, h) * (1000 + skew) + (int64_t)max(x - h, 0) * (1000 - skew);
  };
  const int64_t r = ((int64_t)n * cum(w) + cum(W) - 1) / cum(W);
  const int64_t rt = (r + TILE - 1) / TILE * TILE;
  return (int)(rt < n ? rt : n);
}

struct Ctx {
  float* partial;
  int C, nq, M, Hq, G, b, hkv;
};

__device__ inline int64_t qrow_of(const Ctx& c, int qs) {
  return ((int64_t)c.b * c.Hq + c.hkv * c.G + qs / c.M) * c.M + qs % c.M;
}

// merge the four waves' state through LDS and write one partial record;
// ok = false marks the record invalid (l = NaN)
__device__ __attribute__((always_inline)) inline void flush(State& st, char* lds, const Ctx& c, int slot, bool ok, int lane,
                             int wave) {
  const int i16 = lane & 15, g4 = lane >> 4;
  // full row sums: the four lanes of one query hold partial sums
  st.l += __shfl_xor(st.l, 16, 64);
  st.l += __shfl_xor(st.l, 32, 64);
  __syncthreads();  // the tile area is reused
  float* mo = reinterpret_cast<float*>(lds);  // [WAVES][16][D]
  float* ml = mo + WAVES * 16 * D;            // [WAVES][16] m, then [WAVES][16] l
  if (g4 == 0) {
    ml[wave * 16 + i16] = st.m;
    ml[WAVES * 16 + wave * 16 + i16] = st.l;
  }
#pragma unroll
  for (int d = 0; d < 8; ++d)
#pragma unroll
    for (int j = 0; j < 4; ++j) mo[(wave * 16 + i16) * D + d * 16 + g4 * 4 + j] = st.acc[d][j];
  __syncthreads();
  for (int e = threadIdx.x; e < c.nq * (D + 2); e += blockDim.x) {
    const int qs = e / (D + 2), f = e % (D + 2);
    float mw[WAVES], M_ = -INFINITY;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
      mw[w] = ml[w * 16 + qs];
      M_ = fmaxf(M_, mw[w]);
    }
    float val;
    if (f == 0) {
      val = ok ? M_ : 0.0f;
    } else {
      float a = 0.0f;
#pragma unroll
      for (int w = 0; w < WAVES; ++w) {
        const float wt = mw[w] == -INFINITY ? 0.0f : exp2f(mw[w] - M_);
        a += wt * (f == 1 ? ml[WAVES * 16 + w * 16 + qs] : mo[(w * 16 + qs) * D + (f - 2)]);
      }
      val = (f == 1 && !ok) ? __builtin_nanf("") : a;
    }
    c.partial[(qrow_of(c, qs) * c.C + slot) * (D + 2) + f] = val;
  }
  __syncthreads();  // LDS free again
}

// one workgroup's share [r0, r1) of segment ks for head bh
__device__ __attribute__((always_inline)) inline bool segment_share(State& st, const KSeg& ks, int bh, int r0, int r1, int wave,
                                     int& rot, int lane, const char* lq, float scale_log2,
                                     char* lk, char* lv) {
  if (r1 <= r0) return true;
  if (ks.kind == UC_SEG_DENSE) {
    const int64_t base = (int64_t)bh * ks.row_stride * D;
    dense_loop(st, (const uint16_t*)ks.k + base, (const uint16_t*)ks.v + base, r0, r1,
               (wave - rot) & (WAVES - 1), lane, lq, scale_log2, lk, lv);
    rot += (r1 - r0 + TILE - 1) / TILE;
    return true;
  }
  int bits = 0;
  int64_t off = 0;
  // code widths of 2 and 4 bits only (ks.bits bounds the per-head widths)
  if (!head_codes(ks, bh, D, bits, off) || bits > 4) return false;
  // the per-head entries are the same in every lane: keep them in scalar
  // registers so the buffer descriptors built from them stay scalar
  bits = __builtin_amdgcn_readfirstlane(bits);
  off = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(off >> 32)) << 32) |
                  (uint32_t)__builtin_amdgcn_readfirstlane((int)off));
  // packed rows [0, n_full), then the residual tail rows as dense rows
  const int p1 = min(r1, ks.n_full);
  if (p1 > r0) {
    const int lgG = __builtin_ctz((unsigned)ks.group);
    const int ngk = ks.n_full >> lgG, ngv = D >> lgG;  // live key groups, value groups per row
    const uint32_t cbytes = (uint32_t)ks.n_full * (D * bits / 8);
    PackedSeg P;
    P.ck = rsrc(ks.codes_k + off, cbytes);
    P.cv = rsrc(ks.codes_v + off, cbytes);
    const int64_t sko = (int64_t)bh * ks.kgroups * D, svo = (int64_t)bh * ks.cap_full * ngv;
    P.sk = rsrc(ks.scale_k + sko, (uint32_t)ngk * D * 4);
    P.mk = rsrc(ks.min_k + sko, (uint32_t)ngk * D * 4);
    P.sv = rsrc(ks.scale_v + svo, (uint32_t)ks.n_full * ngv * 4);
    P.mv = rsrc(ks.min_v + svo, (uint32_t)ks.n_full * ngv * 4);
    P.lgG = lgG;
    P.ngv = ngv;
    const int ew = (wave - rot) & (WAVES - 1);
    if (bits == 4) packed_loop<4>(st, P, r0, p1, ew, lane, lq, scale_log2, lk, lv);
    else packed_loop<2>(st, P, r0, p1, ew, lane, lq, scale_log2, lk, lv);
    rot += (p1 - r0) / TILE;
  }
  const int t0 = max(r0, ks.n_full);
  if (r1 > t0) {
    const int64_t base = (int64_t)bh * ks.tail_stride * D;
    dense_loop(st, (const uint16_t*)ks.tail_k + base, (const uint16_t*)ks.tail_v + base,
               t0 - ks.n_full, r1 - ks.n_full, (wave - rot) & (WAVES - 1), lane, lq, scale_log2,
               lk, lv);
    rot += (r1 - t0 + TILE - 1) / TILE;
  }
  return true;
}

// BATCH: requests of different segment layouts in one launch; blockIdx.y is
// (request, h_kv), each request's segments (a one-request layout) come from
// the static descriptors reqs[request] completed with this call's row counts,
// and its query rows follow those of the requests before it (as batch
// elements do)
template <bool BATCH>
__device__ __attribute__((always_inline)) inline void decode_body(
    const KSegs& segs, const BatchDesc* __restrict__ table, const KSeg* __restrict__ flat,
    const DecodePlan& pl, const AppendOp& ap, int w, int bh,
    const uint16_t* __restrict__ q, int Hq, int Hkv, int M, float scale_log2,
    float* __restrict__ partial) {
  __shared__ __attribute__((aligned(16))) char lds[WAVES * 2 * TILEB + QOPB];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int G = Hq / Hkv, nq = G * M, b = bh / Hkv, hkv = bh % Hkv;
  const int W = pl.W;


  // query block: slot i16 = g * M + m  (query head hkv*G + g, row m)
  // (the group's query rows are consecutive; slots past nq read as zeros
  // through the range check, so all four loads issue without branches)
  u4 qop[4];
  {
    const __amdgpu_buffer_rsrc_t rq = rsrc(q + ((int64_t)b * Hq + hkv * G) * M * D,
                                           (uint32_t)nq * D * 2);
#pragma unroll
    for (int t = 0; t < 4; ++t) qop[t] = bload(rq, (i16 * D + t * 32 + g4 * 8) * 2, 0);
  }
  // fused append: this call attends the new rows from k_new / v_new (a
  // segment of their own) and stores them into the protected segment for the
  // calls after it; no workgroup of this launch reads the rows written here
  // (every range ends at the segment's row count before the append).  Issued
  // after the query loads so that both wait out one memory latency together.
  if (!BATCH && ap.n_new > 0 && w == 0) {
    const int per = ap.n_new * ap.row_bytes / 16;
    for (int e = threadIdx.x; e < per; e += blockDim.x) {
      const int64_t src = (int64_t)bh * ap.n_new * ap.row_bytes + (int64_t)e * 16;
      const int64_t dst = ((int64_t)bh * ap.row_stride + ap.pos) * ap.row_bytes + (int64_t)e * 16;
      const u4 kr = *reinterpret_cast<const u4*>(ap.kn + src);  // both loads before
      const u4 vr = *reinterpret_cast<const u4*>(ap.vn + src);  // either store
      *reinterpret_cast<u4*>(ap.kd + dst) = kr;
      *reinterpret_cast<u4*>(ap.vd + dst) = vr;
    }
  }
  char* lk = lds + wave * 2 * TILEB;
  char* lv = lk + TILEB;
  char* lq = lds + WAVES * 2 * TILEB;  // outside the area the record merge reuses
  if (wave == 0) {
#pragma unroll
    for (int t = 0; t < 4; ++t) *reinterpret_cast<u4*>(lq + (t * 64 + lane) * 16) = qop[t];
  }
  __syncthreads();
  Ctx c{partial, pl.per_seg ? pl.n_seg * W : W, nq, M, Hq, G, b, hkv};

  State st;
  state_init(st);
  bool ok = true;
  // tiles go to the waves round-robin, continuing across segments (and from
  // a packed segment's codes into its tail), so no wave collects every
  // segment's remainder tile
  int rot = 0;
  const int first = BATCH ? table[b].first : 0;
  // a batched request splits its rows among its own W_r workgroups; its
  // first workgroup marks the record slots W_r .. W-1 of its rows empty
  const int Wr = BATCH ? table[b].W : W;
  const int n_seg = BATCH ? table[b].n : pl.n_seg;
  if (BATCH && w == 0) {
    for (int e = threadIdx.x; e < nq * (W - Wr); e += blockDim.x)
      c.partial[(qrow_of(c, e / (W - Wr)) * c.C + Wr + e % (W - Wr)) * (D + 2)] = -INFINITY;
  }
  const int sbh = BATCH ? hkv : bh;  // (b, h_kv) within the segments' own layout
  // items: the segments in order, or with a split segment (never with
  // per-segment records) its first part, the others in order, then its
  // second part
  const int split = BATCH ? table[b].split : pl.split;
  const int n_items = split >= 0 ? n_seg + 1 : n_seg;
  for (int it = 0; it < n_items; ++it) {
    int si = it;
    if (split >= 0) si = it == 0 || it == n_items - 1 ? split : (it - 1 < split ? it - 1 : it);
    const KSeg& ks = BATCH ? flat[first + si] : segs.s[si];
    // the appended rows (the last segment) go to the last workgroup, whose
    // shares of the other segments are the remainders; workgroup 0 already
    // holds the start of the protected segment
    const int ws = (!BATCH && ap.n_new > 0 && si == n_seg - 1) ? Wr - 1 - w : w;
    int r0 = share_row_skewed(ks.n_rows, ws, Wr, pl.skew);
    int r1 = share_row_skewed(ks.n_rows, ws + 1, Wr, pl.skew);
    if (split >= 0 && si == split) {
      // r0 is tile-aligned, so both parts start on a tile boundary and only
      // the second can end in a partial tile
      const int rm = r0 + ((r1 - r0) / TILE * ((w + bh) % Wr) / Wr) * TILE;
      if (it == 0) r1 = rm;
      else r0 = rm;
    }
    ok &= segment_share(st, ks, sbh, r0, r1, wave, rot, lane, lq, scale_log2, lk, lv);
    if (pl.per_seg) {
      flush(st, lds, c, si * W + w, ok, lane, wave);
      state_init(st);
      ok = true;
    }
  }
  if (!pl.per_seg) flush(st, lds, c, w, ok, lane, wave);
}

__global__ __launch_bounds__(256, 2) void decode_mfma_kernel(KSegs segs, DecodePlan pl,
                                                             AppendOp ap,
                                                             const uint16_t* __restrict__ q,
                                                             int Hq, int Hkv, int M,
                                                             float scale_log2,
                                                             float* __restrict__ partial) {
  // one-dimensional grid of W * BH workgroups, dispatched in order: the first
  // half of the launch holds workgroups 0 .. W/2-1 of every head, the second
  // half the others, so every head has workgroups of both halves
  const int BH = gridDim.x / pl.W, h = pl.W / 2, L = blockIdx.x;
  int w, bh;
  if (h == 0) {
    w = 0;
    bh = L;
  } else if (L < h * BH) {
    bh = L / h;
    w = L % h;
  } else {
    const int L2 = L - h * BH, hh = pl.W - h;
    bh = L2 / hh;
    w = h + L2 % hh;
  }
  decode_body<false>(segs, nullptr, nullptr, pl, ap, w, bh, q, Hq, Hkv, M, scale_log2, partial);
}

// a batched workgroup: its grid run is the last entry starting at or before
// it (starts ascend); then its request, KV head and share
__device__ __attribute__((always_inline)) inline void batch_entry(
    const BatchDesc* __restrict__ table, const BatchGrid* __restrict__ grid, int n_grid,
    const KSeg* __restrict__ flat, const DecodePlan& pl, const uint16_t* __restrict__ q, int Hq,
    int Hkv, int M, float scale_log2, float* __restrict__ partial) {
  const int g = blockIdx.x;
  int lo = 0, hi = n_grid - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (grid[mid].start <= g) lo = mid;
    else hi = mid - 1;
  }
  const BatchGrid e = grid[lo];
  const int local = g - e.start;
  KSegs none;
  none.n = 0;
  const AppendOp no_append{};
  decode_body<true>(none, table, flat, pl, no_append, e.w0 + local % e.nw,
                    e.req * Hkv + local / e.nw, q, Hq, Hkv, M, scale_log2, partial);
}

// descriptors stored in the workspace
__global__ __launch_bounds__(256, 2) void decode_batch_kernel(const BatchDesc* __restrict__ table,
                                                              const BatchGrid* __restrict__ grid,
                                                              int n_grid,
                                                              const KSeg* __restrict__ flat,
                                                              DecodePlan pl,
                                                              const uint16_t* __restrict__ q,
                                                              int Hq, int Hkv, int M,
                                                              float scale_log2,
                                                              float* __restrict__ partial) {
  batch_entry(table, grid, n_grid, flat, pl, q, Hq, Hkv, M, scale_log2, partial);
}

// descriptors in the kernel arguments
__global__ __launch_bounds__(256, 2) void decode_batch_args_kernel(BatchArgs a, int n_grid,
                                                                   DecodePlan pl,
                                                                   const uint16_t* __restrict__ q,
                                                                   int Hq, int Hkv, int M,
                                                                   float scale_log2,
                                                                   float* __restrict__ partial) {
  batch_entry(a.table, a.grid, n_grid, a.flat, pl, q, Hq, Hkv, M, scale_log2, partial);
}

}  // namespace

int device_cus() {
  static int cus = 0;
  if (!cus) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
      cus = n;
    else
      cus = 256;
  }
  return cus;
}

namespace {

// workgroups per (b, h_kv): two resident workgroups per CU in one round
// Merge of a decode call's partial records into O (and lse) when every
// record belongs to one softmax (no per-segment outputs): one wave per query
// row, four rows per workgroup, each lane owning two of the 128 dims.  A
// record is (m, l, o[D]) with m the base-2 reference of its running sums;
// eight records are loaded at a time, every load issued before any is used,
// and merged online; an empty record (m = -inf, other fields undefined) is
// dropped by selects.
__global__ __launch_bounds__(256) void decode_merge_kernel(int Q, int C,
                                                           const float* __restrict__ partial,
                                                           float* __restrict__ o,
                                                           float* __restrict__ lse) {
  const int qi = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (qi >= Q) return;
  const int lane = threadIdx.x & 63;
  const int ps = D + 2;
  const float* P = partial + (int64_t)qi * C * ps;
  float M = -INFINITY, l = 0.0f;
  f2 acc = f2{0.0f, 0.0f};
  for (int c0 = 0; c0 < C; c0 += 8) {
    f2 ml[8], oc[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int c = min(c0 + r, C - 1);
      ml[r] = *reinterpret_cast<const f2*>(P + (int64_t)c * ps);
      oc[r] = *reinterpret_cast<const f2*>(P + (int64_t)c * ps + 2 + 2 * lane);
    }
#pragma unroll
    for (int r = 0; r < 8; ++r)
      if (c0 + r >= C) ml[r][0] = -INFINITY;
    float mx = M;
#pragma unroll
    for (int r = 0; r < 8; ++r) mx = fmaxf(mx, ml[r][0]);
    const float a = M == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(M - mx);
    l *= a;
    acc *= a;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const bool live = ml[r][0] != -INFINITY;
      const float b = live ? __builtin_amdgcn_exp2f(ml[r][0] - mx) : 0.0f;
      l = fmaf(b, live ? ml[r][1] : 0.0f, l);
      acc[0] = fmaf(b, live ? oc[r][0] : 0.0f, acc[0]);
      acc[1] = fmaf(b, live ? oc[r][1] : 0.0f, acc[1]);
    }
    M = mx;
  }
  const float inv = 1.0f / l;
  *reinterpret_cast<f2*>(o + (int64_t)qi * D + 2 * lane) = acc * inv;
  if (lse && lane == 0) lse[qi] = (M + __log2f(l)) * kLn2;
}

int decode_w(const uc_shape& sh) {
  const int BH = sh.B * sh.Hkv;
  return max(1, (2 * device_cus()) / BH);
}

}  // namespace

bool decode_mfma_eligible(const uc_shape& sh, const KSegs& segs, int q_dt, int M) {
  if (sh.D != D || q_dt != UC_BF16) return false;
  if ((sh.Hq / sh.Hkv) * M > 16) return false;
  for (int i = 0; i < segs.n; ++i) {
    if (segs.s[i].dtype != UC_BF16) return false;
    // packed: 2- or 4-bit codes (bits is the uniform width, or the bound of
    // the per-head widths); key row groups must cover whole 32-row tiles (one
    // scale set per tile; groups are powers of two)
    if (segs.s[i].kind == UC_SEG_PACKED && (segs.s[i].group < TILE || segs.s[i].bits > 4))
      return false;
  }
  return true;
}

// Workspace: the partial records, n_seg * W per query row; the size does not
// depend on row counts.
size_t decode_mfma_workspace(const uc_shape& sh, const KSegs& segs, int M) {
  const size_t slots = (size_t)segs.n * decode_w(sh);
  const size_t bytes = (size_t)sh.B * sh.Hq * M * slots * (D + 2) * sizeof(float);
  return (bytes + 255) & ~(size_t)255;
}

// the segment a workgroup takes around the others: the largest dense one,
// when there is another segment and some packed code rows (else -1)
int decode_split_segment(const KSegs& segs) {
  if (segs.n < 2) return -1;
  bool packed = false;
  int best = -1;
  for (int i = 0; i < segs.n; ++i) {
    const KSeg& s = segs.s[i];
    if (s.kind == UC_SEG_PACKED && s.n_full > 0) packed = true;
    if (s.kind == UC_SEG_DENSE && (best < 0 || s.n_rows > segs.s[best].n_rows)) best = i;
  }
  return packed && best >= 0 && segs.s[best].n_rows > 0 ? best : -1;
}

hipError_t launch_decode_mfma(const uc_shape& sh, const KSegs& segs, const void* q, int M,
                              float sm_scale, float* o, float* lse, float* seg_lse, void* ws,
                              hipStream_t st, const AppendOp* ap) {
  DecodePlan p{};
  const AppendOp none{};
  p.W = decode_w(sh);
  {
    // at least one 32-row tile per wave (four per workgroup): a short
    // context gets fewer workgroups, and the merge fewer records per row
    int tiles = ap && ap->n_new > 0 ? 1 : 0;
    for (int i = 0; i < segs.n; ++i) tiles += (segs.s[i].n_rows + TILE - 1) / TILE;
    p.W = max(1, min(p.W, (tiles + WAVES - 1) / WAVES));
  }
  p.n_seg = segs.n;
  p.per_seg = seg_lse != nullptr;
  // a grid of exactly two workgroups per CU pairs every early workgroup with
  // a late one: the early ones take 1.6 / 2 of a pair's share (the best of
  // weights 0 .. 900 per mille measured on the 64k context)
  p.skew = p.W * sh.B * sh.Hkv == 2 * device_cus() ? 600 : 0;
  // split the largest dense segment around the others when packed rows are
  // present (staggered packed phases, see DecodePlan)
  p.split = p.per_seg ? -1 : decode_split_segment(segs);
  float* partial = (float*)ws;
  hipError_t e = kernel_timer_begin(st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_mfma_kernel, dim3(p.W * sh.B * sh.Hkv), dim3(256), 0, st, segs, p,
                     ap ? *ap : none, (const uint16_t*)q, sh.Hq, sh.Hkv, M, sm_scale * kLog2e,
                     partial);
  e = hipGetLastError();
  if (e == hipSuccess) e = kernel_timer_end(st);
  if (e != hipSuccess) return e;
  if (!p.per_seg) {  // one softmax: the lean merge
    const int Q = sh.B * sh.Hq * M;
    hipLaunchKernelGGL(decode_merge_kernel, dim3((Q + 3) / 4), dim3(256), 0, st, Q, p.W, partial,
                       o, lse);
    return hipGetLastError();
  }
  // per-segment records are segment-major (segment s owns slots [s*W, (s+1)*W))
  ChunkPlan cp{};
  cp.n_chunks = p.per_seg ? segs.n * p.W : p.W;
  for (int i = 0; i <= kMaxSeg; ++i)
    cp.first[i] = p.per_seg ? min(i, segs.n) * p.W : (i == 0 ? 0 : p.W);
  return launch_attend_combine(sh, segs, cp, M, partial, o, lse, seg_lse, st);
}

// Requests of different layouts: sh.B = number of requests; the request
// table, grid runs and flat segment descriptors come in args (a batch within
// kArgReq / kArgSeg) or, when args is null, from the workspace (written by
// the caller through launch_blob_upload); the workspace then holds the
// partial records after the descriptor area; q / o / lse
// are laid out as for sh.B batch elements.  Each request gets workgroups per
// KV head in proportion to its rows (at least one), all of them in one
// one-dimensional grid; the record stride per query row is the largest share
// and the workspace is sized for the budget decode_batch_wgs (so it does not
// depend on row counts).
int decode_batch_wgs(const uc_shape& sh) { return max(1, (2 * device_cus()) / sh.Hkv); }

// descriptor area: request table | grid runs (two per request) | flat segments
size_t decode_batch_table_bytes(int n_req) {
  return (((size_t)n_req * sizeof(BatchDesc)) + 255) & ~(size_t)255;
}
size_t decode_batch_grid_bytes(int n_req) {
  return (((size_t)2 * n_req * sizeof(BatchGrid)) + 255) & ~(size_t)255;
}
size_t decode_batch_desc_bytes(int n_req, int n_segs_total) {
  return decode_batch_table_bytes(n_req) + decode_batch_grid_bytes(n_req) +
         ((((size_t)n_segs_total * sizeof(KSeg)) + 255) & ~(size_t)255);
}

size_t decode_batch_workspace(const uc_shape& sh, int M, int n_segs_total) {
  const size_t rec = (size_t)sh.B * sh.Hq * M * decode_batch_wgs(sh) * (D + 2) * sizeof(float);
  return decode_batch_desc_bytes(sh.B, n_segs_total) + ((rec + 255) & ~(size_t)255);
}

hipError_t launch_decode_batch(const uc_shape& sh, int n_segs_total, int W_max, int n_wgs,
                               int n_grid, int skew, const BatchArgs* args, const void* q, int M,
                               float sm_scale, float* o, float* lse, void* ws, hipStream_t st) {
  DecodePlan p{};
  p.W = W_max;
  p.n_seg = sh.B;
  p.per_seg = 0;
  p.split = -1;  // per request, in the table
  p.skew = skew;
  const BatchDesc* table = (const BatchDesc*)ws;
  const BatchGrid* grid = (const BatchGrid*)((char*)ws + decode_batch_table_bytes(sh.B));
  const KSeg* flat = (const KSeg*)((char*)ws + decode_batch_table_bytes(sh.B) +
                                   decode_batch_grid_bytes(sh.B));
  float* partial = (float*)((char*)ws + decode_batch_desc_bytes(sh.B, n_segs_total));
  hipError_t e = kernel_timer_begin(st);
  if (e != hipSuccess) return e;
  if (args)
    hipLaunchKernelGGL(decode_batch_args_kernel, dim3(n_wgs), dim3(256), 0, st, *args, n_grid, p,
                       (const uint16_t*)q, sh.Hq, sh.Hkv, M, sm_scale * kLog2e, partial);
  else
    hipLaunchKernelGGL(decode_batch_kernel, dim3(n_wgs), dim3(256), 0, st, table, grid, n_grid,
                       flat, p, (const uint16_t*)q, sh.Hq, sh.Hkv, M, sm_scale * kLog2e, partial);
  e = hipGetLastError();
  if (e == hipSuccess) e = kernel_timer_end(st);
  if (e != hipSuccess) return e;
  const int Q = sh.B * sh.Hq * M;
  hipLaunchKernelGGL(decode_merge_kernel, dim3((Q + 3) / 4), dim3(256), 0, st, Q, p.W, partial, o,
                     lse);
  return hipGetLastError();
}

}  // namespace uc
