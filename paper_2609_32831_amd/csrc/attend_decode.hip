// attend_decode.hip -- decode attention (a query block of at most 16 rows per
// KV head: the grouped query heads times M) over bf16 segments on the CDNA4
// matrix cores (App. E, "Attention over heterogeneous cache segments": one
// softmax across all segments, chunk results merged by log-sum-exp).
//
// Work item: W workgroups per (b, h_kv) -- two per CU, one round -- each
// taking the same share of every segment (so every CU mixes bandwidth-bound
// dense tiles with dequantisation-bound packed tiles).  Each of the four
// waves takes every fourth 32-row tile of its share with two register sets
// (A/B): while tile t is computed, the
// loads of tiles t+1 and t+2 are outstanding.  A tile is consumed in two
// halves so its registers are refilled as early as possible:
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
// Dense rows are read with raw buffer loads whose descriptor ends at the
// chunk's last row (reads past it return zeros); packed rows of the last,
// partial tile are clamped to the last valid row.  Either way the loads need
// no branches, and rows past the chunk are masked out of the softmax.
// LDS rows are padded by 32 bytes, which keeps the transposing reads free of
// bank conflicts and their addresses affine in the head dimension.  The four waves merge through LDS and the workgroup writes
// one unnormalised partial (m, l, o) per query row and segment touched; the
// combine kernel merges them.
#include "uc_common.h"

namespace uc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef short s4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int D = 128;
constexpr int TILE = 32;          // rows per tile
constexpr int WAVES = 4;
constexpr int ROWB = D * 2;       // bytes of one bf16 row
constexpr int LROW = ROWB + 32;   // bytes of one staged row in LDS (32 B padding)
constexpr int TILEB = TILE * LROW;
constexpr float kLazy = 8.0f;        // base-2 headroom before the reference max is raised

// byte offset of 16-byte chunk c of row r inside a staged tile.  The 32-byte
// row padding puts row r at bank 8r (mod 64): the eight rows a half-wave
// reads in one transposing load land in disjoint 8-bank groups.
__device__ inline int toff(int r, int c) { return r * LROW + (c << 4); }

// two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32)
__device__ inline uint32_t bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{a, b}, bf16x2));
}

__device__ inline f4 mfma(const u4& a, const u4& b, const f4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

typedef __attribute__((address_space(3))) s4 lds_s4;

__device__ inline u4 ds_tr(const char* p0, const char* p1) {
  s4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p0));
  s4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p1));
  return u4{(uint32_t)(uint16_t)a[0] | ((uint32_t)(uint16_t)a[1] << 16),
            (uint32_t)(uint16_t)a[2] | ((uint32_t)(uint16_t)a[3] << 16),
            (uint32_t)(uint16_t)b[0] | ((uint32_t)(uint16_t)b[1] << 16),
            (uint32_t)(uint16_t)b[2] | ((uint32_t)(uint16_t)b[3] << 16)};
}

// running softmax state of the lane's query (i16) and its O^T accumulators
struct State {
  float m, l;
  f4 acc[8];
};

// softmax over one tile's scores + O^T += V^T P (V from the wave's LDS tile)
__device__ inline void softmax_pv(State& st, const f4& s0, const f4& s1, float scale_log2,
                                  int row0, int r_end, const char* lv, int i16, int g4) {
  float p[8];
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    p[j] = row0 + g4 * 4 + j < r_end ? s0[j] * scale_log2 : -INFINITY;
    p[4 + j] = row0 + 16 + g4 * 4 + j < r_end ? s1[j] * scale_log2 : -INFINITY;
    mx = fmaxf(mx, fmaxf(p[j], p[4 + j]));
  }
  if (__builtin_amdgcn_ballot_w64(mx > st.m + kLazy)) {  // rare: raise the reference max
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(st.m, mx);
    const float alpha = exp2f(st.m - m_new);
    st.l *= alpha;
#pragma unroll
    for (int d = 0; d < 8; ++d) st.acc[d] *= alpha;
    st.m = m_new;
  }
  float e[8], psum = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    e[j] = exp2f(p[j] - st.m);
    psum += e[j];
  }
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    hi[j] = bf2(e[2 * j], e[2 * j + 1]);
    const float h0 = __uint_as_float(hi[j] << 16), h1 = __uint_as_float(hi[j] & 0xFFFF0000u);
    lo[j] = bf2(e[2 * j] - h0, e[2 * j + 1] - h1);
  }
  const u4 phi = u4{hi[0], hi[1], hi[2], hi[3]};
  const u4 plo = u4{lo[0], lo[1], lo[2], lo[3]};
  st.l += psum;
  // lane (i16, g4) reads, for dim tile d, rows g4*4 + i16/4 (+16) at dims d*16 + 4*(i16%4)
  const int rr = g4 * 4 + (i16 >> 2);
  const int cb = (i16 & 3) >> 1, hb8 = (i16 & 1) * 8;
#pragma unroll
  for (int d = 0; d < 8; ++d) {
    const char* a0 = lv + toff(rr, 2 * d + cb) + hb8;
    const char* a1 = lv + toff(rr + 16, 2 * d + cb) + hb8;
    const u4 vt = ds_tr(a0, a1);
    st.acc[d] = mfma(vt, phi, st.acc[d]);
    st.acc[d] = mfma(vt, plo, st.acc[d]);
  }
}

// ---------------------------------------------------------------- dense rows
struct DenseSet {
  u4 k[8];  // A operands: k[blk*4 + t] = row blk*16 + i16, dims t*32 + g4*8 .. +7
  u4 v[8];  // v[i] = row lane/16 + 4*i, 16-byte chunk lane%16
};

// Buffer descriptor over rows [0, n_rows) of one (b, h_kv) of a dense segment:
// loads past the end return zeros (raw buffer, stride 0), so the partial last
// tile needs no clamping and each load needs one 32-bit offset register.
__device__ inline __amdgpu_buffer_rsrc_t rows_rsrc(const uint16_t* base, int n_rows) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), (short)0, n_rows * ROWB,
                                           0x00020000);
}

__device__ inline u4 bload(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(u4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

__device__ inline void dense_issue(__amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv, int row0,
                                   int lane, DenseSet& S) {
  const int i16 = lane & 15, g4 = lane >> 4;
  const int ko = (row0 + i16) * ROWB + g4 * 16;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    S.k[t] = bload(rk, ko, t * 64);
    S.k[4 + t] = bload(rk, ko, 16 * ROWB + t * 64);
  }
  const int vo = (row0 + g4) * ROWB + i16 * 16;
#pragma unroll
  for (int i = 0; i < 8; ++i) S.v[i] = bload(rv, vo, i * 4 * ROWB);
}

__device__ inline void dense_head(const DenseSet& S, char* lv, const u4 (&qop)[4], int lane,
                                  f4& s0, f4& s1) {
  const int i16 = lane & 15, g4 = lane >> 4;
#pragma unroll
  for (int i = 0; i < 8; ++i) *reinterpret_cast<u4*>(lv + toff(g4 + 4 * i, i16)) = S.v[i];
  s0 = f4{0.f, 0.f, 0.f, 0.f};
  s1 = s0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    s0 = mfma(S.k[t], qop[t], s0);
    s1 = mfma(S.k[4 + t], qop[t], s1);
  }
}

__device__ inline void dense_loop(State& st, const KSeg& ks, int bh, int r0, int r1, int n_mine,
                                  int wave, int lane, const u4 (&qop)[4], float scale_log2,
                                  char* lv) {
  const int i16 = lane & 15, g4 = lane >> 4;
  const int64_t base = (int64_t)bh * ks.row_stride * D;
  const __amdgpu_buffer_rsrc_t rk = rows_rsrc((const uint16_t*)ks.k + base, r1);
  const __amdgpu_buffer_rsrc_t rv = rows_rsrc((const uint16_t*)ks.v + base, r1);
  auto row_of = [&](int k) { return r0 + (wave + k * WAVES) * TILE; };
  DenseSet A, B;
  f4 s0, s1;
  if (n_mine > 0) dense_issue(rk, rv, row_of(0), lane, A);
  if (n_mine > 1) dense_issue(rk, rv, row_of(1), lane, B);
  int k = 0;
  // steady state without branches, so the compiler's wait counts keep the
  // other set's loads in flight: consume A, refill A, consume B, refill B
  for (; k + 3 < n_mine; k += 2) {
    dense_head(A, lv, qop, lane, s0, s1);
    dense_issue(rk, rv, row_of(k + 2), lane, A);
    softmax_pv(st, s0, s1, scale_log2, row_of(k), r1, lv, i16, g4);
    dense_head(B, lv, qop, lane, s0, s1);
    dense_issue(rk, rv, row_of(k + 3), lane, B);
    softmax_pv(st, s0, s1, scale_log2, row_of(k + 1), r1, lv, i16, g4);
  }
  const int left = n_mine - k;  // 0..3 tiles; A holds tile k, B tile k+1
  if (left >= 1) {
    dense_head(A, lv, qop, lane, s0, s1);
    if (left == 3) dense_issue(rk, rv, row_of(k + 2), lane, A);
    softmax_pv(st, s0, s1, scale_log2, row_of(k), r1, lv, i16, g4);
  }
  if (left >= 2) {
    dense_head(B, lv, qop, lane, s0, s1);
    softmax_pv(st, s0, s1, scale_log2, row_of(k + 1), r1, lv, i16, g4);
  }
  if (left == 3) {
    dense_head(A, lv, qop, lane, s0, s1);
    softmax_pv(st, s0, s1, scale_log2, row_of(k + 2), r1, lv, i16, g4);
  }
}

// ---------------------------------------------------------------- packed rows
// lane owns channels c8*8 .. c8*8+7 of rows lane/16 + 4*i (i < 8); BITS-bit
// codes of those 8 channels fill BITS bytes (one or two 32-bit words)
template <int BITS>
struct PackedSet {
  static constexpr int W = BITS == 8 ? 2 : 1;
  uint32_t ck[8][W], cv[8][W];
  float sv[8], mv[8];  // value scale/min of the lane's channel group, per row
  float sk[8], mk[8];  // key scale/min of the lane's 8 channels (the tile's row group:
                       // groups span at least one 32-row tile)
};

struct PackedSeg {
  const uint8_t* ck;
  const uint8_t* cv;
  const float* sk;
  const float* mk;
  const float* sv;
  const float* mv;
  const uint16_t* tk;
  const uint16_t* tv;
  int64_t off;
  int lgG, n_full, tail_len, bh;  // group size as a power of two
};

// the 8 codes of a lane's channels as floats (channel e of the lane -> c[e])
template <int BITS>
__device__ inline void codes8(const uint32_t (&w)[BITS == 8 ? 2 : 1], float (&c)[8]) {
  if constexpr (BITS == 4) {
    const uint32_t lo = w[0] & 0x0F0F0F0Fu, hi = (w[0] >> 4) & 0x0F0F0F0Fu;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      c[2 * b] = (float)((lo >> (8 * b)) & 0xFFu);
      c[2 * b + 1] = (float)((hi >> (8 * b)) & 0xFFu);
    }
  } else if constexpr (BITS == 8) {
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      c[b] = (float)((w[0] >> (8 * b)) & 0xFFu);
      c[4 + b] = (float)((w[1] >> (8 * b)) & 0xFFu);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) c[e] = (float)((w[0] >> (2 * e)) & 3u);
  }
}

template <int BITS>
__device__ inline void load_codes(const uint8_t* p, uint32_t (&w)[BITS == 8 ? 2 : 1]) {
  if constexpr (BITS == 8) {
    const uint2 a = *reinterpret_cast<const uint2*>(p);
    w[0] = a.x;
    w[1] = a.y;
  } else if constexpr (BITS == 4) {
    w[0] = *reinterpret_cast<const uint32_t*>(p);
  } else {
    w[0] = *reinterpret_cast<const uint16_t*>(p);
  }
}

template <int BITS>
__device__ inline void packed_issue(const PackedSeg& P, int row0, int last, int lane,
                                    PackedSet<BITS>& S) {
  const int c8 = lane & 15, g4 = lane >> 4;
  constexpr int RB = D * BITS / 8;  // bytes per row
  const int ngk = P.n_full >> P.lgG, lgGv = P.lgG;  // key row groups; value groups of G channels
  const bool any_full = row0 < P.n_full;
  if (any_full) {  // key scales of the tile's first row group
    const int64_t si = ((int64_t)P.bh * ngk + (row0 >> P.lgG)) * D + c8 * 8;
    const u4 a = *reinterpret_cast<const u4*>(P.sk + si);
    const u4 b = *reinterpret_cast<const u4*>(P.sk + si + 4);
    const u4 c = *reinterpret_cast<const u4*>(P.mk + si);
    const u4 d = *reinterpret_cast<const u4*>(P.mk + si + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      S.sk[e] = __uint_as_float(a[e]);
      S.sk[4 + e] = __uint_as_float(b[e]);
      S.mk[e] = __uint_as_float(c[e]);
      S.mk[4 + e] = __uint_as_float(d[e]);
    }
    const int ngv_lg = 7 - lgGv;  // log2(D / G)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = min(row0 + g4 + 4 * i, last);
      const int rq = min(r, P.n_full - 1);  // a valid code row even where r is a tail row
      load_codes<BITS>(P.ck + P.off + (int64_t)rq * RB + c8 * BITS, S.ck[i]);
      load_codes<BITS>(P.cv + P.off + (int64_t)rq * RB + c8 * BITS, S.cv[i]);
      const int64_t vi = (((int64_t)P.bh * P.n_full + rq) << ngv_lg) + ((c8 * 8) >> lgGv);
      S.sv[i] = P.sv[vi];
      S.mv[i] = P.mv[vi];
    }
  }
}

// dequantise one row's 8 channels of K and V into packed bf16 (4 x u32 each)
template <int BITS>
__device__ inline void dequant_row(const PackedSet<BITS>& S, int i, u4& kk, u4& vv) {
  float qk[8], qv[8];
  codes8<BITS>(S.ck[i], qk);
  codes8<BITS>(S.cv[i], qv);
  float xk[8], xv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    xk[e] = fmaf(qk[e], S.sk[e], S.mk[e]);
    xv[e] = fmaf(qv[e], S.sv[i], S.mv[i]);
  }
  kk = u4{bf2(xk[0], xk[1]), bf2(xk[2], xk[3]), bf2(xk[4], xk[5]), bf2(xk[6], xk[7])};
  vv = u4{bf2(xv[0], xv[1]), bf2(xv[2], xv[3]), bf2(xv[4], xv[5]), bf2(xv[6], xv[7])};
}

template <int BITS>
__device__ inline void packed_head(const PackedSeg& P, const PackedSet<BITS>& S, int row0, int last,
                                   char* lk, char* lv, const u4 (&qop)[4], int lane, f4& s0,
                                   f4& s1) {
  const int c8 = lane & 15, g4 = lane >> 4;
  if (row0 + TILE <= P.n_full) {  // whole tile quantised: no per-row branches
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int rr = g4 + 4 * i;
      u4 kk, vv;
      dequant_row<BITS>(S, i, kk, vv);
      *reinterpret_cast<u4*>(lk + toff(rr, c8)) = kk;
      *reinterpret_cast<u4*>(lv + toff(rr, c8)) = vv;
    }
  } else {  // the tile reaches the residual tail (at most once per head)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int rr = g4 + 4 * i;
      const int r = min(row0 + rr, last);
      u4 kk, vv;
      if (r < P.n_full) {
        dequant_row<BITS>(S, i, kk, vv);
      } else {
        const int64_t e = ((int64_t)P.bh * P.tail_len + (r - P.n_full)) * D + c8 * 8;
        kk = *reinterpret_cast<const u4*>(P.tk + e);
        vv = *reinterpret_cast<const u4*>(P.tv + e);
      }
      *reinterpret_cast<u4*>(lk + toff(rr, c8)) = kk;
      *reinterpret_cast<u4*>(lv + toff(rr, c8)) = vv;
    }
  }
  const int i16 = lane & 15;
  s0 = f4{0.f, 0.f, 0.f, 0.f};
  s1 = s0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const u4 k0 = *reinterpret_cast<const u4*>(lk + toff(i16, t * 4 + g4));
    const u4 k1 = *reinterpret_cast<const u4*>(lk + toff(16 + i16, t * 4 + g4));
    s0 = mfma(k0, qop[t], s0);
    s1 = mfma(k1, qop[t], s1);
  }
}

template <int BITS>
__device__ inline void packed_loop(State& st, const PackedSeg& P, int r0, int r1, int n_mine,
                                   int wave, int lane, const u4 (&qop)[4], float scale_log2,
                                   char* lk, char* lv) {
  const int i16 = lane & 15, g4 = lane >> 4;
  const int last = r1 - 1;
  auto row_of = [&](int k) { return r0 + (wave + k * WAVES) * TILE; };
  PackedSet<BITS> A, B;
  f4 s0, s1;
  if (n_mine > 0) packed_issue<BITS>(P, row_of(0), last, lane, A);
  if (n_mine > 1) packed_issue<BITS>(P, row_of(1), last, lane, B);
  int k = 0;
  for (; k + 3 < n_mine; k += 2) {
    packed_head<BITS>(P, A, row_of(k), last, lk, lv, qop, lane, s0, s1);
    packed_issue<BITS>(P, row_of(k + 2), last, lane, A);
    softmax_pv(st, s0, s1, scale_log2, row_of(k), r1, lv, i16, g4);
    packed_head<BITS>(P, B, row_of(k + 1), last, lk, lv, qop, lane, s0, s1);
    packed_issue<BITS>(P, row_of(k + 3), last, lane, B);
    softmax_pv(st, s0, s1, scale_log2, row_of(k + 1), r1, lv, i16, g4);
  }
  const int left = n_mine - k;
  if (left >= 1) {
    packed_head<BITS>(P, A, row_of(k), last, lk, lv, qop, lane, s0, s1);
    if (left == 3) packed_issue<BITS>(P, row_of(k + 2), last, lane, A);
    softmax_pv(st, s0, s1, scale_log2, row_of(k), r1, lv, i16, g4);
  }
  if (left >= 2) {
    packed_head<BITS>(P, B, row_of(k + 1), last, lk, lv, qop, lane, s0, s1);
    softmax_pv(st, s0, s1, scale_log2, row_of(k + 1), r1, lv, i16, g4);
  }
  if (left == 3) {
    packed_head<BITS>(P, A, row_of(k + 2), last, lk, lv, qop, lane, s0, s1);
    softmax_pv(st, s0, s1, scale_log2, row_of(k + 2), r1, lv, i16, g4);
  }
}

// ---------------------------------------------------------------- kernel
// Work split: W workgroups per (b, h_kv) (two per CU, one round).  Workgroup
// w takes the w-th of W equal tile-aligned shares of every segment, so each
// CU mixes bandwidth-bound dense tiles with dequantisation-bound packed
// tiles.  Each workgroup writes one partial record (m, l, o) per segment for
// its query rows (slot s*W + w; m = -inf for an empty share); the combine
// kernel merges them.
struct DecodePlan {
  int W;      // workgroups per (b, h_kv)
  int n_seg;
};

// tile-aligned share w of n rows among W workgroups
__device__ inline int share_row(int n, int w, int W) {
  const int64_t r = ((int64_t)n * w + W - 1) / W;
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

// merge the four waves' state through LDS and write one partial record
__device__ inline void flush(State& st, char* lds, const Ctx& c, int slot, bool ok, int lane,
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

__global__ __launch_bounds__(256, 2) void decode_mfma_kernel(KSegs segs, DecodePlan pl,
                                                             const uint16_t* __restrict__ q,
                                                             int Hq, int Hkv, int M,
                                                             float scale_log2,
                                                             float* __restrict__ partial) {
  __shared__ __attribute__((aligned(16))) char lds[WAVES * 2 * TILEB];
  const int w = blockIdx.x, bh = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int G = Hq / Hkv, nq = G * M, b = bh / Hkv, hkv = bh % Hkv;
  const int W = pl.W;

  // query block: slot i16 = g * M + m  (query head hkv*G + g, row m)
  u4 qop[4];
  {
    const bool live = i16 < nq;
    const int64_t qrow = live ? (((int64_t)b * Hq + hkv * G + i16 / M) * M + i16 % M) : 0;
#pragma unroll
    for (int t = 0; t < 4; ++t)
      qop[t] = live ? *reinterpret_cast<const u4*>(q + qrow * D + t * 32 + g4 * 8) : u4{0, 0, 0, 0};
  }
  char* lk = lds + wave * 2 * TILEB;
  char* lv = lk + TILEB;
  Ctx c{partial, pl.n_seg * W, nq, M, Hq, G, b, hkv};

  for (int si = 0; si < pl.n_seg; ++si) {
    const KSeg& ks = segs.s[si];
    const int r0 = share_row(ks.n_rows, w, W);
    const int r1 = share_row(ks.n_rows, w + 1, W);
    State st;
    st.m = -INFINITY;
    st.l = 0.0f;
#pragma unroll
    for (int d = 0; d < 8; ++d) st.acc[d] = f4{0.f, 0.f, 0.f, 0.f};
    bool ok = true;
    if (r1 > r0) {
      int bits = 0;
      int64_t off = 0;
      if (ks.kind == UC_SEG_PACKED) ok = head_codes(ks, bh, D, bits, off);
      const int n_tiles = ok ? (r1 - r0 + TILE - 1) / TILE : 0;
      const int n_mine = n_tiles > wave ? (n_tiles - wave + WAVES - 1) / WAVES : 0;
      if (ks.kind == UC_SEG_DENSE) {
        dense_loop(st, ks, bh, r0, r1, n_mine, wave, lane, qop, scale_log2, lv);
      } else if (n_mine > 0) {
        PackedSeg P;
        P.ck = ks.codes_k;
        P.cv = ks.codes_v;
        P.sk = ks.scale_k;
        P.mk = ks.min_k;
        P.sv = ks.scale_v;
        P.mv = ks.min_v;
        P.tk = (const uint16_t*)ks.tail_k;
        P.tv = (const uint16_t*)ks.tail_v;
        P.off = off;
        P.lgG = __builtin_ctz((unsigned)ks.group);
        P.n_full = ks.n_full;
        P.tail_len = ks.tail_len;
        P.bh = bh;
        if (bits == 4) packed_loop<4>(st, P, r0, r1, n_mine, wave, lane, qop, scale_log2, lk, lv);
        else packed_loop<2>(st, P, r0, r1, n_mine, wave, lane, qop, scale_log2, lk, lv);
      }
    }
    flush(st, lds, c, si * W + w, ok, lane, wave);
  }

}

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

// workgroups per (b, h_kv): two resident workgroups per CU in one round
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
    // packed: 2- or 4-bit codes of uniform width, key row groups covering
    // whole 32-row tiles (one scale set per tile)
    if (segs.s[i].kind == UC_SEG_PACKED &&
        (segs.s[i].group < TILE || segs.s[i].head_bits || segs.s[i].bits == 8))
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

hipError_t launch_decode_mfma(const uc_shape& sh, const KSegs& segs, const void* q, int M,
                              float sm_scale, float* o, float* lse, float* seg_lse, void* ws,
                              hipStream_t st) {
  DecodePlan p{};
  p.W = decode_w(sh);
  p.n_seg = segs.n;
  float* partial = (float*)ws;
  hipLaunchKernelGGL(decode_mfma_kernel, dim3(p.W, sh.B * sh.Hkv), dim3(256), 0, st, segs, p,
                     (const uint16_t*)q, sh.Hq, sh.Hkv, M, sm_scale * kLog2e, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // records are segment-major: segment s owns slots [s*W, (s+1)*W)
  ChunkPlan cp{};
  cp.n_chunks = segs.n * p.W;
  for (int i = 0; i <= kMaxSeg; ++i) cp.first[i] = min(i, segs.n) * p.W;
  return launch_attend_combine(sh, segs, cp, M, partial, o, lse, seg_lse, st);
}

}  // namespace uc
