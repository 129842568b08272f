// attend_prefill.hip -- multi-query (prefill / denoising) attention over
// bf16 segments on the CDNA4 matrix cores (App. E, "Attention over
// heterogeneous cache segments": one softmax across all segments; packed
// segments are dequantised into a reusable workspace before attention).
//
// Work item: 128 query rows of one (b, h_kv) -- the rows of its G query heads
// are contiguous in q -- in one workgroup of four waves; each wave owns two
// 16-row query tiles.  The workgroup walks every key tile (32 rows) of every
// segment once: the waves stage the K and V rows of later tiles through
// registers (two register sets, so a tile's loads have two iterations to
// arrive) into a four-deep ring of padded LDS tiles.  The loop is a
// three-stage software pipeline: in iteration t a wave issues, interleaved
// (each matrix instruction followed by its share of the softmax),
//   S^T(t+1) = K Q^T    v_mfma_f32_16x16x32_bf16, K rows read from LDS as the
//                       A operand (shared by both query tiles), Q^T in
//                       registers;
//   O^T += V^T P(t-1)   V^T by transposing LDS reads (shared by both query
//                       tiles); fp16 P and V on v_mfma_f32_16x16x32_f16 when
//                       every V value of the call fits fp16 (a range pass sets
//                       a flag the kernel reads), else bf16 V with P as bf16
//                       hi + lo parts;
//   softmax(t)          on the vector ALUs: base-2 exponentials against a
//                       lazily raised reference maximum, running per-segment
//                       sums for seg_lse;
// none of which depends on another, so one wave keeps the matrix cores and
// the vector ALUs busy at once; the probability operands of consecutive
// tiles alternate between two register sets.  The rare raise of the reference
// maximum runs
// after the matrix instructions (it rescales the accumulators they update).
// Outputs (normalised O, lse, per-segment lse) are written directly; no
// split over keys.  Workgroups are mapped so that those of one (b, h_kv) run
// on the same XCD and share its L2 copy of the head's rows.
//
// Packed segments first go through dequant_kernel: codes -> round_to_bf16(
// fmaf(code, scale, min)) into a [B, Hkv, n_full, D] bf16 workspace (once per
// call, where the query blocks of a head would otherwise each decode every
// packed tile again); their residual tails are read in place.  This
// preparation (with the fp16 V copies and the range flag) is a stage of its
// own, so an execution plan over an unchanged cache runs it once.
#include <string.h>

#include <type_traits>

#include "mfma_util.h"
#include "uc_common.h"

namespace uc {
namespace {

using namespace mf;

constexpr int STAGES = 4;                  // stages in LDS: t-1 .. t+1 in use, t+2 staged
constexpr int SUBB = 2 * TILEB;            // one tile: K rows + V rows
// Layouts: W waves per workgroup, TPS tiles per stage (one barrier per
// stage) and QT 16-row query tiles per wave.  <4, 1, 2>: 128 query rows, two
// workgroups per CU; <8, 2, 2>: 256 query rows, one workgroup per CU, half
// the barriers and staging per query row.  (Four query tiles per wave, one
// wave per SIMD, measured slower than two waves per SIMD with two.)
template <int W, int QT>
constexpr int qrows() { return W * QT * 16; }
constexpr float kLazy = 8.0f;
constexpr float kLazyExp = 256.0f;  // 2^kLazy
constexpr int kMaxViews = 2 * kMaxSeg;

// dense row views of the logical sequence, in order; seg = logical segment
struct View {
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* vh;  // the V rows converted to fp16 once per call, [BH, n, D]
  int64_t bh_stride;   // elements between consecutive (b, h_kv) of k and v
  int n;               // rows
  int seg;
};

struct Views {
  View v[kMaxViews];
  int n;
  int tiles;  // total key tiles
};

struct QState {
  float m, l, ls;  // reference max (base 2), row sum, running sum of the current segment
  f4 acc[8];       // O^T, dims d*16 + g4*4 + j of query column i16
};

// tile t of the sequence -> view index and first row
__device__ inline int tile_view(const Views& vs, int t, int& row0) {
  int i = 0;
  while (i + 1 < vs.n && t >= (vs.v[i].n + TILE - 1) / TILE) {
    t -= (vs.v[i].n + TILE - 1) / TILE;
    ++i;
  }
  row0 = t * TILE;
  return i;
}

// A walk over the logical sequence one 32-row tile at a time.  The current
// view's row count, segment and this (b, h_kv)'s K and V rows stay in
// scalars, so a step reads the view table (kernel arguments) only when it
// crosses into the next view.
template <bool F16>
struct Cursor {
  int vi, row0, n, seg;
  const uint16_t* k;
  const uint16_t* v;
  __device__ inline void load(const Views& vs, int bh) {
    const View& w = vs.v[vi];
    n = w.n;
    seg = w.seg;
    k = w.k + bh * w.bh_stride;
    v = F16 ? w.vh + (int64_t)bh * w.n * D : w.v + bh * w.bh_stride;
  }
  __device__ inline void start(const Views& vs, int bh, int t) {
    vi = tile_view(vs, t, row0);
    load(vs, bh);
  }
  __device__ inline void next(const Views& vs, int bh) {
    row0 += TILE;
    if (row0 >= n && vi + 1 < vs.n) {
      ++vi;
      row0 = 0;
      load(vs, bh);
    }
  }
};

// one thread's share of staging the two tiles of a stage: row tid/16,
// chunk tid%16 of each tile's K and V rows
struct Stage {
  u4 k[2], v[2];
};

// A thread stages two 16-byte chunks of K and of V per stage: chunk i is
// global chunk g = tid + i * NT, tile g / 512 of the stage, row (g % 512) / 16,
// column chunk g % 16 (two rows of one tile with 256 threads, one row of each
// of two tiles with 512).  F16: V comes from the view's fp16 copy.
template <bool F16, int NT>
__device__ inline void stage_load(const Cursor<F16>& cu, Stage& S, int i) {
  const __amdgpu_buffer_rsrc_t rk = rsrc(cu.k, (uint32_t)cu.n * ROWB);
  const __amdgpu_buffer_rsrc_t rv = rsrc(cu.v, (uint32_t)cu.n * ROWB);
  const int g = (threadIdx.x + i * NT) & 511, r = g >> 4, c = g & 15;
  const int off = (cu.row0 + r) * ROWB + c * 16;
  S.k[i] = bload(rk, off, 0);
  S.v[i] = bload(rv, off, 0);
}

// chunk i into the LDS tile at buf (K rows, V rows at + TILEB)
template <int NT>
__device__ inline void stage_store(char* buf, const Stage& S, int i) {
  const int g = (threadIdx.x + i * NT) & 511, r = g >> 4, c = g & 15;
  *reinterpret_cast<u4*>(buf + toff(r, c)) = S.k[i];
  *reinterpret_cast<u4*>(buf + TILEB + toff(r, c)) = S.v[i];
}

// LDS tile of tile t of the sequence
template <int TPS>
__device__ inline char* tile_buf(char* lds, int t) {
  return lds + ((t / TPS) % STAGES) * (TPS * SUBB) + (t % TPS) * SUBB;
}

// raw logits of one query tile (8 per lane).  Rows past a view's end were
// staged as zeros (range-checked loads), so their logit is 0 and their V row
// is 0: they add nothing to O, and tile_step removes what they add to the
// row sums.
__device__ inline void tile_logits(const f4& s0, const f4& s1, float (&p)[8]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    p[j] = s0[j];
    p[4 + j] = s1[j];
  }
}

// common path of the softmax of one query tile: probabilities against the
// current reference; returns the lane's sum.  A lane sum above 2^kLazy
// (every logit more than kLazy above the reference makes one, and a first
// tile's -inf reference makes inf or NaN) sends the wave through tile_raise.
__device__ inline float tile_exp(const QState& st, const f4& s0, const f4& s1, float scale_log2,
                                 float (&e)[8]) {
  float p[8];
  tile_logits(s0, s1, p);
#pragma unroll
  for (int j = 0; j < 8; ++j) e[j] = __builtin_amdgcn_exp2f(fmaf(p[j], scale_log2, -st.m));
  return ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
}

// rare path: raise the reference to the column maximum, rescale the running
// state and recompute the probabilities (they stay below 2^kLazy, well inside
// fp16)
__device__ inline float tile_raise(QState& st, const f4& s0, const f4& s1, float scale_log2,
                                   float (&e)[8]) {
  float p[8];
  tile_logits(s0, s1, p);
  // the scale is positive, so the maximum of the raw logits gives the maximum
  float mx = fmaxf(fmaxf(fmaxf(p[0], p[1]), fmaxf(p[2], p[3])),
                   fmaxf(fmaxf(p[4], p[5]), fmaxf(p[6], p[7]))) * scale_log2;
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const float m_new = fmaxf(st.m, mx);
  const float alpha = __builtin_amdgcn_exp2f(st.m - m_new);
  st.l *= alpha;
  st.ls *= alpha;
#pragma unroll
  for (int d = 0; d < 8; ++d) st.acc[d] *= alpha;
  st.m = m_new;
#pragma unroll
  for (int j = 0; j < 8; ++j) e[j] = __builtin_amdgcn_exp2f(fmaf(p[j], scale_log2, -st.m));
  return ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
}

// probability operands of one query tile: fp16 P (F16), else bf16 hi + lo
struct POp {
  u4 hi, lo;
};

template <bool F16>
__device__ inline POp pack_p(const float (&e)[8]) {
  POp r;
  if (F16) {
    r.hi = u4{h2(e[0], e[1]), h2(e[2], e[3]), h2(e[4], e[5]), h2(e[6], e[7])};
    r.lo = r.hi;
  } else {
    split_p(e, r.hi, r.lo);
  }
  return r;
}

// sum of a lane-partial value over the four key-row lanes of a query column
__device__ inline float col_sum(float x) {
  x += __shfl_xor(x, 16, 64);
  x += __shfl_xor(x, 32, 64);
  return x;
}

// K rows of tile buffer lk as A operands (shared by the query tiles)
__device__ inline void load_ka(const char* lk, int i16, int g4, u4 (&ka)[8]) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    ka[k] = *reinterpret_cast<const u4*>(lk + toff(i16, k * 4 + g4));
    ka[4 + k] = *reinterpret_cast<const u4*>(lk + toff(16 + i16, k * 4 + g4));
  }
}

// S^T = K Q^T of one tile for one query tile
__device__ inline void qt_scores(const u4 (&ka)[8], const u4 (&q)[4], f4& s0, f4& s1) {
  s0 = f4{0.f, 0.f, 0.f, 0.f};
  s1 = s0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    s0 = mfma(ka[k], q[k], s0);
    s1 = mfma(ka[4 + k], q[k], s1);
  }
}

// S^T = K Q^T of one tile for every query tile of the wave
template <int QT>
__device__ inline void tile_scores(const u4 (&ka)[8], const u4 (&qop)[QT][4], f4 (&s)[QT][2]) {
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) qt_scores(ka, qop[qt], s[qt][0], s[qt][1]);
}

// O^T += V^T P of one tile (V^T operands read from the tile's LDS V rows)
template <bool F16, int QT>
__device__ inline void tile_pv(const char* lv, const POp (&pp)[QT], QState (&st)[QT], int i16,
                               int g4) {
  const char* vb = vt_base(lv, i16, g4);
#pragma unroll
  for (int d = 0; d < 8; ++d) {
    const u4 vt = vt_operand_at(vb, d);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      if (F16) {
        st[qt].acc[d] = mfma_f16(vt, pp[qt].hi, st[qt].acc[d]);
      } else {
        st[qt].acc[d] = mfma(vt, pp[qt].hi, st[qt].acc[d]);
        st[qt].acc[d] = mfma(vt, pp[qt].lo, st[qt].acc[d]);
      }
    }
  }
}

// Scheduling of one pipeline iteration: N matrix instructions, each followed
// by its even share of about NV vector instructions.
template <int N, int NV, int I = 0>
__device__ inline void interleave() {
  if constexpr (I < N) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    constexpr int v = (I + 1) * NV / N - I * NV / N;
    if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x002, v, 0);  // VALU
    interleave<N, NV, I + 1>();
  }
}

// One iteration of the pipeline (tile t): scores of tile t+1 and, with PV,
// O += V^T P of tile t-1 (operands pp) on the matrix cores, interleaved with
// the softmax common path of tile t on the vector ALUs; then the rare
// reference raise (which recomputes tile t's scores from its K rows, still in
// LDS, so the scores need not stay in registers) and the running sums.  sc
// holds tile t's scores on entry and tile t+1's on exit; tile t's
// probability operands go to pn (the caller alternates two sets, so they
// are never copied).
template <bool F16, int TPS, bool PV, int QT>
__device__ __attribute__((always_inline)) inline void tile_step(
    int t, char* lds, const u4 (&qop)[QT][4], QState (&st)[QT], f4 (&sc)[QT][2],
    const POp (&pp)[QT], POp (&pn)[QT], float scale_log2, int n_valid, int i16, int g4) {
  float psum[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    float e[8];
    psum[qt] = tile_exp(st[qt], sc[qt][0], sc[qt][1], scale_log2, e);
    pn[qt] = pack_p<F16>(e);
  }
  {
    u4 ka[8];
    load_ka(tile_buf<TPS>(lds, t + 1), i16, g4, ka);
    tile_scores(ka, qop, sc);
  }
  if (PV) tile_pv<F16, QT>(tile_buf<TPS>(lds, t - 1) + TILEB, pp, st, i16, g4);
  // matrix and vector instructions in turn (the softmax takes about 26
  // vector instructions per query tile, 30 with the bf16 split)
  interleave<QT * 8 + (PV ? QT * 8 * (F16 ? 1 : 2) : 0), QT * (F16 ? 26 : 30)>();
  bool rare = false;
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) rare = rare || !(psum[qt] <= kLazyExp);
  if (__builtin_amdgcn_ballot_w64(rare)) {  // rare: raise the reference max
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
      if (__builtin_amdgcn_ballot_w64(!(psum[qt] <= kLazyExp))) {
        u4 ka[8];
        load_ka(tile_buf<TPS>(lds, t), i16, g4, ka);
        f4 s0, s1;
        qt_scores(ka, qop[qt], s0, s1);
        float e[8];
        psum[qt] = tile_raise(st[qt], s0, s1, scale_log2, e);
        pn[qt] = pack_p<F16>(e);
      }
  }
  if (n_valid < TILE) {
    // the TILE - n_valid rows past the view's end each added 2^-m to their
    // column's sum (logit 0); a quarter of that comes off each of the
    // column's four lanes.  The fp16 bound above counted them, so their
    // probability operands stay in range too.
    const float gone = 0.25f * (float)(TILE - n_valid);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt)
      psum[qt] = fmaf(-gone, __builtin_amdgcn_exp2f(-st[qt].m), psum[qt]);
  }
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    st[qt].l += psum[qt];
    st[qt].ls += psum[qt];
  }
}

// the key-tile loop of one workgroup (see the file comment).  Returns the
// view of the last tile.
template <bool F16, int W, int TPS, int QT>
__device__ __attribute__((always_inline)) inline int tile_loop(
    const Views& vs, int bh, char* lds, const u4 (&qop)[QT][4], QState (&st)[QT],
    float scale_log2, int r_wave, int nq, int64_t qbase, int nseg, float* seg_lse, int i16,
    int g4) {
  int cur_view = -1, cur_seg = -1;
  const int T = vs.tiles;
  // tiles go through LDS in stages of TPS: stage j holds tiles TPS*j ..
  // TPS*j + TPS - 1; after the last tile of stage j the tiles of stage j + 2
  // are stored, and one barrier per stage publishes them.  During stage j
  // the pipeline reads stages j - 1 .. j + 1.  With two tiles per stage the
  // tiles of stage j + 2 are loaded at the start of stage j; with one, tile
  // t + 3 is loaded at the start of iteration t into the other of two
  // register sets, so a load has two iterations to arrive.
  constexpr int NT = W * 64;
  Cursor<F16> ct, cs;  // tile t (computed) and the next tile to stage
  Stage SA, SB;
  {
    Stage S;
    ct.start(vs, bh, 0);
    cs.start(vs, bh, 0);
    for (int u = 0; u < 2 * TPS && u < T; ++u) {
      // the chunks of tile u (both with one tile per stage)
#pragma unroll
      for (int i = 0; i < 2; ++i)
        if (TPS == 1 || i == 0) stage_load<F16, NT>(cs, S, i);
#pragma unroll
      for (int i = 0; i < 2; ++i)
        if (TPS == 1 || i == 0) stage_store<NT>(tile_buf<TPS>(lds, u), S, i);
      cs.next(vs, bh);
    }
    if (TPS == 1 && T > 2) {
      stage_load<F16, NT>(cs, SA, 0);
      stage_load<F16, NT>(cs, SA, 1);
      cs.next(vs, bh);
    }
  }
  __syncthreads();
  f4 sc[QT][2];
  {
    u4 ka[8];
    load_ka(tile_buf<TPS>(lds, 0), i16, g4, ka);
    tile_scores(ka, qop, sc);
  }
  POp pa[QT], pb[QT];  // probability operands of alternate tiles
  int n_pre = 0;  // tiles of the stage in flight (two tiles per stage)
  // one iteration (PV of tile t-1 from pp, P of tile t into pn; with one
  // tile per stage, tile t+2 stored from Sc and tile t+3 loaded into Sn);
  // the first (no previous tile to multiply with V) is peeled
  auto iter = [&](int t, auto pv, const POp (&pp)[QT], POp (&pn)[QT], Stage& Sc, Stage& Sn) {
    if (TPS == 1) {
      if (t + 3 < T) {
        stage_load<F16, NT>(cs, Sn, 0);
        stage_load<F16, NT>(cs, Sn, 1);
        cs.next(vs, bh);
      }
    } else if (t % TPS == 0 && t + 2 * TPS < T) {  // the tiles of stage t/TPS + 2
      stage_load<F16, NT>(cs, Sn, 0);
      cs.next(vs, bh);
      n_pre = 1;
      if (t + 2 * TPS + 1 < T) {
        stage_load<F16, NT>(cs, Sn, 1);
        cs.next(vs, bh);
        n_pre = 2;
      }
    }
    const int vi = ct.vi;
    const int n_valid = min(TILE, ct.n - ct.row0);
    if (seg_lse && vi != cur_view && cur_view >= 0 && ct.seg != cur_seg) {
      // the previous logical segment ended: its log-sum-exp per query row
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        const float ls = col_sum(st[qt].ls);
        const int r = r_wave + qt * 16 + i16;
        if (g4 == 0 && r < nq)
          seg_lse[(qbase + r) * nseg + cur_seg] =
              ls > 0.0f ? (st[qt].m + __log2f(ls)) * kLn2 : -INFINITY;
        st[qt].ls = 0.0f;
      }
    }
    cur_view = vi;
    cur_seg = ct.seg;
    ct.next(vs, bh);
    // past the last tile the next scores come from a stale buffer and are
    // never used
    tile_step<F16, TPS, decltype(pv)::value, QT>(t, lds, qop, st, sc, pp, pn, scale_log2,
                                                 n_valid, i16, g4);
    if (t % TPS == TPS - 1 || t == T - 1) {  // the stage's last tile
      const int t0 = t - t % TPS + 2 * TPS;  // first tile of the staged stage
      if (TPS == 1) {
        if (t0 < T) {
          stage_store<NT>(tile_buf<TPS>(lds, t0), Sc, 0);
          stage_store<NT>(tile_buf<TPS>(lds, t0), Sc, 1);
        }
      } else {  // Sc and Sn are the same set
        if (n_pre >= 1) stage_store<NT>(tile_buf<TPS>(lds, t0), Sc, 0);
        if (n_pre >= 2) stage_store<NT>(tile_buf<TPS>(lds, t0 + 1), Sc, 1);
      }
      n_pre = 0;
      __syncthreads();
    }
  };
  // with two tiles per stage both register-set roles are SA
  Stage& S1 = TPS == 1 ? SB : SA;
  iter(0, std::false_type{}, pb, pa, SA, S1);
  int t = 1;
  for (; t + 1 < T; t += 2) {
    iter(t, std::true_type{}, pa, pb, S1, SA);
    iter(t + 1, std::true_type{}, pb, pa, SA, S1);
  }
  // the last tile's O += V^T P
  if (t < T) {
    iter(t, std::true_type{}, pa, pb, S1, SA);
    tile_pv<F16, QT>(tile_buf<TPS>(lds, T - 1) + TILEB, pb, st, i16, g4);
  } else {
    tile_pv<F16, QT>(tile_buf<TPS>(lds, T - 1) + TILEB, pa, st, i16, g4);
  }
  return cur_view;
}

template <int W, int TPS, int QT>
__global__ __launch_bounds__(W * 64, W == 4 && QT == 2 ? 2 : 1) void prefill_mfma_kernel(Views vs, const uint16_t* __restrict__ q,
                                                              int Hq, int Hkv, int M, int nseg,
                                                              int n_qblocks, int n_work,
                                                              float scale_log2, float* __restrict__ o,
                                                              float* __restrict__ lse,
                                                              float* __restrict__ seg_lse,
                                                              const int* __restrict__ v_unsafe) {
  __shared__ __attribute__((aligned(16))) char lds[STAGES * TPS * SUBB];
  // XCD-aware work mapping: consecutive work items (the query blocks of one
  // head, which share its K/V rows) go to the same XCD
  const int per_xcd = (n_work + 7) / 8;
  const int work = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (work >= n_work) return;
  const int qb = work % n_qblocks, bh = work / n_qblocks;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i16 = lane & 15, g4 = lane >> 4;
  const int G = Hq / Hkv, nq = G * M, b = bh / Hkv, hkv = bh % Hkv;
  const int64_t qbase = ((int64_t)b * Hq + hkv * G) * M;  // first query row of the head
  const int r_wave = qb * qrows<W, QT>() + wave * QT * 16;  // first row of the wave

  u4 qop[QT][4];
  QState st[QT];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int r = r_wave + t * 16 + i16;
#pragma unroll
    for (int k = 0; k < 4; ++k)
      qop[t][k] = r < nq ? *reinterpret_cast<const u4*>(q + (qbase + r) * D + k * 32 + g4 * 8)
                         : u4{0, 0, 0, 0};
    st[t].m = -INFINITY;
    st[t].l = 0.0f;
    st[t].ls = 0.0f;
#pragma unroll
    for (int d = 0; d < 8; ++d) st[t].acc[d] = f4{0.f, 0.f, 0.f, 0.f};
  }

  // segments without rows never see a tile: their log-sum-exp stays -inf
  if (seg_lse && g4 == 0) {
#pragma unroll
    for (int t = 0; t < QT; ++t) {
      const int r = r_wave + t * 16 + i16;
      if (r < nq)
        for (int a = 0; a < nseg; ++a) seg_lse[(qbase + r) * nseg + a] = -INFINITY;
    }
  }
  const bool f16 = *v_unsafe == 0;
  const int cur_view = f16 ? tile_loop<true, W, TPS, QT>(vs, bh, lds, qop, st, scale_log2, r_wave, nq, qbase,
                                             nseg, seg_lse, i16, g4)
                           : tile_loop<false, W, TPS, QT>(vs, bh, lds, qop, st, scale_log2, r_wave, nq, qbase,
                                              nseg, seg_lse, i16, g4);
  // outputs
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int r = r_wave + qt * 16 + i16;
    const float l = col_sum(st[qt].l);
    const float ls = col_sum(st[qt].ls);
    if (r < nq) {
      const float inv = 1.0f / l;
      float* orow = o + (qbase + r) * D;
#pragma unroll
      for (int d = 0; d < 8; ++d) *reinterpret_cast<f4*>(orow + d * 16 + g4 * 4) = st[qt].acc[d] * inv;
      if (g4 == 0) {
        if (lse) lse[qbase + r] = (st[qt].m + __log2f(l)) * kLn2;
        if (seg_lse && cur_view >= 0)
          seg_lse[(qbase + r) * nseg + vs.v[cur_view].seg] =
              ls > 0.0f ? (st[qt].m + __log2f(ls)) * kLn2 : -INFINITY;
      }
    }
  }
}

// codes -> bf16 values of one packed segment's whole row groups:
// out[b, h, r, c] = round_to_bf16(fmaf(code, scale, min)); one thread per
// 8 channels of one row, K and V: the 8 codes in one 16-, 32- or 64-bit load,
// the key scales and minima in 16-byte loads, one value group (groups are at
// least 8 channels)
__global__ void dequant_kernel(KSeg s, int BH, uint16_t* __restrict__ kout,
                               uint16_t* __restrict__ vout, uint16_t* __restrict__ vhout,
                               int* __restrict__ v_unsafe) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (bh, row, c8)
  const int c8 = (int)(e % (D / 8));
  const int64_t rr = e / (D / 8);
  const int r = (int)(rr % s.n_full), bh = (int)(rr / s.n_full);
  if (bh >= BH) return;
  int bits;
  int64_t off;
  u4 ko, vo;
  if (!head_codes(s, bh, D, bits, off) || (off & 15)) {
    const uint32_t nan2 = 0x7FC07FC0u;
    ko = u4{nan2, nan2, nan2, nan2};
    vo = ko;
  } else {
    const int rb = D * bits / 8, G = s.group;
    const int64_t cb = off + (int64_t)r * rb + c8 * bits;  // 8 channels = bits bytes
    uint64_t wk, wv;
    if (bits == 4) {
      wk = *reinterpret_cast<const uint32_t*>(s.codes_k + cb);
      wv = *reinterpret_cast<const uint32_t*>(s.codes_v + cb);
    } else if (bits == 2) {
      wk = *reinterpret_cast<const uint16_t*>(s.codes_k + cb);
      wv = *reinterpret_cast<const uint16_t*>(s.codes_v + cb);
    } else {
      wk = *reinterpret_cast<const uint64_t*>(s.codes_k + cb);
      wv = *reinterpret_cast<const uint64_t*>(s.codes_v + cb);
    }
    const int mask = (1 << bits) - 1;
    const int64_t kg = ((int64_t)bh * s.kgroups + r / G) * D + c8 * 8;
    const f4 sk0 = *reinterpret_cast<const f4*>(s.scale_k + kg);
    const f4 sk1 = *reinterpret_cast<const f4*>(s.scale_k + kg + 4);
    const f4 mk0 = *reinterpret_cast<const f4*>(s.min_k + kg);
    const f4 mk1 = *reinterpret_cast<const f4*>(s.min_k + kg + 4);
    const float sk[8] = {sk0[0], sk0[1], sk0[2], sk0[3], sk1[0], sk1[1], sk1[2], sk1[3]};
    const float mk[8] = {mk0[0], mk0[1], mk0[2], mk0[3], mk1[0], mk1[1], mk1[2], mk1[3]};
    const int64_t vi = ((int64_t)bh * s.cap_full + r) * (D / G) + (c8 * 8) / G;
    const float sv = s.scale_v[vi], mv = s.min_v[vi];
    uint32_t kw[4], vw[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c0 = 2 * j, c1 = 2 * j + 1;
      const float k0 = fmaf((float)((wk >> (c0 * bits)) & mask), sk[c0], mk[c0]);
      const float k1 = fmaf((float)((wk >> (c1 * bits)) & mask), sk[c1], mk[c1]);
      const float v0 = fmaf((float)((wv >> (c0 * bits)) & mask), sv, mv);
      const float v1 = fmaf((float)((wv >> (c1 * bits)) & mask), sv, mv);
      kw[j] = bf2(k0, k1);
      vw[j] = bf2(v0, v1);
    }
    ko = u4{kw[0], kw[1], kw[2], kw[3]};
    vo = u4{vw[0], vw[1], vw[2], vw[3]};
  }
  const int64_t oi = ((int64_t)bh * s.n_full + r) * D + c8 * 8;
  *reinterpret_cast<u4*>(kout + oi) = ko;
  *reinterpret_cast<u4*>(vout + oi) = vo;
  *reinterpret_cast<u4*>(vhout + oi) =
      u4{bf2_to_h2(vo[0]), bf2_to_h2(vo[1]), bf2_to_h2(vo[2]), bf2_to_h2(vo[3])};
  if (bf2_over_f16(vo[0]) || bf2_over_f16(vo[1]) || bf2_over_f16(vo[2]) || bf2_over_f16(vo[3]))
    atomicOr(v_unsafe, 1);
}

// V rows of a dense view: flag values that fp16 cannot hold
// fp16 copy of a view's bf16 V rows ([BH, n, D], round to nearest even) and
// the range check: a value with no fp16 counterpart sets the flag
__global__ void vconvert_kernel(const uint16_t* __restrict__ v, int64_t bh_stride, int n_rows,
                                uint16_t* __restrict__ vh, int* __restrict__ v_unsafe) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // 8 elements each
  if (e >= (int64_t)n_rows * (D / 8)) return;
  const u4 x = *reinterpret_cast<const u4*>(v + blockIdx.y * bh_stride + e * 8);
  *reinterpret_cast<u4*>(vh + (int64_t)blockIdx.y * n_rows * D + e * 8) =
      u4{bf2_to_h2(x[0]), bf2_to_h2(x[1]), bf2_to_h2(x[2]), bf2_to_h2(x[3])};
  if (bf2_over_f16(x[0]) || bf2_over_f16(x[1]) || bf2_over_f16(x[2]) || bf2_over_f16(x[3]))
    atomicOr(v_unsafe, 1);
}

__global__ void flag_clear_kernel(int* flag) { *flag = 0; }

}  // namespace

bool prefill_mfma_eligible(const uc_shape& sh, const KSegs& segs, int q_dt, int M) {
  if (sh.D != D || q_dt != UC_BF16) return false;
  if ((sh.Hq / sh.Hkv) * M <= 16) return false;  // the decode kernel's range
  for (int i = 0; i < segs.n; ++i)
    if (segs.s[i].dtype != UC_BF16) return false;
  return true;
}

// Workspace: a flag word (some V value outside fp16's range), then bf16 K
// and V plus fp16 V of every packed segment's whole row groups, and the fp16
// V copy of every dense view (dense segments, residual tails).
size_t prefill_mfma_workspace(const uc_shape& sh, const KSegs& segs) {
  const size_t BH = (size_t)sh.B * sh.Hkv;
  auto round = [](size_t x) { return (x + 255) & ~(size_t)255; };
  size_t bytes = 256;
  for (int i = 0; i < segs.n; ++i) {
    const KSeg& s = segs.s[i];
    if (s.kind == UC_SEG_PACKED) {
      bytes += round(BH * s.n_full * D * 2 * 3);
      bytes += round(BH * s.tail_len * D * 2);
    } else {
      bytes += round(BH * s.n_rows * D * 2);
    }
  }
  return bytes;
}

static_assert(sizeof(Views) <= kPrefillViewBytes, "prepared views do not fit their slot");

// Preparation of a call: the range flag, the dequantised rows of every
// packed segment and the fp16 V copies, all in ws; the views the attention
// kernel walks go to views_out (kPrefillViewBytes).  The result depends only
// on the segments' contents and ws, so calls over unchanged segments can
// reuse it (execution plans).
hipError_t launch_prefill_prepare(const uc_shape& sh, const KSegs& segs, void* ws, hipStream_t st,
                                  void* views_out) {
  const int BH = sh.B * sh.Hkv;
  Views vs{};
  int* v_unsafe = (int*)ws;
  char* wp = (char*)ws + 256;
  int tiles = 0;
  // the PV product runs in fp16 when every V value fits fp16 (checked here,
  // decided in the kernel); otherwise in bf16 hi + lo parts
  hipLaunchKernelGGL(flag_clear_kernel, dim3(1), dim3(1), 0, st, v_unsafe);
  for (int i = 0; i < segs.n; ++i) {
    const KSeg& s = segs.s[i];
    auto take = [&](size_t bytes) {
      char* p = wp;
      wp += (bytes + 255) & ~(size_t)255;
      return (uint16_t*)p;
    };
    if (s.kind == UC_SEG_DENSE) {
      vs.v[vs.n++] = View{(const uint16_t*)s.k, (const uint16_t*)s.v,
                          take((size_t)BH * s.n_rows * D * 2), (int64_t)s.row_stride * D, s.n_rows, i};
      continue;
    }
    if (s.n_full > 0) {
      uint16_t* kd = take((size_t)BH * s.n_full * D * 2 * 3);
      uint16_t* vd = kd + (size_t)BH * s.n_full * D;
      uint16_t* vh = vd + (size_t)BH * s.n_full * D;
      const int64_t n_thr = (int64_t)BH * s.n_full * (D / 8);
      hipLaunchKernelGGL(dequant_kernel, dim3((unsigned)((n_thr + 255) / 256)), dim3(256), 0, st,
                         s, BH, kd, vd, vh, v_unsafe);
      vs.v[vs.n++] = View{kd, vd, vh, (int64_t)s.n_full * D, s.n_full, i};
    }
    uint16_t* th = take((size_t)BH * s.tail_len * D * 2);
    if (s.tail_len > 0)
      vs.v[vs.n++] = View{(const uint16_t*)s.tail_k, (const uint16_t*)s.tail_v, th,
                          (int64_t)s.tail_stride * D, s.tail_len, i};
  }
  // drop empty views (their tiles would be empty); keep the order
  int n = 0;
  for (int i = 0; i < vs.n; ++i)
    if (vs.v[i].n > 0) vs.v[n++] = vs.v[i];
  vs.n = n;
  for (int i = 0; i < n; ++i) {
    tiles += (vs.v[i].n + TILE - 1) / TILE;
    if (segs.s[vs.v[i].seg].kind == UC_SEG_PACKED && vs.v[i].v != (const uint16_t*)segs.s[vs.v[i].seg].tail_v)
      continue;  // dequantised rows were converted and checked by the dequant kernel
    const int64_t per = (int64_t)vs.v[i].n * (D / 8);
    hipLaunchKernelGGL(vconvert_kernel, dim3((unsigned)((per + 255) / 256), BH), dim3(256), 0, st,
                       vs.v[i].v, vs.v[i].bh_stride, vs.v[i].n, (uint16_t*)vs.v[i].vh, v_unsafe);
  }
  vs.tiles = tiles;
  memcpy(views_out, &vs, sizeof vs);
  return hipGetLastError();
}

// The attention kernel over prepared views (launch_prefill_prepare on the
// same ws).
hipError_t launch_prefill_run(const uc_shape& sh, int n_segs, const void* views, const void* q,
                              int M, float sm_scale, float* o, float* lse, float* seg_lse,
                              void* ws, hipStream_t st) {
  Views vs;
  memcpy(&vs, views, sizeof vs);
  const int BH = sh.B * sh.Hkv;
  const int* v_unsafe = (const int*)ws;
  hipError_t e;
  const int nq = (sh.Hq / sh.Hkv) * M;
  // the 8-wave layout (one workgroup per CU) when its grid fills every round
  // or runs many rounds; otherwise the 4-wave one (two per CU), whose last
  // round leaves fewer CUs idle
  const int cus = device_cus();
  const int n8 = (nq + qrows<8, 2>() - 1) / qrows<8, 2>() * BH;
  const bool wide = n8 % cus == 0 || n8 >= 8 * cus;
  const int qr = wide ? qrows<8, 2>() : qrows<4, 2>();
  const int n_qblocks = (nq + qr - 1) / qr;
  const int n_work = n_qblocks * BH;
  const int grid = (n_work + 7) / 8 * 8;
  const float sl2 = sm_scale * kLog2e;
  const uint16_t* qp = (const uint16_t*)q;
  if ((e = kernel_timer_begin(st)) != hipSuccess) return e;
  if (wide)
    hipLaunchKernelGGL((prefill_mfma_kernel<8, 2, 2>), dim3(grid), dim3(8 * 64), 0, st, vs, qp,
                       sh.Hq, sh.Hkv, M, n_segs, n_qblocks, n_work, sl2, o, lse, seg_lse, v_unsafe);
  else
    hipLaunchKernelGGL((prefill_mfma_kernel<4, 1, 2>), dim3(grid), dim3(4 * 64), 0, st, vs, qp,
                       sh.Hq, sh.Hkv, M, n_segs, n_qblocks, n_work, sl2, o, lse, seg_lse, v_unsafe);
  e = hipGetLastError();
  return e == hipSuccess ? kernel_timer_end(st) : e;
}

hipError_t launch_prefill_mfma(const uc_shape& sh, const KSegs& segs, const void* q, int M,
                               float sm_scale, float* o, float* lse, float* seg_lse, void* ws,
                               hipStream_t st) {
  alignas(16) char views[kPrefillViewBytes];
  const hipError_t e = launch_prefill_prepare(sh, segs, ws, st, views);
  if (e != hipSuccess) return e;
  return launch_prefill_run(sh, segs.n, views, q, M, sm_scale, o, lse, seg_lse, ws, st);
}

}  // namespace uc
