// mfma_util.h -- building blocks shared by the matrix-core kernels (decode,
// prefill, scoring) for bf16 rows of head dim 128 on gfx950.
//
// v_mfma_f32_16x16x32_bf16 operand layouts (lane l, i16 = l % 16, g4 = l / 16):
//   A (16 x 32):  lane holds A[i16][g4*8 .. g4*8+7]
//   B (32 x 16):  lane holds B[g4*8 .. g4*8+7][i16]
//   C (16 x 16):  lane holds C[g4*4 .. g4*4+3][i16]
// Rows of a staged 32-row tile sit LROW bytes apart in LDS; the 32-byte
// padding puts row r at bank 8r (mod 64), so the eight rows a half-wave reads
// in one transposing load (ds_read_b64_tr_b16) fall in disjoint 8-bank groups.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace uc {
namespace mf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef short s4 __attribute__((ext_vector_type(4)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s4 lds_s4;

constexpr int D = 128;           // head dim of the matrix-core kernels
constexpr int TILE = 32;         // rows per tile
constexpr int ROWB = D * 2;      // bytes of one bf16 row
constexpr int LROW = ROWB + 32;  // bytes of one staged row in LDS (32 B padding)
constexpr int TILEB = TILE * LROW;

// byte offset of 16-byte chunk c of row r inside a staged tile
__device__ inline int toff(int r, int c) { return r * LROW + (c << 4); }

// two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32)
__device__ inline uint32_t bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{a, b}, bf16x2));
}

__device__ inline f4 mfma(const u4& a, const u4& b, const f4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

__device__ inline f4 mfma_f16(const u4& a, const u4& b, const f4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// two floats -> packed fp16 pair, round to nearest even (v_cvt_pk_f16_f32)
__device__ inline uint32_t h2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{a, b}, f16x2));
}

// packed bf16 pair -> packed fp16 pair (exact for magnitudes in fp16's
// normal range; callers check the range)
__device__ inline uint32_t bf2_to_h2(uint32_t w) {
  return h2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
}

// true if some bf16 of the packed word reaches 2^16 in magnitude (or is
// inf/NaN): such a value has no fp16 counterpart (fp16's largest is 65504 and
// the bf16 value below 2^16 is 65280)
__device__ inline bool bf2_over_f16(uint32_t w) {
  return (w & 0x7FFFu) >= 0x4780u || ((w >> 16) & 0x7FFFu) >= 0x4780u;
}

// two transposing 64-bit LDS reads -> one 8 x bf16 operand
__device__ inline u4 ds_tr(const char* p0, const char* p1) {
  s4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p0));
  s4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4*)(p1));
  return u4{(uint32_t)(uint16_t)a[0] | ((uint32_t)(uint16_t)a[1] << 16),
            (uint32_t)(uint16_t)a[2] | ((uint32_t)(uint16_t)a[3] << 16),
            (uint32_t)(uint16_t)b[0] | ((uint32_t)(uint16_t)b[1] << 16),
            (uint32_t)(uint16_t)b[2] | ((uint32_t)(uint16_t)b[3] << 16)};
}

// V^T operand of dim tile d from a staged tile: the A block rows are dims
// d*16 .. d*16+15, its k index runs over the tile's keys in the order the S^T
// C layout hands them to a lane (keys g4*4 + j, then 16 + g4*4 + j)
__device__ inline u4 vt_operand(const char* lv, int d, int i16, int g4) {
  const int rr = g4 * 4 + (i16 >> 2);
  const int cb = (i16 & 3) >> 1, hb8 = (i16 & 1) * 8;
  return ds_tr(lv + toff(rr, 2 * d + cb) + hb8, lv + toff(rr + 16, 2 * d + cb) + hb8);
}

// the same operands from a lane base computed once per tile (vt_base), so
// the dim tiles differ only in the reads' immediate offsets
__device__ inline const char* vt_base(const char* lv, int i16, int g4) {
  return lv + toff(g4 * 4 + (i16 >> 2), (i16 & 3) >> 1) + (i16 & 1) * 8;
}
__device__ inline u4 vt_operand_at(const char* vb, int d) {
  return ds_tr(vb + d * 32, vb + 16 * LROW + d * 32);
}

// probabilities as bf16 hi + lo parts (16 significant bits between them)
__device__ inline void split_p(const float (&e)[8], u4& phi, u4& plo) {
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    hi[j] = bf2(e[2 * j], e[2 * j + 1]);
    const float h0 = __uint_as_float(hi[j] << 16), h1 = __uint_as_float(hi[j] & 0xFFFF0000u);
    lo[j] = bf2(e[2 * j] - h0, e[2 * j + 1] - h1);
  }
  phi = u4{hi[0], hi[1], hi[2], hi[3]};
  plo = u4{lo[0], lo[1], lo[2], lo[3]};
}

// Raw buffer descriptor over `bytes` bytes from `base`: loads at or past the
// end return zeros, and each load needs one 32-bit offset register.
__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, bytes, 0x00020000);
}

// Cache policy of a load: 0 = default; kNT = non-temporal, for data read
// once per launch (the caches are not filled with it, which keeps a long
// stream from evicting lines that are reused)
constexpr int kNT = 2;

template <int AUX = 0>
__device__ inline u4 bload(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(u4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, AUX));
}

template <int AUX = 0>
__device__ inline uint32_t bload32(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, AUX);
}

// a value the compiler cannot see through (keeps byte-extract conversions)
__device__ inline uint32_t opaque(uint32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}

}  // namespace mf
}  // namespace uc
