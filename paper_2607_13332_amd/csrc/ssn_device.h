// Device-side helpers shared by the codec kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ssn {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

// Round-to-nearest-even float -> bf16 (hardware v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f);
}

// Two floats -> one dword of packed bf16 (lo in bits 0..15), each rounded to
// nearest even: one two-source v_cvt_pk_bf16_f32 (the scalar form above
// costs two conversions plus a shift and an or per pair).
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Low / high bf16 of a packed dword, widened to float.
__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// 16x16x32 bf16 MFMA, fp32 accumulate.  Operand layout (64 lanes):
//   A (16 x 32): lane l holds row l%16, K elements 8*(l/16) .. 8*(l/16)+7
//   B (32 x 16): lane l holds column l%16, the same K elements
//   C (16 x 16): lane l holds rows 4*(l/16) .. +3 of column l%16
// Only the pairing of K elements between A and B matters for the result, so
// the kernels are free to choose which physical index each K slot carries.
__device__ __forceinline__ f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// 16x16x4 float32 MFMA.  A (16 x 4): lane l holds row l%16, K element l/16;
// B (4 x 16): lane l holds column l%16, K element l/16; C (16 x 16): lane l
// holds rows 4 (l/16) .. +3 of column l%16.  Only the pairing of K elements
// between A and B matters, so each kernel picks the index a K slot carries.
__device__ __forceinline__ f32x4 mfma16x16x4f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Split 8 floats into bf16 hi + lo parts with x ~= hi + lo to ~2^-17 relative:
// two MFMAs on (hi, lo) carry a float32 operand at close to fp32 accuracy.
__device__ __forceinline__ void split_bf16x8(const float* v, u32x4& hi, u32x4& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    uint32_t h0 = f32_to_bf16(v[2 * m]), h1 = f32_to_bf16(v[2 * m + 1]);
    float r0 = v[2 * m] - __uint_as_float(h0 << 16);
    float r1 = v[2 * m + 1] - __uint_as_float(h1 << 16);
    h[m] = h0 | (h1 << 16);
    l[m] = pack_bf16x2(r0, r1);
  }
  hi = u32x4{h[0], h[1], h[2], h[3]};
  lo = u32x4{l[0], l[1], l[2], l[3]};
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, kWave);
  return v;
}

template <typename T>
__device__ __forceinline__ float load_as_f32(const T* p);
template <>
__device__ __forceinline__ float load_as_f32<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load_as_f32<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }

template <typename T>
__device__ __forceinline__ void store_from_f32(T* p, float v);
template <>
__device__ __forceinline__ void store_from_f32<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_from_f32<uint16_t>(uint16_t* p, float v) { *p = (uint16_t)f32_to_bf16(v); }

// Loads the 8 x KP bf16 block M[row0 .. row0+7][col0 .. col0+KP-1] of a
// row-major matrix with `ld` columns into packed dwords (two columns per
// dword).  FULL: the block never crosses column `ncols` and rows are aligned
// for vector loads (ld == 16*KP-style layouts); otherwise each element is
// loaded under a bounds predicate and missing columns read as zero.
template <int KP, bool FULL>
__device__ __forceinline__ void load_block8(const uint16_t* __restrict__ M, int64_t row0, int col0,
                                            int ld, int ncols, uint32_t (&w)[8][(KP + 1) / 2]) {
  constexpr int KW = (KP + 1) / 2;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const uint16_t* p = M + (row0 + r) * (int64_t)ld + col0;
    if constexpr (FULL && KP == 8) {
      const u32x4 v = *(const u32x4*)p;
      w[r][0] = v[0]; w[r][1] = v[1]; w[r][2] = v[2]; w[r][3] = v[3];
    } else if constexpr (FULL && KP == 4) {
      const u32x2 v = *(const u32x2*)p;
      w[r][0] = v[0]; w[r][1] = v[1];
    } else if constexpr (FULL && (KP % 2) == 0) {
#pragma unroll
      for (int q = 0; q < KW; ++q) w[r][q] = ((const uint32_t*)p)[q];
    } else {
#pragma unroll
      for (int q = 0; q < KW; ++q) {
        const uint32_t lo = (col0 + 2 * q < ncols) ? (uint32_t)p[2 * q] : 0u;
        const uint32_t hi = (2 * q + 1 < KP && col0 + 2 * q + 1 < ncols) ? (uint32_t)p[2 * q + 1] : 0u;
        w[r][q] = lo | (hi << 16);
      }
    }
  }
}

// Column i of a block loaded by load_block8, as one MFMA operand fragment:
// 8 consecutive rows of that column, two bf16 per dword.
template <int KP>
__device__ __forceinline__ u32x4 block8_column(const uint32_t (&w)[8][(KP + 1) / 2], int i) {
  uint32_t f[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const uint32_t a = w[2 * m][i >> 1], b = w[2 * m + 1][i >> 1];
    f[m] = (i & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
  }
  return u32x4{f[0], f[1], f[2], f[3]};
}

// 16-byte global load / store; NT marks streaming data (non-temporal hint) so
// that it does not displace data the kernel re-reads from L2.
template <bool NT>
__device__ __forceinline__ u32x4 ldg(const uint16_t* p) {
  if constexpr (NT) return __builtin_nontemporal_load((const u32x4*)p);
  else return *(const u32x4*)p;
}
template <bool NT>
__device__ __forceinline__ void stg(uint16_t* p, u32x4 v) {
  if constexpr (NT) __builtin_nontemporal_store(v, (u32x4*)p);
  else *(u32x4*)p = v;
}

// LDS transpose read of 4 bf16 per lane (ds_read_b64_tr_b16, gfx950).  Within
// each group of 16 lanes, lane i receives element (i mod 4) of the 8-byte
// words addressed by lanes 4j + i/4, j = 0..3.  So when lane L of a group
// points at row r0 + L/4, columns c0 + 4 (L mod 4) .. +3 of a row-major bf16
// tile in LDS, lane i receives rows r0 .. r0+3 of column c0 + i: the
// row-contiguous tile yields column-contiguous MFMA fragments.
typedef short i16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x2 lds_read_tr16(const uint16_t* p) {
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4*)p);
  return __builtin_bit_cast(u32x2, v);
}

// Rows of k bf16 with k % 8 != 0 start only 2-byte aligned.  Eight
// consecutive elements M[e0 .. e0 + 8) are read as the 4-byte aligned window
// of ten elements that starts at e0 rounded down to even (one 16-byte and one
// 4-byte load), and realigned in registers once the loads have landed, so
// that the loads can run ahead of their use.  Within the last ten elements of
// the buffer (`total` elements) the window is read element by element and
// nothing past the end is touched.
typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));
struct Bf16Window {
  u32x4 v;      // elements a0 .. a0 + 7
  uint32_t x;   // elements a0 + 8, a0 + 9
};
__device__ __forceinline__ Bf16Window load_bf16_window(const uint16_t* __restrict__ M, int64_t e0,
                                                       int64_t total) {
  const int64_t a0 = e0 & ~(int64_t)1;
  Bf16Window w;
  if (a0 + 10 <= total) {
    const uint32_t* p = (const uint32_t*)(M + a0);
    w.v = *(const u32x4_a4*)p;
    w.x = p[4];
  } else {
    uint32_t r[5];
#pragma unroll
    for (int i = 0; i < 5; ++i) {
      const uint32_t lo = (a0 + 2 * i < total) ? (uint32_t)M[a0 + 2 * i] : 0u;
      const uint32_t hi = (a0 + 2 * i + 1 < total) ? (uint32_t)M[a0 + 2 * i + 1] : 0u;
      r[i] = lo | (hi << 16);
    }
    w.v = u32x4{r[0], r[1], r[2], r[3]};
    w.x = r[4];
  }
  return w;
}
// The eight elements starting at e0 (odd: e0 is odd) out of a window loaded
// by load_bf16_window; elements at positions >= nv (past the end of a matrix
// row) become zero.
__device__ __forceinline__ u32x4 realign_bf16_window(const Bf16Window& w, bool odd, int nv) {
  const uint32_t sh = odd ? 16u : 0u;
  uint32_t r[4] = {__builtin_amdgcn_alignbit(w.v[1], w.v[0], sh),
                   __builtin_amdgcn_alignbit(w.v[2], w.v[1], sh),
                   __builtin_amdgcn_alignbit(w.v[3], w.v[2], sh),
                   __builtin_amdgcn_alignbit(w.x, w.v[3], sh)};
#pragma unroll
  for (int i = 0; i < 4; ++i)
    r[i] = (2 * i + 1 < nv) ? r[i] : ((2 * i < nv) ? (r[i] & 0xFFFFu) : 0u);
  return u32x4{r[0], r[1], r[2], r[3]};
}

// The 16-byte window M[a0 .. a0 + 8), a0 = e0 rounded down to even, of a
// buffer of `total` elements (elements past the end read as zero).
__device__ __forceinline__ u32x4 load_bf16x8_even(const uint16_t* __restrict__ M, int64_t e0,
                                                  int64_t total) {
  const int64_t a0 = e0 & ~(int64_t)1;
  if (a0 + 8 <= total) return *(const u32x4_a4*)(M + a0);
  uint32_t r[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t lo = (a0 + 2 * i < total) ? (uint32_t)M[a0 + 2 * i] : 0u;
    const uint32_t hi = (a0 + 2 * i + 1 < total) ? (uint32_t)M[a0 + 2 * i + 1] : 0u;
    r[i] = lo | (hi << 16);
  }
  return u32x4{r[0], r[1], r[2], r[3]};
}
// Elements e0 .. e0 + 8 out of that window and the dword that follows it
// (`next`: elements a0 + 8, a0 + 9), zero at positions >= nv.
__device__ __forceinline__ u32x4 realign_bf16x8(u32x4 v, uint32_t next, bool odd, int nv) {
  return realign_bf16_window(Bf16Window{v, next}, odd, nv);
}

__device__ __forceinline__ int64_t clamp_id(int32_t id, int64_t V) {
  int64_t i = id;
  return i < 0 ? 0 : (i >= V ? V - 1 : i);
}

}  // namespace ssn
