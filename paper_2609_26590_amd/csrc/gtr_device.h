// Device-side helpers shared by the libgtr kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gtr.h"

namespace gtr {

typedef _Float16 h4 __attribute__((ext_vector_type(4)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef float f8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Directional scan order (Sec. 3.1 "Directional scanning").
// pi(s) = spatial index (row-major, i*W + j) of the token visited at step s.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int64_t scan_to_spatial(int64_t s, int32_t H, int32_t W, int dir) {
  const int64_t L = (int64_t)H * W;
  if (dir == GTR_SCAN_ROW_REV || dir == GTR_SCAN_COL_REV) s = L - 1 - s;
  if (dir == GTR_SCAN_COL || dir == GTR_SCAN_COL_REV) {
    const int64_t j = s / H;
    const int64_t i = s - j * H;
    return i * W + j;
  }
  return s;
}

// ---------------------------------------------------------------------------
// bf16 <-> f32 (bf16 is the upper half of an IEEE binary32).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_bits_to_f32(unsigned short b) {
  return __builtin_bit_cast(float, (uint32_t)b << 16);
}

__device__ __forceinline__ unsigned short f32_to_bf16_bits(float f) {
  // round to nearest even; a NaN stays a (quiet) NaN. Branch-free: a select,
  // not a divergent branch per element.
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  const uint32_t rne = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  const uint32_t nan = (u >> 16) | 0x40u;
  return (unsigned short)((u & 0x7fffffffu) > 0x7f800000u ? nan : rne);
}

// Load 8 consecutive elements starting at element offset `off` of a tensor of
// dtype `dt` and widen them to float. `off` must be a multiple of 8 elements
// (16-byte alignment for 16-bit types, 32 bytes for float).
__device__ __forceinline__ void load8(const void* base, int dt, int64_t off, float (&x)[8]) {
  if (dt == GTR_F32) {
    const f4* p = reinterpret_cast<const f4*>(static_cast<const float*>(base) + off);
    const f4 a = p[0], b = p[1];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = a[e];
      x[e + 4] = b[e];
    }
  } else if (dt == GTR_F16) {
    const h8 a = *reinterpret_cast<const h8*>(static_cast<const _Float16*>(base) + off);
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = (float)a[e];
  } else {
    const u16x8 a = *reinterpret_cast<const u16x8*>(static_cast<const unsigned short*>(base) + off);
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = bf16_bits_to_f32(a[e]);
  }
}

// Store n (4 or 8) floats converted to dtype `dt` at element offset `off`.
template <int N>
__device__ __forceinline__ void store_n(void* base, int dt, int64_t off, const float* x) {
  if (dt == GTR_F32) {
    f4* p = reinterpret_cast<f4*>(static_cast<float*>(base) + off);
#pragma unroll
    for (int v = 0; v < N / 4; ++v) p[v] = f4{x[4 * v], x[4 * v + 1], x[4 * v + 2], x[4 * v + 3]};
  } else if (dt == GTR_F16) {
    _Float16* p = static_cast<_Float16*>(base) + off;
    if constexpr (N == 8) {
      h8 h;
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = (_Float16)x[e];
      *reinterpret_cast<h8*>(p) = h;
    } else {
      h4 h;
#pragma unroll
      for (int e = 0; e < 4; ++e) h[e] = (_Float16)x[e];
      *reinterpret_cast<h4*>(p) = h;
    }
  } else {
    unsigned short* p = static_cast<unsigned short*>(base) + off;
    if constexpr (N == 8) {
      u16x8 h;
#pragma unroll
      for (int e = 0; e < 8; ++e) h[e] = f32_to_bf16_bits(x[e]);
      *reinterpret_cast<u16x8*>(p) = h;
    } else {
      typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));
      u16x4 h;
#pragma unroll
      for (int e = 0; e < 4; ++e) h[e] = f32_to_bf16_bits(x[e]);
      *reinterpret_cast<u16x4*>(p) = h;
    }
  }
}

// ---------------------------------------------------------------------------
// Matrix-core products on 16x16 output tiles, float32 accumulation.
//
// Operand layout (both operands of C[16x16] += A[16xK] * B[Kx16]): lane l holds
// row (A) / column (B) index l % 16 and the K-slots 8*(l/16) .. 8*(l/16)+7
// (K = 32) or 4*(l/16) .. 4*(l/16)+3 (K = 16). The accumulator lane l holds
// C[4*(l/16) + e][l % 16], e = 0..3. Which physical K index a K-slot stands for
// is up to the caller, as long as A and B agree.
// ---------------------------------------------------------------------------
__device__ __forceinline__ f4 mma32(const h8& a, const h8& b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// float32 variant: eight K=4 steps; in step e lane group l/16 supplies K-slot
// 8*(l/16)+e, so the slot assignment matches the f16 form above.
__device__ __forceinline__ f4 mma32(const f8& a, const f8& b, f4 c) {
#pragma unroll
  for (int e = 0; e < 8; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], c, 0, 0, 0);
  return c;
}

__device__ __forceinline__ f4 mma16(const h4& a, const h4& b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f4 mma16(const f4& a, const f4& b, f4 c) {
#pragma unroll
  for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], c, 0, 0, 0);
  return c;
}

template <bool F16>
struct Op;
template <>
struct Op<true> {
  typedef h8 frag8;
  typedef h4 frag4;
  typedef _Float16 elem;
  static __device__ __forceinline__ frag8 pack8(const float (&x)[8]) {
    frag8 r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = (_Float16)x[e];
    return r;
  }
  static __device__ __forceinline__ frag4 pack4(const f4& x) {
    return frag4{(_Float16)x[0], (_Float16)x[1], (_Float16)x[2], (_Float16)x[3]};
  }
};
template <>
struct Op<false> {
  typedef f8 frag8;
  typedef f4 frag4;
  typedef float elem;
  static __device__ __forceinline__ frag8 pack8(const float (&x)[8]) {
    frag8 r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = x[e];
    return r;
  }
  static __device__ __forceinline__ frag4 pack4(const f4& x) { return x; }
};

// ---------------------------------------------------------------------------
// Lane exchange inside a 16-lane row (DPP row operations).
// ---------------------------------------------------------------------------
template <int SHIFT>
__device__ __forceinline__ float row_shr(float x) {
  // lanes whose source is outside the row receive 0
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x),
                                                               0x110 + SHIFT, 0xf, 0xf, false));
}

// Inclusive prefix sum over the 16 lanes of each row.
__device__ __forceinline__ float row_inclusive_scan(float x) {
  x += row_shr<1>(x);
  x += row_shr<2>(x);
  x += row_shr<4>(x);
  x += row_shr<8>(x);
  return x;
}

// Value of lane N (0..15) of this lane's 16-lane row (DPP row_newbcast). Every
// lane receives a value, so the move needs no initialised destination.
template <int N>
__device__ __forceinline__ float row_bcast(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x150 + N, 0xf, 0xf, false));
}

// Maximum over the 64 lanes, as a wave-uniform value: a running maximum along
// each 16-lane row with DPP row shifts (a lane whose source is outside its row
// keeps its own value), then the four row maxima (lanes 15, 31, 47, 63) read
// into scalar registers. No LDS round trips.
template <int SHIFT>
__device__ __forceinline__ float row_shr_keep(float x) {
  const int b = __builtin_bit_cast(int, x);
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(b, b, 0x110 + SHIFT, 0xf, 0xf, false));
}
__device__ __forceinline__ float wave_max_uniform(float x) {
  x = fmaxf(x, row_shr_keep<1>(x));
  x = fmaxf(x, row_shr_keep<2>(x));
  x = fmaxf(x, row_shr_keep<4>(x));
  x = fmaxf(x, row_shr_keep<8>(x));
  const int b = __builtin_bit_cast(int, x);
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 15));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 31));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 47));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(b, 63));
  return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

}  // namespace gtr
