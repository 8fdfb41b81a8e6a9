// The small kernels of one GTR block (Sec. 3.1) around the GLA call and the
// Spatial SwiGLU: the layer normalisation before each of them, the head
// split of the projections and the head concat before W_o, and the residual
// add after the Spatial SwiGLU. All of them move 16-byte vectors of eight
// 16-bit elements; the arithmetic is float32.
#include <hip/hip_runtime.h>

#include "gtr.h"
#include "gtr_device.h"
#include "gtr_internal.h"

namespace gtr {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void unpack8(v4u raw, int dt, float (&x)[8]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const unsigned u = raw[e];
    if (dt == GTR_F16) {
      x[2 * e] = (float)__builtin_bit_cast(_Float16, (unsigned short)(u & 0xffffu));
      x[2 * e + 1] = (float)__builtin_bit_cast(_Float16, (unsigned short)(u >> 16));
    } else {
      x[2 * e] = __builtin_bit_cast(float, u << 16);
      x[2 * e + 1] = __builtin_bit_cast(float, u & 0xffff0000u);
    }
  }
}

// Sum over the 64 lanes as a wave-uniform value: a prefix sum along each
// 16-lane row with DPP row shifts, then the four row totals (lanes 15, 31, 47,
// 63) read into scalar registers. No LDS round trips.
__device__ __forceinline__ float wave_sum(float x) {
  const int s = __builtin_bit_cast(int, row_inclusive_scan(x));
  const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(s, 15));
  const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(s, 31));
  const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(s, 47));
  const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(s, 63));
  return (r0 + r1) + (r2 + r3);
}

// One wave per row of d channels (d / 8 vectors, at most 4 per lane). The
// affine weights are loaded with the row, so the two reductions (mean, then the
// centred sum of squares) are the only steps between the loads and the store.
constexpr int kLnMaxVec = 4;
__global__ void __launch_bounds__(256) layernorm_kernel(const v4u* __restrict__ x, const float* __restrict__ w,
                                                        const float* __restrict__ b, void* __restrict__ y, int64_t M,
                                                        int d, float eps, int dt) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= M) return;
  const int nv = d / 8;
  float v[kLnMaxVec][8], wv[kLnMaxVec][8], bv[kLnMaxVec][8];
  float s = 0.f;
#pragma unroll
  for (int q = 0; q < kLnMaxVec; ++q) {
    const int i = lane + 64 * q;
    if (i < nv) {
      unpack8(x[row * nv + i], dt, v[q]);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const f4 wq = w ? reinterpret_cast<const f4*>(w)[2 * i + h] : f4{1.f, 1.f, 1.f, 1.f};
        const f4 bq = b ? reinterpret_cast<const f4*>(b)[2 * i + h] : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          wv[q][4 * h + e] = wq[e];
          bv[q][4 * h + e] = bq[e];
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[q][e];
    }
  }
  const float mean = wave_sum(s) / (float)d;
  float ss = 0.f;
#pragma unroll
  for (int q = 0; q < kLnMaxVec; ++q)
    if (lane + 64 * q < nv)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float t = v[q][e] - mean;
        ss = fmaf(t, t, ss);
      }
  const float rs = rsqrtf(wave_sum(ss) / (float)d + eps);
#pragma unroll
  for (int q = 0; q < kLnMaxVec; ++q) {
    const int i = lane + 64 * q;
    if (i < nv) {
      float o8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o8[e] = (v[q][e] - mean) * rs * wv[q][e] + bv[q][e];
      store_n<8>(y, dt, (row * nv + i) * 8, o8);
    }
  }
}

// split: vector t of dst in [parts][B][H][L][dh / 8] order; merge: vector t of
// dst in [B][L][H][dh / 8] order. One 16-byte vector per thread.
__global__ void __launch_bounds__(256) heads_kernel(const v4u* __restrict__ src, v4u* __restrict__ dst,
                                                    int64_t total, int B, int H, int64_t L, int dv8, int64_t ld8,
                                                    int parts, int merge) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= total) return;
  const int64_t jv = t % dv8;
  int64_t r = t / dv8;
  if (merge) {
    const int64_t h = r % H;
    r /= H;
    const int64_t l = r % L, bb = r / L;  // dst row bb * L + l, column block h
    dst[t] = src[((bb * H + h) * L + l) * dv8 + jv];
  } else {
    const int64_t l = r % L;
    r /= L;
    const int64_t h = r % H;
    r /= H;
    const int64_t bb = r % B, p = r / B;
    dst[t] = src[(bb * L + l) * ld8 + (p * H + h) * dv8 + jv];
  }
}

__global__ void __launch_bounds__(256) add_kernel(const v4u* __restrict__ a, const v4u* __restrict__ b,
                                                  void* __restrict__ y, int64_t nv, int dt) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= nv) return;
  float xa[8], xb[8];
  unpack8(a[i], dt, xa);
  unpack8(b[i], dt, xb);
#pragma unroll
  for (int e = 0; e < 8; ++e) xa[e] += xb[e];
  store_n<8>(y, dt, i * 8, xa);
}

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
static bool overlaps(const void* p, size_t pb, const void* q, size_t qb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(p), y = reinterpret_cast<uintptr_t>(q);
  return x < y + qb && y < x + pb;
}
static unsigned blocks_for(int64_t n) { return (unsigned)((n + 255) / 256); }

}  // namespace gtr

using namespace gtr;

extern "C" gtr_status gtr_layernorm(const void* x, const float* w, const float* b, void* y, int64_t M, int32_t d,
                                    float eps, gtr_dtype dtype, hipStream_t stream) {
  if (M <= 0 || d <= 0) return GTR_ERR_SHAPE;
  if (d % 8 || d > 8 * 64 * kLnMaxVec || (dtype != GTR_F16 && dtype != GTR_BF16)) return GTR_ERR_UNSUPPORTED;
  if (M > ((int64_t)1 << 33)) return GTR_ERR_SHAPE;
  if (!x || !y) return GTR_ERR_NULL;
  if (!aligned16(x) || !aligned16(y) || (w && !aligned16(w)) || (b && !aligned16(b))) return GTR_ERR_UNSUPPORTED;
  const size_t bytes = (size_t)M * d * 2;
  if (x != y && overlaps(x, bytes, y, bytes)) return GTR_ERR_ALIAS;
  if ((w && overlaps(w, (size_t)d * 4, y, bytes)) || (b && overlaps(b, (size_t)d * 4, y, bytes))) return GTR_ERR_ALIAS;
  hipLaunchKernelGGL(layernorm_kernel, dim3((unsigned)((M + 3) / 4)), dim3(256), 0, stream,
                     static_cast<const v4u*>(x), w, b, y, M, (int)d, eps, (int)dtype);
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}

static gtr_status heads_launch(const void* src, void* dst, int32_t parts, int32_t B, int32_t H, int64_t L,
                               int32_t dh, int64_t ld, gtr_dtype dtype, int merge, hipStream_t stream) {
  if (parts <= 0 || B <= 0 || H <= 0 || L <= 0 || dh <= 0) return GTR_ERR_SHAPE;
  if (dh % 8 || ld % 8 || ld < (int64_t)parts * H * dh || (dtype != GTR_F16 && dtype != GTR_BF16))
    return GTR_ERR_UNSUPPORTED;
  int64_t n;
  if (__builtin_mul_overflow((int64_t)parts * B * H, L, &n) || __builtin_mul_overflow(n, (int64_t)dh, &n) ||
      n > ((int64_t)1 << 38) || (int64_t)B * L * ld > ((int64_t)1 << 38))
    return GTR_ERR_SHAPE;
  if (!src || !dst) return GTR_ERR_NULL;
  if (!aligned16(src) || !aligned16(dst)) return GTR_ERR_UNSUPPORTED;
  const size_t sb = merge ? (size_t)n * 2 : (size_t)B * L * ld * 2;
  if (overlaps(src, sb, dst, (size_t)n * 2)) return GTR_ERR_ALIAS;
  const int64_t total = n / 8;
  hipLaunchKernelGGL(heads_kernel, dim3(blocks_for(total)), dim3(256), 0, stream, static_cast<const v4u*>(src),
                     static_cast<v4u*>(dst), total, (int)B, (int)H, L, (int)(dh / 8), ld / 8, (int)parts, merge);
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}

extern "C" gtr_status gtr_heads_split(const void* src, void* dst, int32_t parts, int32_t B, int32_t H, int64_t L,
                                      int32_t dh, int64_t ld, gtr_dtype dtype, hipStream_t stream) {
  return heads_launch(src, dst, parts, B, H, L, dh, ld, dtype, 0, stream);
}

extern "C" gtr_status gtr_heads_merge(const void* src, void* dst, int32_t B, int32_t H, int64_t L, int32_t dh,
                                      gtr_dtype dtype, hipStream_t stream) {
  return heads_launch(src, dst, 1, B, H, L, dh, (int64_t)H * dh, dtype, 1, stream);
}

extern "C" gtr_status gtr_add(const void* a, const void* b, void* y, int64_t n, gtr_dtype dtype, hipStream_t stream) {
  if (n <= 0) return GTR_ERR_SHAPE;
  if (n % 8 || (dtype != GTR_F16 && dtype != GTR_BF16)) return GTR_ERR_UNSUPPORTED;
  if (n > ((int64_t)1 << 38)) return GTR_ERR_SHAPE;
  if (!a || !b || !y) return GTR_ERR_NULL;
  if (!aligned16(a) || !aligned16(b) || !aligned16(y)) return GTR_ERR_UNSUPPORTED;
  const size_t bytes = (size_t)n * 2;
  if ((y != a && overlaps(y, bytes, a, bytes)) || (y != b && overlaps(y, bytes, b, bytes))) return GTR_ERR_ALIAS;
  hipLaunchKernelGGL(add_kernel, dim3(blocks_for(n / 8)), dim3(256), 0, stream, static_cast<const v4u*>(a),
                     static_cast<const v4u*>(b), y, n / 8, (int)dtype);
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}
