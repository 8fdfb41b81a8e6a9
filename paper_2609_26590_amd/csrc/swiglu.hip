// Spatial SwiGLU for gfx950 (MI355X): paper Sec. 3.1, "Spatial SwiGLU",
//   Y = [SiLU(X W_g) * DWConv3x3(X W_v)] W_o,
// X the patch tokens of one image in row-major grid order, the value branch
// convolved depthwise over the H x W grid (zero padding), the gate tokenwise.
//
// Three launches:
//   1. gemm_nt_kernel (z = 0, 1): G = X W_g^T and V = X W_v^T, float32 out,
//      MFMA on the input dtype's operands (fp16 or bf16), float32 accumulation;
//   2. conv_gate_kernel: H = SiLU(G) * (DWConv3x3(V) + bias), rounded to fp16,
//      the operand type of the next product;
//   3. gemm_nt_kernel: Y = H W_o^T (fp16 operands; bf16 weights are widened).
// Weights use the layout of a linear layer (output features first), so both
// operands of every product are read along K in 16-byte pieces.
#include <hip/hip_runtime.h>

#include "gtr.h"
#include "gtr_device.h"
#include "gtr_internal.h"

namespace gtr {

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef unsigned int w4 __attribute__((ext_vector_type(4)));

// 8 consecutive K elements of one row as an MFMA operand. DT is the dtype of
// the matrix in memory, MT the operand type (GTR_F16 or GTR_BF16).
template <int DT, int MT>
struct Operand;
template <>
struct Operand<GTR_F16, GTR_F16> {
  typedef h8 T;
  static __device__ __forceinline__ T get(w4 raw) { return __builtin_bit_cast(T, raw); }
};
template <>
struct Operand<GTR_BF16, GTR_BF16> {
  typedef bf8 T;
  static __device__ __forceinline__ T get(w4 raw) { return __builtin_bit_cast(T, raw); }
};
template <>
struct Operand<GTR_BF16, GTR_F16> {  // bf16 weights against fp16 activations
  typedef h8 T;
  static __device__ __forceinline__ T get(w4 raw) {
    T r;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const unsigned int u = raw[e];
      r[2 * e] = (_Float16)__builtin_bit_cast(float, u << 16);
      r[2 * e + 1] = (_Float16)__builtin_bit_cast(float, u & 0xffff0000u);
    }
    return r;
  }
};

__device__ __forceinline__ f4 mfma(const h8& a, const h8& b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f4 mfma(const bf8& a, const bf8& b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// C[M][N] = A[M][K] * B[N][K]^T, row-major, K a multiple of 32, N a multiple
// of 64. Work-group tile 64 x 64 (4 waves of 32 x 32, 2 x 2 MFMA tiles each);
// rows past M are read from row M-1 and not stored. blockIdx.z selects one of
// two (B, C) pairs, so G and V come out of one launch.
struct GemmArgs {
  const void* A;
  const void* B[2];
  void* C[2];
  int M, N, K;
  int cdt;  // dtype of C (GTR_F32 / GTR_F16 / GTR_BF16)
};

template <int ADT, int BDT, int MT>
__global__ void __launch_bounds__(256) gemm_nt_kernel(GemmArgs g) {
  typedef Operand<ADT, MT> OA;
  typedef Operand<BDT, MT> OB;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, kq = lane >> 4;
  const int m0 = blockIdx.x * 64 + 32 * (w >> 1), n0 = blockIdx.y * 64 + 32 * (w & 1);
  const unsigned short* A = static_cast<const unsigned short*>(g.A);
  const unsigned short* B = static_cast<const unsigned short*>(g.B[blockIdx.z]);
  const int64_t K = g.K;
  const int64_t ra0 = min(m0 + r16, g.M - 1), ra1 = min(m0 + 16 + r16, g.M - 1);
  const int64_t rb0 = n0 + r16, rb1 = n0 + 16 + r16;
  const w4* pa0 = reinterpret_cast<const w4*>(A + ra0 * K + 8 * kq);
  const w4* pa1 = reinterpret_cast<const w4*>(A + ra1 * K + 8 * kq);
  const w4* pb0 = reinterpret_cast<const w4*>(B + rb0 * K + 8 * kq);
  const w4* pb1 = reinterpret_cast<const w4*>(B + rb1 * K + 8 * kq);
  f4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
  // one K-step of 32 elements is 4 pieces of 16 bytes per row
  w4 a0 = pa0[0], a1 = pa1[0], b0 = pb0[0], b1 = pb1[0];
  for (int64_t k = 32; k <= K; k += 32) {
    // prefetch the next step while this one multiplies (the last prefetch
    // re-reads the final step and is not used)
    const int64_t kn = (k < K ? k : k - 32) / 8;
    const w4 na0 = pa0[kn], na1 = pa1[kn], nb0 = pb0[kn], nb1 = pb1[kn];
    const typename OA::T fa0 = OA::get(a0), fa1 = OA::get(a1);
    const typename OB::T fb0 = OB::get(b0), fb1 = OB::get(b1);
    acc[0][0] = mfma(fa0, fb0, acc[0][0]);
    acc[0][1] = mfma(fa0, fb1, acc[0][1]);
    acc[1][0] = mfma(fa1, fb0, acc[1][0]);
    acc[1][1] = mfma(fa1, fb1, acc[1][1]);
    a0 = na0;
    a1 = na1;
    b0 = nb0;
    b1 = nb1;
  }
  // lane holds C[row 16i + 4kq + e][column 16j + r16] of this wave's 32 x 32
  void* C = g.C[blockIdx.z];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = m0 + 16 * i + 4 * kq + e;
      if (m >= g.M) continue;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int64_t off = (int64_t)m * g.N + n0 + 16 * j + r16;
        const float x = acc[i][j][e];
        if (g.cdt == GTR_F32)
          static_cast<float*>(C)[off] = x;
        else if (g.cdt == GTR_F16)
          static_cast<_Float16*>(C)[off] = (_Float16)x;
        else
          static_cast<unsigned short*>(C)[off] = f32_to_bf16_bits(x);
      }
    }
}

// H[b][t][c] = SiLU(G[b][t][c]) * (sum_{u,v} V[b][t + (u-1, v-1)][c] * cw[c][u][v] + cb[c]),
// one thread per token and 8 channels; neighbours outside the grid are zero.
__global__ void __launch_bounds__(256) conv_gate_kernel(const float* G, const float* V, const float* cw,
                                                        const float* cb, _Float16* Hout, int B, int Hh, int W,
                                                        int hidden) {
  const int groups = hidden / 8;
  const int64_t n = (int64_t)B * Hh * W * groups;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;  // launched with 256 threads
  if (idx >= n) return;
  const int cg = (int)(idx % groups);
  const int64_t tok = idx / groups;  // b * L + t
  const int64_t L = (int64_t)Hh * W;
  const int64_t b = tok / L, t = tok - b * L;
  const int i = (int)(t / W), j = (int)(t - (int64_t)(t / W) * W);
  const int c = 8 * cg;
  float acc[8];
  if (cb) {
    const f4 lo = *reinterpret_cast<const f4*>(cb + c), hi = *reinterpret_cast<const f4*>(cb + c + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[e] = lo[e];
      acc[e + 4] = hi[e];
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  }
  // the 72 weights of channels c .. c+7 are contiguous ([hidden][3][3])
  float wt[72];
#pragma unroll
  for (int q = 0; q < 18; ++q) {
    const f4 x = *reinterpret_cast<const f4*>(cw + (int64_t)c * 9 + 4 * q);
#pragma unroll
    for (int e = 0; e < 4; ++e) wt[4 * q + e] = x[e];
  }
#pragma unroll
  for (int u = 0; u < 3; ++u) {
    const int ii = i + u - 1;
#pragma unroll
    for (int v = 0; v < 3; ++v) {
      const int jj = j + v - 1;
      if (ii < 0 || ii >= Hh || jj < 0 || jj >= W) continue;
      const float* p = V + ((b * L + (int64_t)ii * W + jj) * hidden + c);
      const f4 lo = *reinterpret_cast<const f4*>(p), hi = *reinterpret_cast<const f4*>(p + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[e] = fmaf(lo[e], wt[9 * e + 3 * u + v], acc[e]);
        acc[e + 4] = fmaf(hi[e], wt[9 * (e + 4) + 3 * u + v], acc[e + 4]);
      }
    }
  }
  const float* pg = G + tok * hidden + c;
  const f4 glo = *reinterpret_cast<const f4*>(pg), ghi = *reinterpret_cast<const f4*>(pg + 4);
  h8 out;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float z = e < 4 ? glo[e] : ghi[e - 4];
    out[e] = (_Float16)(z * __builtin_amdgcn_rcpf(1.f + __expf(-z)) * acc[e]);
  }
  *reinterpret_cast<h8*>(Hout + tok * hidden + c) = out;
}

struct SwigluLayout {
  size_t g_off, v_off, h_off, total;
};

static SwigluLayout swiglu_layout(int64_t M, int64_t hidden) {
  auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  SwigluLayout l;
  l.g_off = 0;
  l.v_off = a256((size_t)M * hidden * 4);
  l.h_off = a256(l.v_off + (size_t)M * hidden * 4);
  l.total = a256(l.h_off + (size_t)M * hidden * 2);
  return l;
}

// All checks but the workspace size and the pointers when !check_pointers.
static gtr_status swiglu_check(const gtr_swiglu_args* a, int64_t* M_out, bool check_pointers) {
  if (a->B <= 0 || a->H <= 0 || a->W <= 0 || a->d <= 0 || a->hidden <= 0) return GTR_ERR_SHAPE;
  if (a->d % 64 || a->hidden % 64) return GTR_ERR_UNSUPPORTED;
  if (a->dtype != GTR_F16 && a->dtype != GTR_BF16) return GTR_ERR_UNSUPPORTED;
  if (a->y_dtype != a->dtype && a->y_dtype != GTR_F32) return GTR_ERR_UNSUPPORTED;
  int64_t L, M, n;
  if (__builtin_mul_overflow((int64_t)a->H, (int64_t)a->W, &L) || __builtin_mul_overflow(L, (int64_t)a->B, &M))
    return GTR_ERR_SHAPE;
  if (M > 0x7fffffff - 64 || __builtin_mul_overflow(M, (int64_t)a->hidden, &n) || n > ((int64_t)1 << 40))
    return GTR_ERR_SHAPE;
  *M_out = M;
  if (!check_pointers) return GTR_OK;
  if (!a->x || !a->w_gate || !a->w_value || !a->w_out || !a->conv_w || !a->y) return GTR_ERR_NULL;
  const uintptr_t mis = reinterpret_cast<uintptr_t>(a->x) | reinterpret_cast<uintptr_t>(a->w_gate) |
                        reinterpret_cast<uintptr_t>(a->w_value) | reinterpret_cast<uintptr_t>(a->w_out) |
                        reinterpret_cast<uintptr_t>(a->conv_w) | reinterpret_cast<uintptr_t>(a->conv_b) |
                        reinterpret_cast<uintptr_t>(a->y);
  if (mis & 15u) return GTR_ERR_UNSUPPORTED;
  const SwigluLayout lay = swiglu_layout(M, a->hidden);
  if (!a->workspace || (reinterpret_cast<uintptr_t>(a->workspace) & 255u)) return GTR_ERR_WORKSPACE;
  if (a->workspace_bytes < lay.total) return GTR_ERR_WORKSPACE;
  const size_t es = dtype_size(a->dtype);
  struct R {
    uintptr_t lo, hi;
  };
  auto rng = [](const void* p, size_t bytes) {
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return R{lo, lo + bytes};
  };
  auto ovl = [](R x, R y) { return x.lo < y.hi && y.lo < x.hi; };
  const R ry = rng(a->y, (size_t)M * a->d * dtype_size(a->y_dtype));
  const R rw = rng(a->workspace, lay.total);
  const R ins[] = {rng(a->x, (size_t)M * a->d * es), rng(a->w_gate, (size_t)a->hidden * a->d * es),
                   rng(a->w_value, (size_t)a->hidden * a->d * es), rng(a->w_out, (size_t)a->d * a->hidden * es),
                   rng(a->conv_w, (size_t)a->hidden * 9 * 4),
                   a->conv_b ? rng(a->conv_b, (size_t)a->hidden * 4) : R{0, 0}};
  for (const R& r : ins)
    if (ovl(ry, r) || ovl(rw, r)) return GTR_ERR_ALIAS;
  if (ovl(ry, rw)) return GTR_ERR_ALIAS;
  return GTR_OK;
}

}  // namespace gtr

using namespace gtr;

extern "C" size_t gtr_spatial_swiglu_workspace_size(const gtr_swiglu_args* a) {
  int64_t M;
  if (!a || swiglu_check(a, &M, false) != GTR_OK) return 0;
  return swiglu_layout(M, a->hidden).total;
}

extern "C" gtr_status gtr_spatial_swiglu(const gtr_swiglu_args* a, hipStream_t stream) {
  if (!a) return GTR_ERR_NULL;
  int64_t M;
  gtr_status st = swiglu_check(a, &M, true);
  if (st != GTR_OK) return st;
  const SwigluLayout lay = swiglu_layout(M, a->hidden);
  char* ws = static_cast<char*>(a->workspace);
  float* G = reinterpret_cast<float*>(ws + lay.g_off);
  float* V = reinterpret_cast<float*>(ws + lay.v_off);
  _Float16* Hb = reinterpret_cast<_Float16*>(ws + lay.h_off);
  const bool bf = a->dtype == GTR_BF16;

  GemmArgs g1{a->x, {a->w_gate, a->w_value}, {G, V}, (int)M, a->hidden, a->d, GTR_F32};
  const dim3 grid1((unsigned)((M + 63) / 64), (unsigned)(a->hidden / 64), 2);
  if (bf)
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_BF16, GTR_BF16, GTR_BF16>), grid1, dim3(256), 0, stream, g1);
  else
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_F16, GTR_F16, GTR_F16>), grid1, dim3(256), 0, stream, g1);
  if (hipGetLastError() != hipSuccess) return GTR_ERR_HIP;

  const int64_t threads = M * (a->hidden / 8);
  hipLaunchKernelGGL(conv_gate_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream, G, V,
                     a->conv_w, a->conv_b, Hb, a->B, a->H, a->W, a->hidden);
  if (hipGetLastError() != hipSuccess) return GTR_ERR_HIP;

  GemmArgs g3{Hb, {a->w_out, a->w_out}, {a->y, a->y}, (int)M, a->d, a->hidden, a->y_dtype};
  const dim3 grid3((unsigned)((M + 63) / 64), (unsigned)(a->d / 64), 1);
  if (bf)
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_F16, GTR_BF16, GTR_F16>), grid3, dim3(256), 0, stream, g3);
  else
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_F16, GTR_F16, GTR_F16>), grid3, dim3(256), 0, stream, g3);
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}
