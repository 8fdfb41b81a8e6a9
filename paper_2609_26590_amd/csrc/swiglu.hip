// Spatial SwiGLU for gfx950 (MI355X): paper Sec. 3.1, "Spatial SwiGLU",
//   Y = [SiLU(X W_g) * DWConv3x3(X W_v)] W_o,
// X the patch tokens of one image in row-major grid order, the value branch
// convolved depthwise over the H x W grid (zero padding), the gate tokenwise.
//
// Three launches (four when the output product splits K):
//   1. gemm_nt_kernel (z = 0, 1): G = X W_g^T and V = X W_v^T, MFMA on the
//      input dtype's operands (fp16 or bf16), float32 accumulation, stored as
//      fp16 (the type H is rounded to anyway);
//   2. conv_gate_kernel: H = SiLU(G) * (DWConv3x3(V) + bias), rounded to fp16,
//      the operand type of the next product;
//   3. gemm_nt_kernel: Y = H W_o^T (fp16 operands; bf16 weights are widened),
//      float32 partial products per K slice summed by ksplit_reduce_kernel.
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
// of BN. Work-group tile BM x BN, 4 waves in a 2 x 2 grid, each wave a
// (BM/2) x (BN/2) block of 16 x 16 MFMA tiles. Every K-step of 32 stages the
// A and B tiles in LDS once (each element is read from memory by one thread
// and from LDS by every wave that needs it); the loads of the next step are in
// flight while the current one multiplies (two LDS buffers). Rows past M are
// read from row M-1 and not stored. blockIdx.z selects one of two (B, C) pairs
// (G and V come out of one launch) or, with ksplit > 1, a slice of K whose
// partial product goes to C[1] + slice * M * N (float32) for a reduction.
struct GemmArgs {
  const void* A;
  const void* B[2];
  void* C[2];
  int M, N, K;
  int cdt;     // dtype of C (GTR_F32 / GTR_F16 / GTR_BF16)
  int ksplit;  // number of K slices (1: none)
};

constexpr int KB = 4;     // minimum K-steps per slice when splitting K
// LDS tiles: rows of 32 K elements (64 bytes, no padding); the 16-byte piece
// c of row r sits at piece c ^ kSwz(r). Measured on gfx950, ds_read_b128 serves
// 32 lanes per cycle from 32 distinct 16-byte slots (address / 16 mod 32) and
// ds_write_b128 16 lanes from 16 slots (mod 16): with this swizzle the operand
// reads (lanes = 16 rows x 2 pieces) and the staging writes (lanes = 4 rows x
// 4 pieces) both hit distinct slots.
constexpr int kPitch = 32;
__device__ __forceinline__ int kSwz(int r) { return (r >> 2) & 2; }

template <int ADT, int BDT, int MT, int BM, int BN>
__global__ void __launch_bounds__(256) gemm_nt_kernel(GemmArgs g) {
  typedef Operand<ADT, MT> OA;
  typedef Operand<BDT, MT> OB;
  constexpr int TI = BM / 32, TJ = BN / 32;   // MFMA tiles per wave
  constexpr int PA = BM * 4 / 256, PB = BN * 4 / 256;  // 16-byte pieces per thread per step
  __shared__ __attribute__((aligned(16))) unsigned short As[2][BM * kPitch];
  __shared__ __attribute__((aligned(16))) unsigned short Bs[2][BN * kPitch];

  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, kq = lane >> 4;
  const int mb = blockIdx.x * BM, nb = blockIdx.y * BN;
  const int wm = (w >> 1) * (BM / 2), wn = (w & 1) * (BN / 2);
  const int pair = g.ksplit > 1 ? 0 : blockIdx.z;
  const unsigned short* A = static_cast<const unsigned short*>(g.A);
  const unsigned short* B = static_cast<const unsigned short*>(g.B[pair]);
  const int64_t K = g.K;
  const int steps = g.K / 32;
  const int s_per = (steps + g.ksplit - 1) / g.ksplit;
  const int s0 = g.ksplit > 1 ? blockIdx.z * s_per : 0;
  const int s1 = min(s0 + s_per, steps);

  // global pieces of this thread: piece p -> row p / 4, 16-byte column p % 4
  const w4* ga[PA];
  const w4* gb[PB];
  int la[PA], lb[PB];
#pragma unroll
  for (int q = 0; q < PA; ++q) {
    const int p = threadIdx.x + 256 * q, row = p >> 2, col = p & 3;
    ga[q] = reinterpret_cast<const w4*>(A + (int64_t)min(mb + row, g.M - 1) * K + 8 * col);
    la[q] = row * kPitch + 8 * (col ^ kSwz(row));
  }
#pragma unroll
  for (int q = 0; q < PB; ++q) {
    const int p = threadIdx.x + 256 * q, row = p >> 2, col = p & 3;
    gb[q] = reinterpret_cast<const w4*>(B + (int64_t)(nb + row) * K + 8 * col);
    lb[q] = row * kPitch + 8 * (col ^ kSwz(row));
  }
  f4 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  // D K-steps of global loads in flight: a ring of register slots, each staged
  // to LDS the step before it is multiplied (the loop is unrolled by D so
  // every slot index is a compile-time constant)
  constexpr int D = 4;
  w4 ra[D][PA], rb[D][PB];
  auto fetch = [&](int st, w4 (&a)[PA], w4 (&b)[PB]) {
#pragma unroll
    for (int q = 0; q < PA; ++q) a[q] = ga[q][4 * st];
#pragma unroll
    for (int q = 0; q < PB; ++q) b[q] = gb[q][4 * st];
  };
  auto stage = [&](int buf, const w4 (&a)[PA], const w4 (&b)[PB]) {
#pragma unroll
    for (int q = 0; q < PA; ++q) *reinterpret_cast<w4*>(&As[buf][la[q]]) = a[q];
#pragma unroll
    for (int q = 0; q < PB; ++q) *reinterpret_cast<w4*>(&Bs[buf][lb[q]]) = b[q];
  };
#pragma unroll
  for (int q = 0; q < D; ++q)
    if (s0 + q < s1) fetch(s0 + q, ra[q], rb[q]);
  if (s0 < s1) stage(0, ra[0], rb[0]);
  __syncthreads();
  for (int sb = s0; sb < s1; sb += D) {
#pragma unroll
    for (int q = 0; q < D; ++q) {
      const int st = sb + q;
      if (st < s1) {
        const int buf = (st - s0) & 1;
        if (st + D < s1) fetch(st + D, ra[q], rb[q]);  // slot q was staged before this step
        typename OA::T fa[TI];
        typename OB::T fb[TJ];
#pragma unroll
        for (int i = 0; i < TI; ++i)
          fa[i] = OA::get(*reinterpret_cast<const w4*>(&As[buf][(wm + 16 * i + r16) * kPitch + 8 * (kq ^ kSwz(r16))]));
#pragma unroll
        for (int j = 0; j < TJ; ++j)
          fb[j] = OB::get(*reinterpret_cast<const w4*>(&Bs[buf][(wn + 16 * j + r16) * kPitch + 8 * (kq ^ kSwz(r16))]));
#pragma unroll
        for (int i = 0; i < TI; ++i)
#pragma unroll
          for (int j = 0; j < TJ; ++j) acc[i][j] = mfma(fb[j], fa[i], acc[i][j]);  // C^T tiles
        if (st + 1 < s1) stage(buf ^ 1, ra[(q + 1) % D], rb[(q + 1) % D]);  // nobody reads buf ^ 1 now
        __syncthreads();
      }
    }
  }

  // lane holds C[row 16i + r16][columns 16j + 4kq .. 16j + 4kq + 3] of this
  // wave's block (the products above are C^T tiles): one 4-element store each
  void* C = g.ksplit > 1 ? static_cast<void*>(static_cast<float*>(g.C[1]) + (int64_t)blockIdx.z * g.M * g.N)
                         : g.C[blockIdx.z];
  const int cdt = g.ksplit > 1 ? (int)GTR_F32 : g.cdt;
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    const int m = mb + wm + 16 * i + r16;
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int64_t off = (int64_t)m * g.N + nb + wn + 16 * j + 4 * kq;
      const float x[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      store_n<4>(C, cdt, off, x);
    }
  }
}

// C = sum over the ksplit float32 partial products, converted to C's dtype;
// 4 elements per thread.
__global__ void __launch_bounds__(256) ksplit_reduce_kernel(const float* part, void* C, int64_t n4, int ksplit,
                                                            int cdt) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  f4 s = reinterpret_cast<const f4*>(part)[i];
  for (int z = 1; z < ksplit; ++z) s += reinterpret_cast<const f4*>(part)[(int64_t)z * n4 + i];
  if (cdt == GTR_F32) {
    reinterpret_cast<f4*>(C)[i] = s;
  } else {
    float x[4] = {s[0], s[1], s[2], s[3]};
    store_n<4>(C, cdt, 4 * i, x);
  }
}

// H[b][t][c] = SiLU(G[b][t][c]) * (sum_{u,v} V[b][t + (u-1, v-1)][c] * cw[c][u][v] + cb[c]).
// One work-group per tile of kCT x kCT tokens and kCC channels. The
// (kCT + 2)^2-token halo of V (zero outside the grid) is staged in LDS with
// every global load of the work-group issued before any is used; each thread
// then forms 8 channels of two tokens of the tile from LDS (a wave reads one
// tile row of 8 tokens x 128 contiguous bytes per tap).
constexpr int kCT = 8;            // tile edge in tokens
constexpr int kCC = 64;           // channels per work-group (8 pieces of 8)
constexpr int kHalo = kCT + 2;    // halo tile edge
constexpr int kHaloPieces = kHalo * kHalo * (kCC / 8);
constexpr int kHaloPer = (kHaloPieces + 255) / 256;

__global__ void __launch_bounds__(256) conv_gate_kernel(const _Float16* G, const _Float16* V, const float* cw,
                                                        const float* cb, _Float16* Hout, int Hh, int W,
                                                        int hidden) {
  __shared__ __attribute__((aligned(16))) _Float16 vs[kHalo * kHalo * kCC];
  __shared__ __attribute__((aligned(16))) float wsm[kCC * 9];
  __shared__ __attribute__((aligned(16))) float bsm[kCC];
  const int tiles_x = (W + kCT - 1) / kCT, tiles_y = (Hh + kCT - 1) / kCT;
  const int tx = (int)(blockIdx.x % tiles_x);
  const int ty = (int)((blockIdx.x / tiles_x) % tiles_y);
  const int64_t b = blockIdx.x / ((unsigned)tiles_x * tiles_y);
  const int c0 = blockIdx.y * kCC;
  const int64_t L = (int64_t)Hh * W;
  const int tid = threadIdx.x;

  // halo pieces (token of the halo tile, 16-byte piece of its kCC channels)
  w4 hv[kHaloPer];
#pragma unroll
  for (int q = 0; q < kHaloPer; ++q) {
    const int p = tid + 256 * q;
    const int ht = p >> 3, pc = p & 7;
    const int gy = ty * kCT - 1 + ht / kHalo, gx = tx * kCT - 1 + ht % kHalo;
    const bool in = p < kHaloPieces && gy >= 0 && gy < Hh && gx >= 0 && gx < W;
    hv[q] = w4{0u, 0u, 0u, 0u};
    if (in) hv[q] = *reinterpret_cast<const w4*>(V + (b * L + (int64_t)gy * W + gx) * hidden + c0 + 8 * pc);
  }
  // this thread's outputs: channel piece pc, tile column rx, tile rows ry and ry + kCT / 2
  const int pc = tid & 7, rx = (tid >> 3) % kCT, ry = (tid >> 3) / kCT;
  w4 gv[2];
  bool own[2];
  int64_t tok[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int gy = ty * kCT + ry + k * (kCT / 2), gx = tx * kCT + rx;
    own[k] = gy < Hh && gx < W;
    tok[k] = b * L + (int64_t)gy * W + gx;
    gv[k] = w4{0u, 0u, 0u, 0u};
    if (own[k]) gv[k] = *reinterpret_cast<const w4*>(G + tok[k] * hidden + c0 + 8 * pc);
  }
  // weights [kCC][9] and bias of the work-group's channels
  f4 wv = {0.f, 0.f, 0.f, 0.f}, bv = {0.f, 0.f, 0.f, 0.f};
  constexpr int WQ = kCC * 9 / 4, BQ = kCC / 4;
  if (tid < WQ) wv = reinterpret_cast<const f4*>(cw + (int64_t)c0 * 9)[tid];
  if (cb && tid >= WQ && tid < WQ + BQ) bv = reinterpret_cast<const f4*>(cb + c0)[tid - WQ];

#pragma unroll
  for (int q = 0; q < kHaloPer; ++q) {
    const int p = tid + 256 * q;
    if (p < kHaloPieces) *reinterpret_cast<w4*>(&vs[8 * p]) = hv[q];
  }
  if (tid < WQ) reinterpret_cast<f4*>(wsm)[tid] = wv;
  if (tid >= WQ && tid < WQ + BQ) reinterpret_cast<f4*>(bsm)[tid - WQ] = bv;
  __syncthreads();

  float wt[72];  // wt[9 e + 3 u + v]: tap (u, v) of channel 8 pc + e
#pragma unroll
  for (int q = 0; q < 18; ++q) {
    const f4 x = reinterpret_cast<const f4*>(wsm + 72 * pc)[q];
#pragma unroll
    for (int e = 0; e < 4; ++e) wt[4 * q + e] = x[e];
  }
  const f4 blo = reinterpret_cast<const f4*>(bsm + 8 * pc)[0], bhi = reinterpret_cast<const f4*>(bsm + 8 * pc)[1];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    float acc[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[e] = blo[e];
      acc[e + 4] = bhi[e];
    }
    const int hy = ry + k * (kCT / 2);
#pragma unroll
    for (int u = 0; u < 3; ++u)
#pragma unroll
      for (int v = 0; v < 3; ++v) {
        const h8 x = *reinterpret_cast<const h8*>(&vs[((hy + u) * kHalo + rx + v) * kCC + 8 * pc]);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf((float)x[e], wt[9 * e + 3 * u + v], acc[e]);
      }
    const h8 g8 = __builtin_bit_cast(h8, gv[k]);
    h8 out;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float z = (float)g8[e];
      out[e] = (_Float16)(z * __builtin_amdgcn_rcpf(1.f + __expf(-z)) * acc[e]);
    }
    if (own[k]) *reinterpret_cast<h8*>(Hout + tok[k] * hidden + c0 + 8 * pc) = out;
  }
}

// K slices of the output product: enough work-groups to give every SIMD a few
// waves when M x d alone does not (d is small next to hidden).
static int out_ksplit(int64_t M, int d, int hidden) {
  const int64_t wgs = ((M + 127) / 128) * (d / (d % 128 == 0 ? 128 : 64));
  int s = 1;
  while (wgs * s < 1024 && s < 8 && hidden / 32 >= 2 * s * KB) s *= 2;
  return s;
}

struct SwigluLayout {
  size_t g_off, v_off, h_off, part_off, total;
};

static SwigluLayout swiglu_layout(int64_t M, int d, int64_t hidden) {
  auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  SwigluLayout l;
  l.g_off = 0;
  l.v_off = a256((size_t)M * hidden * 2);
  l.h_off = a256(l.v_off + (size_t)M * hidden * 2);
  l.part_off = a256(l.h_off + (size_t)M * hidden * 2);
  const int ks = out_ksplit(M, d, (int)hidden);
  l.total = a256(l.part_off + (ks > 1 ? (size_t)ks * M * d * 4 : 0));
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
  const SwigluLayout lay = swiglu_layout(M, a->d, a->hidden);
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
  return swiglu_layout(M, a->d, a->hidden).total;
}

extern "C" gtr_status gtr_spatial_swiglu(const gtr_swiglu_args* a, hipStream_t stream) {
  if (!a) return GTR_ERR_NULL;
  int64_t M;
  gtr_status st = swiglu_check(a, &M, true);
  if (st != GTR_OK) return st;
  const SwigluLayout lay = swiglu_layout(M, a->d, a->hidden);
  char* ws = static_cast<char*>(a->workspace);
  _Float16* G = reinterpret_cast<_Float16*>(ws + lay.g_off);
  _Float16* V = reinterpret_cast<_Float16*>(ws + lay.v_off);
  _Float16* Hb = reinterpret_cast<_Float16*>(ws + lay.h_off);
  const bool bf = a->dtype == GTR_BF16;

  GemmArgs g1{a->x, {a->w_gate, a->w_value}, {G, V}, (int)M, a->hidden, a->d, GTR_F16, 1};
  const bool n128 = a->hidden % 128 == 0;
  const dim3 grid1((unsigned)((M + 127) / 128), (unsigned)(a->hidden / (n128 ? 128 : 64)), 2);
  if (bf && n128)
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_BF16, GTR_BF16, GTR_BF16, 128, 128>), grid1, dim3(256), 0, stream, g1);
  else if (bf)
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_BF16, GTR_BF16, GTR_BF16, 128, 64>), grid1, dim3(256), 0, stream, g1);
  else if (n128)
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_F16, GTR_F16, GTR_F16, 128, 128>), grid1, dim3(256), 0, stream, g1);
  else
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_F16, GTR_F16, GTR_F16, 128, 64>), grid1, dim3(256), 0, stream, g1);
  if (hipGetLastError() != hipSuccess) return GTR_ERR_HIP;

  const int64_t tiles = (int64_t)a->B * ((a->H + kCT - 1) / kCT) * ((a->W + kCT - 1) / kCT);
  hipLaunchKernelGGL(conv_gate_kernel, dim3((unsigned)tiles, (unsigned)(a->hidden / kCC)), dim3(256), 0, stream,
                     G, V, a->conv_w, a->conv_b, Hb, a->H, a->W, a->hidden);
  if (hipGetLastError() != hipSuccess) return GTR_ERR_HIP;

  const int ks = out_ksplit(M, a->d, a->hidden);
  float* part = reinterpret_cast<float*>(ws + lay.part_off);
  GemmArgs g3{Hb, {a->w_out, a->w_out}, {a->y, ks > 1 ? static_cast<void*>(part) : a->y}, (int)M, a->d,
              a->hidden, a->y_dtype, ks};
  const bool d128 = a->d % 128 == 0;
  const dim3 grid3((unsigned)((M + 127) / 128), (unsigned)(a->d / (d128 ? 128 : 64)), (unsigned)ks);
  if (bf && d128)
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_F16, GTR_BF16, GTR_F16, 128, 128>), grid3, dim3(256), 0, stream, g3);
  else if (bf)
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_F16, GTR_BF16, GTR_F16, 128, 64>), grid3, dim3(256), 0, stream, g3);
  else if (d128)
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_F16, GTR_F16, GTR_F16, 128, 128>), grid3, dim3(256), 0, stream, g3);
  else
    hipLaunchKernelGGL((gemm_nt_kernel<GTR_F16, GTR_F16, GTR_F16, 128, 64>), grid3, dim3(256), 0, stream, g3);
  if (hipGetLastError() != hipSuccess) return GTR_ERR_HIP;
  if (ks > 1) {
    const int64_t n4 = M * a->d / 4;
    hipLaunchKernelGGL(ksplit_reduce_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream, part, a->y,
                       n4, ks, (int)a->y_dtype);
  }
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}
