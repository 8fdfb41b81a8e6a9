// Spatial SwiGLU for gfx950 (MI355X): paper Sec. 3.1, "Spatial SwiGLU",
//   Y = [SiLU(X W_g) * DWConv3x3(X W_v)] W_o,
// X the patch tokens of one image in row-major grid order, the value branch
// convolved depthwise over the H x W grid (zero padding), the gate tokenwise.
//
// Two launches (three when the output product splits K):
//   1. gated_conv_kernel: H = SiLU(X W_g^T) * (DWConv3x3(X W_v^T) + bias) per
//      tile of tokens, both products on MFMA with the input dtype's operands
//      (fp16 or bf16) and float32 accumulation, rounded to fp16 on chip, the
//      convolution's halo recomputed per tile; H is stored in fp16, the
//      operand type of the next product;
//   2. gemm_nt_kernel: Y = H W_o^T (fp16 operands; bf16 weights are widened),
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

// C[M][N] = A[M][K] * B[N][K]^T, row-major, K a multiple of 64, N a multiple
// of BN. Work-group tile BM x BN, 4 waves in a 2 x 2 grid, each wave a
// (BM/2) x (BN/2) block of 16 x 16 MFMA tiles. Every K-step of 64 stages the
// A and B tiles in LDS once (each element is read from memory by one thread
// and from LDS by every wave that needs it) and runs two 32-deep MFMA passes
// over them; the loads of the next steps are in flight while the current one
// multiplies (two LDS buffers). Rows past M are read from row M-1 and not
// stored. With ksplit > 1, K is cut into ksplit slices whose partial products
// go to part + slice * M * N (float32) for ksplit_reduce_kernel; with
// ksplit = 1 the product goes to C.
// The grid is one-dimensional, gx * gy * ksplit work-groups (gx = ceil(M / BM),
// gy = N / BN). Work-group b runs on XCD b % 8 (round-robin dispatch), and each
// XCD takes a contiguous range of the tile order (slice, row block, column
// block), column blocks fastest: the work-groups that read the same rows of A
// (all column blocks of a row block and slice) share one XCD's L2 instead of
// fetching those rows once per XCD.
struct GemmArgs {
  const void* A;
  const void* B;
  void* C;
  float* part;
  int M, N, K;
  int cdt;     // dtype of C (GTR_F32 / GTR_F16 / GTR_BF16)
  int ksplit;  // number of K slices (1: none)
  const float* bias;  // [N] float32 added to every row, or null (ksplit = 1 only)
  const void* res;    // [M][N] in C's dtype added elementwise (a residual), or null (ksplit = 1 only)
  // head-major operands (ksplit = 1 only; 0: row-major):
  int64_t a_tokens;   // A is [M / a_tokens][K / 64][a_tokens][64]: row m = (image m / a_tokens, token
                      // m % a_tokens), K step s = head s (a head concat read in place)
  int64_t c_tokens;   // C is written [N / (c_heads c_dim)][M / c_tokens][c_heads][c_tokens][c_dim]
  int c_heads, c_dim;
  float ln_eps;       // the row normalisation's epsilon (kernels with LN = 1)
  int pad_;
};

// 8 consecutive 16-bit elements of dtype DT (one 16-byte piece) as floats.
template <int DT>
__device__ __forceinline__ void unpack_piece(const w4& v, float (&x)[8]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const unsigned u = v[e];
    if (DT == GTR_F16) {
      x[2 * e] = (float)__builtin_bit_cast(_Float16, (unsigned short)(u & 0xffffu));
      x[2 * e + 1] = (float)__builtin_bit_cast(_Float16, (unsigned short)(u >> 16));
    } else {
      x[2 * e] = __builtin_bit_cast(float, u << 16);
      x[2 * e + 1] = __builtin_bit_cast(float, u & 0xffff0000u);
    }
  }
}

// 4 consecutive elements of dtype dt at element offset off, as floats.
__device__ __forceinline__ void load4(const void* base, int dt, int64_t off, float (&x)[4]) {
  if (dt == GTR_F32) {
    const f4 v = *reinterpret_cast<const f4*>(static_cast<const float*>(base) + off);
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = v[e];
  } else if (dt == GTR_F16) {
    const h4 v = *reinterpret_cast<const h4*>(static_cast<const _Float16*>(base) + off);
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = (float)v[e];
  } else {
    typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));
    const u16x4 v = *reinterpret_cast<const u16x4*>(static_cast<const unsigned short*>(base) + off);
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = bf16_bits_to_f32(v[e]);
  }
}

constexpr int KB = 4;     // minimum 64-wide K-steps per slice when splitting K
// LDS tiles: rows of 32 K elements (64 bytes, no padding); the 16-byte piece
// c of row r sits at piece c ^ kSwz(r). Measured on gfx950, ds_read_b128 serves
// 32 lanes per cycle from 32 distinct 16-byte slots (address / 16 mod 32) and
// ds_write_b128 16 lanes from 16 slots (mod 16): with this swizzle the operand
// reads (lanes = 16 rows x 2 pieces) and the staging writes (lanes = 4 rows x
// 4 pieces) both hit distinct slots.
constexpr int kPitch = 32;
__device__ __forceinline__ int kSwz(int r) { return (r >> 2) & 2; }
// The output product's 64-wide rows (128 bytes, 8 pieces): piece c of row r at
// c ^ kSwz64(r). Operand reads (16 rows x 2 pieces per 32 lanes) then hit 32
// distinct slots (rows r, r + 4, r + 8, r + 12 share address / 16 mod 32 up to
// the piece, and the swizzle gives them 4 disjoint piece pairs); staging writes
// (2 rows x 8 pieces per 16 lanes) hit 16.
constexpr int kPitch64 = 64;
__device__ __forceinline__ int kSwz64(int r) { return ((r >> 2) & 3) << 1; }

// With LN = 1 every row of A is normalised over its K columns (A' = (A - mu)
// / sqrt(var + eps), a layer normalisation without affine weights, which the
// caller folds into B and the bias) inside the product: the MFMAs multiply the
// raw A, the row sums and squares of A and the row sums of B (colsum of B^T)
// are taken from the pieces as they pass through registers on their way to
// LDS, and the epilogue forms rs_m (C_mn - mu_m colsum_n), which is A' B^T in
// real arithmetic. The squares are taken about a shift (the row's first
// element) so that a row mean large next to its spread costs no precision.
// LN = 1 needs K in one slice and a row-major A.
template <int ADT, int BDT, int MT, int BM, int BN, int KW, int LN>
__global__ void __launch_bounds__(256 * KW) gemm_nt_kernel(GemmArgs g) {
  typedef Operand<ADT, MT> OA;
  typedef Operand<BDT, MT> OB;
  constexpr int NT = 256 * KW;                // threads
  constexpr int TI = BM / 32, TJ = BN / 32;   // MFMA tiles per wave
  constexpr int PA = BM * 8 / NT, PB = BN * 8 / NT;  // 16-byte pieces per thread per step
  static_assert((KW == 1 || KW == 2) && PA >= 1 && PB >= 1 && BM * 8 % NT == 0 && BN * 8 % NT == 0,
                "tiles split evenly over the threads");
  static_assert(KW == 1 || BM * BN * 4 <= 2 * BM * kPitch64 * 2, "the K halves' partial sums fit in As");
  __shared__ __attribute__((aligned(16))) unsigned short As[2][BM * kPitch64];
  __shared__ __attribute__((aligned(16))) unsigned short Bs[2][BN * kPitch64];
  __shared__ float lnst[LN ? 2 * BM : 1];  // per tile row: mean, 1 / sqrt(var + eps)
  __shared__ float lncs[LN ? BN : 1];      // per tile column: the row sum of B

  // wave w of the 2 x 2 grid over the tile; with KW = 2 the waves kh = 0 and
  // kh = 1 take the first and the second 32-deep half of every K step
  const int w = (threadIdx.x >> 6) & 3, kh = threadIdx.x >> 8, lane = threadIdx.x & 63;
  const int r16 = lane & 15, kq = lane >> 4;
  // tile of this work-group: XCD k = b % 8 takes positions [start_k, start_k +
  // count_k) of the tile order, count_k = ceil((T - k) / 8)
  const int gx = (g.M + BM - 1) / BM, gy = g.N / BN;
  const int T = gx * gy * g.ksplit, xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int j = xcd * (T >> 3) + min(xcd, T & 7) + slot;
  const int by = j % gy, bxz = j / gy, bx = bxz % gx, bz = bxz / gx;
  const int mb = bx * BM, nb = by * BN;
  const int wm = (w >> 1) * (BM / 2), wn = (w & 1) * (BN / 2);
  const unsigned short* A = static_cast<const unsigned short*>(g.A);
  const unsigned short* B = static_cast<const unsigned short*>(g.B);
  const int64_t K = g.K;
  const int steps = g.K / 64;
  const int s_per = (steps + g.ksplit - 1) / g.ksplit;
  const int s0 = g.ksplit > 1 ? bz * s_per : 0;
  const int s1 = min(s0 + s_per, steps);

  // global pieces of this thread: piece p -> row p / 8, 16-byte column p % 8
  const w4* ga[PA];
  const w4* gb[PB];
  int la[PA], lb[PB];
#pragma unroll
  for (int q = 0; q < PA; ++q) {
    const int p = threadIdx.x + NT * q, row = p >> 3, col = p & 7;
    const unsigned m = (unsigned)min(mb + row, g.M - 1), at = g.a_tokens ? (unsigned)g.a_tokens : 1u;
    ga[q] = reinterpret_cast<const w4*>(
        A + (g.a_tokens ? ((int64_t)(m / at) * (K / 64) * at + m % at) * 64 : (int64_t)m * K) + 8 * col);
    la[q] = row * kPitch64 + 8 * (col ^ kSwz64(row));
  }
#pragma unroll
  for (int q = 0; q < PB; ++q) {
    const int p = threadIdx.x + NT * q, row = p >> 3, col = p & 7;
    gb[q] = reinterpret_cast<const w4*>(B + (int64_t)(nb + row) * K + 8 * col);
    lb[q] = row * kPitch64 + 8 * (col ^ kSwz64(row));
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
  const int64_t ast = g.a_tokens ? 8 * g.a_tokens : 8;  // 16-byte pieces from one K step of A to the next
  w4 ra[D][PA], rb[D][PB];
  auto fetch = [&](int st, w4 (&a)[PA], w4 (&b)[PB]) {
#pragma unroll
    for (int q = 0; q < PA; ++q) a[q] = ga[q][ast * st];
#pragma unroll
    for (int q = 0; q < PB; ++q) b[q] = gb[q][8 * st];
  };
  auto stage = [&](int buf, const w4 (&a)[PA], const w4 (&b)[PB]) {
#pragma unroll
    for (int q = 0; q < PA; ++q) *reinterpret_cast<w4*>(&As[buf][la[q]]) = a[q];
#pragma unroll
    for (int q = 0; q < PB; ++q) *reinterpret_cast<w4*>(&Bs[buf][lb[q]]) = b[q];
  };
  // row statistics (LN = 1) of the steps staged so far: per piece of A the
  // sum and the sum of squares about the row's shift, per piece of B its sum
  float sh[PA], sa[PA], sq[PA], cb[PB];
#pragma unroll
  for (int q = 0; q < PA; ++q) sh[q] = sa[q] = sq[q] = 0.f;
#pragma unroll
  for (int q = 0; q < PB; ++q) cb[q] = 0.f;
  auto stats = [&](const w4 (&a)[PA], const w4 (&b)[PB]) {
    if constexpr (LN != 0) {
#pragma unroll
      for (int q = 0; q < PA; ++q) {
        float x[8];
        unpack_piece<ADT>(a[q], x);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = x[e] - sh[q];
          sa[q] += d;
          sq[q] = fmaf(d, d, sq[q]);
        }
      }
#pragma unroll
      for (int q = 0; q < PB; ++q) {
        float x[8];
        unpack_piece<BDT>(b[q], x);
#pragma unroll
        for (int e = 0; e < 8; ++e) cb[q] += x[e];
      }
    }
  };
  auto mma = [&](int buf) {
#pragma unroll
    for (int hh = 0; hh < 2 / KW; ++hh) {  // the 32-deep halves of the step this wave takes
      const int h = KW == 1 ? hh : kh;
      const int pc = (4 * h + kq) ^ kSwz64(r16);
      typename OA::T fa[TI];
      typename OB::T fb[TJ];
#pragma unroll
      for (int i = 0; i < TI; ++i)
        fa[i] = OA::get(*reinterpret_cast<const w4*>(&As[buf][(wm + 16 * i + r16) * kPitch64 + 8 * pc]));
#pragma unroll
      for (int j = 0; j < TJ; ++j)
        fb[j] = OB::get(*reinterpret_cast<const w4*>(&Bs[buf][(wn + 16 * j + r16) * kPitch64 + 8 * pc]));
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) acc[i][j] = mfma(fb[j], fa[i], acc[i][j]);  // C^T tiles
    }
  };
  // The loop runs whole groups of D steps in which every step issues the same
  // loads (past the slice's last step they re-read that step, never used):
  // with no load under a branch the compiler's waits count exactly, so a step
  // waits for the loads of the step it stages, not for the newer ones (which
  // matters where few work-groups run, each a chain of K steps). The last
  // (steps mod D) steps follow with their loads already in flight.
  if (s1 > s0) {
#pragma unroll
    for (int q = 0; q < D; ++q) fetch(min(s0 + q, s1 - 1), ra[q], rb[q]);
    if constexpr (LN != 0) {  // the shift of each row: its first element, from the row's column-0 lane
#pragma unroll
      for (int q = 0; q < PA; ++q) {
        float x[8];
        unpack_piece<ADT>(ra[0][q], x);
        sh[q] = __shfl(x[0], lane & ~7, kWave);
      }
    }
    stage(0, ra[0], rb[0]);
    stats(ra[0], rb[0]);
    __syncthreads();
    int sb = s0;
    for (; sb + D <= s1; sb += D) {
#pragma unroll
      for (int q = 0; q < D; ++q) {
        const int st = sb + q, buf = (st - s0) & 1;
        fetch(min(st + D, s1 - 1), ra[q], rb[q]);  // slot q was staged before this step
        mma(buf);
        stage(buf ^ 1, ra[(q + 1) % D], rb[(q + 1) % D]);  // nobody reads buf ^ 1 now
        if (st + 1 < s1) stats(ra[(q + 1) % D], rb[(q + 1) % D]);  // past the last step: a re-read
        __syncthreads();
      }
    }
#pragma unroll
    for (int q = 0; q < D - 1; ++q) {
      const int st = sb + q, buf = (st - s0) & 1;
      if (st < s1) {
        mma(buf);
        if (st + 1 < s1) {
          stage(buf ^ 1, ra[(q + 1) % D], rb[(q + 1) % D]);
          stats(ra[(q + 1) % D], rb[(q + 1) % D]);
        }
        __syncthreads();
      }
    }
  }

  if constexpr (LN != 0) {  // the 8 lanes of a row combine; lane 0 of each stores
#pragma unroll
    for (int o = 1; o < 8; o <<= 1) {
#pragma unroll
      for (int q = 0; q < PA; ++q) {
        sa[q] += __shfl_xor(sa[q], o, kWave);
        sq[q] += __shfl_xor(sq[q], o, kWave);
      }
#pragma unroll
      for (int q = 0; q < PB; ++q) cb[q] += __shfl_xor(cb[q], o, kWave);
    }
    if ((lane & 7) == 0) {
      const float inv = 1.f / (float)g.K;
#pragma unroll
      for (int q = 0; q < PA; ++q) {
        const int row = (threadIdx.x + NT * q) >> 3;
        const float m1 = sa[q] * inv;
        lnst[2 * row] = sh[q] + m1;
        lnst[2 * row + 1] = rsqrtf(fmaxf(sq[q] * inv - m1 * m1, 0.f) + g.ln_eps);
      }
#pragma unroll
      for (int q = 0; q < PB; ++q) lncs[(threadIdx.x + NT * q) >> 3] = cb[q];
    }
    if (KW == 1) __syncthreads();
  }
  if (KW == 2) {  // the second K half's sums join the first's through LDS
    f4* red = reinterpret_cast<f4*>(&As[0][0]);
    __syncthreads();  // every wave is past the K loop's last LDS read
    if (kh == 1) {
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j) red[((w * TI + i) * TJ + j) * 64 + lane] = acc[i][j];
    }
    __syncthreads();
    if (kh == 1) return;
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int j = 0; j < TJ; ++j) acc[i][j] += red[((w * TI + i) * TJ + j) * 64 + lane];
  }

  // lane holds C[row 16i + r16][columns 16j + 4kq .. 16j + 4kq + 3] of this
  // wave's block (the products above are C^T tiles): one 4-element store each
  void* C = g.ksplit > 1 ? static_cast<void*>(g.part + (int64_t)bz * g.M * g.N) : g.C;
  const int cdt = g.ksplit > 1 ? (int)GTR_F32 : g.cdt;
  // head-major C: element (m, n) at (((p img + b) heads + h) tokens + t) dim + c
  // with m = b tokens + t, n = (p heads + h) dim + c; the divisions are 32-bit
  // (the host keeps M below 2^31) and taken once per row and column block
  const bool hmc = g.ksplit == 1 && g.c_tokens != 0;
  const unsigned tokens = hmc ? (unsigned)g.c_tokens : 1u, cdim = hmc ? (unsigned)g.c_dim : 1u;
  const unsigned hd = hmc ? (unsigned)(g.c_heads * g.c_dim) : 1u, img = (unsigned)g.M / tokens;
  int64_t rowoff[TI], coloff[TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    const unsigned m = (unsigned)(mb + wm + 16 * i + r16);
    rowoff[i] = hmc ? ((int64_t)(m / tokens) * g.c_heads * tokens + m % tokens) * cdim : (int64_t)m * g.N;
  }
#pragma unroll
  for (int j = 0; j < TJ; ++j) {
    const unsigned n0 = (unsigned)(nb + wn + 16 * j + 4 * kq);
    const unsigned p = n0 / hd, r = n0 - p * hd, h = r / cdim;
    coloff[j] = hmc ? ((int64_t)p * img * g.c_heads * tokens + (int64_t)h * tokens) * cdim + (r - h * cdim) : n0;
  }
#pragma unroll
  for (int i = 0; i < TI; ++i) {
    const int m = mb + wm + 16 * i + r16;
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int n0 = nb + wn + 16 * j + 4 * kq;
      const int64_t off = rowoff[i] + coloff[j];
      float x[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      if constexpr (LN != 0) {
        const int lr = wm + 16 * i + r16, lc = wn + 16 * j + 4 * kq;
        const float mu = lnst[2 * lr], rs = lnst[2 * lr + 1];
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = rs * (x[e] - mu * lncs[lc + e]);
      }
      if (g.ksplit == 1 && g.bias) {
        const f4 bv = *reinterpret_cast<const f4*>(g.bias + n0);
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] += bv[e];
      }
      if (g.ksplit == 1 && g.res) {  // (row-major C)
        float rv[4];
        load4(g.res, cdt, off, rv);
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] += rv[e];
      }
      store_n<4>(C, cdt, off, x);
    }
  }
}

// C = sum over the ksplit float32 partial products, converted to C's dtype;
// 4 elements per thread.
__global__ void __launch_bounds__(256) ksplit_reduce_kernel(const float* part, void* C, int64_t n4, int ksplit,
                                                            int cdt, const void* res) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n4) return;
  f4 s = reinterpret_cast<const f4*>(part)[i];
  for (int z = 1; z < ksplit; ++z) s += reinterpret_cast<const f4*>(part)[(int64_t)z * n4 + i];
  if (res) {  // a residual in C's dtype
    float r[4];
    load4(res, cdt, 4 * i, r);
#pragma unroll
    for (int e = 0; e < 4; ++e) s[e] += r[e];
  }
  if (cdt == GTR_F32) {
    reinterpret_cast<f4*>(C)[i] = s;
  } else {
    float x[4] = {s[0], s[1], s[2], s[3]};
    store_n<4>(C, cdt, 4 * i, x);
  }
}

// H[b][t][c] = SiLU(G[b][t][c]) * (sum_{u,v} V[b][t + (u-1, v-1)][c] * cw[c][u][v] + cb[c]),
// G = X W_g^T and V = X W_v^T, in one launch. A work-group owns a tile of
// kFH x kFW tokens of one image and kFN channels. Its K loop multiplies the
// tile's (kFH + 2) x (kFW + 2)-token halo of X (rows outside the image are
// zero) by the kFN rows of W_v, and the tile's own tokens (each tile row is a
// run of 16 consecutive halo rows) by the kFN rows of W_g, with the load ring,
// LDS swizzle and C^T accumulator layout of gemm_nt_kernel. The epilogue
// rounds both products to fp16 into the LDS the K loop used and forms the
// gated convolution there: G and V never leave the chip, and the halo's extra
// V rows are the price (180 V rows per 128 tokens). One-dimensional grid of
// tiles * (hidden / kFN) work-groups; as in gemm_nt_kernel each XCD takes a
// contiguous range of the order (tile, channel block), channel blocks
// fastest, so the work-groups that read the same X halo share one XCD's L2.
// (Measured at 40x40 tokens, one image, us per SwiGLU call: GTR-L 34.4, GTR-X
// 45.9 with this order; 35.1 / 46.9 with channel blocks slowest; 34.2 / 46.6
// with the plain two-dimensional grid.)
constexpr int kFH = 8, kFW = 16;         // tile: 8 rows of 16 tokens
constexpr int kFHW = kFW + 2;            // halo row length
constexpr int kFV = (kFH + 2) * kFHW;    // halo tokens (180)
constexpr int kFVT = (kFV + 15) / 16;    // MFMA row blocks of V (12; rows 180..191 are zero padding)
constexpr int kFN = 64;                  // channels per work-group
constexpr int kFA = kFVT * 16 * 4 / 256; // 16-byte A pieces per thread per K step (3)
constexpr int kFB = kFN * 4 * 2 / 256;   // 16-byte pieces of the W_g and W_v tiles per thread per K step
constexpr int kFP = kFN / 8;             // 16-byte pieces (8 channels) of one token's kFN channels
static_assert(kFB >= 1 && kFN * 4 * 2 % 256 == 0 && (kFP & (kFP - 1)) == 0, "weight tiles split evenly over 256 threads");
static_assert(kFVT % 4 == 0 && kFH % 4 == 0, "row blocks split evenly over 4 waves");

struct GatedConvArgs {
  const void* X;
  const void* Wg;
  const void* Wv;
  const float* cw;  // [hidden][9]
  const float* cb;  // [hidden] or null
  _Float16* H;      // [B * Hh * W][hidden]
  int Hh, W, d, hidden;
  int B;            // images
};

template <int DT>
__global__ void __launch_bounds__(256) gated_conv_kernel(GatedConvArgs f) {
  typedef Operand<DT, DT> OP;
  constexpr int SA = kFVT * 16 * kPitch, SB = kFN * kPitch;  // 16-bit elements per stage
  constexpr int VT = kFVT / 4, GT = kFH / 4;                 // row blocks of V and G per wave
  constexpr int NJ = kFN / 16;                               // column blocks (all waves)
  static_assert(2 * (SA + 2 * SB) >= (kFVT * 16 + kFH * kFW) * kFN, "epilogue tiles fit the stage buffers");
  __shared__ __attribute__((aligned(16))) unsigned short stg[2][SA + 2 * SB];
  __shared__ __attribute__((aligned(16))) float wsm[kFN * 9 + kFN];

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, kq = lane >> 4;
  const int tiles_x = (f.W + kFW - 1) / kFW, tiles_y = (f.Hh + kFH - 1) / kFH;
  const int tiles = f.B * tiles_x * tiles_y;
  const int T = tiles * (f.hidden / kFN), xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int ncb = f.hidden / kFN;
  const int j = xcd * (T >> 3) + min(xcd, T & 7) + slot;  // position in the (tile, channel block) order
  const int tile = j / ncb;
  const int tx = tile % tiles_x;
  const int ty = (tile / tiles_x) % tiles_y;
  const int64_t b = tile / (tiles_x * tiles_y);
  const int y0 = ty * kFH, x0 = tx * kFW;
  const int c0 = (j % ncb) * kFN;
  const int64_t L = (int64_t)f.Hh * f.W, K = f.d;
  const unsigned short* X = static_cast<const unsigned short*>(f.X);

  // conv weights and bias of the work-group's channels (read in the epilogue)
  if (tid < kFN * 9 / 4) reinterpret_cast<f4*>(wsm)[tid] = reinterpret_cast<const f4*>(f.cw + (int64_t)c0 * 9)[tid];
  if (tid >= 160 && tid < 160 + kFN / 4) {
    const int q = tid - 160;
    reinterpret_cast<f4*>(wsm + kFN * 9)[q] =
        f.cb ? reinterpret_cast<const f4*>(f.cb + c0)[q] : f4{0.f, 0.f, 0.f, 0.f};
  }

  // this thread's 16-byte pieces of the A (halo) and B (weight) tiles
  const w4* ga[kFA];
  unsigned am[kFA];  // all-ones for a token of the image, zero otherwise
  int la[kFA];
#pragma unroll
  for (int q = 0; q < kFA; ++q) {
    const int p = tid + 256 * q, row = p >> 2, col = p & 3;
    const int hy = row / kFHW, hx = row - hy * kFHW;
    const int y = y0 - 1 + hy, x = x0 - 1 + hx;
    const bool in = row < kFV && y >= 0 && y < f.Hh && x >= 0 && x < f.W;
    ga[q] = reinterpret_cast<const w4*>(X + (in ? (b * L + (int64_t)y * f.W + x) * K : 0) + 8 * col);
    am[q] = in ? 0xffffffffu : 0u;
    la[q] = row * kPitch + 8 * (col ^ kSwz(row));
  }
  // weight pieces: piece p < 4 kFN of the W_g tile, then the W_v tile
  const w4* gb[kFB];
  int lb[kFB];
#pragma unroll
  for (int q = 0; q < kFB; ++q) {
    const int p = tid + 256 * q, v = p / (kFN * 4), r = (p % (kFN * 4)) >> 2, col = p & 3;
    gb[q] = reinterpret_cast<const w4*>(static_cast<const unsigned short*>(v ? f.Wv : f.Wg) + (int64_t)(c0 + r) * K +
                                        8 * col);
    lb[q] = SA + v * SB + r * kPitch + 8 * (col ^ kSwz(r));
  }

  f4 av[VT][NJ], ag[GT][NJ];
#pragma unroll
  for (int t = 0; t < VT; ++t)
#pragma unroll
    for (int j = 0; j < NJ; ++j) av[t][j] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < GT; ++t)
#pragma unroll
    for (int j = 0; j < NJ; ++j) ag[t][j] = f4{0.f, 0.f, 0.f, 0.f};

  constexpr int D = 4;
  w4 ra[D][kFA], rb[D][kFB];
  auto fetch = [&](int s, w4 (&a)[kFA], w4 (&b)[kFB]) {
#pragma unroll
    for (int q = 0; q < kFA; ++q) a[q] = ga[q][4 * s];
#pragma unroll
    for (int q = 0; q < kFB; ++q) b[q] = gb[q][4 * s];
  };
  auto stage = [&](int buf, const w4 (&a)[kFA], const w4 (&b)[kFB]) {
    unsigned short* S = stg[buf];
#pragma unroll
    for (int q = 0; q < kFA; ++q) *reinterpret_cast<w4*>(&S[la[q]]) = a[q] & am[q];  // zero outside the image
#pragma unroll
    for (int q = 0; q < kFB; ++q) *reinterpret_cast<w4*>(&S[lb[q]]) = b[q];
  };
  auto frag = [&](const unsigned short* S, int row) {
    return OP::get(*reinterpret_cast<const w4*>(&S[row * kPitch + 8 * (kq ^ kSwz(row))]));
  };
  const int steps = f.d / 32;
#pragma unroll
  for (int q = 0; q < D; ++q)
    if (q < steps) fetch(q, ra[q], rb[q]);
  stage(0, ra[0], rb[0]);
  __syncthreads();
  for (int sb = 0; sb < steps; sb += D) {
#pragma unroll
    for (int q = 0; q < D; ++q) {
      const int s = sb + q;
      if (s < steps) {
        const unsigned short* S = stg[s & 1];
        if (s + D < steps) fetch(s + D, ra[q], rb[q]);  // slot q was staged before this step
        typename OP::T fg[NJ], fv[NJ];
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          fg[j] = frag(S + SA, 16 * j + r16);
          fv[j] = frag(S + SA + SB, 16 * j + r16);
        }
#pragma unroll
        for (int t = 0; t < VT; ++t) {
          const typename OP::T fa = frag(S, 16 * (VT * w + t) + r16);
#pragma unroll
          for (int j = 0; j < NJ; ++j) av[t][j] = mfma(fv[j], fa, av[t][j]);  // V^T tiles
        }
#pragma unroll
        for (int t = 0; t < GT; ++t) {
          const int ci = GT * w + t;  // tile row: halo rows (ci + 1) * kFHW + 1 .. + 16
          const typename OP::T fa = frag(S, (ci + 1) * kFHW + 1 + r16);
#pragma unroll
          for (int j = 0; j < NJ; ++j) ag[t][j] = mfma(fg[j], fa, ag[t][j]);  // G^T tiles
        }
        if (s + 1 < steps) stage((s & 1) ^ 1, ra[(q + 1) % D], rb[(q + 1) % D]);
        __syncthreads();
      }
    }
  }

  // epilogue: V [192 halo rows][kFN] and G [128 tile tokens][kFN] in fp16, in
  // the stage buffers (every wave passed the K loop's last barrier). The
  // 16-byte piece p of row r sits at piece p ^ eswz(r): the C^T writes (16
  // rows x 2 half-pieces per 32 lanes) and the convolution's reads (4
  // consecutive rows x 8 pieces per 32 lanes) then both spread over all banks;
  // unswizzled, the writes of rows r, r + 2, r + 4, ... hit the same banks.
  _Float16* Vt = reinterpret_cast<_Float16*>(&stg[0][0]);
  _Float16* Gt = Vt + kFVT * 16 * kFN;
  auto eswz = [](int row) { return (row >> 1) & (kFP - 1); };
#pragma unroll
  for (int t = 0; t < VT; ++t)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int row = 16 * (VT * w + t) + r16;
      const h4 hv = {(_Float16)av[t][j][0], (_Float16)av[t][j][1], (_Float16)av[t][j][2], (_Float16)av[t][j][3]};
      *reinterpret_cast<h4*>(&Vt[row * kFN + 8 * ((2 * j + (kq >> 1)) ^ eswz(row)) + 4 * (kq & 1)]) = hv;
    }
#pragma unroll
  for (int t = 0; t < GT; ++t)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int row = 16 * (GT * w + t) + r16;
      const h4 hg = {(_Float16)ag[t][j][0], (_Float16)ag[t][j][1], (_Float16)ag[t][j][2], (_Float16)ag[t][j][3]};
      *reinterpret_cast<h4*>(&Gt[row * kFN + 8 * ((2 * j + (kq >> 1)) ^ eswz(row)) + 4 * (kq & 1)]) = hg;
    }
  __syncthreads();

  // gated convolution: 8 channels (piece pc) of kFH kFW kFP / 256 tile tokens per thread
  const int pc = tid & (kFP - 1), tg = tid / kFP;
  float wt[72];  // wt[9 e + 3 u + v]: tap (u, v) of channel 8 pc + e
#pragma unroll
  for (int q = 0; q < 18; ++q) {
    const f4 x = reinterpret_cast<const f4*>(wsm + 72 * pc)[q];
#pragma unroll
    for (int e = 0; e < 4; ++e) wt[4 * q + e] = x[e];
  }
  const f4 blo = reinterpret_cast<const f4*>(wsm + kFN * 9 + 8 * pc)[0];
  const f4 bhi = reinterpret_cast<const f4*>(wsm + kFN * 9 + 8 * pc)[1];
#pragma unroll
  for (int m = 0; m < kFH * kFW * kFP / 256; ++m) {
    const int ct = tg + 256 / kFP * m, ci = ct / kFW, cj = ct % kFW;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[e] = blo[e];
      acc[e + 4] = bhi[e];
    }
#pragma unroll
    for (int u = 0; u < 3; ++u)
#pragma unroll
      for (int v = 0; v < 3; ++v) {
        const int row = (ci + u) * kFHW + cj + v;
        const h8 x = *reinterpret_cast<const h8*>(&Vt[row * kFN + 8 * (pc ^ eswz(row))]);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf((float)x[e], wt[9 * e + 3 * u + v], acc[e]);
      }
    const h8 g8 = *reinterpret_cast<const h8*>(&Gt[ct * kFN + 8 * (pc ^ eswz(ct))]);
    h8 out;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float z = (float)g8[e];
      out[e] = (_Float16)(z * __builtin_amdgcn_rcpf(1.f + __expf(-z)) * acc[e]);
    }
    const int y = y0 + ci, x = x0 + cj;
    if (y < f.Hh && x < f.W) *reinterpret_cast<h8*>(f.H + (b * L + (int64_t)y * f.W + x) * f.hidden + c0 + 8 * pc) = out;
  }
}

// Both products on gemm_nt_kernel (the Spatial SwiGLU's output product and
// gtr_gemm) use 64 x 64 work-group tiles (4 waves of 32 x 32). The K loop of a
// work-group is a chain of dependent steps, so at the token counts of one or a
// few images the number of work-groups sets the time more than the operand
// reuse of a larger tile. Measured at one 40x40 image (us): the output product
// 1600 x 384 x 1536 alone 10.3 with 64 x 64 tiles (150 work-groups) against
// 15.1 with 128 x 64 (78); the whole Spatial SwiGLU 27.3 against 30.4 (128 x 64
// tiles with K split in 2 and the reduction) at GTR-L and 40.5 against 41.3 at
// GTR-X; 32 x 64 tiles 28.9 / 42.2; at 3200 and 12800 tokens the two tile
// sizes are on par. K is split into the fewest slices that give 64 work-groups
// when M x d alone does not (small grids only): every slice costs a float32
// partial product and its share of the reduction. (With 8-wave tiles below 256
// tiles, a target of 64 against 128 took the GTR-S block from 48.9 to 47.3 us:
// its 75-tile output product no longer splits; 256 was slower at every width.)
constexpr int kGemmBM = 64, kGemmBN = 64;

// A grid of fewer tiles than the chip's 256 compute units leaves CUs idle, and
// each work-group's K loop is a chain of dependent steps: there, 8 waves per
// tile (the two 32-deep halves of every K step on separate waves, their sums
// joined through LDS at the end) run the chain faster. Larger grids keep 4
// waves per tile. Measured (us): 1600 x 384 x 1536 (150 tiles) 9.5 against
// 10.1, 1600 x 384 x 384 5.0 against 5.3, the Spatial SwiGLU 26.4 / 38.5
// against 27.2 / 40.6 (GTR-L / GTR-X); 1600 x 1920 x 384 (750 tiles) 10.8
// against 9.3, 12800 x 384 x 1536 37.4 against 36.5.
constexpr int kKHalvesBelow = 256;
template <int ADT, int BDT, int MT, int LN>
static void launch_gemm(const GemmArgs& g, unsigned tiles, hipStream_t stream) {
  if (tiles < (unsigned)kKHalvesBelow)
    hipLaunchKernelGGL((gemm_nt_kernel<ADT, BDT, MT, kGemmBM, kGemmBN, 2, LN>), dim3(tiles), dim3(512), 0, stream, g);
  else
    hipLaunchKernelGGL((gemm_nt_kernel<ADT, BDT, MT, kGemmBM, kGemmBN, 1, LN>), dim3(tiles), dim3(256), 0, stream, g);
}
static int out_ksplit(int64_t M, int d, int hidden) {
  const int64_t wgs = ((M + kGemmBM - 1) / kGemmBM) * (d / kGemmBN);
  int s = 1;
  while (wgs * s < 64 && s < 8 && hidden / 64 >= 2 * s * KB) s *= 2;
  return s;
}

struct SwigluLayout {
  size_t h_off, part_off, total;
};

static SwigluLayout swiglu_layout(int64_t M, int d, int64_t hidden) {
  auto a256 = [](size_t x) { return (x + 255) & ~(size_t)255; };
  SwigluLayout l;
  l.h_off = 0;
  l.part_off = a256((size_t)M * hidden * 2);
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
  // both launches number their work-groups with 32-bit ints
  const int64_t tiles = (int64_t)a->B * ((a->H + kFH - 1) / kFH) * ((a->W + kFW - 1) / kFW);
  if (tiles * (a->hidden / kFN) > 0x7fffffff || ((M + kGemmBM - 1) / kGemmBM) * (a->d / kGemmBN) * 8 > 0x7fffffff)
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
  if (a->residual) {  // read-only like the inputs, or y itself (each element read, then written, by one thread)
    if (reinterpret_cast<uintptr_t>(a->residual) & 15u) return GTR_ERR_UNSUPPORTED;
    const R rr = rng(a->residual, (size_t)M * a->d * dtype_size(a->y_dtype));
    if ((a->residual != a->y && ovl(rr, ry)) || ovl(rr, rw)) return GTR_ERR_ALIAS;
  }
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
  _Float16* Hb = reinterpret_cast<_Float16*>(ws + lay.h_off);
  const bool bf = a->dtype == GTR_BF16;

  const GatedConvArgs gc{a->x, a->w_gate, a->w_value, a->conv_w, a->conv_b, Hb, a->H, a->W, a->d, a->hidden, a->B};
  const int64_t tiles = (int64_t)a->B * ((a->H + kFH - 1) / kFH) * ((a->W + kFW - 1) / kFW);
  const dim3 grid1((unsigned)(tiles * (a->hidden / kFN)));
  if (bf)
    hipLaunchKernelGGL(gated_conv_kernel<GTR_BF16>, grid1, dim3(256), 0, stream, gc);
  else
    hipLaunchKernelGGL(gated_conv_kernel<GTR_F16>, grid1, dim3(256), 0, stream, gc);
  if (hipGetLastError() != hipSuccess) return GTR_ERR_HIP;

  const int ks = out_ksplit(M, a->d, a->hidden);
  float* part = reinterpret_cast<float*>(ws + lay.part_off);
  GemmArgs g3{Hb, a->w_out, a->y, part, (int)M, a->d, a->hidden, a->y_dtype, ks, nullptr, ks == 1 ? a->residual : nullptr};
  const unsigned tiles3 = (unsigned)(((M + kGemmBM - 1) / kGemmBM) * (a->d / kGemmBN) * ks);
  if (bf)
    launch_gemm<GTR_F16, GTR_BF16, GTR_F16, 0>(g3, tiles3, stream);
  else
    launch_gemm<GTR_F16, GTR_F16, GTR_F16, 0>(g3, tiles3, stream);
  if (hipGetLastError() != hipSuccess) return GTR_ERR_HIP;
  if (ks > 1) {
    const int64_t n4 = M * a->d / 4;
    hipLaunchKernelGGL(ksplit_reduce_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream, part, a->y,
                       n4, ks, (int)a->y_dtype, a->residual);
  }
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}

// ---------------------------------------------------------------------------
// gtr_gemm: C = A B^T (+ bias) (+ res) on gemm_nt_kernel, 64 x 64 tiles, no
// K split (the block's products have K = d or 64).
// ---------------------------------------------------------------------------
static gtr_status gemm_check(const gtr_gemm_args* a) {
  if (a->M <= 0 || a->N <= 0 || a->K <= 0 || a->a_tokens < 0 || a->c_tokens < 0) return GTR_ERR_SHAPE;
  if (a->N % 64 || a->K % 64) return GTR_ERR_UNSUPPORTED;
  if (a->a_tokens && a->M % a->a_tokens) return GTR_ERR_SHAPE;
  if (a->c_tokens) {
    if (a->c_heads <= 0 || a->c_head_dim <= 0 || a->M % a->c_tokens) return GTR_ERR_SHAPE;
    if (a->c_head_dim % 4 || a->N % ((int64_t)a->c_heads * a->c_head_dim) || a->res) return GTR_ERR_UNSUPPORTED;
  }
  if ((a->a_dtype != GTR_F16 && a->a_dtype != GTR_BF16) || a->b_dtype != a->a_dtype) return GTR_ERR_UNSUPPORTED;
  if (a->c_dtype != GTR_F16 && a->c_dtype != GTR_BF16 && a->c_dtype != GTR_F32) return GTR_ERR_UNSUPPORTED;
  if (a->row_norm && (a->row_norm != 1 || a->a_tokens || !(a->row_norm_eps >= 0.f && a->row_norm_eps < 1e30f)))
    return GTR_ERR_UNSUPPORTED;
  if (a->M > 0x7fffffff - 128 || ((a->M + kGemmBM - 1) / kGemmBM) * (a->N / kGemmBN) > 0x7fffffff)
    return GTR_ERR_SHAPE;
  if (!a->a || !a->b || !a->c) return GTR_ERR_NULL;
  const uintptr_t mis = reinterpret_cast<uintptr_t>(a->a) | reinterpret_cast<uintptr_t>(a->b) |
                        reinterpret_cast<uintptr_t>(a->c) | reinterpret_cast<uintptr_t>(a->bias) |
                        reinterpret_cast<uintptr_t>(a->res);
  if (mis & 15u) return GTR_ERR_UNSUPPORTED;
  const size_t es = dtype_size(a->a_dtype);
  auto ovl = [](const void* p, size_t pb, const void* q, size_t qb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(p), y = reinterpret_cast<uintptr_t>(q);
    return q && x < y + qb && y < x + pb;
  };
  const size_t cb = (size_t)a->M * a->N * dtype_size(a->c_dtype);
  // C may be res itself (an in-place residual: each element is read, then
  // written, by one thread), not any other input
  if (ovl(a->c, cb, a->a, (size_t)a->M * a->K * es) || ovl(a->c, cb, a->b, (size_t)a->N * a->K * es) ||
      ovl(a->c, cb, a->bias, (size_t)a->N * 4) || (a->res != a->c && ovl(a->c, cb, a->res, cb)))
    return GTR_ERR_ALIAS;
  return GTR_OK;
}

extern "C" gtr_status gtr_gemm(const gtr_gemm_args* a, hipStream_t stream) {
  if (!a) return GTR_ERR_NULL;
  const gtr_status st = gemm_check(a);
  if (st != GTR_OK) return st;
  GemmArgs g{a->a, a->b, a->c, nullptr, (int)a->M, a->N, a->K, (int)a->c_dtype, 1, a->bias, a->res,
             a->a_tokens, a->c_tokens, a->c_tokens ? a->c_heads : 0, a->c_tokens ? a->c_head_dim : 0,
             a->row_norm ? a->row_norm_eps : 0.f, 0};
  const unsigned tiles = (unsigned)(((a->M + kGemmBM - 1) / kGemmBM) * (a->N / kGemmBN));
  if (a->a_dtype == GTR_BF16) {
    if (a->row_norm)
      launch_gemm<GTR_BF16, GTR_BF16, GTR_BF16, 1>(g, tiles, stream);
    else
      launch_gemm<GTR_BF16, GTR_BF16, GTR_BF16, 0>(g, tiles, stream);
  } else {
    if (a->row_norm)
      launch_gemm<GTR_F16, GTR_F16, GTR_F16, 1>(g, tiles, stream);
    else
      launch_gemm<GTR_F16, GTR_F16, GTR_F16, 0>(g, tiles, stream);
  }
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}
