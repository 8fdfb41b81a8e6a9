// One-launch chunkwise GLA forward for 16-bit inputs (fp16 / bf16) on gfx950,
// chunk size 64.
//
// The method, its numerics and its hand-off protocol are those of the
// one-launch kernel in gla_fwd.hip (paper Sec. 3.3: Eq. chunk_boundary_main and
// the chunk-output formula; the look-back and its bounded waits are shared
// through gla_common.h). What differs is the layout, chosen for the matrix
// cores and for few vector instructions:
//  * Tiles that a product needs token-contiguous (v for the summary and for
//    P V, k 2^(T_R - a) for the summary, S_[c] for the readout) are written to
//    LDS in their natural row-major form with 16-byte stores and read back with
//    the transposing LDS read ds_read_b64_tr_b16: 16 lanes that point at the
//    rows m = 0..3 and the column quads q = 0..3 of a 4 x 16 block receive, lane
//    i, the column i of those four rows.
//  * The outputs are computed transposed, O^T = V^T P^T + S^T Qt^T, so each
//    lane ends with four consecutive value columns of one token row, which it
//    stores straight to memory; no output staging.
//  * The gate's cumulative sums are kept in base-2 units, so every factor is
//    one hardware exp2.
//  * The q operand is q 2^(a_r) (a_r: the inclusive sum of the log2-decays
//    within the 16-token sub-chunk, <= 0); the off-diagonal score blocks scale
//    it by 2^(sum of the totals of the sub-chunks in between) and the diagonal
//    block by the mid-point factor 2^(-T_R/2), every exponent bounded as in
//    gla_fwd.hip.
#include <hip/hip_runtime.h>

#include "gla_common.h"
#include "gtr.h"
#include "gtr_device.h"
#include "gtr_internal.h"

namespace gtr {

constexpr float kLog2e = 1.4426950408889634f;

typedef short s16x4 __attribute__((ext_vector_type(4)));

// Four 16-bit elements through the transposing LDS read (see the file header
// for the lane layout). `p` is this lane's LDS address (8-byte aligned).
__device__ __forceinline__ h4 ld_tr(const _Float16* p) {
  return __builtin_bit_cast(
      h4, __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p)));
}
__device__ __forceinline__ h8 cat(const h4& a, const h4& b) { return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7); }
__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int DK, int DV, int C, int IN, int OCC>
struct Lean {
  static_assert(IN == GTR_F16 || IN == GTR_BF16, "16-bit inputs only");
  static_assert(C == 64, "chunk 64 only");
  static constexpr bool F16 = true;  // fp16 products and fp16 summaries (shared look-back)
  static constexpr int kLookRegs = OCC >= 4 ? 40 : 80;  // registers of loads per look-back batch
  static constexpr int kDK = DK, kDV = DV;
  static constexpr int NW = C / 16;
  static constexpr int NT = NW * kWave;
  static constexpr int KS = DK / 32;  // 32-wide key steps
  static constexpr int VS = DV / 32;  // 32-wide value steps
  static constexpr int KB = DK / 16;  // 16-wide key blocks
  static constexpr int VB = DV / 16;  // 16-wide value blocks
  static constexpr int RP = DK + 8;   // row pitch (elements) of the key tile
  static constexpr int VP = DV + 8;   // row pitch of the value tile
  static constexpr int SPp = DV + 8;  // row pitch of the state tile
  static constexpr int NF = NW + 2;   // factor rows per sub-chunk
  static constexpr int RS = 2 * DK;   // chunk record stride (floats): (d_c[i], scale) pairs
  static constexpr int SQ8 = DK * DV / 8;
  static constexpr int SPER = (SQ8 + NT - 1) / NT;
  static constexpr int TPR = DV / (8 * SPER);
  static constexpr int NTILE = KB * VB / NW;  // summary tiles per wave, all in value block w % VB
  static_assert(DV % (8 * SPER) == 0 && NW % VB == 0 && (KB * VB) % NW == 0, "tile split");
  // factor rows
  static constexpr int kFq = 0;    // 2^(sum of the totals before R): readout
  static constexpr int kFk = 1;    // 2^(sum of the totals after R): summary
  static constexpr int kFh = 2;    // 2^(-T_R / 2): diagonal mid-point
  static constexpr int kFoff = 3;  // + J: 2^(sum of the totals between J and R), J < R

  struct Smem {
    union alignas(16) {
      _Float16 ke[C * RP];   // k 2^(T_R - a), token-major
      _Float16 st[DK * SPp];  // S_[c] / tsc, key-dim-major (after the look-back)
    };
    alignas(16) _Float16 v[C * VP];  // v (fp16), token-major
    float T[NW][DK];         // sub-chunk totals of the log2-decays
    float F[NW][NF][DK];     // factors per sub-chunk and key dim
    float Pt[NW][16][17];    // exact diagonal blocks
    float M[NW][2];          // per wave: max |q|, |k|; max |v|
    float smax[NW];
    float dc[DK];
    int okw[NW];
  };

  int w, lane, tr, g, r;
  float qh[KS][8];   // q 2^(a_r)
  float ke[KS][8];   // k 2^(T_R - a_r)
  h8 qt[KS];         // q 2^(A_r), the readout operand
  float spanmax;     // wave-uniform: widest log2-decay across the sub-chunk
  float absmax;      // wave-uniform: largest |q|, |k| of the sub-chunk
  float usc;         // chunk-uniform: U_c travels as fp16(U_c / usc)
  float pup;         // wave-uniform: the fp16 score tile holds P / pup
  float tsc;         // chunk-uniform: the fp16 state tile holds S_[c] / tsc
  bool range_bad;    // chunk-uniform: a bf16 input lies outside the fp16 range

  // ---- the state in pieces of 8 elements, as in gla_fwd.hip's Chunk ----
  __device__ __forceinline__ static int piece_n0(int m) { return 8 * (SPER * ((int)threadIdx.x % TPR) + m); }
  __device__ __forceinline__ static int piece_i(int) { return (int)threadIdx.x / TPR; }
  __device__ __forceinline__ static bool piece_ok(int) { return (int)threadIdx.x < DK * TPR; }
  __device__ __forceinline__ static uint32_t piece_elem(int m) { return (uint32_t)(piece_i(m) * DV + piece_n0(m)); }

  __device__ __forceinline__ void lanes() {
    w = threadIdx.x >> 6;
    lane = threadIdx.x & 63;
    tr = lane & 15;
    g = lane >> 4;
    r = 16 * w + tr;
  }

  static __device__ __forceinline__ int64_t token(const GlaParams& P, int64_t pos, bool& valid) {
    valid = pos < P.L;
    return valid ? scan_to_spatial(pos, P.H, P.W, P.scan) : 0;
  }

  // LDS address for the transposing read that gives lane (g, i) the column
  // c0 + i of rows r0 + 0..3 of a row-major tile with pitch `pitch`.
  __device__ __forceinline__ const _Float16* tr_addr(const _Float16* tile, int pitch, int r0, int c0) const {
    return tile + (r0 + (tr >> 2)) * pitch + c0 + 4 * (tr & 3);
  }

  // Loads and per-token work; ends with the barrier after which every wave's
  // key and value rows, sub-chunk totals and maxima are in shared memory.
  template <class S>
  __device__ __forceinline__ void load(const GlaParams& P, S& sm, int bh, int c) {
    lanes();
    bool valid;
    const int64_t t = token(P, (int64_t)c * C + r, valid);
    const uint32_t gs = P.gdt == GTR_F32 ? 4 : 2;
    const int64_t L = P.L;
    const char* qb = static_cast<const char*>(P.q) + (int64_t)bh * L * DK * 2;
    const char* kb = static_cast<const char*>(P.k) + (int64_t)bh * L * DK * 2;
    const char* vb = static_cast<const char*>(P.v) + (int64_t)bh * L * P.dvp * 2;
    const char* gb = static_cast<const char*>(P.g) + (int64_t)bh * L * DK * gs;
    const __amdgpu_buffer_rsrc_t qr = make_rsrc(qb, (uint32_t)(L * DK * 2));
    const __amdgpu_buffer_rsrc_t kr = make_rsrc(kb, (uint32_t)(L * DK * 2));
    const __amdgpu_buffer_rsrc_t vr = make_rsrc(vb, (uint32_t)(L * P.dvp * 2));
    const __amdgpu_buffer_rsrc_t gr = make_rsrc(gb, (uint32_t)(L * DK * gs));
    Raw rq[KS], rk[KS], rg[KS], rv[VS];
#pragma unroll
    for (int s = 0; s < KS; ++s) ld_raw_buf(gr, P.gdt, valid ? ((uint32_t)t * DK + 32 * s + 8 * g) * gs : kOutOfRange, rg[s]);
#pragma unroll
    for (int s = 0; s < KS; ++s) ld_raw_buf(kr, IN, valid ? ((uint32_t)t * DK + 32 * s + 8 * g) * 2 : kOutOfRange, rk[s]);
#pragma unroll
    for (int s = 0; s < VS; ++s)
      ld_raw_buf(vr, IN, valid ? ((uint32_t)t * P.dvp + 32 * s + 8 * g) * 2 : kOutOfRange, rv[s]);
#pragma unroll
    for (int s = 0; s < KS; ++s) ld_raw_buf(qr, IN, valid ? ((uint32_t)t * DK + 32 * s + 8 * g) * 2 : kOutOfRange, rq[s]);

    // log2-decays and their inclusive sums within the sub-chunk
    float a[KS][8], tot[KS][8];
    float spn = 0.f, am = 0.f, vm = 0.f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      float gx[8];
      cvt_raw(rg[s], P.gdt, gx);
      if (P.gkind == GTR_GATE_LOGITS) {
#pragma unroll
        for (int e = 0; e < 8; ++e) gx[e] = log_decay(P, gx[e]);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        a[s][e] = row_inclusive_scan(gx[e] * kLog2e);
        tot[s][e] = row_bcast<15>(a[s][e]);
        spn = fmaxf(spn, -tot[s][e]);
      }
    }
    // key rows k 2^(T - a) (exponent <= 0) and the q operand q 2^(a) (<= 0)
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      float kx[8], qx[8];
      cvt_raw(rk[s], IN, kx);
      cvt_raw(rq[s], IN, qx);
      h8 kh;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        am = fmaxf(am, fmaxf(fabsf(kx[e]), fabsf(qx[e])));
        ke[s][e] = kx[e] * fexp2(tot[s][e] - a[s][e]);
        qh[s][e] = qx[e] * fexp2(a[s][e]);
        kh[e] = (_Float16)ke[s][e];
      }
      *reinterpret_cast<h8*>(&sm.ke[r * RP + 32 * s + 8 * g]) = kh;
      if (tr == 15) {
        *reinterpret_cast<f4*>(&sm.T[w][32 * s + 8 * g]) = f4{tot[s][0], tot[s][1], tot[s][2], tot[s][3]};
        *reinterpret_cast<f4*>(&sm.T[w][32 * s + 8 * g + 4]) = f4{tot[s][4], tot[s][5], tot[s][6], tot[s][7]};
      }
    }
    // value rows in fp16
#pragma unroll
    for (int s = 0; s < VS; ++s) {
      h8 vh;
      if constexpr (IN == GTR_F16) {
        vh = __builtin_bit_cast(h8, rv[s].a);
#pragma unroll
        for (int e = 0; e < 8; ++e) vm = fmaxf(vm, fabsf((float)vh[e]));
      } else {
        float vx[8];
        cvt_raw(rv[s], IN, vx);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          vm = fmaxf(vm, fabsf(vx[e]));
          vh[e] = (_Float16)vx[e];
        }
      }
      *reinterpret_cast<h8*>(&sm.v[r * VP + 32 * s + 8 * g]) = vh;
    }
    spanmax = wave_max_uniform(spn);
    absmax = wave_max_uniform(am);
    vm = wave_max_uniform(vm);
    if (lane == 0) {
      sm.M[w][0] = absmax;
      sm.M[w][1] = vm;
    }
    __syncthreads();
    float amx = 0.f, vmx = 0.f;
#pragma unroll
    for (int K = 0; K < NW; ++K) {
      amx = fmaxf(amx, sm.M[K][0]);
      vmx = fmaxf(vmx, sm.M[K][1]);
    }
    // |U_c| <= C max|k| max|v|; NaN maxima (non-finite inputs) count as out of range
    range_bad = IN == GTR_BF16 && !(amx <= kF16Safe && vmx <= kF16Safe);
    usc = exp2i(fp16_exponent((float)C * amx * vmx));
  }

  // Factors per key dim (lane d of each wave for its sub-chunk), d_c, and the
  // readout operand; ends with the barrier after which every wave's factors
  // are visible (the summary scales each sub-chunk's keys by its own).
  template <class S>
  __device__ __forceinline__ void factors(S& sm) {
    if (lane < DK) {
      const int d = lane;
      float tK[NW];
      float before = 0.f, after = 0.f, all = 0.f;
#pragma unroll
      for (int K = 0; K < NW; ++K) {
        tK[K] = sm.T[K][d];
        before += K < w ? tK[K] : 0.f;
        after += K > w ? tK[K] : 0.f;
        all += tK[K];
      }
      sm.F[w][kFq][d] = fexp2(before);
      sm.F[w][kFk][d] = fexp2(after);
      sm.F[w][kFh][d] = fexp2(-0.5f * tK[w]);
      float acc = 0.f;  // sum of the totals strictly between J and w, J = w-1, w-2, ...
#pragma unroll
      for (int J = NW - 2; J >= 0; --J) {
        if (J < w) {
          sm.F[w][kFoff + J][d] = fexp2(acc);
          acc += tK[J];
        }
      }
      if (w == 0) sm.dc[d] = fexp2(all);
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const f4 lo = *reinterpret_cast<const f4*>(&sm.F[w][kFq][32 * s + 8 * g]);
      const f4 hi = *reinterpret_cast<const f4*>(&sm.F[w][kFq][32 * s + 8 * g + 4]);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        qt[s][e] = (_Float16)(qh[s][e] * lo[e]);
        qt[s][e + 4] = (_Float16)(qh[s][e + 4] * hi[e]);
      }
    }
  }

  // U_c to `U` ([DK][DV], fp16(U_c / usc), stores not waited for; `local`:
  // plain stores that stay in this XCD's L2, else agent-coherent ones):
  // U^T = V^T Khat over the chunk's tokens, Khat = k 2^(A_last - A_r) formed
  // from the key rows and the k-hat factor of each token's sub-chunk.
  template <class S>
  __device__ __forceinline__ void summary(const S& sm, void* U, bool local) const {
    const int jb = w % VB;
    f4 acc[NTILE];
#pragma unroll
    for (int m = 0; m < NTILE; ++m) acc[m] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < C / 32; ++ks) {
      const int t0 = 32 * ks + 8 * g;  // this lane's tokens t0 .. t0 + 7
      const h8 A = cat(ld_tr(tr_addr(sm.v, VP, t0, 16 * jb)), ld_tr(tr_addr(sm.v, VP, t0 + 4, 16 * jb)));
      const int Rk = t0 / 16;
#pragma unroll
      for (int m = 0; m < NTILE; ++m) {
        const int ib = (w + NW * m) / VB;
        const h8 Bk = cat(ld_tr(tr_addr(sm.ke, RP, t0, 16 * ib)), ld_tr(tr_addr(sm.ke, RP, t0 + 4, 16 * ib)));
        const _Float16 f = (_Float16)sm.F[Rk][kFk][16 * ib + tr];
        acc[m] = mma32(A, Bk * f, acc[m]);
      }
    }
    // lane (g, i): acc[m][e] = U[16 ib + i][16 jb + 4 g + e]
    const float down = range_bad ? __builtin_nanf("") : 1.f / usc;
    const __amdgpu_buffer_rsrc_t ur = make_rsrc(U, DK * DV * 2);
#pragma unroll
    for (int m = 0; m < NTILE; ++m) {
      const int ib = (w + NW * m) / VB;
      const h4 hv = {(_Float16)(acc[m][0] * down), (_Float16)(acc[m][1] * down), (_Float16)(acc[m][2] * down),
                     (_Float16)(acc[m][3] * down)};
      const int off = ((16 * ib + tr) * DV + 16 * jb + 4 * g) * 2;
      if (local)
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, hv), ur, off, 0, 0);
      else
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, hv), ur, off, 0, kAgentCoherent);
    }
  }

  // Exact diagonal block for sub-chunks whose decay span is too wide for the
  // mid-point factors: P^T[j][r] = sum_d q_r k_j exp(a_r - a_j), j <= r, from
  // the raw q, k, g of the sub-chunk (reloaded; rare).
  __device__ __forceinline__ f4 exact_diagonal(const GlaParams& P, float (*pt)[17], int bh, int c) const {
    bool valid;
    const int64_t t = token(P, (int64_t)c * C + r, valid);
    const int64_t kb = ((int64_t)bh * P.L + t) * DK;
    float qx[KS][8], kx[KS][8], ax[KS][8];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const u32x4 z = {0u, 0u, 0u, 0u};
      Raw rq = Raw{z, z}, rk = Raw{z, z}, rg = Raw{z, z};
      if (valid) {
        ld_raw(P.q, IN, kb + 32 * s + 8 * g, rq);
        ld_raw(P.k, IN, kb + 32 * s + 8 * g, rk);
        ld_raw(P.g, P.gdt, kb + 32 * s + 8 * g, rg);
      }
      float gx[8];
      cvt_raw(rq, IN, qx[s]);
      cvt_raw(rk, IN, kx[s]);
      cvt_raw(rg, P.gdt, gx);
#pragma unroll
      for (int e = 0; e < 8; ++e) gx[e] = log_decay(P, gx[e]);
#pragma unroll
      for (int e = 0; e < 8; ++e) ax[s][e] = row_inclusive_scan(gx[e]);
    }
#pragma unroll 1
    for (int j = 0; j < 16; ++j) {
      const int src = ((g << 4) | j) << 2;
      float acc = 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float kj = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src, __builtin_bit_cast(int, kx[s][e])));
          const float aj = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src, __builtin_bit_cast(int, ax[s][e])));
          acc += (j <= tr) ? qx[s][e] * kj * expf(ax[s][e] - aj) : 0.f;
        }
      acc += __shfl_xor(acc, 16, kWave);
      acc += __shfl_xor(acc, 32, kWave);
      if (g == (j >> 2)) pt[j][tr] = acc;  // P^T[j][r]
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
    __builtin_amdgcn_wave_barrier();
    f4 res;
#pragma unroll
    for (int e = 0; e < 4; ++e) res[e] = pt[4 * g + e][tr];
    return res;
  }

  // Intra-chunk part, transposed: O^T[n][r] = sum_{j <= r} V^T[n][j] P^T[j][r] / pup
  // for this wave's rows r; lane (g, i) gets O[jb][e] = O[r = 16 w + i][16 jb + 4 g + e].
  template <class S>
  __device__ __forceinline__ void intra(const GlaParams& P, S& sm, int bh, int c, f4 (&O)[VB]) {
    f4 PT[NW];
    // off-diagonal blocks J < w: P^T = KE_J (q 2^(a) 2^(sum of the totals between))^T
#pragma unroll
    for (int J = 0; J < NW; ++J) {
      PT[J] = f4{0.f, 0.f, 0.f, 0.f};
      if (J < w) {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const f4 lo = *reinterpret_cast<const f4*>(&sm.F[w][kFoff + J][32 * s + 8 * g]);
          const f4 hi = *reinterpret_cast<const f4*>(&sm.F[w][kFoff + J][32 * s + 8 * g + 4]);
          h8 b;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            b[e] = (_Float16)(qh[s][e] * lo[e]);
            b[e + 4] = (_Float16)(qh[s][e + 4] * hi[e]);
          }
          const h8 a = *reinterpret_cast<const h8*>(&sm.ke[(16 * J + tr) * RP + 32 * s + 8 * g]);
          PT[J] = mma32(a, b, PT[J]);
        }
      }
    }
    // diagonal block: mid-point factors 2^(-T_R/2) on both sides while they
    // stay well inside the fp16 range, float32 operands up to e^30, else exact
    {
      f4 D = {0.f, 0.f, 0.f, 0.f};
      constexpr float kSpanF16b = kSpanF16 * kLog2e, kSpanF32b = kSpanF32 * kLog2e;
      if (spanmax <= kSpanF16b && absmax <= 256.f) {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const f4 lo = *reinterpret_cast<const f4*>(&sm.F[w][kFh][32 * s + 8 * g]);
          const f4 hi = *reinterpret_cast<const f4*>(&sm.F[w][kFh][32 * s + 8 * g + 4]);
          h8 a, b;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            a[e] = (_Float16)(ke[s][e] * lo[e]);
            a[e + 4] = (_Float16)(ke[s][e + 4] * hi[e]);
            b[e] = (_Float16)(qh[s][e] * lo[e]);
            b[e + 4] = (_Float16)(qh[s][e + 4] * hi[e]);
          }
          D = mma32(a, b, D);
        }
      } else if (spanmax <= kSpanF32b) {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const f4 lo = *reinterpret_cast<const f4*>(&sm.F[w][kFh][32 * s + 8 * g]);
          const f4 hi = *reinterpret_cast<const f4*>(&sm.F[w][kFh][32 * s + 8 * g + 4]);
          f8 a, b;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            a[e] = ke[s][e] * lo[e];
            a[e + 4] = ke[s][e + 4] * hi[e];
            b[e] = qh[s][e] * lo[e];
            b[e + 4] = qh[s][e + 4] * hi[e];
          }
          D = mma32(a, b, D);
        }
      } else {
        D = exact_diagonal(P, sm.Pt[w], bh, c);
      }
      // causal mask: lane holds P^T[j = 4g + e][r = tr]
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (4 * g + e > tr) D[e] = 0.f;
#pragma unroll
      for (int J = 0; J < NW; ++J)
        if (J == w) PT[J] = D;
    }
    // power-of-two scale of the fp16 score tile: its largest magnitude below 2^15
    float pm = 0.f;
#pragma unroll
    for (int J = 0; J < NW; ++J)
      if (J <= w)
#pragma unroll
        for (int e = 0; e < 4; ++e) pm = fmaxf(pm, fabsf(PT[J][e]));
    const int ex = fp16_exponent(wave_max_uniform(pm));
    pup = exp2i(ex);
    const float down = exp2i(-ex);
#pragma unroll
    for (int jb = 0; jb < VB; ++jb) O[jb] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int J = 0; J < NW; ++J) {
      if (J <= w) {
        const h4 pb = {(_Float16)(PT[J][0] * down), (_Float16)(PT[J][1] * down), (_Float16)(PT[J][2] * down),
                       (_Float16)(PT[J][3] * down)};
#pragma unroll
        for (int jb = 0; jb < VB; ++jb) O[jb] = mma16(ld_tr(tr_addr(sm.v, VP, 16 * J + 4 * g, 16 * jb)), pb, O[jb]);
      }
    }
  }

  // Grouped look-back, at the last chunk c of a group: the group aggregate
  // A = Diag(d_c) acc + U_c (acc: the summaries of the group's other chunks,
  // decayed to chunk c) and D = run d_c go to the state slot of chunk c - 1 as
  // an fp16 tile with a power-of-two scale per row, and the record (D[i],
  // scale[i]) after it; then the chunk's kFlagGroup. `ok` false (the own
  // group's wait ran out) stores NaN, which poisons every chunk that uses it.
  template <class S>
  __device__ __forceinline__ void publish_aggregate(const GlaParams& P, S& sm, int seq, int c, const void* U,
                                                    const float (&acc)[SPER][8], float run, bool ok,
                                                    unsigned* flag) const {
    const __amdgpu_buffer_rsrc_t ur = make_rsrc(U, DK * DV * 2);
    const __amdgpu_buffer_rsrc_t sr =
        make_rsrc(P.states + ((size_t)seq * P.nchunks + c - 1) * (DK * DV), DK * DV * 4);
    const bool mine = piece_ok(0);
    const int row = mine ? piece_i(0) : 0;
    const float dc = sm.dc[row];
    Piece<true> own[SPER];
#pragma unroll
    for (int m = 0; m < SPER; ++m)
      if (mine) own[m].load(ur, piece_elem(m));
    float a[SPER][8];
    float mx = 0.f;
#pragma unroll
    for (int m = 0; m < SPER; ++m) {
#pragma unroll
      for (int e = 0; e < 8; ++e) a[m][e] = ok ? acc[m][e] * dc : __builtin_nanf("");
      if (mine) own[m].fma_into(a[m], usc);
#pragma unroll
      for (int e = 0; e < 8; ++e) mx = fmaxf(mx, fabsf(a[m][e]));
    }
    // the row's largest |A| over its TPR neighbouring lanes
#pragma unroll
    for (int o = 1; o < TPR; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
    const int ex = fp16_exponent(mx);
    const float inv = exp2i(-ex);
    if (mine) {
#pragma unroll
      for (int m = 0; m < SPER; ++m) {
        h8 h;
#pragma unroll
        for (int e = 0; e < 8; ++e) h[e] = (_Float16)(a[m][e] * inv);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, h), sr, (int)piece_elem(m) * 2, 0,
                                               kAgentCoherent);
      }
      if ((int)threadIdx.x % TPR == 0)
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, f2{run * dc, exp2i(ex)}), sr,
                                              DK * DV * 2 + row * 8, 0, kAgentCoherent);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) __hip_atomic_fetch_or(flag, kFlagGroup, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // S_[c] pieces -> the shared state tile (rows i, fp16 of S / tsc, tsc = 2^e
  // from the largest |S_[c]| of the work-group). No barrier.
  template <class S>
  __device__ __forceinline__ void state_tile(S& sm, const float (&acc)[SPER][8], float wg_max) {
    const int ex = fp16_exponent(wg_max);
    tsc = exp2i(ex);
    const float down = exp2i(-ex);
#pragma unroll
    for (int m = 0; m < SPER; ++m)
      if (piece_ok(m)) {
        h8 h;
#pragma unroll
        for (int e = 0; e < 8; ++e) h[e] = (_Float16)(acc[m][e] * down);
        *reinterpret_cast<h8*>(&sm.st[piece_i(m) * SPp + piece_n0(m)]) = h;
      }
  }

  // O^T += S^T Qt^T (times tsc); reads the shared state tile.
  template <class S>
  __device__ __forceinline__ void readout(const S& sm, f4 (&O)[VB]) const {
#pragma unroll
    for (int jb = 0; jb < VB; ++jb) {
      f4 R = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const h8 A = cat(ld_tr(tr_addr(sm.st, SPp, 32 * s + 8 * g, 16 * jb)),
                         ld_tr(tr_addr(sm.st, SPp, 32 * s + 8 * g + 4, 16 * jb)));
        R = mma32(A, qt[s], R);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) O[jb][e] = fmaf(R[e], tsc, O[jb][e]);
    }
  }

  // The output-gate pre-activation for this lane's row and columns (loaded
  // early, with the other inputs; only when P.gate is set).
  __device__ __forceinline__ void prefetch_gate(const GlaParams& P, int bh, int c, Raw (&rz)[VB]) const {
    bool valid;
    const int64_t t = token(P, (int64_t)c * C + r, valid);
#pragma unroll
    for (int jb = 0; jb < VB; ++jb) {
      const int64_t off = ((int64_t)bh * P.L + t) * P.dvp + 16 * jb + 4 * g;
      if (P.gatedt == GTR_F32) {
        rz[jb].a = *reinterpret_cast<const u32x4*>(static_cast<const float*>(P.gate) + off);
      } else {
        const u32x2 x = *reinterpret_cast<const u32x2*>(static_cast<const unsigned short*>(P.gate) + off);
        rz[jb].a = u32x4{x[0], x[1], 0u, 0u};
      }
    }
  }

  // Scale, the optional output-gate epilogue (Sec. 3.1: u = SiLU(z) * RMSNorm(o)
  // over the DV channels of one token) and the store of this lane's four
  // columns per value block; `poison` stores NaN instead.
  __device__ __forceinline__ void store(const GlaParams& P, int bh, int c, const f4 (&O)[VB], const Raw (&rz)[VB],
                                        bool poison) const {
    bool valid;
    const int64_t t = token(P, (int64_t)c * C + r, valid);
    const float mul = poison ? __builtin_nanf("") : P.scale;
    float x[VB][4];
#pragma unroll
    for (int jb = 0; jb < VB; ++jb)
#pragma unroll
      for (int e = 0; e < 4; ++e) x[jb][e] = mul * O[jb][e];
    if (P.gate) {
      float ss = 0.f;
#pragma unroll
      for (int jb = 0; jb < VB; ++jb)
#pragma unroll
        for (int e = 0; e < 4; ++e) ss = fmaf(x[jb][e], x[jb][e], ss);
      ss += __shfl_xor(ss, 16, kWave);
      ss += __shfl_xor(ss, 32, kWave);
      const float rs = rsqrtf(ss * (1.f / DV) + P.eps);
#pragma unroll
      for (int jb = 0; jb < VB; ++jb) {
        float z[4];
        if (P.gatedt == GTR_F32) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const unsigned u = rz[jb].a[e];
            z[e] = __builtin_bit_cast(float, u);
          }
        } else if (P.gatedt == GTR_F16) {
          const h4 h = __builtin_bit_cast(h4, u32x2{rz[jb].a[0], rz[jb].a[1]});
#pragma unroll
          for (int e = 0; e < 4; ++e) z[e] = (float)h[e];
        } else {
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const unsigned u = rz[jb].a[e];
            z[2 * e] = __builtin_bit_cast(float, u << 16);
            z[2 * e + 1] = __builtin_bit_cast(float, u & 0xffff0000u);
          }
        }
        float wt[4] = {1.f, 1.f, 1.f, 1.f};
        if (P.nw) {
          const f4 q = *reinterpret_cast<const f4*>(P.nw + 16 * jb + 4 * g);
#pragma unroll
          for (int e = 0; e < 4; ++e) wt[e] = q[e];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
          x[jb][e] = z[e] * __builtin_amdgcn_rcpf(1.f + __expf(-z[e])) * (x[jb][e] * rs) * wt[e];
      }
    }
    if (!valid) return;
    const int64_t off = ((int64_t)bh * P.L + t) * P.dvp + 4 * g;
#pragma unroll
    for (int jb = 0; jb < VB; ++jb) store_n<4>(P.o, P.odt, off + 16 * jb, x[jb]);
  }
};

// ---------------------------------------------------------------------------
// The kernel: same grid, flags, look-back, poison and hand-off protocol as
// gla_chain_kernel in gla_fwd.hip.
// ---------------------------------------------------------------------------
// OCC work-groups per CU: at most 168 registers for 3 (look-back batches of
// about 80 registers), 128 for 4 (batches of about 40).
template <int DK, int DV, int C, int IN, int OCC>
__global__ void __launch_bounds__(tile_threads(C)) __attribute__((amdgpu_waves_per_eu(OCC)))
gla_lean_kernel(GlaParams P) {
  typedef Lean<DK, DV, C, IN, OCC> T;
  __shared__ typename T::Smem sm;
  const int NC = P.nchunks;
  const int b = blockIdx.x;
  int row, seq;
  if (P.nxcd > 1) {
    // sequence-per-XCD grid: block b runs on XCD b % nxcd (round-robin
    // dispatch), which holds the sequences x, x + nxcd, ..., chunk major
    const int x = b % P.nxcd, k = b / P.nxcd;
    const int nx = (P.ns - x + P.nxcd - 1) / P.nxcd;
    if (k >= nx * NC) return;  // padding of the XCDs with fewer sequences
    row = k / nx;
    seq = x + P.nxcd * (k - row * nx);
  } else {
    row = b / P.ns;
    seq = b - row * P.ns;
  }
  const int c = P.desc ? NC - 1 - row : row;
  const int bh = seq / P.vparts, vp = seq - bh * P.vparts;
  // the XCD this block runs on; its summary goes through the XCD's L2 when
  // that is the XCD of its sequence (every chunk of the sequence reads it
  // there), through memory otherwise
  const unsigned xcc = __builtin_amdgcn_s_getreg((3 << 11) | 20);  // HW_REG_XCC_ID bits 3:0
  const bool local = P.nxcd > 1 && (int)xcc == b % P.nxcd;
  if (P.vparts > 1) {
    P.v = static_cast<const char*>(P.v) + (int64_t)vp * DV * 2;
    P.o = static_cast<char*>(P.o) + (int64_t)vp * DV * (P.odt == GTR_F32 ? 4 : 2);
    if (P.s_final) P.s_final += vp * DV;
  }
  const int64_t sc = (int64_t)seq * NC + c;
  unsigned* flag = P.flags + (size_t)seq * kMaxChainChunks + c;

  T ch;
  ch.load(P, sm, bh, c);
  ch.factors(sm);
  // the chunk record (d_c, the summary's scale) for the chunks after this one
  if (ch.w == 0 && ch.lane < DK) {
    const u32x2 rv = __builtin_bit_cast(u32x2, f2{sm.dc[ch.lane], ch.usc});
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(P.rec + sc * T::RS, T::RS * 4);
    if (local)
      __builtin_amdgcn_raw_buffer_store_b64(rv, rr, ch.lane * 8, 0, 0);
    else
      __builtin_amdgcn_raw_buffer_store_b64(rv, rr, ch.lane * 8, 0, kAgentCoherent);
  }
  void* U = static_cast<char*>(P.agg) + sc * (DK * DV) * 2;
  ch.summary(sm, U, local);

  // the intra part runs while the summary stores are acknowledged
  f4 O[T::VB];
  ch.intra(P, sm, bh, c, O);
#pragma unroll
  for (int jb = 0; jb < T::VB; ++jb) O[jb] *= ch.pup;
  // every wave's summary tiles (and the record) are acknowledged before the
  // chunk's flag goes up
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0)
    __hip_atomic_fetch_or(flag, kFlagSummary | (local ? kFlagLocal | (xcc << 8) : 0u), __ATOMIC_RELAXED,
                          __HIP_MEMORY_SCOPE_AGENT);

  float acc[T::SPER][8];
  int base;
  if (P.group) {
    // grouped: the summaries of the own group, then (at a group's last chunk)
    // the group's aggregate, then one aggregate per earlier group back to the
    // nearest inclusive state
    const int lo = c - c % kGroup;
    const int st = wait_own_group(P, ch, seq, lo, c, xcc);
#pragma unroll
    for (int m = 0; m < T::SPER; ++m)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[m][e] = 0.f;
    float run = 1.f;
    if (st == 0) sum_items<T, false>(P, seq, c - 1, c - lo, acc, run);
    if (c % kGroup == kGroup - 1 && c < NC - 1) ch.publish_aggregate(P, sm, seq, c, U, acc, run, st == 0, flag);
    int naggs = 0;
    base = st == 0 ? wait_groups(P, ch, seq, c / kGroup, naggs) : st;
    if (base >= -1) {
      sum_items<T, true>(P, seq, c / kGroup - 1, naggs, acc, run);
      add_base<T>(P, seq, base, run, acc);
    }
  } else {
    base = lookback_base(P, ch, seq, c, xcc);
    if (base >= -1) lookback_sum(P, ch, seq, c, base, acc);
  }
  // the output gate's loads overlap the exchange, the state tile and the
  // readout (issued earlier they would hold registers through every phase)
  Raw rz[T::VB];
  if (P.gate) ch.prefetch_gate(P, bh, c, rz);
  const bool okw = base >= -1;
  // one exchange makes the outcome uniform (a wait that ran out, or a NaN
  // state handed over by a poisoned chunk before it, poisons everything this
  // chunk writes) and gives the largest |S_[c]| for the state tile's scale
  bool nan_in = false;
  float mx = 0.f;
#pragma unroll
  for (int m = 0; m < T::SPER; ++m)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (!okw) acc[m][e] = 0.f;
      nan_in = nan_in || acc[m][e] != acc[m][e];
      mx = fmaxf(mx, T::piece_ok(m) ? fabsf(acc[m][e]) : 0.f);
    }
  const bool wave_nan = __builtin_amdgcn_ballot_w64(nan_in) != 0;
  mx = wave_max_uniform(mx);
  if (ch.lane == 0) {
    sm.okw[ch.w] = (okw ? 0 : 1) | (wave_nan ? 2 : 0);
    sm.smax[ch.w] = mx;
  }
  __syncthreads();
  int bad = 0;
  mx = 0.f;
#pragma unroll
  for (int K = 0; K < T::NW; ++K) {
    bad |= sm.okw[K];
    mx = fmaxf(mx, sm.smax[K]);
  }
  const bool ok = (bad & 1) == 0;
  const bool poison = bad != 0 || ch.range_bad;
  if (poison)
#pragma unroll
    for (int m = 0; m < T::SPER; ++m)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[m][e] = __builtin_nanf("");
  if (threadIdx.x == 0 && poison)
    __hip_atomic_fetch_or(P.fault,
                          (ok ? 0u : (base == -3 ? kFaultPlace : kFaultWait)) | (ch.range_bad ? kFaultRange : 0u),
                          __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  // S_[c+1] = Diag(d_c) S_[c] + U_c for the chunks after this one (FUSED), or
  // S_final after the last chunk; U_c is read back from the acknowledged stores
  const int every = P.group ? kGroup : kPublishEvery;
  const bool next = c < NC - 1 ? P.publish != 0 && c % every == every - 1 : P.s_final != nullptr;
  if (next) {
    Piece<true> own[T::SPER];
    const __amdgpu_buffer_rsrc_t ur = make_rsrc(U, DK * DV * 2);
#pragma unroll
    for (int m = 0; m < T::SPER; ++m)
      if (T::piece_ok(m)) own[m].load(ur, T::piece_elem(m));
    float nx[T::SPER][8];
#pragma unroll
    for (int m = 0; m < T::SPER; ++m) {
      const float dc = sm.dc[T::piece_ok(m) ? T::piece_i(m) : 0];
#pragma unroll
      for (int e = 0; e < 8; ++e) nx[m][e] = acc[m][e] * dc;
      if (T::piece_ok(m)) own[m].fma_into(nx[m], ch.usc);
    }
    if (c < NC - 1) {
      const __amdgpu_buffer_rsrc_t sr = make_rsrc(P.states + sc * (DK * DV), DK * DV * 4);
#pragma unroll
      for (int m = 0; m < T::SPER; ++m)
        if (T::piece_ok(m)) {
          coh_store4(sr, T::piece_elem(m) * 4, f4{nx[m][0], nx[m][1], nx[m][2], nx[m][3]});
          coh_store4(sr, T::piece_elem(m) * 4 + 16, f4{nx[m][4], nx[m][5], nx[m][6], nx[m][7]});
        }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (threadIdx.x == 0) __hip_atomic_fetch_or(flag, kFlagInclusive, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
#pragma unroll
      for (int m = 0; m < T::SPER; ++m)
        if (T::piece_ok(m)) {
          f4* dst = reinterpret_cast<f4*>(P.s_final + ((size_t)bh * DK + T::piece_i(m)) * P.dvp + T::piece_n0(m));
          dst[0] = f4{nx[m][0], nx[m][1], nx[m][2], nx[m][3]};
          dst[1] = f4{nx[m][4], nx[m][5], nx[m][6], nx[m][7]};
        }
    }
  }

  if (c > 0 || P.s0) {
    // the key tile (which the state tile overwrites) is dead: every wave is
    // past its summary and intra part (the exchange above)
    ch.state_tile(sm, acc, mx);
    __syncthreads();
    ch.readout(sm, O);
  }
  ch.store(P, bh, c, O, rz, poison);

  if (threadIdx.x == 0) {
    unsigned* done = P.sync + 4 * seq;
    const unsigned prev = __hip_atomic_fetch_add(done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == (unsigned)NC - 1) {  // last one out: leave the flags and the count zeroed
      unsigned* fl = P.flags + (size_t)seq * kMaxChainChunks;
      for (int j = 0; j < NC; ++j) __hip_atomic_store(&fl[j], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

template <int DK, int DV, int IN>
static void lean_set(LeanKernels* o) {
  o->whole3 = reinterpret_cast<const void*>(&gla_lean_kernel<DK, DV, 64, IN, 3>);
  o->whole4 = reinterpret_cast<const void*>(&gla_lean_kernel<DK, DV, 64, IN, 4>);
  if constexpr (DV == 64) {
    o->split3 = reinterpret_cast<const void*>(&gla_lean_kernel<DK, 32, 64, IN, 3>);
    o->split4 = reinterpret_cast<const void*>(&gla_lean_kernel<DK, 32, 64, IN, 4>);
  }
}

template <int IN>
static bool lean_dims(int dk, int dv, LeanKernels* o) {
  if (dk == 64 && dv == 64) return lean_set<64, 64, IN>(o), true;
  if (dk == 32 && dv == 64) return lean_set<32, 64, IN>(o), true;
  if (dk == 32 && dv == 32) return lean_set<32, 32, IN>(o), true;
  return false;
}

bool lean_kernels(int qdt, int dk, int dv, int chunk, LeanKernels* o) {
  *o = LeanKernels{nullptr, nullptr, nullptr, nullptr};
  if (chunk != 64) return false;
  if (qdt == GTR_F16) return lean_dims<GTR_F16>(dk, dv, o);
  if (qdt == GTR_BF16) return lean_dims<GTR_BF16>(dk, dv, o);
  return false;
}

}  // namespace gtr
