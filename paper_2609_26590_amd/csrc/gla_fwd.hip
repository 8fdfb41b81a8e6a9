// Chunkwise key-only GLA forward for gfx950 (MI355X).
//
// Method (paper Sec. 3.3, Eq. chunk_boundary_main, and the chunk-output formula
// that follows it): the token sequence of one head, in scan order, is cut into
// chunks of C tokens. For chunk c with cumulative log-decay A_r = sum_{i<=r} g_i:
//   U_c  = sum_r (k_r * exp(A_last - A_r))^T v_r          (chunk summary)
//   d_c  = exp(A_last)                                     (chunk decay)
//   S_[c+1] = Diag(d_c) S_[c] + U_c                        (boundary states)
//   o_r  = scale * ( (q_r * exp(A_r)) S_[c]
//                    + sum_{j<=r} (sum_i q_r[i] k_j[i] exp(A_r[i]-A_j[i])) v_j )
//
// Numerics differ from the paper's q*exp(A), k*exp(-A) factorisation, which
// overflows half precision as soon as |A| > 11. The chunk is split into
// 16-token sub-chunks R (one wave each). Local cumulative sums a_r (within R),
// sub-chunk totals T_R and the value g0_R of a at the first token of R are kept
// in fp32; every exponent is a sum of these small terms, never a difference of
// two large cumulative sums.
//   * Off-diagonal score blocks (J < R) use q_r*exp(a_r - g0_R) and
//     k_j*exp(T_J - a_j)*exp(g0_R + sum_{J<K<R} T_K): every exponent <= 0, so
//     both matrix operands are bounded by |q| and |k|.
//   * Diagonal blocks use a mid-point reference, both factors within
//     exp(+-span/2), span = decay across the 16 tokens: fp16 operands for
//     span <= kSpanF16, float32 operands for span <= kSpanF32, and the exact
//     per-element exp(a_r - a_j) on the vector ALUs beyond that.
//   * The summary uses k_j exp(A_last - A_j) and the readout q_r exp(A_r), both
//     with exponents <= 0.
// Half-precision operands that are not bounded by an input (the score tile P,
// the summaries U_c, the boundary state S_[c]) are scaled by powers of two
// before they are rounded to fp16 (per wave, per chunk and per state column
// respectively), and the scale is undone in float32: exact, and no overflow
// whatever the magnitudes the inputs' range allows.
//
// Schedules:
//   * one launch (look-back): one work-group per (sequence, chunk). It stores
//     its summary U_c and d_c and raises its chunk's flag to 1 (aggregate
//     ready), then finds S_[c] by looking back over the chunks before it,
//     nearest first: the summary of every chunk whose flag is 1, until it meets
//     a chunk whose flag is 2 (its inclusive state S_[j+1] is ready) or the start
//     of the sequence (S_0). With `publish` it then stores S_[c+1] in float32 and
//     raises its flag to 2, which lets the chunks after it stop there. Without
//     `publish` every chunk reads all the summaries before it (the paper's
//     inline-prefix form for short sequences). Every wait is bounded: a
//     work-group that gives up marks the call's fault word and writes NaN in
//     place of everything that depends on it.
//   * staged: summary kernel -> boundary-state scan kernel -> output kernel.
// Hand-offs between work-groups are agent-coherent (cache policy sc1) stores
// and loads; a work-group waits for its stores to be acknowledged (vmcnt(0))
// before it raises a flag. No release/acquire fence is used: on this GPU those
// write back / invalidate the whole L2 of the XCD.
// Hand-off precision: with fp16/bf16 inputs the summaries travel in fp16 with a
// power-of-two scale per chunk; inclusive states travel in float32 (so no
// rounding accumulates along the chain of chunks); every combination
// accumulates in float32, and S_final is float32. With float32 inputs
// everything is float32.
#include <hip/hip_runtime.h>

#include <mutex>
#include <type_traits>

#include "gla_common.h"
#include "gtr.h"
#include "gtr_device.h"
#include "gtr_internal.h"

namespace gtr {

// One chunk of one sequence: C tokens, one wave per 16-token sub-chunk.
// IN is the dtype of q, k, v (GTR_F32 / GTR_F16 / GTR_BF16); DV the value
// columns of this work-group (d_v, or d_v / 2 under the value split).
template <int DK, int DV, int C, int IN>
struct Chunk {
  static constexpr int kLookRegs = 80;  // registers of loads per look-back batch
  static constexpr bool F16 = IN != GTR_F32;  // matrix operands: fp16 (else float32)
  static constexpr int kDK = DK, kDV = DV;
  static constexpr int NW = C / 16;
  static constexpr int NT = NW * kWave;
  static constexpr int KS = DK / 32;
  static constexpr int VS = DV / 32;
  static constexpr int KP = DK + 4;  // padded fp32 row pitch (k rows / output rows)
  static constexpr int OP = DV + 4;
  static constexpr int BUFW = KP > OP ? KP : OP;
  static constexpr int TP = F16 ? C + 8 : C + 4;    // transposed-tile pitch (elements)
  static constexpr int SP = F16 ? DK + 8 : DK + 4;  // boundary-state tile pitch
  static constexpr int NF = 3 + (NW > 1 ? NW - 1 : 1);  // factor-table rows per wave
  static constexpr int RS = 2 * DK;                 // record stride (floats): (d_c[i], scale) pairs
  // summaries and boundary states are [DK][DV] (key dim i, value column n), in
  // 8-element pieces: piece p holds row i = p / (DV/8), columns 8 (p % (DV/8)) ..
  static constexpr int SQ8 = DK * DV / 8;
  static constexpr int SPER = (SQ8 + NT - 1) / NT;  // pieces per thread
  static constexpr int TPR = DV / (8 * SPER);       // threads per state row
  static_assert(DV % (8 * SPER) == 0, "the pieces of one thread lie in one row");
  typedef typename Op<F16>::elem E;
  typedef typename Op<F16>::frag8 F8;
  typedef typename Op<F16>::frag4 F4;

  // Shared memory of the one-launch kernel (every part). The staged kernels
  // use the subsets below: the summary kernel has no k rows, state or
  // diagonal staging, the output kernel no k-hat tile.
  struct Smem {
    float buf[C * BUFW];   // k*exp(T-a) rows [C][KP]; later the output tile [C][OP]
    // three tiles that are never live at once share one region, each phase
    // separated from the next by a barrier: the k-hat tile (factors, summary),
    // the exact diagonal staging (intra), the state tile (readout)
    union {
      E kT[DK * TP];         // (k * exp(A_last - A_r))^T  [DK][TP]
      float Pt[NW][16][17];  // exact diagonal blocks, P^T staging
      E sT[DV * SP];         // S_[c]^T                   [DV][SP]
    };
    E vT[DV * TP];         // v^T                       [DV][TP]
    float T[NW][DK];       // sub-chunk totals of g
    float G0[NW][DK];      // g at the first token of each sub-chunk
    float F[NW][NF][DK];   // per-wave factor table (rows kFq, kFk, kFh, kFoff + J)
    float M[NW][2];        // per-wave maxima of |q|,|k| and of |v|
    float smax[NW];        // per-wave maxima of |S_[c]|
    float dc[DK];          // d_c
    int okw[NW];           // per wave: 1 its look-back gave up, 2 it met a NaN state
  };
  struct SmemSummary {
    E kT[DK * TP];
    E vT[DV * TP];
    float T[NW][DK];
    float G0[NW][DK];
    float F[NW][NF][DK];
    float M[NW][2];
    float dc[DK];
  };
  struct SmemOutput {
    float buf[C * BUFW];
    E vT[DV * TP];
    E sT[DV * SP];  // written before the intra part, read after it: not shared with Pt
    float T[NW][DK];
    float G0[NW][DK];
    float F[NW][NF][DK];
    float Pt[NW][16][17];
    float M[NW][2];
    float smax[NW];
  };
  // rows of the factor table of sub-chunk R, per dimension d:
  static constexpr int kFq = 0;    // exp(A before R + g0_R): q readout factor
  static constexpr int kFk = 1;    // exp(sum of totals after R): k-hat factor
  static constexpr int kFh = 2;    // exp((g0_R - T_R) / 2): diagonal mid-point factor
  static constexpr int kFoff = 3;  // + J: exp(g0_R + sum_{J<K<R} T_K), J < R

  int w, lane, tr, gq, r;
  float qh[KS][8];  // q * exp(a - g0)
  float ke[KS][8];  // k * exp(T - a)
  float g0[KS][8];  // a at the first token of this sub-chunk (= g there)
  float tw[KS][8];  // total of g over this sub-chunk
  float qt[KS][8];  // q * exp(A_r), the readout operand (set by factors())
  float spanmax;    // wave-uniform: widest decay span of this sub-chunk
  float absmax;     // wave-uniform: largest |q|, |k| of this sub-chunk
  float usc;        // chunk-uniform: U_c is handed over as fp16(U_c / usc) (1 for float32 inputs)
  float pup;        // wave-uniform: the fp16 score tile holds P / pup
  float tsc;        // chunk-uniform: the fp16 state tile holds S_[c]^T / tsc
  bool range_bad;   // chunk-uniform: a bf16 input lies outside the fp16 range

  __device__ __forceinline__ int dim(int s, int e) const { return 32 * s + 8 * gq + e; }

  __device__ __forceinline__ void lanes() {
    w = threadIdx.x >> 6;
    lane = threadIdx.x & 63;
    tr = lane & 15;
    gq = lane >> 4;
    r = 16 * w + tr;
  }

  // Spatial token index of scan position `pos` (0 past the end) and whether
  // the position exists.
  static __device__ __forceinline__ int64_t token(const GlaParams& P, int64_t pos, bool& valid) {
    valid = pos < P.L;
    return valid ? scan_to_spatial(pos, P.H, P.W, P.scan) : 0;
  }

  // Loads and per-token work. Writes v^T, the sub-chunk totals, the per-wave
  // maxima and (ROWS) the k*exp(T-a) rows. Ends with a barrier, after which the
  // chunk-uniform summary scale and range flag are set.
  template <bool ROWS, class S>
  __device__ __forceinline__ void load(const GlaParams& P, S& sm, int bh, int c) {
    lanes();
    bool valid;
    const int64_t t = token(P, (int64_t)c * C + r, valid);

    // issue every load before converting any of them; a position past the end
    // of the sequence reads zeros through the descriptors' range check
    constexpr uint32_t ES = F16 ? 2 : 4;
    const uint32_t gs = P.gdt == GTR_F32 ? 4 : 2;
    const int64_t L = P.L;
    const char* qb = static_cast<const char*>(P.q) + (int64_t)bh * L * DK * ES;
    const char* kb = static_cast<const char*>(P.k) + (int64_t)bh * L * DK * ES;
    const char* vb = static_cast<const char*>(P.v) + (int64_t)bh * L * P.dvp * ES;
    const char* gb = static_cast<const char*>(P.g) + (int64_t)bh * L * DK * gs;
    const __amdgpu_buffer_rsrc_t qr = make_rsrc(qb, (uint32_t)(L * DK * ES));
    const __amdgpu_buffer_rsrc_t kr = make_rsrc(kb, (uint32_t)(L * DK * ES));
    const __amdgpu_buffer_rsrc_t vr = make_rsrc(vb, (uint32_t)(L * P.dvp * ES));
    const __amdgpu_buffer_rsrc_t gr = make_rsrc(gb, (uint32_t)(L * DK * gs));
    Raw rq[KS], rk[KS], rg[KS], rv[VS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const uint32_t e = (uint32_t)t * DK + 32 * s + 8 * gq;
      ld_raw_buf(qr, IN, valid ? e * ES : kOutOfRange, rq[s]);
      ld_raw_buf(kr, IN, valid ? e * ES : kOutOfRange, rk[s]);
      ld_raw_buf(gr, P.gdt, valid ? e * gs : kOutOfRange, rg[s]);
    }
#pragma unroll
    for (int s = 0; s < VS; ++s)
      ld_raw_buf(vr, IN, valid ? ((uint32_t)t * P.dvp + 32 * s + 8 * gq) * ES : kOutOfRange, rv[s]);

    // v^T tile
    float vmax = 0.f;
#pragma unroll
    for (int s = 0; s < VS; ++s) {
      float x[8];
      cvt_raw(rv[s], IN, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        vmax = fmaxf(vmax, fabsf(x[e]));
        sm.vT[(32 * s + 8 * gq + e) * TP + r] = (E)x[e];
      }
    }

    float smax = 0.f, amax = 0.f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      float qx[8], kx[8], gx[8];
      cvt_raw(rq[s], IN, qx);
      cvt_raw(rk[s], IN, kx);
      cvt_raw(rg[s], P.gdt, gx);
#pragma unroll
      for (int e = 0; e < 8; ++e) gx[e] = log_decay(P, gx[e]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // local inclusive cumulative sum over the 16 tokens of this sub-chunk
        const float a = row_inclusive_scan(gx[e]);
        const float T = row_bcast<15>(a);
        const float f = row_bcast<0>(a);
        g0[s][e] = f;
        tw[s][e] = T;
        smax = fmaxf(smax, f - T);
        amax = fmaxf(amax, fmaxf(fabsf(qx[e]), fabsf(kx[e])));
        qh[s][e] = qx[e] * gexp<F16>(a - f);  // exp(A_r - A_first) <= 1
        ke[s][e] = kx[e] * gexp<F16>(T - a);  // exp(A_last(R) - A_r) <= 1
      }
      if (tr == 0) {
        *reinterpret_cast<f4*>(&sm.T[w][32 * s + 8 * gq]) = f4{tw[s][0], tw[s][1], tw[s][2], tw[s][3]};
        *reinterpret_cast<f4*>(&sm.T[w][32 * s + 8 * gq + 4]) = f4{tw[s][4], tw[s][5], tw[s][6], tw[s][7]};
        *reinterpret_cast<f4*>(&sm.G0[w][32 * s + 8 * gq]) = f4{g0[s][0], g0[s][1], g0[s][2], g0[s][3]};
        *reinterpret_cast<f4*>(&sm.G0[w][32 * s + 8 * gq + 4]) = f4{g0[s][4], g0[s][5], g0[s][6], g0[s][7]};
      }
      if constexpr (ROWS) {
        *reinterpret_cast<f4*>(&sm.buf[r * KP + 32 * s + 8 * gq]) = f4{ke[s][0], ke[s][1], ke[s][2], ke[s][3]};
        *reinterpret_cast<f4*>(&sm.buf[r * KP + 32 * s + 8 * gq + 4]) = f4{ke[s][4], ke[s][5], ke[s][6], ke[s][7]};
      }
    }
    spanmax = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, wave_max_uniform(smax))));
    absmax = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, wave_max_uniform(amax))));
    const float vm = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, wave_max_uniform(vmax))));
    if (lane == 0) {
      sm.M[w][0] = absmax;
      sm.M[w][1] = vm;
    }
    __syncthreads();
    float am = 0.f, vv = 0.f;
#pragma unroll
    for (int K = 0; K < NW; ++K) {
      am = fmaxf(am, sm.M[K][0]);
      vv = fmaxf(vv, sm.M[K][1]);
    }
    // |U_c| <= C max|k| max|v|; NaN maxima (non-finite inputs) count as out of range
    range_bad = IN == GTR_BF16 && !(am <= kF16Safe && vv <= kF16Safe);
    usc = F16 ? exp2i(fp16_exponent((float)C * am * vv)) : 1.f;
  }

  // This lane's 8 consecutive dims of factor-table row `row`, for K-step s.
  template <class S>
  __device__ __forceinline__ void frow(const S& sm, int row, int s, float (&x)[8]) const {
    const f4 lo = *reinterpret_cast<const f4*>(&sm.F[w][row][32 * s + 8 * gq]);
    const f4 hi = *reinterpret_cast<const f4*>(&sm.F[w][row][32 * s + 8 * gq + 4]);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[e] = lo[e];
      x[e + 4] = hi[e];
    }
  }

  // Chunk-level factors. Lane d of each wave fills dimension d of its
  // sub-chunk's factor table (one exponential per factor and dimension); the
  // wave then reads back what its lanes need. READOUT: qt = q exp(A_r).
  // SUMMARY: the transposed k-hat tile, and the chunk record (d_c and the
  // summary scale, written by wave 0 through `rec` unless it is null) and d_c
  // in shared memory, followed by a barrier.
  template <bool READOUT, bool SUMMARY, class S>
  __device__ __forceinline__ void factors(S& sm, float* rec) {
    if (lane < DK) {
      const int d = lane;
      float tK[NW];
      float before = 0.f, after = 0.f;
#pragma unroll
      for (int K = 0; K < NW; ++K) {
        tK[K] = sm.T[K][d];
        before += K < w ? tK[K] : 0.f;
        after += K > w ? tK[K] : 0.f;
      }
      const float g0d = sm.G0[w][d];
      sm.F[w][kFq][d] = gexp<F16>(before + g0d);
      sm.F[w][kFk][d] = gexp<F16>(after);
      sm.F[w][kFh][d] = gexp<F16>(0.5f * (g0d - sm.T[w][d]));
      float acc = g0d;  // exp(g0_R + sum_{J<K<R} T_K) for J = R-1, R-2, ...
#pragma unroll
      for (int J = NW - 2; J >= 0; --J) {
        if (J < w) {
          sm.F[w][kFoff + J][d] = gexp<F16>(acc);
          acc += tK[J];
        }
      }
      if (SUMMARY && w == 0) {
        const float dc = gexp<F16>(before + sm.T[0][d] + after);
        if (rec) *reinterpret_cast<f2*>(rec + 2 * d) = f2{dc, usc};
        if constexpr (std::is_same<S, Smem>::value || std::is_same<S, SmemSummary>::value) sm.dc[d] = dc;
      }
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the table writes of this wave are done
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      float f[8];
      if constexpr (READOUT) {
        frow(sm, kFq, s, f);
#pragma unroll
        for (int e = 0; e < 8; ++e) qt[s][e] = qh[s][e] * f[e];
      }
      if constexpr (SUMMARY) {
        frow(sm, kFk, s, f);
#pragma unroll
        for (int e = 0; e < 8; ++e) sm.kT[dim(s, e) * TP + r] = (E)(ke[s][e] * f[e]);
      }
    }
    if constexpr (SUMMARY) __syncthreads();
  }

  // U_c ([DK][DV], row i = key dim) to `U`: float32 for float32 inputs, else
  // fp16(U / usc); coherent (agent scope) or plain. Computed as U^T = v^T khat,
  // so each lane holds 4 consecutive value columns of one row.
  template <bool COH, class S>
  __device__ __forceinline__ void summary_out(const S& sm, void* U) {
    constexpr int NTI = (DK / 16) * (DV / 16);
    // a power of two (exact); NaN poisons the summary of a chunk with an
    // out-of-range input, and through it every state after the chunk
    const float down = range_bad ? __builtin_nanf("") : 1.f / usc;
    for (int tau = w; tau < NTI; tau += NW) {
      const int ib = tau / (DV / 16), jb = tau % (DV / 16);
      f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < C / 32; ++ks) {
        const F8 a = *reinterpret_cast<const F8*>(&sm.vT[(16 * jb + tr) * TP + 32 * ks + 8 * gq]);
        const F8 b = *reinterpret_cast<const F8*>(&sm.kT[(16 * ib + tr) * TP + 32 * ks + 8 * gq]);
        acc = mma32(a, b, acc);
      }
      // lane holds U^T[16jb + 4gq + e][16ib + tr] = U[16ib + tr][16jb + 4gq + e]
      const int off = (16 * ib + tr) * DV + 16 * jb + 4 * gq;
      if constexpr (F16) {
        const h4 hv = {(_Float16)(acc[0] * down), (_Float16)(acc[1] * down), (_Float16)(acc[2] * down),
                       (_Float16)(acc[3] * down)};
        if constexpr (COH)
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, hv), make_rsrc(U, DK * DV * 2), off * 2, 0,
                                                kAgentCoherent);
        else
          *reinterpret_cast<h4*>(static_cast<_Float16*>(U) + off) = hv;
      } else if constexpr (COH) {
        coh_store4(make_rsrc(U, DK * DV * 4), off * 4, acc);
      } else {
        *reinterpret_cast<f4*>(static_cast<float*>(U) + off) = acc;
      }
    }
  }

  // Exact diagonal block for sub-chunks whose decay span is too wide for the
  // mid-point factors: P[r][j] = sum_d q_r k_j exp(a_r - a_j), j <= r. Rare:
  // the raw q, k and g of the sub-chunk are reloaded and the token loop is kept
  // rolled to keep the code small.
  __device__ __forceinline__ f4 exact_diagonal(const GlaParams& P, float (*pt)[17], int bh, int c) {
    bool valid;
    const int64_t t = token(P, (int64_t)c * C + r, valid);
    const int64_t kb = ((int64_t)bh * P.L + t) * DK;
    float qx[KS][8], kx[KS][8], ax[KS][8];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const u32x4 z = {0u, 0u, 0u, 0u};
      Raw rq = Raw{z, z}, rk = Raw{z, z}, rg = Raw{z, z};
      if (valid) {
        ld_raw(P.q, IN, kb + 32 * s + 8 * gq, rq);
        ld_raw(P.k, IN, kb + 32 * s + 8 * gq, rk);
        ld_raw(P.g, P.gdt, kb + 32 * s + 8 * gq, rg);
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
      const int src = ((gq << 4) | j) << 2;
      float acc = 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float kj = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src, __builtin_bit_cast(int, kx[s][e])));
          const float aj = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src, __builtin_bit_cast(int, ax[s][e])));
          acc += (j <= tr) ? qx[s][e] * kj * gexp<F16>(ax[s][e] - aj) : 0.f;
        }
      acc += __shfl_xor(acc, 16, kWave);
      acc += __shfl_xor(acc, 32, kWave);
      if (gq == (j >> 2)) pt[j][tr] = acc;  // P^T[j][r]
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
    __builtin_amdgcn_wave_barrier();
    f4 res;
#pragma unroll
    for (int e = 0; e < 4; ++e) res[e] = pt[4 * gq + e][tr];
    return res;
  }

  // Intra-chunk part: O = sum_{j<=r} P[r][j] v_j / pup for this wave's 16 rows
  // (16-bit inputs: the score tile is scaled by a power of two before it is
  // rounded to fp16). Needs the k rows written by load<true>().
  template <class S>
  __device__ __forceinline__ void intra(const GlaParams& P, S& sm, int bh, int c, f4 (&O)[DV / 16]) {
    f4 PT[NW];
    F8 qhf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) qhf[s] = Op<F16>::pack8(qh[s]);

    // off-diagonal blocks J < R = w, with the pair factors of the table
#pragma unroll
    for (int J = 0; J < NW; ++J) {
      PT[J] = f4{0.f, 0.f, 0.f, 0.f};
      if (J < w) {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const float* row = &sm.buf[(16 * J + tr) * KP + 32 * s + 8 * gq];
          const f4 lo = *reinterpret_cast<const f4*>(row);
          const f4 hi = *reinterpret_cast<const f4*>(row + 4);
          float fo[8], x[8];
          frow(sm, kFoff + J, s, fo);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            x[e] = lo[e] * fo[e];
            x[e + 4] = hi[e] * fo[e + 4];
          }
          // P^T[j][r] = sum_d (k_j exp(T_J - a_j) Foff)[d] (q_r exp(a_r - g0_R))[d]
          PT[J] = mma32(Op<F16>::pack8(x), qhf[s], PT[J]);
        }
      }
    }

    // diagonal block: fp16 operands only if the mid-point factors keep them well
    // inside fp16 range
    {
      f4 D = {0.f, 0.f, 0.f, 0.f};
      if (F16 && spanmax <= kSpanF16 && absmax <= 256.f) {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          float a[8], b[8], h[8];
          frow(sm, kFh, s, h);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            a[e] = ke[s][e] * h[e];
            b[e] = qh[s][e] * h[e];
          }
          D = mma32(Op<F16>::pack8(a), Op<F16>::pack8(b), D);
        }
      } else if (spanmax <= kSpanF32) {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          f8 a, b;
          float h[8];
          frow(sm, kFh, s, h);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            a[e] = ke[s][e] * h[e];
            b[e] = qh[s][e] * h[e];
          }
          D = mma32(a, b, D);
        }
      } else {
        D = exact_diagonal(P, sm.Pt[w], bh, c);
      }
      // causal mask: lane holds P^T[j = 4gq + e][r = tr]
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (4 * gq + e > tr) D[e] = 0.f;
#pragma unroll
      for (int J = 0; J < NW; ++J)
        if (J == w) PT[J] = D;
    }

    // power-of-two scale of the fp16 score tile: its largest magnitude below 2^15
    pup = 1.f;
    if constexpr (F16) {
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
      for (int J = 0; J < NW; ++J)
#pragma unroll
        for (int e = 0; e < 4; ++e) PT[J][e] *= down;
    }

#pragma unroll
    for (int jb = 0; jb < DV / 16; ++jb) O[jb] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int J = 0; J < NW; ++J) {
      if (J <= w) {
        const F4 a = Op<F16>::pack4(PT[J]);
#pragma unroll
        for (int jb = 0; jb < DV / 16; ++jb) {
          const F4 b = *reinterpret_cast<const F4*>(&sm.vT[(16 * jb + tr) * TP + 16 * J + 4 * gq]);
          O[jb] = mma16(a, b, O[jb]);
        }
      }
    }
  }

  // ---- boundary states in pieces of 8 elements: the SPER pieces of a thread
  // are consecutive columns n0(m) .. n0(m) + 7 of one row i of the [DK][DV]
  // state (TPR threads per row), so one decay per tile serves them all ----
  __device__ __forceinline__ static int piece_n0(int m) { return 8 * (SPER * ((int)threadIdx.x % TPR) + m); }
  __device__ __forceinline__ static int piece_i(int m) { return (int)threadIdx.x / TPR; }
  __device__ __forceinline__ static bool piece_ok(int m) { return (int)threadIdx.x < DK * TPR; }
  __device__ __forceinline__ static uint32_t piece_elem(int m) {
    return (uint32_t)(piece_i(m) * DV + piece_n0(m));
  }

  // S_[c] pieces -> the shared state tile S^T ([DV][SP]). For 16-bit inputs the
  // whole tile is divided by tsc = 2^e, e = fp16_exponent of `wg_max`, the
  // largest |S_[c]| over the work-group. No barrier.
  template <class S>
  __device__ __forceinline__ void state_tile(S& sm, const float (&acc)[SPER][8], float wg_max) {
    float down = 1.f;
    tsc = 1.f;
    if constexpr (F16) {
      const int ex = fp16_exponent(wg_max);
      tsc = exp2i(ex);
      down = exp2i(-ex);
    }
#pragma unroll
    for (int m = 0; m < SPER; ++m)
      if (piece_ok(m)) {
        const int i = piece_i(m), n0 = piece_n0(m);
#pragma unroll
        for (int e = 0; e < 8; ++e) sm.sT[(n0 + e) * SP + i] = (E)(acc[m][e] * down);
      }
  }

  // The largest |S_[c]| of this thread's pieces, over the work-group: one
  // barrier (the staged output kernel; the one-launch kernel folds it into its
  // own exchange).
  template <class S>
  __device__ __forceinline__ float state_max(S& sm, const float (&acc)[SPER][8]) const {
    float mx = 0.f;
#pragma unroll
    for (int m = 0; m < SPER; ++m)
#pragma unroll
      for (int e = 0; e < 8; ++e) mx = fmaxf(mx, piece_ok(m) ? fabsf(acc[m][e]) : 0.f);
    mx = wave_max_uniform(mx);
    if (lane == 0) sm.smax[w] = mx;
    __syncthreads();
    mx = 0.f;
#pragma unroll
    for (int K = 0; K < NW; ++K) mx = fmaxf(mx, sm.smax[K]);
    return mx;
  }

  // O += (q_r exp(A_r)) S_[c]: the tile's product times tsc. Reads the shared
  // state tile.
  template <class S>
  __device__ __forceinline__ void readout(const S& sm, f4 (&O)[DV / 16]) {
    F8 qtf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) qtf[s] = Op<F16>::pack8(qt[s]);
#pragma unroll
    for (int jb = 0; jb < DV / 16; ++jb) {
      f4 R = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const F8 b = *reinterpret_cast<const F8*>(&sm.sT[(16 * jb + tr) * SP + 32 * s + 8 * gq]);
        R = mma32(qtf[s], b, R);
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) O[jb][e] = fmaf(R[e], tsc, O[jb][e]);
    }
  }

  // Stage the output tile through LDS and write whole rows back in spatial order.
  // Gate values of the output-gate epilogue for the rows this thread stores,
  // loaded early (with the other inputs) so that the epilogue does not wait
  // for memory at the end of the kernel. Only when P.gate is set.
  static constexpr int SITER = C * (DV / 8) / NT;  // store iterations per thread
  static constexpr int PIECES = DV / 8;            // 8-element pieces of an output row
  __device__ __forceinline__ void prefetch_gate(const GlaParams& P, int bh, int c, Raw (&rz)[SITER]) const {
#pragma unroll
    for (int it = 0; it < SITER; ++it) {
      const int idx = threadIdx.x + it * NT;
      const int rr = idx / PIECES, pc = idx % PIECES;
      bool valid;
      const int64_t t = token(P, (int64_t)c * C + rr, valid);
      ld_raw(P.gate, P.gatedt, ((int64_t)bh * P.L + t) * P.dvp + 8 * pc, rz[it]);
    }
  }

  // O holds the output rows of this wave (before the scale); `poison` stores
  // NaN instead. BARRIER: wait first until every wave is done with the k rows
  // in buf (which the output tile overwrites).
  template <bool BARRIER, class S>
  __device__ __forceinline__ void store(const GlaParams& P, S& sm, int bh, int c, const f4 (&O)[DV / 16],
                                        const Raw (&rz)[SITER], bool poison) {
    if constexpr (BARRIER) __syncthreads();
    const float mul = poison ? __builtin_nanf("") : P.scale;
#pragma unroll
    for (int jb = 0; jb < DV / 16; ++jb)
#pragma unroll
      for (int e = 0; e < 4; ++e) sm.buf[(16 * w + 4 * gq + e) * OP + 16 * jb + tr] = mul * O[jb][e];
    __syncthreads();
    // C * PIECES is a multiple of NT, so every lane runs the same number of
    // iterations, and the PIECES lanes of a row are consecutive lanes of one wave
    static_assert((C * PIECES) % NT == 0 && kWave % PIECES == 0, "row groups");
#pragma unroll
    for (int it = 0; it < SITER; ++it) {
      const int idx = threadIdx.x + it * NT;
      const int rr = idx / PIECES, pc = idx % PIECES;
      bool valid;
      const int64_t t = token(P, (int64_t)c * C + rr, valid);
      const int64_t off = ((int64_t)bh * P.L + t) * P.dvp + 8 * pc;  // token 0 past the end: in bounds
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = sm.buf[rr * OP + 8 * pc + e];
      if (P.gate) epilogue(P, rz[it], pc, x);
      if (valid) store_n<8>(P.o, P.odt, off, x);
    }
  }

  // Output-gate epilogue (Sec. 3.1): u = SiLU(z) * o / sqrt(mean(o^2) + eps) * w
  // over the DV channels of one token; x holds this lane's 8 channels of o.
  // Called by every lane (the row sum is a cross-lane reduction).
  __device__ __forceinline__ void epilogue(const GlaParams& P, const Raw& rz, int pc, float (&x)[8]) const {
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf(x[e], x[e], ss);
#pragma unroll
    for (int m = 1; m < PIECES; m <<= 1) ss += __shfl_xor(ss, m, kWave);
    const float rs = rsqrtf(ss * (1.f / DV) + P.eps);
    float z[8], wt[8];
    cvt_raw(rz, P.gatedt, z);
    if (P.nw) {
      const f4 lo = *reinterpret_cast<const f4*>(P.nw + 8 * pc);
      const f4 hi = *reinterpret_cast<const f4*>(P.nw + 8 * pc + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        wt[e] = lo[e];
        wt[e + 4] = hi[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) wt[e] = 1.f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = z[e] * __builtin_amdgcn_rcpf(1.f + __expf(-z[e])) * (x[e] * rs) * wt[e];
  }
};

// ---------------------------------------------------------------------------
// staged schedule
// ---------------------------------------------------------------------------
template <int DK, int DV, int C, int IN>
__global__ void __launch_bounds__(tile_threads(C)) gla_summary_kernel(GlaParams P) {
  typedef Chunk<DK, DV, C, IN> T;
  __shared__ typename T::SmemSummary sm;
  T ch;
  const int c = blockIdx.x, bh = blockIdx.y;
  const int64_t sc = (int64_t)bh * P.nchunks + c;
  ch.template load<false>(P, sm, bh, c);
  if (ch.range_bad && threadIdx.x == 0) __hip_atomic_fetch_or(P.fault, kFaultRange, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  ch.template factors<false, true>(sm, P.rec + sc * T::RS);
  ch.template summary_out<false>(sm, static_cast<char*>(P.agg) + sc * (DK * DV) * (T::F16 ? 2 : 4));
}

// Boundary-state scan over chunks (Eq. chunk_boundary_main) for 256 state
// elements of one sequence per work-group (128 threads, two adjacent value
// columns of one row each, element e = i * DV + n): reads the summaries (fp16
// times their scale, or float32) and the decays, writes S_[c] in float32 and
// S_final.
template <int DK, int DV, bool H16>
__global__ void __launch_bounds__(128) gla_scan_kernel(GlaParams P) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  constexpr int RS = 2 * DK;
  const int bh = blockIdx.y;
  const int e = blockIdx.x * 256 + 2 * threadIdx.x;
  if (e >= DK * DV) return;
  const int NC = P.nchunks;
  float* st = P.states + (int64_t)bh * NC * (DK * DV);
  const char* ag = static_cast<const char*>(P.agg) + (int64_t)bh * NC * (DK * DV) * (H16 ? 2 : 4);
  const float* rc = P.rec + (int64_t)bh * NC * RS;
  const int i = e / DV;
  f2 s = {0.f, 0.f};
  if (P.s0) s = *reinterpret_cast<const f2*>(&P.s0[(int64_t)bh * DK * DV + e]);
  for (int c0 = 0; c0 < NC; c0 += 16) {
    // raw loads first (all 16 in flight), conversions only where the values
    // are used: a conversion next to its load would wait for that load
    typedef typename std::conditional<H16, h2, f2>::type U2;
    U2 u[16];
    float d[16], sc[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      if (c0 + m < NC) {
        u[m] = *reinterpret_cast<const U2*>(ag + ((int64_t)(c0 + m) * (DK * DV) + e) * (H16 ? 2 : 4));
        const f2 r = *reinterpret_cast<const f2*>(&rc[(int64_t)(c0 + m) * RS + 2 * i]);
        d[m] = r[0];
        sc[m] = r[1];
      }
    }
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      if (c0 + m < NC) {
        *reinterpret_cast<f2*>(&st[(int64_t)(c0 + m) * (DK * DV) + e]) = s;
        s[0] = fmaf(d[m], s[0], sc[m] * (float)u[m][0]);
        s[1] = fmaf(d[m], s[1], sc[m] * (float)u[m][1]);
      }
    }
  }
  if (P.s_final) *reinterpret_cast<f2*>(&P.s_final[(int64_t)bh * DK * DV + e]) = s;
}

template <int DK, int DV, int C, int IN>
__global__ void __launch_bounds__(tile_threads(C)) gla_output_kernel(GlaParams P) {
  typedef Chunk<DK, DV, C, IN> T;
  __shared__ typename T::SmemOutput sm;
  T ch;
  const int c = blockIdx.x, bh = blockIdx.y;
  const bool have_state = c > 0 || P.s0;
  const int64_t sc = (int64_t)bh * P.nchunks + c;
  Piece32 sp[T::SPER];
  if (have_state) {
    const __amdgpu_buffer_rsrc_t sr = make_rsrc(P.states + sc * (DK * DV), DK * DV * 4);
#pragma unroll
    for (int m = 0; m < T::SPER; ++m)
      if (T::piece_ok(m)) sp[m].load(sr, T::piece_elem(m));
  }
  ch.template load<true>(P, sm, bh, c);
  Raw rz[T::SITER];
  if (P.gate) ch.prefetch_gate(P, bh, c, rz);
  if (have_state) {
    float acc[T::SPER][8];
#pragma unroll
    for (int m = 0; m < T::SPER; ++m) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[m][e] = sp[m].a[e];
        acc[m][e + 4] = sp[m].b[e];
      }
    }
    ch.state_tile(sm, acc, ch.state_max(sm, acc));
  }
  ch.template factors<true, false>(sm, nullptr);
  f4 O[DV / 16];
  ch.intra(P, sm, bh, c, O);
#pragma unroll
  for (int jb = 0; jb < DV / 16; ++jb) O[jb] *= ch.pup;
  if (have_state) {
    __syncthreads();  // state tile complete
    ch.readout(sm, O);
  }
  ch.template store<true>(P, sm, bh, c, O, rz, ch.range_bad);
}

// ---------------------------------------------------------------------------
// one-launch schedule (look-back)
// ---------------------------------------------------------------------------
// Work-group -> (sequence, chunk): the grid is chunk major over all sequences.
// In ascending chunk order every block waits only on blocks with smaller
// indices; work-groups are handed to the 8 XCDs round robin and each XCD starts
// its blocks in index order, so the smallest unfinished block is always running
// and the grid drains however few work-groups fit at once. When every
// work-group of the grid is resident at once (P.desc) the chunks go in
// descending order instead: the chunks with the longest look-backs start first.
// Value split (P.vparts = 2): the work-groups of a chunk each take DV of the
// head's 2 DV value columns, so a head runs as two sequences with their own
// summaries, flags and boundary states (columns of S) over the same q, k, g.
template <int DK, int DV, int C, int IN>
__global__ void __launch_bounds__(tile_threads(C)) gla_chain_kernel(GlaParams P) {
  typedef Chunk<DK, DV, C, IN> T;
  __shared__ typename T::Smem sm;
  const int NC = P.nchunks;
  const int b = blockIdx.x;
  const int row = b / P.ns;
  const int seq = b - row * P.ns;
  const int c = P.desc ? NC - 1 - row : row;
  const int bh = seq / P.vparts, vp = seq - bh * P.vparts;
  if (P.vparts > 1) {
    P.v = static_cast<const char*>(P.v) + (int64_t)vp * DV * (T::F16 ? 2 : 4);
    P.o = static_cast<char*>(P.o) + (int64_t)vp * DV * (P.odt == GTR_F32 ? 4 : 2);
    if (P.s_final) P.s_final += vp * DV;
  }
  const int64_t sc = (int64_t)seq * NC + c;
  unsigned* flag = P.flags + (size_t)seq * kMaxChainChunks + c;

  T ch;
  ch.template load<true>(P, sm, bh, c);
  Raw rz[T::SITER];
  if (P.gate) ch.prefetch_gate(P, bh, c, rz);
  // the chunk record (d_c, the summary's scale) for the chunks after this one
  ch.template factors<true, true>(sm, nullptr);
  if (ch.w == 0 && ch.lane < DK)
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, f2{sm.dc[ch.lane], ch.usc}),
                                          make_rsrc(P.rec + sc * T::RS, T::RS * 4), ch.lane * 8, 0, kAgentCoherent);
  void* U = static_cast<char*>(P.agg) + sc * (DK * DV) * (T::F16 ? 2 : 4);
  ch.template summary_out<true>(sm, U);

  // the intra part runs while the summary stores are acknowledged
  f4 O[DV / 16];
  ch.intra(P, sm, bh, c, O);
#pragma unroll
  for (int jb = 0; jb < DV / 16; ++jb) O[jb] *= ch.pup;
  // every wave's summary tiles (and the record) are acknowledged before the
  // chunk's flag goes up
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_or(flag, kFlagSummary, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

  float acc[T::SPER][8];
  const int base = lookback_base(P, ch, seq, c);
  const bool okw = base >= -1;
  if (okw) lookback_sum(P, ch, seq, c, base, acc);
  // one exchange makes the outcome uniform: a wait that ran out (bit 0 of a
  // wave's word) poisons the whole state, and so does a NaN state handed over
  // by a poisoned chunk before it (bit 1): either way every row of this chunk
  // and everything it hands over is NaN. The same exchange gives the largest
  // |S_[c]| for the scale of the fp16 state tile.
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
    __hip_atomic_fetch_or(P.fault, (ok ? 0u : kFaultWait) | (ch.range_bad ? kFaultRange : 0u), __ATOMIC_RELAXED,
                          __HIP_MEMORY_SCOPE_AGENT);

  // S_[c+1] = Diag(d_c) S_[c] + U_c: the inclusive state for the chunks after
  // this one (the flag goes up once every wave's pieces are acknowledged), or
  // S_final after the last chunk. U_c is read back from the stores every wave
  // had acknowledged before the flag went up.
  const bool next = c < NC - 1 ? P.publish != 0 && c % kPublishEvery == kPublishEvery - 1 : P.s_final != nullptr;
  if (next) {
    Piece<T::F16> own[T::SPER];
    const __amdgpu_buffer_rsrc_t ur = make_rsrc(U, DK * DV * (T::F16 ? 2 : 4));
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
    ch.state_tile(sm, acc, mx);
    __syncthreads();  // state tile complete
    ch.readout(sm, O);
  }
  // every wave is past the intra part (the exchange above): the k rows in buf
  // are dead, so the output tile needs no barrier before it
  ch.template store<false>(P, sm, bh, c, O, rz, poison);

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

__global__ void zero_fill_kernel(uint4* p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
    p[i] = uint4{0u, 0u, 0u, 0u};
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
struct KernelSet {
  const void* summary;
  const void* output;
  const void* scan;
  const void* chain;
  const void* chain_split;  // one launch with d_v split in two (d_v = 64 only), else null
  int threads;
  const void* lean;         // one launch for 16-bit inputs at chunk 64 (gla_lean.hip), else null
  const void* lean_split;   // the same with d_v split in two, else null
  const void* lean4;        // the same at four work-groups per CU
  const void* lean4_split;
  // the one-launch kernels that run: the lean ones where they exist (occ4:
  // the four-per-CU instantiation)
  const void* one(bool occ4 = false) const { return lean ? (occ4 ? lean4 : lean) : chain; }
  const void* one_split(bool occ4 = false) const {
    return lean_split ? (occ4 ? lean4_split : lean_split) : chain_split;
  }
};

template <int DK, int DV, int C, int IN>
static KernelSet kernels_for() {
  const void* split = nullptr;
  if constexpr (DV == 64) split = reinterpret_cast<const void*>(&gla_chain_kernel<DK, DV / 2, C, IN>);
  return KernelSet{reinterpret_cast<const void*>(&gla_summary_kernel<DK, DV, C, IN>),
                   reinterpret_cast<const void*>(&gla_output_kernel<DK, DV, C, IN>),
                   reinterpret_cast<const void*>(&gla_scan_kernel<DK, DV, IN != GTR_F32>),
                   reinterpret_cast<const void*>(&gla_chain_kernel<DK, DV, C, IN>), split, tile_threads(C)};
}

template <int DK, int DV, int IN>
static bool pick_chunk(int chunk, KernelSet* ks) {
  switch (chunk) {
    case 32: *ks = kernels_for<DK, DV, 32, IN>(); return true;
    case 64: *ks = kernels_for<DK, DV, 64, IN>(); return true;
    case 128: *ks = kernels_for<DK, DV, 128, IN>(); return true;
    default: return false;
  }
}

template <int IN>
static bool pick_dims(int dk, int dv, int chunk, KernelSet* ks) {
  if (dk == 32 && dv == 32) return pick_chunk<32, 32, IN>(chunk, ks);
  if (dk == 32 && dv == 64) return pick_chunk<32, 64, IN>(chunk, ks);
  if (dk == 64 && dv == 64) return pick_chunk<64, 64, IN>(chunk, ks);
  return false;
}

static bool select_kernels(const GlaShape& s, KernelSet* ks) {
  bool ok = false;
  switch (s.qdt) {
    case GTR_F32: ok = pick_dims<GTR_F32>(s.dk, s.dv, s.chunk, ks); break;
    case GTR_F16: ok = pick_dims<GTR_F16>(s.dk, s.dv, s.chunk, ks); break;
    case GTR_BF16: ok = pick_dims<GTR_BF16>(s.dk, s.dv, s.chunk, ks); break;
    default: return false;
  }
  if (ok) {
    LeanKernels lk;
    lean_kernels(s.qdt, s.dk, s.dv, s.chunk, &lk);
    ks->lean = lk.whole3;
    ks->lean_split = lk.split3;
    ks->lean4 = lk.whole4;
    ks->lean4_split = lk.split4;
  }
  return ok;
}

// Work-groups of `kernel` resident per CU and the device's CU count (0 if a
// query fails). The occupancy answer depends only on the kernel and the
// device, so it is kept in a small table that is filled once per (device,
// kernel) pair and never changes afterwards.
static int resident_per_cu(const void* kernel, int threads, int* cus) {
  struct Entry {
    int dev;
    const void* k;
    int per_cu, cus;
  };
  static std::mutex mu;
  static Entry cache[256];
  static int n = 0;
  int dev = 0;
  *cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  {
    std::lock_guard<std::mutex> lk(mu);
    for (int i = 0; i < n; ++i)
      if (cache[i].dev == dev && cache[i].k == kernel) {
        *cus = cache[i].cus;
        return cache[i].per_cu;
      }
  }
  int per_cu = 0, ncu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  *cus = ncu;
  std::lock_guard<std::mutex> lk(mu);
  if (n < 256) cache[n++] = Entry{dev, kernel, per_cu, ncu};
  return per_cu;
}

// XCDs of the current device (1 if the query fails): the one-launch kernel for
// 16-bit inputs lays out its grid so that every chunk of a sequence runs on one
// XCD. Kept per device like the occupancy answers.
static int xcd_count() {
  static std::mutex mu;
  static int cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1;
  std::lock_guard<std::mutex> lk(mu);
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeNumberOfXccs, dev) != hipSuccess || n < 1 || n > 16) n = 1;
    cache[dev] = n;
  }
  return cache[dev];
}

struct Plan {
  int sched;    // GTR_PATH_FUSED (one launch, look-back), GTR_PATH_INLINE (one launch, no inclusive states)
                // or GTR_PATH_STAGED
  int vparts;   // value split of the one-launch schedules
  int desc;     // chunks in descending order (every work-group resident at once)
  int nxcd;     // sequence-per-XCD grid of the 16-bit kernel (0: chunk-major grid)
  int group;    // grouped look-back (16-bit kernel, FUSED)
  int occ4;     // 16-bit kernel at four work-groups per CU
  int64_t blocks;
};

// Length-aware dispatch (the paper's operator appendix switches to inline
// prefixes for short sequences and co-runs the scan with the outputs
// otherwise):
//   * one launch whenever the flags fit (at most kSyncSeqs sequences of at
//     most kMaxChainChunks chunks); INLINE (every chunk reads all summaries
//     before it, no inclusive states) while a sequence has at most
//     kInlineMaxChunks chunks and the whole grid is resident at once, FUSED
//     (look-back to the nearest inclusive state) otherwise: up to
//     kFusedMaxChunks chunks on the float32 kernel (STAGED beyond), up to
//     kMaxChainChunks on the 16-bit kernel at chunk 64, which looks back by
//     groups of kGroup chunks once a sequence is longer than kInlineMaxChunks;
//   * the value split (d_v = 64 in two halves, no output gate: its RMSNorm needs
//     whole rows) when the doubled grid still gives every work-group a CU of
//     its own;
//   * the chunk-major grid, in descending chunk order when every work-group is
//     resident at once (ascending for the grouped look-back).
// An explicit path that does not fit is GTR_ERR_UNSUPPORTED; STAGED always fits.
constexpr int64_t kInlineMaxChunks = 32;
constexpr int64_t kFusedMaxChunks = 64;  // longer sequences: the staged kernels are faster (float32 kernel)
// FUSED, 16-bit kernel: the grouped look-back for sequences longer than this
// (shorter ones, which are not all resident, find an inclusive state within
// kPublishEvery chunks)
constexpr int64_t kGroupMinChunks = kInlineMaxChunks + 1;

static gtr_status plan_call(const GlaShape& s, int path, bool gate, const KernelSet& ks, Plan* pl) {
  pl->sched = GTR_PATH_STAGED;
  pl->vparts = 1;
  pl->desc = 0;
  pl->nxcd = 0;
  pl->group = 0;
  pl->occ4 = 0;
  pl->blocks = 0;
  if (path == GTR_PATH_STAGED) return GTR_OK;
  const bool fits = s.nchunks <= kMaxChainChunks && s.BH <= kSyncSeqs;
  if (!fits) return path == GTR_PATH_AUTO ? GTR_OK : GTR_ERR_UNSUPPORTED;
  int cus = 0;
  const int per_cu = resident_per_cu(ks.one(), ks.threads, &cus);
  int64_t resident = (int64_t)per_cu * cus;  // 0 without a usable device
  if (!gate && ks.one_split() && 2 * s.BH <= kSyncSeqs && cus > 0 && 2 * s.BH * s.nchunks <= cus) {
    int c2 = 0;
    const int per_cu2 = resident_per_cu(ks.one_split(), ks.threads, &c2);
    if (per_cu2 > 0) {
      pl->vparts = 2;
      resident = (int64_t)per_cu2 * c2;
    }
  }
  const int64_t ns = s.BH * pl->vparts;
  bool all_resident = resident > 0 && ns * s.nchunks <= resident;
  const int nx = (pl->vparts > 1 ? ks.lean_split : ks.lean) ? xcd_count() : 1;
  if (nx > 1 && cus >= nx && (ns + nx - 1) / nx * s.nchunks <= cus / nx) {
    // every XCD runs ceil(ns / nx) sequences, one work-group per CU: the
    // summaries stay in the XCD's L2. (Where the sequences do not spread
    // evenly or need more than one round of an XCD's CUs, the chunk-major grid
    // over all XCDs is faster.)
    pl->nxcd = nx;
    all_resident = true;
  }
  if (path == GTR_PATH_AUTO) {
    if (all_resident && s.nchunks <= kInlineMaxChunks)
      pl->sched = GTR_PATH_INLINE;
    else
      pl->sched = s.nchunks <= (ks.lean ? kMaxChainChunks : kFusedMaxChunks) ? GTR_PATH_FUSED : GTR_PATH_STAGED;
  } else {
    pl->sched = path;
  }
  if (pl->sched == GTR_PATH_STAGED) {
    pl->vparts = 1;
    pl->nxcd = 0;
    return GTR_OK;
  }
  const bool lean = (pl->vparts > 1 ? ks.lean_split : ks.lean) != nullptr;
  pl->group = pl->sched == GTR_PATH_FUSED && lean && s.nchunks >= kGroupMinChunks ? 1 : 0;
  // four work-groups per CU (shorter look-back batches) where the grid is more
  // than one round of work-groups or the key width is 32; the inline schedule
  // at d_k = 64, whose look-backs are the longest, keeps the longer batches
  pl->occ4 = lean && (pl->sched == GTR_PATH_FUSED || s.dk == 32) ? 1 : 0;
  // descending chunk order when every work-group is resident (the chunks that
  // wait longest start first), except for the grouped look-back, whose
  // aggregates come from the low chunks
  pl->desc = all_resident && !pl->group ? 1 : 0;
  pl->blocks = pl->nxcd > 1 ? (int64_t)pl->nxcd * ((ns + pl->nxcd - 1) / pl->nxcd) * s.nchunks : ns * s.nchunks;
  return GTR_OK;
}

}  // namespace gtr

using namespace gtr;

extern "C" size_t gtr_gla_workspace_size(const gtr_gla_args* a) {
  GlaShape s;
  if (!a || gla_shape_from_args(a, &s, /*check_pointers=*/false) != GTR_OK) return 0;
  return gla_workspace_layout(s).total;
}

extern "C" gtr_status gtr_gla_workspace_init(void* workspace, size_t bytes, hipStream_t stream) {
  if (!workspace) return GTR_ERR_NULL;
  if (bytes == 0) return GTR_OK;
  if ((reinterpret_cast<uintptr_t>(workspace) & 255u) || (bytes & 15u)) return GTR_ERR_WORKSPACE;
  const size_t n16 = bytes / 16;
  const int blocks = (int)((n16 + 255) / 256 < 1024 ? (n16 + 255) / 256 : 1024);
  hipLaunchKernelGGL(zero_fill_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<uint4*>(workspace), n16);
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}

extern "C" int gtr_gla_workspace_fault(const void* workspace, size_t bytes) {
  if (!workspace || bytes < 256) return -1;
  unsigned v = 0;
  if (hipMemcpy(&v, workspace, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess) return -1;
  return (int)(v & 0xffu);
}

static int plan_query(const gtr_gla_args* a, Plan* pl) {
  GlaShape s;
  KernelSet ks;
  if (!a || gla_shape_from_args(a, &s, /*check_pointers=*/false) != GTR_OK || !select_kernels(s, &ks)) return -1;
  if (plan_call(s, a->path, a->out_gate != nullptr, ks, pl) != GTR_OK) return -1;
  return 0;
}

extern "C" int gtr_gla_schedule(const gtr_gla_args* a) {
  Plan pl;
  return plan_query(a, &pl) ? -1 : pl.sched;
}

extern "C" int gtr_gla_value_parts(const gtr_gla_args* a) {
  Plan pl;
  return plan_query(a, &pl) ? -1 : pl.vparts;
}

// Launches the schedule for arguments already validated (workspace included).
static gtr_status gla_launch(const gtr_gla_args* a, const GlaShape& s, hipStream_t stream) {
  gtr_status st;
  KernelSet ks;
  if (!select_kernels(s, &ks)) return GTR_ERR_UNSUPPORTED;
  Plan pl;
  st = plan_call(s, a->path, a->out_gate != nullptr, ks, &pl);
  if (st != GTR_OK) return st;

  const WorkspaceLayout lay = gla_workspace_layout(s);
  char* ws = static_cast<char*>(a->workspace);
  GlaParams P;
  P.q = a->q;
  P.k = a->k;
  P.v = a->v;
  P.g = a->g;
  P.o = a->o;
  P.s0 = a->s0;
  P.s_final = a->s_final;
  P.qdt = a->qkv_dtype;
  P.gdt = a->g_dtype;
  P.odt = a->o_dtype;
  P.BH = (int)s.BH;
  P.H = a->H;
  P.W = a->W;
  P.L = s.L;
  P.nchunks = (int)s.nchunks;
  P.scale = a->scale;
  P.scan = a->scan;
  P.fault = reinterpret_cast<unsigned*>(ws + lay.fault_off);
  P.sync = reinterpret_cast<unsigned*>(ws + lay.sync_off);
  P.flags = reinterpret_cast<unsigned*>(ws + lay.flags_off);
  P.agg = ws + lay.agg_off;
  P.rec = reinterpret_cast<float*>(ws + lay.rec_off);
  P.states = reinterpret_cast<float*>(ws + lay.states_off);
  P.gkind = a->g_kind;
  P.inv_tau = a->g_kind == GTR_GATE_LOGITS ? 1.f / a->gate_tau : 1.f;
  P.gate = a->out_gate;
  P.nw = a->out_gate ? a->norm_weight : nullptr;
  P.gatedt = a->out_gate_dtype;
  P.eps = a->norm_eps;
  P.dvp = s.dv;
  P.vparts = pl.vparts;
  P.ns = (int)(s.BH * pl.vparts);
  P.desc = pl.desc;
  P.publish = pl.sched == GTR_PATH_FUSED;
  P.nxcd = pl.nxcd;
  P.spin = a->spin_limit ? a->spin_limit : kSpinDefault;
  P.group = pl.group;

  void* kargs[] = {&P};
  hipError_t err;
  if (pl.sched != GTR_PATH_STAGED) {
    const void* k = pl.vparts > 1 ? ks.one_split(pl.occ4) : ks.one(pl.occ4);
    err = hipLaunchKernel(k, dim3((unsigned)pl.blocks), dim3(ks.threads), kargs, 0, stream);
  } else {
    err = hipLaunchKernel(ks.summary, dim3((unsigned)s.nchunks, (unsigned)s.BH), dim3(ks.threads), kargs, 0, stream);
    if (err == hipSuccess) {
      const unsigned eb = (unsigned)((s.dk * s.dv + 255) / 256);
      err = hipLaunchKernel(ks.scan, dim3(eb, (unsigned)s.BH), dim3(128), kargs, 0, stream);
    }
    if (err == hipSuccess)
      err = hipLaunchKernel(ks.output, dim3((unsigned)s.nchunks, (unsigned)s.BH), dim3(ks.threads), kargs, 0, stream);
  }
  if (err != hipSuccess) return GTR_ERR_HIP;
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}

extern "C" gtr_status gtr_gla_fwd(const gtr_gla_args* a, hipStream_t stream) {
  if (!a) return GTR_ERR_NULL;
  GlaShape s;
  const gtr_status st = gla_shape_from_args(a, &s, /*check_pointers=*/true);
  if (st != GTR_OK) return st;
  return gla_launch(a, s, stream);
}

// ---------------------------------------------------------------------------
// The entry point that allocates nothing: the workspace is a file-scope device
// array of fixed size (one copy per device, zero at load; every completed call
// leaves its synchronisation words zeroed again). In host code `scratch` only
// names the symbol: its device address on each device comes from
// hipGetSymbolAddress, taken once per device with that device current.
// ---------------------------------------------------------------------------
namespace gtr {
constexpr size_t kNoAllocBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

static void* scratch_on_current_device() {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* ptr[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(mu);
  if (!ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    ptr[dev] = p;
  }
  return ptr[dev];
}
}  // namespace gtr

extern "C" gtr_status gtr_gla_fwd_noalloc(const gtr_gla_args* a, hipStream_t stream) {
  if (!a) return GTR_ERR_NULL;
  GlaShape s;
  gtr_status st = gla_shape_from_args(a, &s, /*check_pointers=*/false);
  if (st != GTR_OK) return st;
  if (gla_workspace_layout(s).total > kNoAllocBytes) return GTR_ERR_SCRATCH;
  void* ws = scratch_on_current_device();
  if (!ws) return GTR_ERR_HIP;
  gtr_gla_args b = *a;
  b.workspace = ws;
  b.workspace_bytes = kNoAllocBytes;
  st = gla_shape_from_args(&b, &s, /*check_pointers=*/true);
  if (st != GTR_OK) return st;
  return gla_launch(&b, s, stream);
}
