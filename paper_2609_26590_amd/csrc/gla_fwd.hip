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
// The factors that depend only on (sub-chunk, dimension) are computed once per
// dimension (lane d of the wave for dimension d) into a small per-wave table in
// LDS, from the shared table of sub-chunk totals, and read back by the lanes
// that use them.
//
// Schedules:
//   * staged: summary kernel -> boundary-state scan kernel -> output kernel.
//   * inline: one launch; each work-group publishes its summary and, once all
//     summaries of its sequence are in, rebuilds its own boundary state from
//     the summaries of the chunks before it,
//       S_[c] = (prod_{m<c} Diag(d_m)) S_0 + sum_{j<c} (prod_{j<m<c} Diag(d_m)) U_j,
//     which costs c reads of a summary but only one hand-off (short sequences).
//   * fused : one launch; each work-group owns one (sequence, chunk), publishes
//     its summary, and the work-groups of one sequence then run the boundary
//     state scan cooperatively (each takes a slice of the d_k x d_v state) before
//     reading their own S_[c]. Two per-sequence counters order the phases.
//     Everything one work-group hands to another (summaries, decays, boundary
//     states) is written and read with agent-coherent accesses (cache policy
//     sc1), and a work-group waits for its own stores to be acknowledged
//     (vmcnt(0)) before it bumps a counter. No release/acquire fence is used: on
//     this GPU those write back / invalidate the whole L2 of the XCD, which cost
//     more than the rest of the kernel.
// Hand-off precision: with fp16/bf16 inputs the summaries U_c and the boundary
// states S_[c] travel in fp16 (the readout's MFMA operand type); every scan and
// rebuild accumulates in float32, and S_final is the float32 accumulator. With
// float32 inputs everything stays float32.
#include <hip/hip_runtime.h>

#include <mutex>
#include <type_traits>

#include "gtr.h"
#include "gtr_device.h"
#include "gtr_internal.h"

namespace gtr {

constexpr float kSpanF16 = 10.f;           // mid-point factors within e^5: fp16 operands
constexpr float kSpanF32 = 60.f;           // within e^30: float32 operands
constexpr unsigned kSpinLimit = 1u << 22;  // bounded waits (fused schedule)

struct GlaParams {
  const void* q;
  const void* k;
  const void* v;
  const void* g;
  void* o;
  const float* s0;
  float* s_final;
  int qdt, gdt, odt;
  int BH;
  int H, W;
  int64_t L;
  int nchunks;
  float scale;
  int scan;
  float* states;    // [BH][nchunks][DV][DK] float32 U_c^T, then S_[c]^T (float32 inputs only)
  float* decays;    // [BH][nchunks][DK]
  unsigned* sync;   // [BH][4]: arrive1, arrive2, leave, spare
  unsigned* fault;  // one word
  int groups;       // ceil(BH / 8), fused mapping
  int gkind;        // GTR_GATE_LOG_DECAY or GTR_GATE_LOGITS (g holds the gate logits)
  float inv_tau;    // 1 / tau of the gate fusion
  const void* gate;  // output-gate pre-activation [BH][L][DV] (spatial), or null: no epilogue
  const float* nw;   // RMSNorm weight [DV], or null (ones)
  int gatedt;        // dtype of gate
  float eps;         // RMSNorm epsilon
  unsigned short* states16;  // [BH][nchunks][DV][DK] fp16 U_c^T, then S_[c]^T (16-bit inputs only)
  int dvp;     // row pitch (elements) of v, o, the gate, S0 and S_final: the full d_v
  int vparts;  // value split of the inline schedule: work-groups per chunk, each d_v / vparts columns
};

constexpr int tile_threads(int chunk) { return chunk / 16 * kWave; }

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// Agent-coherent buffer accesses (cache policy sc1: no stale copy in the CU's
// L1 is used, stores are written through). The buffer descriptor bounds every
// access to [base, base + bytes): outside it loads return 0 and stores are
// dropped.
// ---------------------------------------------------------------------------
constexpr int kAgentCoherent = 16;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ void coh_store4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, f4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, (int)byte_off, 0, kAgentCoherent);
}
__device__ __forceinline__ f4 coh_load4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, kAgentCoherent));
}
__device__ __forceinline__ void coh_store1(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, (int)byte_off, 0, kAgentCoherent);
}
__device__ __forceinline__ float coh_load1(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)byte_off, 0, kAgentCoherent));
}

// Raw bits of 8 consecutive elements (32 bytes for float32, 16 for 16-bit types).
struct Raw {
  u32x4 a, b;
};

__device__ __forceinline__ void ld_raw(const void* base, int dt, int64_t off, Raw& r) {
  if (dt == GTR_F32) {
    const u32x4* p = reinterpret_cast<const u32x4*>(static_cast<const float*>(base) + off);
    r.a = p[0];
    r.b = p[1];
  } else {
    r.a = *reinterpret_cast<const u32x4*>(static_cast<const unsigned short*>(base) + off);
  }
}

// The same through a buffer descriptor over one sequence's rows: a byte offset
// at or beyond the descriptor's range (kOutOfRange) reads zeros, which is what
// the positions past the end of a sequence must hold.
constexpr uint32_t kOutOfRange = 0x7fffff00u;  // the host keeps every sequence's rows below this many bytes
__device__ __forceinline__ void ld_raw_buf(__amdgpu_buffer_rsrc_t rs, int dt, uint32_t byte_off, Raw& r) {
  r.a = __builtin_amdgcn_raw_buffer_load_b128(rs, (int)byte_off, 0, 0);
  if (dt == GTR_F32) r.b = __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(byte_off + 16u), 0, 0);
}

__device__ __forceinline__ void cvt_raw(const Raw& r, int dt, float (&x)[8]) {
  if (dt == GTR_F32) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      // copy the lanes to scalars first: this compiler reads element 0 when
      // __builtin_bit_cast is given a vector-element lvalue directly
      const unsigned int ua = r.a[e], ub = r.b[e];
      x[e] = __builtin_bit_cast(float, ua);
      x[e + 4] = __builtin_bit_cast(float, ub);
    }
  } else if (dt == GTR_F16) {
    const h8 h = __builtin_bit_cast(h8, r.a);
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = (float)h[e];
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const unsigned int u = r.a[e];
      x[2 * e] = __builtin_bit_cast(float, u << 16);
      x[2 * e + 1] = __builtin_bit_cast(float, u & 0xffff0000u);
    }
  }
}

template <bool F16>
__device__ __forceinline__ float gexp(float x) {
  if constexpr (F16)
    return __expf(x);
  else
    return expf(x);
}

// Log-decay of one key dimension from what g holds: log gamma itself, or (gate
// fusion) the logit a of gamma = sigmoid(a)^(1/tau) (Sec. 3.1), giving
// log gamma = logsigmoid(a) / tau = (min(a, 0) - log1p(exp(-|a|))) / tau.
// log1p(e) for e in (0, 1] as log(u) * e / (u - 1), u = 1 + e rounded: the
// factor e / (u - 1) undoes the rounding of u (u - 1 is exact), which keeps the
// result within a few ulp with one log and one reciprocal.
// Hardware log2 and reciprocal (about 1 ulp each); when u rounds to 1 the
// quotient is not used (a select, not a branch).
__device__ __forceinline__ float log_decay(const GlaParams& P, float x) {
  if (P.gkind != GTR_GATE_LOGITS) return x;
  constexpr float kLn2 = 0.693147180559945309f;
  const float e = __expf(-fabsf(x));
  const float u = 1.f + e;
  const float d = u - 1.f;
  const float r = __builtin_amdgcn_logf(u) * kLn2 * e * __builtin_amdgcn_rcpf(d);
  const float l1p = d == 0.f ? e : r;
  return (fminf(x, 0.f) - l1p) * P.inv_tau;
}

// One chunk of one sequence: C tokens, one wave per 16-token sub-chunk.
// IN is the dtype of q, k, v (GTR_F32 / GTR_F16 / GTR_BF16).
template <int DK, int DV, int C, int IN>
struct Chunk {
  static constexpr bool F16 = IN != GTR_F32;  // matrix operands: fp16 (else float32)
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
  typedef typename Op<F16>::elem E;
  typedef typename Op<F16>::frag8 F8;
  typedef typename Op<F16>::frag4 F4;

  // Shared memory of the one-launch schedules (every part). The staged
  // kernels use the subsets below, so that more of their work-groups fit on a
  // CU at once: the summary kernel has no k rows, state or diagonal staging,
  // the output kernel no k-hat tile.
  struct Smem {
    float buf[C * BUFW];   // k*exp(T-a) rows [C][KP]; later the output tile [C][OP]
    E kT[DK * TP];         // (k * exp(A_last - A_r))^T  [DK][TP]
    E vT[DV * TP];         // v^T                       [DV][TP]
    E sT[DV * SP];         // S_[c]^T                   [DV][SP]
    float T[NW][DK];       // sub-chunk totals of g
    float G0[NW][DK];      // g at the first token of each sub-chunk
    float F[NW][NF][DK];   // per-wave factor table (rows kFq, kFk, kFh, kFoff + J)
    float Pt[NW][16][17];  // exact diagonal blocks, P^T staging
  };
  struct SmemSummary {
    E kT[DK * TP];
    E vT[DV * TP];
    float T[NW][DK];
    float G0[NW][DK];
    float F[NW][NF][DK];
  };
  struct SmemOutput {
    float buf[C * BUFW];
    E vT[DV * TP];
    E sT[DV * SP];
    float T[NW][DK];
    float G0[NW][DK];
    float F[NW][NF][DK];
    float Pt[NW][16][17];
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

  // Loads and per-token work. Writes v^T, the sub-chunk totals and (ROWS) the
  // k*exp(T-a) rows. Ends with a barrier.
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
#pragma unroll
    for (int s = 0; s < VS; ++s) {
      float x[8];
      cvt_raw(rv[s], IN, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) sm.vT[(32 * s + 8 * gq + e) * TP + r] = (E)x[e];
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
    __syncthreads();
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
  // SUMMARY: the transposed k-hat tile and d_c (written by wave 0 through
  // `dec`, coherent or plain), followed by a barrier.
  template <bool READOUT, bool SUMMARY, bool COH, class S>
  __device__ __forceinline__ void factors(S& sm, float* dec) {
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
        if constexpr (COH)
          coh_store1(make_rsrc(dec, DK * 4), d * 4, dc);
        else
          dec[d] = dc;
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

  // U_c as U^T ([DV][DK]) to `U` in float32 or, with U16 (16-bit inputs), to
  // `U16p` rounded to fp16, the type the states are handed over in; coherent
  // (agent scope) or plain.
  template <bool COH, bool U16 = false, class S>
  __device__ __forceinline__ void summary_out(const S& sm, float* U, unsigned short* U16p = nullptr) {
    constexpr int NTI = (DK / 16) * (DV / 16);
    const __amdgpu_buffer_rsrc_t ur = make_rsrc(U, DK * DV * 4);
    for (int tau = w; tau < NTI; tau += NW) {
      const int ib = tau / (DV / 16), jb = tau % (DV / 16);
      f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < C / 32; ++ks) {
        const F8 a = *reinterpret_cast<const F8*>(&sm.kT[(16 * ib + tr) * TP + 32 * ks + 8 * gq]);
        const F8 b = *reinterpret_cast<const F8*>(&sm.vT[(16 * jb + tr) * TP + 32 * ks + 8 * gq]);
        acc = mma32(a, b, acc);
      }
      // lane holds U[16ib + 4gq + e][16jb + tr]
      const int off = (16 * jb + tr) * DK + 16 * ib + 4 * gq;
      if constexpr (U16) {
        const h4 hv = {(_Float16)acc[0], (_Float16)acc[1], (_Float16)acc[2], (_Float16)acc[3]};
        if constexpr (COH)
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, hv), make_rsrc(U16p, DK * DV * 2), off * 2, 0,
                                                kAgentCoherent);
        else
          *reinterpret_cast<h4*>(reinterpret_cast<_Float16*>(U16p) + off) = hv;
      } else if constexpr (COH)
        coh_store4(ur, off * 4, acc);
      else
        *reinterpret_cast<f4*>(&U[off]) = acc;
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

  // Intra-chunk part: o_r = sum_{j<=r} P[r][j] v_j for this wave's 16 rows.
  // Needs the k rows written by load<true>().
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

  // Boundary state S_[c]^T ([DV][DK] fp32) -> shared tile, in two steps so the
  // loads can be issued early: each thread moves whole 16-byte pieces. No
  // barrier.
  static constexpr int SQ4 = DK * DV / 4;           // 16-byte pieces in one state
  static constexpr int SPER = (SQ4 + NT - 1) / NT;  // pieces per thread
  template <bool COH>
  __device__ __forceinline__ void state_load(const float* ST, f4 (&buf)[SPER]) {
    const __amdgpu_buffer_rsrc_t sr = make_rsrc(ST, DK * DV * 4);
#pragma unroll
    for (int m = 0; m < SPER; ++m) {
      const int q4 = threadIdx.x + m * NT;
      if (q4 < SQ4) {
        if constexpr (COH)
          buf[m] = coh_load4(sr, q4 * 16);
        else
          buf[m] = reinterpret_cast<const f4*>(ST)[q4];
      }
    }
  }
  // 16-bit inputs: the states are handed over already rounded to the fp16 MFMA
  // operand type (what state_store would do), so 16-byte pieces of 8 elements
  // move straight to the tile.
  static constexpr int SQ8 = DK * DV / 8;
  static constexpr int SPER8 = (SQ8 + NT - 1) / NT;
  template <bool COH = false>
  __device__ __forceinline__ void state_load16(const unsigned short* ST, u32x4 (&buf)[SPER8]) const {
    const __amdgpu_buffer_rsrc_t sr = make_rsrc(ST, DK * DV * 2);
#pragma unroll
    for (int m = 0; m < SPER8; ++m) {
      const int q8 = threadIdx.x + m * NT;
      if (q8 < SQ8) {
        if constexpr (COH)
          buf[m] = __builtin_amdgcn_raw_buffer_load_b128(sr, q8 * 16, 0, kAgentCoherent);
        else
          buf[m] = reinterpret_cast<const u32x4*>(ST)[q8];
      }
    }
  }
  template <class S>
  __device__ __forceinline__ void state_store16(S& sm, const u32x4 (&buf)[SPER8]) {
    static_assert(F16 && (SP * 2) % 16 == 0, "16-byte rows of fp16 elements");
#pragma unroll
    for (int m = 0; m < SPER8; ++m) {
      const int q8 = threadIdx.x + m * NT;
      if (q8 < SQ8) {
        const int dv = (q8 * 8) / DK, i = (q8 * 8) % DK;
        *reinterpret_cast<u32x4*>(&sm.sT[dv * SP + i]) = buf[m];
      }
    }
  }
  template <class S>
  __device__ __forceinline__ void state_store(S& sm, const f4 (&buf)[SPER]) {
#pragma unroll
    for (int m = 0; m < SPER; ++m) {
      const int q4 = threadIdx.x + m * NT;  // piece index in [DV][DK]
      if (q4 < SQ4) {
        const int dv = (q4 * 4) / DK, i = (q4 * 4) % DK;
#pragma unroll
        for (int e = 0; e < 4; ++e) sm.sT[dv * SP + i + e] = (E)buf[m][e];
      }
    }
  }

  // o_r += (q_r exp(A_r)) S_[c]. Reads the shared state tile.
  template <class S>
  __device__ __forceinline__ void readout(const S& sm, f4 (&O)[DV / 16]) {
    F8 qtf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) qtf[s] = Op<F16>::pack8(qt[s]);
#pragma unroll
    for (int jb = 0; jb < DV / 16; ++jb)
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const F8 b = *reinterpret_cast<const F8*>(&sm.sT[(16 * jb + tr) * SP + 32 * s + 8 * gq]);
        O[jb] = mma32(qtf[s], b, O[jb]);
      }
  }

  // Stage the output tile through LDS and write whole rows back in spatial order.
  // Gate values of the output-gate epilogue for the rows this thread stores,
  // loaded early (with the other inputs) so that the epilogue does not wait
  // for memory at the end of the kernel. Only when P.gate is set.
  static constexpr int SITER = C * (DV / 8) / NT;  // store iterations per thread
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

  template <class S>
  __device__ __forceinline__ void store(const GlaParams& P, S& sm, int bh, int c, const f4 (&O)[DV / 16],
                                        const Raw (&rz)[SITER]) {
    __syncthreads();  // all waves are done with the k rows in buf
#pragma unroll
    for (int jb = 0; jb < DV / 16; ++jb)
#pragma unroll
      for (int e = 0; e < 4; ++e) sm.buf[(16 * w + 4 * gq + e) * OP + 16 * jb + tr] = P.scale * O[jb][e];
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
  static constexpr int PIECES = DV / 8;  // 8-element pieces of an output row

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
    float z[8], w[8];
    cvt_raw(rz, P.gatedt, z);
    if (P.nw) {
      const f4 lo = *reinterpret_cast<const f4*>(P.nw + 8 * pc);
      const f4 hi = *reinterpret_cast<const f4*>(P.nw + 8 * pc + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        w[e] = lo[e];
        w[e + 4] = hi[e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) w[e] = 1.f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = z[e] * __builtin_amdgcn_rcpf(1.f + __expf(-z[e])) * (x[e] * rs) * w[e];
  }
};

// ---------------------------------------------------------------------------
// Boundary-state scan over chunks (Eq. chunk_boundary_main) for elements
// [e0, e1) of one sequence's state (S^T layout, element e = dv*DK + i). Reads
// U_c^T and writes S_[c]^T in place, float32, or, for 16-bit inputs (H16),
// fp16 in and out (the summaries as the summary kernel rounded them, the states
// as the output kernel's readout consumes them), accumulating in float32.
// S_final gets the float32 state after the last chunk.
// ---------------------------------------------------------------------------
template <int DK, int DV, bool H16>
__device__ __forceinline__ void scan_plain(const GlaParams& P, int bh, int e0, int e1, int tid, int nt) {
  // two adjacent elements (dims i, i + 1 of one d_v row) per thread: 8-byte
  // loads of U and of the decays, 4-byte fp16 (or 8-byte float32) stores
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  static_assert(DK % 2 == 0, "element pairs share a d_v row");
  float* st = P.states + (int64_t)bh * P.nchunks * (DK * DV);
  _Float16* st16 = reinterpret_cast<_Float16*>(P.states16) + (int64_t)bh * P.nchunks * (DK * DV);
  const float* dec = P.decays + (int64_t)bh * P.nchunks * DK;
  const int NC = P.nchunks;
  for (int e = e0 + 2 * tid; e < e1; e += 2 * nt) {
    const int dv = e / DK, i = e - dv * DK;
    f2 s = {0.f, 0.f};
    if (P.s0) {
      s[0] = P.s0[((int64_t)bh * DK + i) * DV + dv];
      s[1] = P.s0[((int64_t)bh * DK + i + 1) * DV + dv];
    }
    for (int c0 = 0; c0 < NC; c0 += 32) {
      // raw loads first (all 32 in flight), conversions only where the values
      // are used: a conversion next to its load would wait for that load
      typedef typename std::conditional<H16, h2, f2>::type U2;
      U2 u[32];
      f2 d[32];
#pragma unroll
      for (int m = 0; m < 32; ++m) {
        if (c0 + m < NC) {
          if constexpr (H16)
            u[m] = *reinterpret_cast<const h2*>(&st16[(int64_t)(c0 + m) * (DK * DV) + e]);
          else
            u[m] = *reinterpret_cast<const f2*>(&st[(int64_t)(c0 + m) * (DK * DV) + e]);
          d[m] = *reinterpret_cast<const f2*>(&dec[(int64_t)(c0 + m) * DK + i]);
        }
      }
#pragma unroll
      for (int m = 0; m < 32; ++m) {
        if (c0 + m < NC) {
          if constexpr (H16)
            *reinterpret_cast<h2*>(&st16[(int64_t)(c0 + m) * (DK * DV) + e]) = h2{(_Float16)s[0], (_Float16)s[1]};
          else
            *reinterpret_cast<f2*>(&st[(int64_t)(c0 + m) * (DK * DV) + e]) = s;
          s[0] = d[m][0] * s[0] + (float)u[m][0];
          s[1] = d[m][1] * s[1] + (float)u[m][1];
        }
      }
    }
    if (P.s_final) {
      P.s_final[((int64_t)bh * DK + i) * DV + dv] = s[0];
      P.s_final[((int64_t)bh * DK + i + 1) * DV + dv] = s[1];
    }
  }
}

// The same with agent-coherent accesses, for the fused schedule. One sequence's
// states span nchunks * DK * DV * 4 bytes, which the host keeps below 2^31.
template <int DK, int DV>
__device__ __forceinline__ void scan_coherent(const GlaParams& P, int bh, int e0, int e1, int tid, int nt) {
  const int NC = P.nchunks;
  const __amdgpu_buffer_rsrc_t sr = make_rsrc(P.states + (int64_t)bh * NC * (DK * DV), (uint32_t)NC * DK * DV * 4);
  const __amdgpu_buffer_rsrc_t dr = make_rsrc(P.decays + (int64_t)bh * NC * DK, (uint32_t)NC * DK * 4);
  for (int e = e0 + tid; e < e1; e += nt) {
    const int dv = e / DK, i = e - dv * DK;
    float s = P.s0 ? P.s0[((int64_t)bh * DK + i) * DV + dv] : 0.f;
    for (int c0 = 0; c0 < NC; c0 += 32) {
      float u[32], d[32];
#pragma unroll
      for (int m = 0; m < 32; ++m) {
        if (c0 + m < NC) {
          u[m] = coh_load1(sr, ((uint32_t)(c0 + m) * (DK * DV) + e) * 4);
          d[m] = coh_load1(dr, ((uint32_t)(c0 + m) * DK + i) * 4);
        }
      }
#pragma unroll
      for (int m = 0; m < 32; ++m) {
        if (c0 + m < NC) {
          coh_store1(sr, ((uint32_t)(c0 + m) * (DK * DV) + e) * 4, s);
          s = d[m] * s + u[m];
        }
      }
    }
    if (P.s_final) P.s_final[((int64_t)bh * DK + i) * DV + dv] = s;
  }
}

// The same over fp16 summaries and states (16-bit inputs), two adjacent
// elements per thread, accumulating in float32.
template <int DK, int DV>
__device__ __forceinline__ void scan_coherent16(const GlaParams& P, int bh, int e0, int e1, int tid, int nt) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  const int NC = P.nchunks;
  const __amdgpu_buffer_rsrc_t sr = make_rsrc(P.states16 + (int64_t)bh * NC * (DK * DV), (uint32_t)NC * DK * DV * 2);
  const __amdgpu_buffer_rsrc_t dr = make_rsrc(P.decays + (int64_t)bh * NC * DK, (uint32_t)NC * DK * 4);
  for (int e = e0 + 2 * tid; e < e1; e += 2 * nt) {
    const int dv = e / DK, i = e - dv * DK;
    f2 s = {0.f, 0.f};
    if (P.s0) {
      s[0] = P.s0[((int64_t)bh * DK + i) * DV + dv];
      s[1] = P.s0[((int64_t)bh * DK + i + 1) * DV + dv];
    }
    for (int c0 = 0; c0 < NC; c0 += 32) {
      unsigned u[32];
      u32x2 d[32];
#pragma unroll
      for (int m = 0; m < 32; ++m) {
        if (c0 + m < NC) {
          u[m] = __builtin_amdgcn_raw_buffer_load_b32(sr, (int)(((uint32_t)(c0 + m) * (DK * DV) + e) * 2), 0,
                                                      kAgentCoherent);
          d[m] = __builtin_amdgcn_raw_buffer_load_b64(dr, (int)(((uint32_t)(c0 + m) * DK + i) * 4), 0, kAgentCoherent);
        }
      }
#pragma unroll
      for (int m = 0; m < 32; ++m) {
        if (c0 + m < NC) {
          const h2 hs = {(_Float16)s[0], (_Float16)s[1]};
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, hs), sr,
                                                (int)(((uint32_t)(c0 + m) * (DK * DV) + e) * 2), 0, kAgentCoherent);
          const h2 hu = __builtin_bit_cast(h2, u[m]);
          const f2 dd = __builtin_bit_cast(f2, d[m]);
          s[0] = dd[0] * s[0] + (float)hu[0];
          s[1] = dd[1] * s[1] + (float)hu[1];
        }
      }
    }
    if (P.s_final) {
      P.s_final[((int64_t)bh * DK + i) * DV + dv] = s[0];
      P.s_final[((int64_t)bh * DK + i + 1) * DV + dv] = s[1];
    }
  }
}

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
  ch.template factors<false, true, false>(sm, P.decays + sc * DK);
  if constexpr (T::F16)
    ch.template summary_out<false, true>(sm, nullptr, P.states16 + sc * (DK * DV));
  else
    ch.template summary_out<false>(sm, P.states + sc * (DK * DV));
}

// 128 threads per work-group, two elements each: 256 elements per work-group.
template <int DK, int DV, bool H16>
__global__ void __launch_bounds__(128) gla_scan_kernel(GlaParams P) {
  const int bh = blockIdx.y;
  const int e0 = blockIdx.x * 256;
  const int e1 = min(e0 + 256, DK * DV);
  scan_plain<DK, DV, H16>(P, bh, e0, e1, threadIdx.x, 128);
}

template <int DK, int DV, int C, int IN>
__global__ void __launch_bounds__(tile_threads(C)) gla_output_kernel(GlaParams P) {
  typedef Chunk<DK, DV, C, IN> T;
  __shared__ typename T::SmemOutput sm;
  T ch;
  const int c = blockIdx.x, bh = blockIdx.y;
  const bool have_state = c > 0 || P.s0;
  const int64_t sc = (int64_t)bh * P.nchunks + c;
  f4 sbuf[T::F16 ? 1 : T::SPER];
  u32x4 hbuf[T::F16 ? T::SPER8 : 1];
  if (have_state) {
    if constexpr (T::F16)
      ch.state_load16(P.states16 + sc * (DK * DV), hbuf);
    else
      ch.template state_load<false>(P.states + sc * (DK * DV), sbuf);
  }
  ch.template load<true>(P, sm, bh, c);
  Raw rz[T::SITER];
  if (P.gate) ch.prefetch_gate(P, bh, c, rz);
  if (have_state) {
    if constexpr (T::F16)
      ch.state_store16(sm, hbuf);
    else
      ch.state_store(sm, sbuf);
  }
  ch.template factors<true, false, false>(sm, nullptr);
  f4 O[DV / 16];
  ch.intra(P, sm, bh, c, O);
  if (have_state) {
    __syncthreads();  // state tile complete
    ch.readout(sm, O);
  }
  ch.store(P, sm, bh, c, O, rz);
}

// ---------------------------------------------------------------------------
// fused schedule
// ---------------------------------------------------------------------------
// A work-group's coherent stores are acknowledged before its one increment.
__device__ __forceinline__ void seq_arrive(unsigned* ctr) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Bounded wait until `ctr` reaches `target`; on time-out the fault word is set
// (the results of the call are then invalid) and the work-group goes on.
__device__ __forceinline__ void seq_wait(unsigned* ctr, unsigned target, unsigned* fault) {
  if (threadIdx.x == 0) {
    unsigned n = 0;
    while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      __builtin_amdgcn_s_sleep(1);
      if (++n > kSpinLimit) {
        __hip_atomic_store(fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
  }
  __syncthreads();
}

// S_[c]^T ([DV][DK]) rebuilt from the summaries and decays of chunks 0..c-1 of
// one sequence (agent-coherent loads) straight into the shared state tile
// (STATE), walking the chunks backwards so that the weight of each summary is
// one more decay factor than the one after it; FINAL also writes
// S_final = Diag(d_c) S_[c] + U_c for the last chunk. Thread t owns the
// 16-byte pieces t, t + NT, ...; with NT a multiple of DK / 4 they all share
// dims i..i+3, so one decay load per chunk serves all of them. No barrier.
// `seq` indexes the summaries (a head's value part under the value split),
// `bh` the decays, S0 and S_final (the head; P's S0 and S_final pointers
// already start at the part's first column).
template <int DK, int DV, int NT, typename Sm, typename E, int SP>
__device__ __forceinline__ void state_inline(const GlaParams& P, Sm& sm, int seq, int bh, int c, bool state,
                                             bool final) {
  constexpr int SQ4 = DK * DV / 4;
  constexpr int SPER = (SQ4 + NT - 1) / NT;
  static_assert(NT % (DK / 4) == 0, "the pieces of one thread must share their dims");
  const int NC = P.nchunks;
  const __amdgpu_buffer_rsrc_t sr = make_rsrc(P.states + (int64_t)seq * NC * (DK * DV), (uint32_t)NC * DK * DV * 4);
  const __amdgpu_buffer_rsrc_t dr = make_rsrc(P.decays + (int64_t)bh * NC * DK, (uint32_t)NC * DK * 4);
  const int i0 = (4 * (int)threadIdx.x) % DK;
  f4 acc[SPER], wgt = {1.f, 1.f, 1.f, 1.f};
#pragma unroll
  for (int m = 0; m < SPER; ++m) acc[m] = f4{0.f, 0.f, 0.f, 0.f};
  constexpr int B = SPER >= 16 ? 1 : 16 / SPER;  // chunks per batch of loads
  for (int j1 = c; j1 > 0; j1 -= B) {
    f4 u[B][SPER], d[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const int j = j1 - 1 - b;
      if (j >= 0) {
        d[b] = coh_load4(dr, ((uint32_t)j * DK + i0) * 4);
#pragma unroll
        for (int m = 0; m < SPER; ++m) {
          const int q4 = threadIdx.x + m * NT;
          if (q4 < SQ4) u[b][m] = coh_load4(sr, ((uint32_t)j * (DK * DV) + 4 * q4) * 4);
        }
      }
    }
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const int j = j1 - 1 - b;
      if (j >= 0) {
#pragma unroll
        for (int m = 0; m < SPER; ++m) acc[m] += wgt * u[b][m];
        wgt *= d[b];
      }
    }
  }
  const f4 dc = final ? coh_load4(dr, ((uint32_t)c * DK + i0) * 4) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int m = 0; m < SPER; ++m) {
    const int q4 = threadIdx.x + m * NT;
    if (q4 < SQ4) {
      const int dv = (4 * q4) / DK;
      if (P.s0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[m][e] += wgt[e] * P.s0[((int64_t)bh * DK + i0 + e) * P.dvp + dv];
      }
      if (state) {
#pragma unroll
        for (int e = 0; e < 4; ++e) sm.sT[dv * SP + i0 + e] = (E)acc[m][e];
      }
      if (final) {
        const f4 uc = coh_load4(sr, ((uint32_t)c * (DK * DV) + 4 * q4) * 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) P.s_final[((int64_t)bh * DK + i0 + e) * P.dvp + dv] = dc[e] * acc[m][e] + uc[e];
      }
    }
  }
}

// The same from fp16 summaries (16-bit inputs): 16-byte pieces of 8 elements,
// which share dims i..i+7 when NT is a multiple of DK / 8; float32 sums.
template <int DK, int DV, int NT, typename Sm, typename E, int SP>
__device__ __forceinline__ void state_inline16(const GlaParams& P, Sm& sm, int seq, int bh, int c, bool state,
                                               bool final) {
  constexpr int SQ8 = DK * DV / 8;
  constexpr int SPER = (SQ8 + NT - 1) / NT;
  static_assert(NT % (DK / 8) == 0, "the pieces of one thread must share their dims");
  const int NC = P.nchunks;
  const __amdgpu_buffer_rsrc_t sr = make_rsrc(P.states16 + (int64_t)seq * NC * (DK * DV), (uint32_t)NC * DK * DV * 2);
  const __amdgpu_buffer_rsrc_t dr = make_rsrc(P.decays + (int64_t)bh * NC * DK, (uint32_t)NC * DK * 4);
  const int i0 = (8 * (int)threadIdx.x) % DK;
  float acc[SPER][8], wgt[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) wgt[e] = 1.f;
#pragma unroll
  for (int m = 0; m < SPER; ++m)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[m][e] = 0.f;
  constexpr int B = SPER >= 16 ? 1 : 16 / SPER;  // chunks per batch of loads
  for (int j1 = c; j1 > 0; j1 -= B) {
    u32x4 u[B][SPER];
    f4 d[B][2];
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const int j = j1 - 1 - b;
      if (j >= 0) {
        d[b][0] = coh_load4(dr, ((uint32_t)j * DK + i0) * 4);
        d[b][1] = coh_load4(dr, ((uint32_t)j * DK + i0 + 4) * 4);
#pragma unroll
        for (int m = 0; m < SPER; ++m) {
          const int q8 = threadIdx.x + m * NT;
          if (q8 < SQ8)
            u[b][m] = __builtin_amdgcn_raw_buffer_load_b128(sr, (int)(((uint32_t)j * (DK * DV) + 8 * q8) * 2), 0,
                                                            kAgentCoherent);
        }
      }
    }
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const int j = j1 - 1 - b;
      if (j >= 0) {
#pragma unroll
        for (int m = 0; m < SPER; ++m) {
          const h8 hv = __builtin_bit_cast(h8, u[b][m]);
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[m][e] += wgt[e] * (float)hv[e];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          wgt[e] *= d[b][0][e];
          wgt[e + 4] *= d[b][1][e];
        }
      }
    }
  }
  f4 dc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  if (final) {
    dc[0] = coh_load4(dr, ((uint32_t)c * DK + i0) * 4);
    dc[1] = coh_load4(dr, ((uint32_t)c * DK + i0 + 4) * 4);
  }
#pragma unroll
  for (int m = 0; m < SPER; ++m) {
    const int q8 = threadIdx.x + m * NT;
    if (q8 < SQ8) {
      const int dv = (8 * q8) / DK;
      if (P.s0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[m][e] += wgt[e] * P.s0[((int64_t)bh * DK + i0 + e) * P.dvp + dv];
      }
      if (state) {
#pragma unroll
        for (int e = 0; e < 8; ++e) sm.sT[dv * SP + i0 + e] = (E)acc[m][e];
      }
      if (final) {
        const h8 uc = __builtin_bit_cast(
            h8, __builtin_amdgcn_raw_buffer_load_b128(sr, (int)(((uint32_t)c * (DK * DV) + 8 * q8) * 2), 0,
                                                      kAgentCoherent));
#pragma unroll
        for (int e = 0; e < 8; ++e)
          P.s_final[((int64_t)bh * DK + i0 + e) * P.dvp + dv] = dc[e >> 2][e & 3] * acc[m][e] + (float)uc[e];
      }
    }
  }
}

// Work-group -> (sequence, chunk). Work-groups are handed to the 8 XCDs round
// robin, so block b runs on XCD b % 8; all chunks of a sequence get the same
// b % 8 and therefore share one L2. Blocks whose sequence index is past the end
// exit at once.
// Value split (inline schedule, P.vparts = 2): the work-groups of a chunk each
// take DV of the head's 2 DV value columns, so a head runs as two sequences
// with their own summaries, counters and boundary states (columns of S) over
// the same q, k, g; both write the chunk decays, with identical values. The
// grid is then exactly (sequences x chunks), chunks in descending order: the
// chunks with the longest rebuilds start first, and the work-groups that
// share a CU once every CU has one are the first chunks of their sequences.
template <int DK, int DV, int C, int IN, bool INLINE>
__global__ void __launch_bounds__(tile_threads(C)) gla_fused_kernel(GlaParams P) {
  typedef Chunk<DK, DV, C, IN> T;
  __shared__ typename T::Smem sm;
  const int NC = P.nchunks;
  const int b = blockIdx.x;
  int seq, c, bh;
  if (INLINE && P.vparts > 1) {
    const int ns = P.BH * P.vparts;
    const int row = b / ns;
    seq = b - row * ns;
    c = NC - 1 - row;
    bh = seq / P.vparts;
    const int vp = seq - bh * P.vparts;
    P.v = static_cast<const char*>(P.v) + (int64_t)vp * DV * (T::F16 ? 2 : 4);
    P.o = static_cast<char*>(P.o) + (int64_t)vp * DV * (P.odt == GTR_F32 ? 4 : 2);
    if (P.s0) P.s0 += vp * DV;
    if (P.s_final) P.s_final += vp * DV;
  } else {
    const int x = b & 7, slot = b >> 3;
    const int grp = slot / NC;
    c = slot - grp * NC;
    seq = bh = grp * 8 + x;
    if (bh >= P.BH) return;
  }
  unsigned* sync = P.sync + 4 * seq;
  const int64_t sc = (int64_t)seq * NC + c;

  T ch;
  ch.template load<true>(P, sm, bh, c);
  Raw rz[T::SITER];
  if (P.gate) ch.prefetch_gate(P, bh, c, rz);
  ch.template factors<true, true, true>(sm, P.decays + ((int64_t)bh * NC + c) * DK);
  if constexpr (T::F16)
    ch.template summary_out<true, true>(sm, nullptr, P.states16 + sc * (DK * DV));
  else
    ch.template summary_out<true>(sm, P.states + sc * (DK * DV));
  seq_arrive(&sync[0]);

  f4 O[DV / 16];
  ch.intra(P, sm, bh, c, O);

  seq_wait(&sync[0], (unsigned)NC, P.fault);
  if constexpr (INLINE) {
    const bool state = c > 0 || P.s0;
    const bool final = P.s_final && c == NC - 1;
    if (state || final) {
      if constexpr (T::F16)
        state_inline16<DK, DV, T::NT, typename T::Smem, typename T::E, T::SP>(P, sm, seq, bh, c, state, final);
      else
        state_inline<DK, DV, T::NT, typename T::Smem, typename T::E, T::SP>(P, sm, seq, bh, c, state, final);
    }
    if (state) {
      __syncthreads();
      ch.readout(sm, O);
    }
  } else {
    if constexpr (T::F16) {
      const int per = 2 * ((DK * DV / 2 + NC - 1) / NC);  // element pairs
      const int e0 = min(c * per, DK * DV), e1 = min(e0 + per, DK * DV);
      scan_coherent16<DK, DV>(P, bh, e0, e1, threadIdx.x, T::NT);
    } else {
      const int per = (DK * DV + NC - 1) / NC;
      const int e0 = min(c * per, DK * DV), e1 = min(e0 + per, DK * DV);
      scan_coherent<DK, DV>(P, bh, e0, e1, threadIdx.x, T::NT);
    }
    seq_arrive(&sync[1]);
    seq_wait(&sync[1], (unsigned)NC, P.fault);

    if (c > 0 || P.s0) {
      if constexpr (T::F16) {
        u32x4 hbuf[T::SPER8];
        ch.template state_load16<true>(P.states16 + sc * (DK * DV), hbuf);
        ch.state_store16(sm, hbuf);
      } else {
        f4 sbuf[T::SPER];
        ch.template state_load<true>(P.states + sc * (DK * DV), sbuf);
        ch.state_store(sm, sbuf);
      }
      __syncthreads();
      ch.readout(sm, O);
    }
  }
  ch.store(P, sm, bh, c, O, rz);

  if (threadIdx.x == 0) {
    const unsigned prev = __hip_atomic_fetch_add(&sync[2], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == (unsigned)NC - 1) {  // last one out: leave the counters zeroed
      __hip_atomic_store(&sync[0], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&sync[1], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&sync[2], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
  const void* fused;
  const void* inlined;
  const void* inlined_split;  // inline schedule with d_v split in two (d_v = 64 only), else null
  const void* scan;
  int threads;
};

template <int DK, int DV, int C, int IN>
static KernelSet kernels_for() {
  const void* split = nullptr;
  if constexpr (DV == 64) split = reinterpret_cast<const void*>(&gla_fused_kernel<DK, DV / 2, C, IN, true>);
  return KernelSet{reinterpret_cast<const void*>(&gla_summary_kernel<DK, DV, C, IN>),
                   reinterpret_cast<const void*>(&gla_output_kernel<DK, DV, C, IN>),
                   reinterpret_cast<const void*>(&gla_fused_kernel<DK, DV, C, IN, false>),
                   reinterpret_cast<const void*>(&gla_fused_kernel<DK, DV, C, IN, true>),
                   split,
                   reinterpret_cast<const void*>(&gla_scan_kernel<DK, DV, IN != GTR_F32>), tile_threads(C)};
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
  switch (s.qdt) {
    case GTR_F32: return pick_dims<GTR_F32>(s.dk, s.dv, s.chunk, ks);
    case GTR_F16: return pick_dims<GTR_F16>(s.dk, s.dv, s.chunk, ks);
    case GTR_BF16: return pick_dims<GTR_BF16>(s.dk, s.dv, s.chunk, ks);
    default: return false;
  }
}

// AUTO takes the inline schedule while the summaries of one sequence take at
// most this many bytes (nchunks * dk * dv elements, float32 for float32 inputs,
// fp16 otherwise): rebuilding a boundary state reads every summary before it,
// so the cost grows with their total size (measured with float32 summaries:
// d_k = d_v = 64 at 25 chunks, 400 KB, faster fused; d_k = 32, d_v = 64 at 25
// chunks, 200 KB, faster inline).
constexpr int64_t kInlineMaxSummaryBytes = 262144;

// Largest number of work-groups of one kernel that can be resident on one XCD
// at once (8 XCDs per device), and the XCD's CU count (0 for both if a query
// fails); cached per (device, kernel).
static int fused_capacity_per_xcd(const void* kernel, int threads, int* cus_per_xcd = nullptr) {
  struct Entry {
    int dev;
    const void* k;
    int cap, cus;
  };
  static std::mutex mu;
  static Entry cache[128];
  static int n = 0;
  int dev = 0;
  if (cus_per_xcd) *cus_per_xcd = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  {
    std::lock_guard<std::mutex> lk(mu);
    for (int i = 0; i < n; ++i)
      if (cache[i].dev == dev && cache[i].k == kernel) {
        if (cus_per_xcd) *cus_per_xcd = cache[i].cus;
        return cache[i].cap;
      }
  }
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  const int cap = per_cu * (cus / 8);
  if (cus_per_xcd) *cus_per_xcd = cus / 8;
  std::lock_guard<std::mutex> lk(mu);
  if (n < 128) cache[n++] = Entry{dev, kernel, cap, cus / 8};
  return cap;
}

// The fused schedule addresses one sequence's states through a buffer
// descriptor with a 32-bit range: nchunks * 64 * 64 * 4 bytes must stay below
// 2^31.
constexpr int64_t kFusedMaxChunks = 4096;

// Length-aware dispatch: short sequences rebuild each boundary state from the
// summaries (one hand-off), longer ones split the scan over their chunks'
// work-groups (two hand-offs). Both need every chunk of a sequence resident at
// once on one XCD, and both lose to the three-launch schedule as soon as an XCD
// has to run more than one sequence (more than 8 sequences): then the sequences
// compete for the XCD's slots and partly resident ones spin while they wait for
// the rest, so AUTO takes the staged schedule there. An explicit one-launch
// path that does not fit is GTR_ERR_UNSUPPORTED.
// The inline schedule splits d_v = 64 over two work-groups per chunk (half the
// value work and half the summary bytes that each chunk's rebuild reads) when
// there is no output-gate epilogue (its RMSNorm needs whole rows) and the
// doubled grid still gives every work-group a CU of its own (the split grid is
// spread over all XCDs: work-group b runs on XCD b % 8). Measured at 40x40
// tokens, fp16, d_k = d_v = 64: 4 heads 11.5 against 13.2 us, 2 heads 11.4
// against 12.9; at 6 heads (300 work-groups, some CUs running two) no gain, and
// for d_k = 32 at 6 heads 13.3 against 10.7 us. *vparts is 1 or 2.
static gtr_status choose_schedule(const GlaShape& s, int path, bool gate, const KernelSet& ks, int* sched,
                                  int* vparts) {
  *sched = GTR_PATH_STAGED;
  *vparts = 1;
  const bool auto_one_launch = path == GTR_PATH_AUTO && s.BH <= 8;
  if (path == GTR_PATH_FUSED || path == GTR_PATH_INLINE || auto_one_launch) {
    const bool inl = path == GTR_PATH_INLINE ||
                     (path == GTR_PATH_AUTO &&
                      s.nchunks * s.dk * s.dv * (s.qdt == GTR_F32 ? 4 : 2) <= kInlineMaxSummaryBytes);
    const int cap = fused_capacity_per_xcd(inl ? ks.inlined : ks.fused, ks.threads);
    const bool fits = cap > 0 && s.nchunks <= cap && s.nchunks <= kFusedMaxChunks && s.BH <= kSyncSeqs;
    if (path != GTR_PATH_AUTO && !fits) return GTR_ERR_UNSUPPORTED;
    if (fits) *sched = inl ? GTR_PATH_INLINE : GTR_PATH_FUSED;
    if (fits && inl && !gate && ks.inlined_split && 2 * s.BH <= kSyncSeqs) {
      int cus = 0;
      const int scap = fused_capacity_per_xcd(ks.inlined_split, ks.threads, &cus);
      const int64_t per_xcd = (2 * s.BH * s.nchunks + 7) / 8;
      if (per_xcd <= scap && per_xcd <= cus) *vparts = 2;
    }
  }
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
  return v != 0;
}

extern "C" int gtr_gla_schedule(const gtr_gla_args* a) {
  GlaShape s;
  KernelSet ks;
  int sched = -1, vparts = 1;
  if (!a || gla_shape_from_args(a, &s, /*check_pointers=*/false) != GTR_OK || !select_kernels(s, &ks)) return -1;
  if (choose_schedule(s, a->path, a->out_gate != nullptr, ks, &sched, &vparts) != GTR_OK) return -1;
  return sched;
}

extern "C" int gtr_gla_value_parts(const gtr_gla_args* a) {
  GlaShape s;
  KernelSet ks;
  int sched = -1, vparts = 1;
  if (!a || gla_shape_from_args(a, &s, /*check_pointers=*/false) != GTR_OK || !select_kernels(s, &ks)) return -1;
  if (choose_schedule(s, a->path, a->out_gate != nullptr, ks, &sched, &vparts) != GTR_OK) return -1;
  return vparts;
}

extern "C" gtr_status gtr_gla_fwd(const gtr_gla_args* a, hipStream_t stream) {
  if (!a) return GTR_ERR_NULL;
  GlaShape s;
  gtr_status st = gla_shape_from_args(a, &s, /*check_pointers=*/true);
  if (st != GTR_OK) return st;
  KernelSet ks;
  if (!select_kernels(s, &ks)) return GTR_ERR_UNSUPPORTED;

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
  P.states = reinterpret_cast<float*>(ws + lay.states_off);
  P.decays = reinterpret_cast<float*>(ws + lay.decays_off);
  P.states16 = lay.states16_off ? reinterpret_cast<unsigned short*>(ws + lay.states16_off) : nullptr;
  P.groups = (int)((s.BH + 7) / 8);
  P.gkind = a->g_kind;
  P.inv_tau = a->g_kind == GTR_GATE_LOGITS ? 1.f / a->gate_tau : 1.f;
  P.gate = a->out_gate;
  P.nw = a->out_gate ? a->norm_weight : nullptr;
  P.gatedt = a->out_gate_dtype;
  P.eps = a->norm_eps;
  P.dvp = s.dv;

  int sched = GTR_PATH_STAGED;
  const gtr_status cs = choose_schedule(s, a->path, a->out_gate != nullptr, ks, &sched, &P.vparts);
  if (cs != GTR_OK) return cs;
  const void* one_launch = sched == GTR_PATH_INLINE ? (P.vparts > 1 ? ks.inlined_split : ks.inlined)
                           : sched == GTR_PATH_FUSED ? ks.fused
                                                     : nullptr;

  void* kargs[] = {&P};
  hipError_t err;
  if (one_launch) {
    const int64_t blocks = P.vparts > 1 ? (int64_t)P.vparts * s.BH * s.nchunks : (int64_t)8 * P.groups * s.nchunks;
    err = hipLaunchKernel(one_launch, dim3((unsigned)blocks), dim3(ks.threads), kargs, 0, stream);
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
