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
// Per-(sub-chunk, dimension) factors are computed once per chunk into a small
// shared table.
//
// Schedules:
//   * staged: summary kernel -> boundary-state scan kernel -> output kernel.
//   * fused : one launch; each work-group owns one (sequence, chunk), publishes
//     its summary, and the work-groups of one sequence then run the boundary
//     state scan cooperatively (each takes a slice of the d_k x d_v state) before
//     reading their own S_[c]. Two per-sequence counters order the phases.
#include <hip/hip_runtime.h>

#include <mutex>

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
  float* states;    // [BH][nchunks][DV][DK]: U_c^T, then S_[c]^T in place
  float* decays;    // [BH][nchunks][DK]
  unsigned* sync;   // [BH][4]: arrive1, arrive2, leave, spare
  unsigned* fault;  // one word
  int groups;       // ceil(BH / 8), fused mapping
};

constexpr int tile_threads(int chunk) { return chunk / 16 * kWave; }

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

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
      x[2 * e] = __builtin_bit_cast(float, r.a[e] << 16);
      x[2 * e + 1] = __builtin_bit_cast(float, r.a[e] & 0xffff0000u);
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
  static constexpr int NPAIR = NW * (NW - 1) / 2 > 0 ? NW * (NW - 1) / 2 : 1;
  typedef typename Op<F16>::elem E;
  typedef typename Op<F16>::frag8 F8;
  typedef typename Op<F16>::frag4 F4;

  struct Smem {
    float buf[C * BUFW];      // k*exp(T-a) rows [C][KP]; later the output tile [C][OP]
    E kT[DK * TP];            // (k * exp(A_last - A_r))^T  [DK][TP]
    E vT[DV * TP];            // v^T                       [DV][TP]
    E sT[DV * SP];            // S_[c]^T                   [DV][SP]
    float T[NW][DK];          // sub-chunk totals of g
    float G0[NW][DK];         // g at the first token of each sub-chunk
    float Fq[NW][DK];         // exp(A at the first token of R)
    float Fk[NW][DK];         // exp(sum of totals after R)
    float Fh[NW][DK];         // exp(span_R / 2)
    float Foff[NPAIR][DK];    // exp(g0_R + sum_{J<K<R} T_K), pair (R, J), J < R
    float Fdec[DK];           // exp(sum of all totals) = d_c
    float Pt[NW][16][17];     // exact diagonal blocks, P^T staging
  };

  int w, lane, tr, gq, r;
  int64_t pos;
  float qraw[KS][8], kraw[KS][8], aloc[KS][8];
  float qh[KS][8];   // q * exp(a - g0)
  float ke[KS][8];   // k * exp(T - a)
  float spanmax;     // wave-uniform: widest decay span of this sub-chunk
  float absmax;      // wave-uniform: largest |q|, |k| of this sub-chunk

  __device__ __forceinline__ int dim(int s, int e) const { return 32 * s + 8 * gq + e; }

  static __device__ __forceinline__ int pair(int R, int J) { return R * (R - 1) / 2 + J; }

  // Loads and per-token work; writes T, G0 and v^T. Ends with a barrier.
  __device__ __forceinline__ void load(const GlaParams& P, Smem& sm, int bh, int c) {
    w = threadIdx.x >> 6;
    lane = threadIdx.x & 63;
    tr = lane & 15;
    gq = lane >> 4;
    r = 16 * w + tr;
    pos = (int64_t)c * C + r;
    const bool valid = pos < P.L;
    const int64_t t = valid ? scan_to_spatial(pos, P.H, P.W, P.scan) : 0;
    const int64_t kb = ((int64_t)bh * P.L + t) * DK;
    const int64_t vb = ((int64_t)bh * P.L + t) * DV;

    // issue every load before converting any of them
    Raw rq[KS], rk[KS], rg[KS], rv[VS];
    if (valid) {
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        ld_raw(P.q, IN, kb + 32 * s + 8 * gq, rq[s]);
        ld_raw(P.k, IN, kb + 32 * s + 8 * gq, rk[s]);
        ld_raw(P.g, P.gdt, kb + 32 * s + 8 * gq, rg[s]);
      }
#pragma unroll
      for (int s = 0; s < VS; ++s) ld_raw(P.v, IN, vb + 32 * s + 8 * gq, rv[s]);
    } else {
      const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int s = 0; s < KS; ++s) rq[s] = rk[s] = rg[s] = Raw{z, z};
#pragma unroll
      for (int s = 0; s < VS; ++s) rv[s] = Raw{z, z};
    }

    float gv[KS][8];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      cvt_raw(rq[s], IN, qraw[s]);
      cvt_raw(rk[s], IN, kraw[s]);
      cvt_raw(rg[s], P.gdt, gv[s]);
    }
    // v^T tile
#pragma unroll
    for (int s = 0; s < VS; ++s) {
      float x[8];
      cvt_raw(rv[s], IN, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) sm.vT[(32 * s + 8 * gq + e) * TP + r] = (E)x[e];
    }

    // local inclusive cumulative sums over the 16 tokens of this sub-chunk
    float smax = 0.f, amax = 0.f;
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float a = row_inclusive_scan(gv[s][e]);
        const float T = row_read(a, 15);
        const float g0 = row_read(a, 0);
        aloc[s][e] = a;
        smax = fmaxf(smax, g0 - T);
        amax = fmaxf(amax, fmaxf(fabsf(qraw[s][e]), fabsf(kraw[s][e])));
        qh[s][e] = qraw[s][e] * gexp<F16>(a - g0);  // exp(A_r - A_first) <= 1
        ke[s][e] = kraw[s][e] * gexp<F16>(T - a);   // exp(A_last(R) - A_r) <= 1
        if (tr == 0) {
          sm.T[w][dim(s, e)] = T;
          sm.G0[w][dim(s, e)] = g0;
        }
      }
    spanmax = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, wave_max(smax))));
    absmax = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, wave_max(amax))));
    __syncthreads();
  }

  // The per-(sub-chunk, dimension) factor table. Ends with a barrier.
  __device__ __forceinline__ void factors(Smem& sm) {
    constexpr int N1 = NW * DK;          // Fq, Fk, Fh
    constexpr int N2 = NW * (NW - 1) / 2 * DK;  // Foff
    constexpr int N = N1 + N2 + DK;
    for (int idx = threadIdx.x; idx < N; idx += NT) {
      if (idx < N1) {
        const int R = idx / DK, d = idx - R * DK;
        float before = 0.f, after = 0.f;
        for (int K = 0; K < R; ++K) before += sm.T[K][d];
        for (int K = R + 1; K < NW; ++K) after += sm.T[K][d];
        const float g0 = sm.G0[R][d];
        sm.Fq[R][d] = gexp<F16>(before + g0);
        sm.Fk[R][d] = gexp<F16>(after);
        sm.Fh[R][d] = gexp<F16>(0.5f * (g0 - sm.T[R][d]));
      } else if (idx < N1 + N2) {
        const int p = (idx - N1) / DK, d = (idx - N1) - p * DK;
        int R = 1;
        while (pair(R + 1, 0) <= p) ++R;
        const int J = p - pair(R, 0);
        float between = sm.G0[R][d];
        for (int K = J + 1; K < R; ++K) between += sm.T[K][d];
        sm.Foff[p][d] = gexp<F16>(between);
      } else {
        const int d = idx - N1 - N2;
        float tot = 0.f;
        for (int K = 0; K < NW; ++K) tot += sm.T[K][d];
        sm.Fdec[d] = gexp<F16>(tot);
      }
    }
    __syncthreads();
  }

  // Writes the k rows (and, for the summary, the transposed k-hat tile).
  // Ends with a barrier.
  __device__ __forceinline__ void stage_k(Smem& sm, bool summary) {
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = dim(s, e);
        sm.buf[r * KP + d] = ke[s][e];
        if (summary) sm.kT[d * TP + r] = (E)(ke[s][e] * sm.Fk[w][d]);
      }
    __syncthreads();
  }

  // U_c (as U^T, [DV][DK]) and d_c to the workspace.
  __device__ __forceinline__ void summary_out(const GlaParams& P, Smem& sm, int bh, int c) {
    constexpr int NTI = (DK / 16) * (DV / 16);
    float* U = P.states + ((int64_t)bh * P.nchunks + c) * (DK * DV);
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
      *reinterpret_cast<f4*>(&U[(16 * jb + tr) * DK + 16 * ib + 4 * gq]) = acc;
    }
    float* dec = P.decays + ((int64_t)bh * P.nchunks + c) * DK;
    for (int d = threadIdx.x; d < DK; d += NT) dec[d] = sm.Fdec[d];
  }

  // Exact diagonal block for sub-chunks whose decay span is too wide for the
  // mid-point factors: P[r][j] = sum_d q_r k_j exp(a_r - a_j), j <= r.
  // Rare; the token loop is kept rolled to keep the code small.
  __device__ __forceinline__ f4 exact_diagonal(float (*pt)[17]) {
#pragma unroll 1
    for (int j = 0; j < 16; ++j) {
      const int src = ((gq << 4) | j) << 2;
      float acc = 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float kj = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src, __builtin_bit_cast(int, kraw[s][e])));
          const float aj = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(src, __builtin_bit_cast(int, aloc[s][e])));
          acc += (j <= tr) ? qraw[s][e] * kj * gexp<F16>(aloc[s][e] - aj) : 0.f;
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
  __device__ __forceinline__ void intra(Smem& sm, f4 (&O)[DV / 16]) {
    f4 PT[NW];
    F8 qhf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) qhf[s] = Op<F16>::pack8(qh[s]);

#pragma unroll
    for (int J = 0; J < NW; ++J) {
      PT[J] = f4{0.f, 0.f, 0.f, 0.f};
      if (J < w) {
        // P^T[j][r] = sum_d (k_j exp(T_J - a_j) Foff[R,J])[d] (q_r exp(a_r - g0_R))[d]
        const float* fo = sm.Foff[pair(w, J)];
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          float x[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] = sm.buf[(16 * J + tr) * KP + dim(s, e)] * fo[dim(s, e)];
          PT[J] = mma32(Op<F16>::pack8(x), qhf[s], PT[J]);
        }
      } else if (J == w) {
        // fp16 operands only if the mid-point factors keep them well inside fp16 range
        if (F16 && spanmax <= kSpanF16 && absmax <= 256.f) {
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            float a[8], b[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float h = sm.Fh[w][dim(s, e)];
              a[e] = ke[s][e] * h;
              b[e] = qh[s][e] * h;
            }
            PT[J] = mma32(Op<F16>::pack8(a), Op<F16>::pack8(b), PT[J]);
          }
        } else if (spanmax <= kSpanF32) {
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            f8 a, b;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float h = sm.Fh[w][dim(s, e)];
              a[e] = ke[s][e] * h;
              b[e] = qh[s][e] * h;
            }
            PT[J] = mma32(a, b, PT[J]);
          }
        } else {
          PT[J] = exact_diagonal(sm.Pt[w]);
        }
        // causal mask: lane holds P^T[j = 4gq + e][r = tr]
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (4 * gq + e > tr) PT[J][e] = 0.f;
      }
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

  // Boundary state S_[c]^T ([DV][DK] fp32 in the workspace) -> shared tile, in
  // two steps so the loads can be issued early: each thread moves whole
  // 16-byte pieces. No barrier.
  static constexpr int SQ4 = DK * DV / 4;          // 16-byte pieces in one state
  static constexpr int SPER = (SQ4 + NT - 1) / NT;  // pieces per thread
  __device__ __forceinline__ void stage_state_load(const float* ST, f4 (&buf)[SPER]) {
#pragma unroll
    for (int m = 0; m < SPER; ++m) {
      const int q4 = threadIdx.x + m * NT;
      if (q4 < SQ4) buf[m] = reinterpret_cast<const f4*>(ST)[q4];
    }
  }
  __device__ __forceinline__ void stage_state_store(Smem& sm, const f4 (&buf)[SPER]) {
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
  __device__ __forceinline__ void readout(Smem& sm, f4 (&O)[DV / 16]) {
    F8 qtf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      float x[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = qh[s][e] * sm.Fq[w][dim(s, e)];
      qtf[s] = Op<F16>::pack8(x);
    }
#pragma unroll
    for (int jb = 0; jb < DV / 16; ++jb)
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const F8 b = *reinterpret_cast<const F8*>(&sm.sT[(16 * jb + tr) * SP + 32 * s + 8 * gq]);
        O[jb] = mma32(qtf[s], b, O[jb]);
      }
  }

  // Stage the output tile through LDS and write whole rows back in spatial order.
  __device__ __forceinline__ void store(const GlaParams& P, Smem& sm, int bh, int c, const f4 (&O)[DV / 16]) {
    __syncthreads();  // all waves are done with the k rows in buf
#pragma unroll
    for (int jb = 0; jb < DV / 16; ++jb)
#pragma unroll
      for (int e = 0; e < 4; ++e) sm.buf[(16 * w + 4 * gq + e) * OP + 16 * jb + tr] = P.scale * O[jb][e];
    __syncthreads();
    constexpr int PIECES = DV / 8;
    for (int idx = threadIdx.x; idx < C * PIECES; idx += NT) {
      const int rr = idx / PIECES, pc = idx % PIECES;
      const int64_t p = (int64_t)c * C + rr;
      if (p < P.L) {
        const int64_t t = scan_to_spatial(p, P.H, P.W, P.scan);
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = sm.buf[rr * OP + 8 * pc + e];
        store_n<8>(P.o, P.odt, ((int64_t)bh * P.L + t) * DV + 8 * pc, x);
      }
    }
  }
};

// ---------------------------------------------------------------------------
// boundary-state scan over chunks for elements [e0, e1) of one sequence's
// state (S^T layout, element e = dv*DK + i). In place: U_c^T -> S_[c]^T.
// ---------------------------------------------------------------------------
template <int DK, int DV>
__device__ __forceinline__ void scan_elements(const GlaParams& P, int bh, int e0, int e1, int tid, int nt) {
  float* st = P.states + (int64_t)bh * P.nchunks * (DK * DV);
  const float* dec = P.decays + (int64_t)bh * P.nchunks * DK;
  const int NC = P.nchunks;
  for (int e = e0 + tid; e < e1; e += nt) {
    const int dv = e / DK, i = e - dv * DK;
    float s = P.s0 ? P.s0[((int64_t)bh * DK + i) * DV + dv] : 0.f;
    int c = 0;
    for (; c + 8 <= NC; c += 8) {
      float u[8], d[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        u[m] = st[(int64_t)(c + m) * (DK * DV) + e];
        d[m] = dec[(int64_t)(c + m) * DK + i];
      }
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        st[(int64_t)(c + m) * (DK * DV) + e] = s;
        s = d[m] * s + u[m];
      }
    }
    for (; c < NC; ++c) {
      const float u = st[(int64_t)c * (DK * DV) + e];
      const float d = dec[(int64_t)c * DK + i];
      st[(int64_t)c * (DK * DV) + e] = s;
      s = d * s + u;
    }
    if (P.s_final) P.s_final[((int64_t)bh * DK + i) * DV + dv] = s;
  }
}

// ---------------------------------------------------------------------------
// staged schedule
// ---------------------------------------------------------------------------
template <int DK, int DV, int C, int IN>
__global__ void __launch_bounds__(tile_threads(C)) gla_summary_kernel(GlaParams P) {
  typedef Chunk<DK, DV, C, IN> T;
  __shared__ typename T::Smem sm;
  T ch;
  const int c = blockIdx.x, bh = blockIdx.y;
  ch.load(P, sm, bh, c);
  ch.factors(sm);
  ch.stage_k(sm, true);
  ch.summary_out(P, sm, bh, c);
}

template <int DK, int DV>
__global__ void __launch_bounds__(256) gla_scan_kernel(GlaParams P) {
  const int bh = blockIdx.y;
  const int e0 = blockIdx.x * 256;
  const int e1 = min(e0 + 256, DK * DV);
  scan_elements<DK, DV>(P, bh, e0, e1, threadIdx.x, 256);
}

template <int DK, int DV, int C, int IN>
__global__ void __launch_bounds__(tile_threads(C)) gla_output_kernel(GlaParams P) {
  typedef Chunk<DK, DV, C, IN> T;
  __shared__ typename T::Smem sm;
  T ch;
  const int c = blockIdx.x, bh = blockIdx.y;
  const bool have_state = c > 0 || P.s0;
  f4 sbuf[T::SPER];
  if (have_state) ch.stage_state_load(P.states + ((int64_t)bh * P.nchunks + c) * (DK * DV), sbuf);
  ch.load(P, sm, bh, c);
  if (have_state) ch.stage_state_store(sm, sbuf);
  ch.factors(sm);
  ch.stage_k(sm, false);
  f4 O[DV / 16];
  ch.intra(sm, O);
  if (have_state) ch.readout(sm, O);
  ch.store(P, sm, bh, c, O);
}

// ---------------------------------------------------------------------------
// fused schedule
// ---------------------------------------------------------------------------
__device__ __forceinline__ void seq_arrive(unsigned* ctr) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void seq_wait(unsigned* ctr, unsigned target, unsigned* fault) {
  if (threadIdx.x == 0) {
    unsigned n = 0;
    while (__hip_atomic_load(ctr, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target) {
      __builtin_amdgcn_s_sleep(1);
      if (++n > kSpinLimit) {
        __hip_atomic_store(fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
  }
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

// Work-group -> (sequence, chunk). Work-groups are handed to the 8 XCDs round
// robin, so block b runs on XCD b % 8; all chunks of a sequence get the same
// b % 8 and therefore share one L2 for their summaries and boundary states.
// Blocks whose sequence index is past the end exit at once.
template <int DK, int DV, int C, int IN>
__global__ void __launch_bounds__(tile_threads(C)) gla_fused_kernel(GlaParams P) {
  typedef Chunk<DK, DV, C, IN> T;
  __shared__ typename T::Smem sm;
  const int NC = P.nchunks;
  const int b = blockIdx.x;
  const int x = b & 7, slot = b >> 3;
  const int grp = slot / NC, c = slot - grp * NC;
  const int bh = grp * 8 + x;
  if (bh >= P.BH) return;
  unsigned* sync = P.sync + 4 * bh;

  T ch;
  ch.load(P, sm, bh, c);
  ch.factors(sm);
  ch.stage_k(sm, true);
  ch.summary_out(P, sm, bh, c);
  seq_arrive(&sync[0]);

  f4 O[DV / 16];
  ch.intra(sm, O);

  seq_wait(&sync[0], (unsigned)NC, P.fault);
  {
    const int per = (DK * DV + NC - 1) / NC;
    const int e0 = min(c * per, DK * DV), e1 = min(e0 + per, DK * DV);
    scan_elements<DK, DV>(P, bh, e0, e1, threadIdx.x, T::NT);
  }
  seq_arrive(&sync[1]);
  seq_wait(&sync[1], (unsigned)NC, P.fault);

  if (c > 0 || P.s0) {
    f4 sbuf[T::SPER];
    ch.stage_state_load(P.states + ((int64_t)bh * NC + c) * (DK * DV), sbuf);
    ch.stage_state_store(sm, sbuf);
    __syncthreads();
    ch.readout(sm, O);
  }
  ch.store(P, sm, bh, c, O);

  if (threadIdx.x == 0) {
    const unsigned prev = __hip_atomic_fetch_add(&sync[2], 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
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
  const void* scan;
  int threads;
};

template <int DK, int DV, int C, int IN>
static KernelSet kernels_for() {
  return KernelSet{reinterpret_cast<const void*>(&gla_summary_kernel<DK, DV, C, IN>),
                   reinterpret_cast<const void*>(&gla_output_kernel<DK, DV, C, IN>),
                   reinterpret_cast<const void*>(&gla_fused_kernel<DK, DV, C, IN>),
                   reinterpret_cast<const void*>(&gla_scan_kernel<DK, DV>), tile_threads(C)};
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

// Largest number of work-groups of one sequence that can be resident on one XCD
// at once (8 XCDs per device); cached per (device, kernel).
static int fused_capacity_per_xcd(const void* kernel, int threads) {
  struct Entry {
    int dev;
    const void* k;
    int cap;
  };
  static std::mutex mu;
  static Entry cache[128];
  static int n = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  {
    std::lock_guard<std::mutex> lk(mu);
    for (int i = 0; i < n; ++i)
      if (cache[i].dev == dev && cache[i].k == kernel) return cache[i].cap;
  }
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  const int cap = per_cu * (cus / 8);
  std::lock_guard<std::mutex> lk(mu);
  if (n < 128) cache[n++] = Entry{dev, kernel, cap};
  return cap;
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
  P.groups = (int)((s.BH + 7) / 8);

  bool fused = false;
  if (a->path == GTR_PATH_FUSED || a->path == GTR_PATH_AUTO) {
    const int cap = fused_capacity_per_xcd(ks.fused, ks.threads);
    const bool fits = cap > 0 && s.nchunks <= cap;
    if (a->path == GTR_PATH_FUSED && !fits) return GTR_ERR_UNSUPPORTED;
    fused = fits;
  }

  void* kargs[] = {&P};
  hipError_t err;
  if (fused) {
    const int64_t blocks = (int64_t)8 * P.groups * s.nchunks;
    err = hipLaunchKernel(ks.fused, dim3((unsigned)blocks), dim3(ks.threads), kargs, 0, stream);
  } else {
    err = hipLaunchKernel(ks.summary, dim3((unsigned)s.nchunks, (unsigned)s.BH), dim3(ks.threads), kargs, 0, stream);
    if (err == hipSuccess) {
      const unsigned eb = (unsigned)((s.dk * s.dv + 255) / 256);
      err = hipLaunchKernel(ks.scan, dim3(eb, (unsigned)s.BH), dim3(256), kargs, 0, stream);
    }
    if (err == hipSuccess)
      err = hipLaunchKernel(ks.output, dim3((unsigned)s.nchunks, (unsigned)s.BH), dim3(ks.threads), kargs, 0, stream);
  }
  if (err != hipSuccess) return GTR_ERR_HIP;
  return hipGetLastError() == hipSuccess ? GTR_OK : GTR_ERR_HIP;
}
