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
// overflows half precision as soon as |A| > 11: every exponent evaluated here is
// <= 0 except on the diagonal 16x16 blocks (see below), so all rescaled matrix
// operands are bounded by |q| and |k|.
//   * The chunk is split into 16-token sub-chunks R. Local cumulative sums a_r
//     (within R), sub-chunk totals T_R and a per-dimension reference at the first
//     token of R are kept in fp32 registers; every exponent is built from sums of
//     these small terms, never as a difference of two large cumulative sums.
//   * Off-diagonal score blocks (J < R) use q_r*exp(A_r - A_f(R)) and
//     k_j*exp(A_f(R) - A_j), both with exponent <= 0, on fp16 matrix cores
//     (float32 cores for float32 inputs).
//   * Diagonal blocks use a mid-point reference: both factors lie within
//     exp(+-span/2), span = decay across the 16 tokens; they run on float32 matrix
//     cores. If span exceeds kSpanLimit the block falls back to exact per-element
//     exp(a_r - a_j) on the vector ALUs.
//
// Schedules:
//   * staged: summary kernel -> boundary-state scan kernel -> output kernel.
//   * fused : one launch; each work-group owns one (sequence, chunk), publishes
//     its summary, and the work-groups of one sequence then run the boundary
//     state scan cooperatively (each takes a slice of the d_k x d_v state) before
//     reading their own S_[c]. Two per-sequence counters order the phases.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "gtr.h"
#include "gtr_device.h"
#include "gtr_internal.h"

namespace gtr {

constexpr float kSpanLimit = 60.f;     // diagonal blocks: mid-point factors stay within e^30
constexpr unsigned kSpinLimit = 1u << 22;  // bounded waits (fused schedule)
constexpr bool kFusedEnabled = false;     // see gtr_gla_fwd

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

template <bool F16>
__device__ __forceinline__ float gexp(float x) {
  if constexpr (F16)
    return __expf(x);
  else
    return expf(x);
}

template <int DK, int DV, int C, bool F16>
struct Tile {
  static constexpr int NW = C / 16;  // one wave per 16-token sub-chunk
  static constexpr int NT = NW * kWave;
  static constexpr int KS = DK / 32;
  static constexpr int VS = DV / 32;
  static constexpr int KP = DK + 4;  // padded fp32 row pitch (k rows / output rows)
  static constexpr int OP = DV + 4;
  static constexpr int BUFW = KP > OP ? KP : OP;
  static constexpr int TP = F16 ? C + 8 : C + 4;  // transposed-tile pitch (elements)
  typedef typename Op<F16>::elem E;
  typedef typename Op<F16>::frag8 F8;
  typedef typename Op<F16>::frag4 F4;

  struct Smem {
    float buf[C * BUFW];  // k*exp(T-a) rows [C][KP]; later the output tile [C][OP]
    E kT[DK * TP];        // (k * exp(A_last - A_r))^T  [DK][TP]
    E vT[DV * TP];        // v^T                       [DV][TP]
    float T[NW * DK];     // sub-chunk totals of g
  };

  // per-lane state after the prologue
  int w, lane, tr, gq;
  int64_t L;
  float qh[KS][8];   // q * exp(a - a_first)                  (off-diagonal B operand)
  float qt[KS][8];   // q * exp(A_r)                          (state readout)
  float qd[KS][8];   // mid-point diagonal factors
  float kd[KS][8];
  float g0[KS][8];   // a at the first token of this sub-chunk (= g there)
  float spanmax;     // wave-uniform
  bool exact_diag;
  float qraw[KS][8], kraw[KS][8], aloc[KS][8];  // kept for the exact diagonal path

  __device__ __forceinline__ int dim(int s, int e) const { return 32 * s + 8 * gq + e; }

  // Load the chunk, build the cumulative sums and rescaled operands; fills the
  // shared tiles. `summary` also builds the transposed k-hat tile.
  __device__ __forceinline__ void prologue(const GlaParams& P, Smem& sm, int bh, int c, bool summary) {
    w = threadIdx.x >> 6;
    lane = threadIdx.x & 63;
    tr = lane & 15;
    gq = lane >> 4;
    L = P.L;
    const int r = 16 * w + tr;
    const int64_t pos = (int64_t)c * C + r;
    const bool valid = pos < L;
    const int64_t t = valid ? scan_to_spatial(pos, P.H, P.W, P.scan) : 0;
    const int64_t kb = ((int64_t)bh * L + t) * DK;
    const int64_t vb = ((int64_t)bh * L + t) * DV;

    float gv[KS][8], vv[VS][8];
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      if (valid) {
        load8(P.q, P.qdt, kb + 32 * s + 8 * gq, qraw[s]);
        load8(P.k, P.qdt, kb + 32 * s + 8 * gq, kraw[s]);
        load8(P.g, P.gdt, kb + 32 * s + 8 * gq, gv[s]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qraw[s][e] = kraw[s][e] = gv[s][e] = 0.f;
      }
    }
#pragma unroll
    for (int s = 0; s < VS; ++s) {
      if (valid) {
        load8(P.v, P.qdt, vb + 32 * s + 8 * gq, vv[s]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) vv[s][e] = 0.f;
      }
    }

    // local inclusive cumulative sums over the 16 tokens of this sub-chunk
    float T[KS][8];
    float smax = 0.f;
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float a = row_inclusive_scan(gv[s][e]);
        aloc[s][e] = a;
        T[s][e] = row_read(a, 15);
        g0[s][e] = row_read(a, 0);
        smax = fmaxf(smax, g0[s][e] - T[s][e]);
      }
    spanmax = wave_max(smax);
    exact_diag = !(spanmax <= kSpanLimit);

    if (tr == 0) {
#pragma unroll
      for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int e = 0; e < 8; ++e) sm.T[w * DK + dim(s, e)] = T[s][e];
    }
    // transposed v tile
#pragma unroll
    for (int s = 0; s < VS; ++s)
#pragma unroll
      for (int e = 0; e < 8; ++e) sm.vT[(32 * s + 8 * gq + e) * TP + r] = (E)vv[s][e];
    __syncthreads();

    // chunk-level prefix of sub-chunk totals
#pragma unroll
    for (int s = 0; s < KS; ++s) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = dim(s, e);
        float before = 0.f, after = 0.f;  // sum of totals before / after sub-chunk w
        for (int K = 0; K < NW; ++K) {
          const float tk = sm.T[K * DK + d];
          if (K < w) before += tk;
          if (K > w) after += tk;
        }
        const float a = aloc[s][e];
        const float e_q = gexp<F16>(a - g0[s][e]);      // exp(A_r - A_first) <= 1
        const float e_k = gexp<F16>(T[s][e] - a);       // exp(A_last(R) - A_r) <= 1
        const float qhv = qraw[s][e] * e_q;
        const float kev = kraw[s][e] * e_k;
        qh[s][e] = qhv;
        qt[s][e] = qhv * gexp<F16>(before + g0[s][e]);  // exp(A_r) = e_q * exp(A_first)
        const float half = gexp<F16>(0.5f * (g0[s][e] - T[s][e]));
        qd[s][e] = qhv * half;
        kd[s][e] = kev * half;
        sm.buf[r * KP + d] = kev;
        if (summary) sm.kT[d * TP + r] = (E)(kev * gexp<F16>(after));  // exp(A_last - A_r)
      }
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
    if (w == 0 && tr == 0) {
      float* dec = P.decays + ((int64_t)bh * P.nchunks + c) * DK;
#pragma unroll
      for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int d = dim(s, e);
          float tot = 0.f;
          for (int K = 0; K < NW; ++K) tot += sm.T[K * DK + d];
          dec[d] = gexp<F16>(tot);
        }
    }
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
        // P^T[j][r] = sum_d (k_j exp(A_f(R) - A_j))[d] (q_r exp(A_r - A_f(R)))[d]
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          float x[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int d = dim(s, e);
            float between = g0[s][e];  // A_f(R) - A_last(J) = g_f(R) + totals in between
            for (int K = J + 1; K < w; ++K) between += sm.T[K * DK + d];
            x[e] = sm.buf[(16 * J + tr) * KP + d] * gexp<F16>(between);
          }
          PT[J] = mma32(Op<F16>::pack8(x), qhf[s], PT[J]);
        }
      } else if (J == w) {
        if (!exact_diag) {
#pragma unroll
          for (int s = 0; s < KS; ++s) {
            f8 a, b;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              a[e] = kd[s][e];
              b[e] = qd[s][e];
            }
            PT[J] = mma32(a, b, PT[J]);
          }
        } else {
          PT[J] = exact_diagonal();
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

  // Exact diagonal block, P^T layout; only for sub-chunks whose decay span is
  // beyond what the mid-point factors can carry.
  __device__ __forceinline__ f4 exact_diagonal() {
    float part[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) part[j] = 0.f;
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const float kj = row_read(kraw[s][e], j);
          const float aj = row_read(aloc[s][e], j);
          if (j <= tr) part[j] += qraw[s][e] * kj * gexp<F16>(aloc[s][e] - aj);
        }
      }
    f4 res = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      float x = part[j];
      x += __shfl_xor(x, 16, kWave);
      x += __shfl_xor(x, 32, kWave);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (4 * gq + e == j) res[e] = x;
    }
    return res;
  }

  // o_r += (q_r exp(A_r)) S_[c]; S^T read from the workspace ([DV][DK] fp32).
  __device__ __forceinline__ void readout(const float* ST, f4 (&O)[DV / 16]) {
    F8 qtf[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s) qtf[s] = Op<F16>::pack8(qt[s]);
#pragma unroll
    for (int jb = 0; jb < DV / 16; ++jb) {
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const f4* p = reinterpret_cast<const f4*>(&ST[(16 * jb + tr) * DK + 32 * s + 8 * gq]);
        const f4 x0 = p[0], x1 = p[1];
        float x[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
        O[jb] = mma32(qtf[s], Op<F16>::pack8(x), O[jb]);
      }
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
      const int r = idx / PIECES, pc = idx % PIECES;
      const int64_t pos = (int64_t)c * C + r;
      if (pos < P.L) {
        const int64_t t = scan_to_spatial(pos, P.H, P.W, P.scan);
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = sm.buf[r * OP + 8 * pc + e];
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
template <int DK, int DV, int C, bool F16>
__global__ void __launch_bounds__(tile_threads(C)) gla_summary_kernel(GlaParams P) {
  typedef Tile<DK, DV, C, F16> T;
  __shared__ typename T::Smem sm;
  T tile;
  const int c = blockIdx.x, bh = blockIdx.y;
  tile.prologue(P, sm, bh, c, true);
  tile.summary_out(P, sm, bh, c);
}

template <int DK, int DV>
__global__ void __launch_bounds__(256) gla_scan_kernel(GlaParams P) {
  const int bh = blockIdx.y;
  const int e0 = blockIdx.x * 256;
  const int e1 = min(e0 + 256, DK * DV);
  scan_elements<DK, DV>(P, bh, e0, e1, threadIdx.x, 256);
}

template <int DK, int DV, int C, bool F16>
__global__ void __launch_bounds__(tile_threads(C)) gla_output_kernel(GlaParams P) {
  typedef Tile<DK, DV, C, F16> T;
  __shared__ typename T::Smem sm;
  T tile;
  const int c = blockIdx.x, bh = blockIdx.y;
  tile.prologue(P, sm, bh, c, false);
  f4 O[DV / 16];
  tile.intra(sm, O);
  if (c > 0 || P.s0) tile.readout(P.states + ((int64_t)bh * P.nchunks + c) * (DK * DV), O);
  tile.store(P, sm, bh, c, O);
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
template <int DK, int DV, int C, bool F16>
__global__ void __launch_bounds__(tile_threads(C)) gla_fused_kernel(GlaParams P) {
  typedef Tile<DK, DV, C, F16> T;
  __shared__ typename T::Smem sm;
  const int NC = P.nchunks;
  const int b = blockIdx.x;
  const int x = b & 7, slot = b >> 3;
  const int grp = slot / NC, c = slot - grp * NC;
  const int bh = grp * 8 + x;
  if (bh >= P.BH) return;
  unsigned* sync = P.sync + 4 * bh;

  T tile;
  tile.prologue(P, sm, bh, c, true);
  tile.summary_out(P, sm, bh, c);
  seq_arrive(&sync[0]);

  f4 O[DV / 16];
  tile.intra(sm, O);

  seq_wait(&sync[0], (unsigned)NC, P.fault);
  {
    const int per = (DK * DV + NC - 1) / NC;
    const int e0 = min(c * per, DK * DV), e1 = min(e0 + per, DK * DV);
    scan_elements<DK, DV>(P, bh, e0, e1, threadIdx.x, T::NT);
  }
  seq_arrive(&sync[1]);
  seq_wait(&sync[1], (unsigned)NC, P.fault);

  if (c > 0 || P.s0) tile.readout(P.states + ((int64_t)bh * NC + c) * (DK * DV), O);
  tile.store(P, sm, bh, c, O);

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

template <int DK, int DV, int C, bool F16>
static KernelSet kernels_for() {
  return KernelSet{reinterpret_cast<const void*>(&gla_summary_kernel<DK, DV, C, F16>),
                   reinterpret_cast<const void*>(&gla_output_kernel<DK, DV, C, F16>),
                   reinterpret_cast<const void*>(&gla_fused_kernel<DK, DV, C, F16>),
                   reinterpret_cast<const void*>(&gla_scan_kernel<DK, DV>), Tile<DK, DV, C, F16>::NT};
}

template <int DK, int DV, bool F16>
static bool pick_chunk(int chunk, KernelSet* ks) {
  switch (chunk) {
    case 32: *ks = kernels_for<DK, DV, 32, F16>(); return true;
    case 64: *ks = kernels_for<DK, DV, 64, F16>(); return true;
    case 128: *ks = kernels_for<DK, DV, 128, F16>(); return true;
    default: return false;
  }
}

template <bool F16>
static bool pick_dims(int dk, int dv, int chunk, KernelSet* ks) {
  if (dk == 32 && dv == 32) return pick_chunk<32, 32, F16>(chunk, ks);
  if (dk == 32 && dv == 64) return pick_chunk<32, 64, F16>(chunk, ks);
  if (dk == 64 && dv == 64) return pick_chunk<64, 64, F16>(chunk, ks);
  return false;
}

static bool select_kernels(const GlaShape& s, KernelSet* ks) {
  if (s.qdt == GTR_F32) return pick_dims<false>(s.dk, s.dv, s.chunk, ks);
  return pick_dims<true>(s.dk, s.dv, s.chunk, ks);
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
  static Entry cache[64];
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
  if (n < 64) cache[n++] = Entry{dev, kernel, cap};
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

  // The fused schedule is switched off: its first run on a 12-sequence bf16
  // workload ended in a GPU memory-aperture fault whose cause has not been
  // found. Until it is, only the staged schedule runs.
  if (a->path == GTR_PATH_FUSED && !kFusedEnabled) return GTR_ERR_UNSUPPORTED;
  bool fused = false;
  if (kFusedEnabled && (a->path == GTR_PATH_FUSED || a->path == GTR_PATH_AUTO)) {
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
