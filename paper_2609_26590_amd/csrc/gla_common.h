// Device code shared by the chunkwise GLA kernels (gla_fwd.hip, gla_lean.hip):
// the call parameters, agent-coherent buffer accesses, raw loads and their
// conversion, the gate log-decay, and the boundary-state look-back of the
// one-launch schedule.
#pragma once

#include <hip/hip_runtime.h>

#include "gtr.h"
#include "gtr_device.h"
#include "gtr_internal.h"

namespace gtr {

constexpr float kSpanF16 = 10.f;           // mid-point factors within e^5: fp16 operands
constexpr float kSpanF32 = 60.f;           // within e^30: float32 operands
constexpr unsigned kSpinDefault = 1u << 22;  // polls of a bounded wait before it gives up
constexpr unsigned kFlagSummary = 1u;      // chunk flag: the summary U_c and the chunk record are stored
constexpr unsigned kFlagInclusive = 2u;    // chunk flag: the inclusive state S_[c+1] is stored
constexpr unsigned kFlagLocal = 4u;        // the summary and record went to the L2 of XCD (flag >> 8) & 15
// FUSED schedule: every kPublishEvery-th chunk (and no other) stores its
// inclusive state S_[c+1]; a look-back sums at most about that many summaries
// before it meets one, and the other chunks skip the store.
constexpr int kPublishEvery = 8;
// Grouped look-back (16-bit kernel, long sequences): the chunks form groups of
// kGroup; the last chunk e of a group stores the group's aggregate
//   A_g = sum_{j in group} (prod_{j<l<=e} Diag(d_l)) U_j,  D_g = prod_{j in group} d_j,
// so a chunk sums the summaries of its own group and then one aggregate per
// earlier group instead of every summary. Inclusive states are then stored at
// group ends only.
constexpr int kGroup = 16;
constexpr unsigned kFlagGroup = 8u;        // chunk flag (group ends): the group aggregate and its record are stored
constexpr float kF16Safe = 65504.f;        // bf16 inputs must stay within the fp16 range

// fault word bits (the workspace's first word; sticky until the workspace is
// initialised again)
constexpr unsigned kFaultWait = 1u;   // a bounded wait ran out
constexpr unsigned kFaultRange = 2u;  // a bf16 input lies outside the fp16 range
constexpr unsigned kFaultPlace = 4u;  // a chunk ran on another XCD than the summaries it needed

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
  void* agg;        // [NS][NC][DK][DVp] chunk summaries U_c: fp16 scaled (16-bit inputs) or float32
  float* rec;       // [NS][NC][DK][2] per chunk and key dim i: (d_c[i], the summary's scale)
  float* states;    // [NS][NC][DK][DVp] float32: S_[c+1] (one launch) or S_[c] (staged)
  unsigned* sync;   // [kSyncSeqs][4]: work-groups done per sequence
  unsigned* flags;  // [kSyncSeqs][kMaxChainChunks]: kFlagSummary | kFlagInclusive per chunk
  unsigned* fault;  // one word
  int gkind;        // GTR_GATE_LOG_DECAY or GTR_GATE_LOGITS (g holds the gate logits)
  float inv_tau;    // 1 / tau of the gate fusion
  const void* gate;  // output-gate pre-activation [BH][L][DV] (spatial), or null: no epilogue
  const float* nw;   // RMSNorm weight [DV], or null (ones)
  int gatedt;        // dtype of gate
  float eps;         // RMSNorm epsilon
  int dvp;      // row pitch (elements) of v, o, the gate, S0 and S_final: the full d_v
  int vparts;   // value split: work-groups per chunk, each d_v / vparts columns
  int ns;       // sequences: BH * vparts
  int desc;     // one launch: chunks in descending order (every work-group resident at once)
  int publish;  // one launch: store inclusive states
  int nxcd;     // one launch, 16-bit kernel: XCDs of the sequence-per-XCD grid (0: plain chunk-major grid)
  unsigned spin;  // polls of a bounded wait
  int group;      // one launch, 16-bit kernel: grouped look-back (kGroup chunks per group)
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
__device__ __forceinline__ u32x4 coh_load16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, kAgentCoherent);
}
__device__ __forceinline__ f4 coh_load4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(f4, coh_load16(r, byte_off));
}
__device__ __forceinline__ void coh_store1(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, (int)byte_off, 0, kAgentCoherent);
}
__device__ __forceinline__ float coh_load1(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)byte_off, 0, kAgentCoherent));
}

// Powers of two from an exponent in [-126, 127] (bit patterns, exact).
__device__ __forceinline__ float exp2i(int e) { return __builtin_bit_cast(float, (unsigned)(127 + e) << 23); }
// Exponent e such that m * 2^-e lies in [2^14, 2^15) for a finite m > 0 (0 for
// m = 0), clamped to [-100, 100]: scaling by 2^-e keeps the largest magnitude
// of a tile well inside the fp16 range and every other value at full fp16
// precision unless it is below 2^-24 of the largest.
__device__ __forceinline__ int fp16_exponent(float m) {
  const int b = (int)((__builtin_bit_cast(unsigned, m) >> 23) & 0xffu);
  const int e = m > 0.f ? b - 127 - 14 : 0;
  return e < -100 ? -100 : (e > 100 ? 100 : e);
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

// Maximum over the groups of N consecutive lanes (N = 4 or 8) with DPP
// (quad permutations, then the half-row mirror); every lane gets its group's
// maximum.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xf, 0xf, false));
}
template <int N>
__device__ __forceinline__ float group_max(float x) {
  x = fmaxf(x, dpp_mov<0xB1>(x));  // quad_perm [1,0,3,2]
  x = fmaxf(x, dpp_mov<0x4E>(x));  // quad_perm [2,3,0,1]
  if constexpr (N == 8) x = fmaxf(x, dpp_mov<0x141>(x));  // row_half_mirror: lane i <-> 7 - i
  return x;
}

// 8 elements of a summary piece (fp16 bits or float32) times w, added to acc.
template <bool F16>
struct Piece;
template <>
struct Piece<true> {
  u32x4 a;
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t elem) { a = coh_load16(r, elem * 2); }
  __device__ __forceinline__ void plain(const void* base, uint32_t elem) {
    a = *reinterpret_cast<const u32x4*>(static_cast<const _Float16*>(base) + elem);
  }
  __device__ __forceinline__ void fma_into(float (&acc)[8], float wt) const {
    const h8 h = __builtin_bit_cast(h8, a);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = fmaf(wt, (float)h[e], acc[e]);
  }
};
template <>
struct Piece<false> {
  u32x4 a, b;
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t elem) {
    a = coh_load16(r, elem * 4);
    b = coh_load16(r, elem * 4 + 16);
  }
  __device__ __forceinline__ void plain(const void* base, uint32_t elem) {
    const u32x4* p = reinterpret_cast<const u32x4*>(static_cast<const float*>(base) + elem);
    a = p[0];
    b = p[1];
  }
  __device__ __forceinline__ void fma_into(float (&acc)[8], float wt) const {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const unsigned ua = a[e], ub = b[e];
      acc[e] = fmaf(wt, __builtin_bit_cast(float, ua), acc[e]);
      acc[e + 4] = fmaf(wt, __builtin_bit_cast(float, ub), acc[e + 4]);
    }
  }
};
// 8 float32 elements of a state piece.
struct Piece32 {
  f4 a, b;
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t r, uint32_t elem) {
    a = coh_load4(r, elem * 4);
    b = coh_load4(r, elem * 4 + 16);
  }
  __device__ __forceinline__ void fma_into(float (&acc)[8], float wt) const {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[e] = fmaf(wt, a[e], acc[e]);
      acc[e + 4] = fmaf(wt, b[e], acc[e + 4]);
    }
  }
};

// ---------------------------------------------------------------------------
// Boundary state of chunk c by look-back (one launch):
//   S_[c] = sum_{j<c} (prod_{j<l<c} Diag(d_l)) U_j + (prod_{l<c} Diag(d_l)) S_0.
// The summaries of the chunks before c are summed nearest first; the sum stops
// at the nearest chunk j that has already stored its inclusive state S_[j+1]
// (FUSED schedule), which it takes with the decay product of the chunks in
// between, else it goes back to S_0.
// lookback_base: each wave polls the chunk flags, 64 chunks back at a time
// (lane l watches the l-th chunk back), until every summary after the nearest
// inclusive state is stored, and returns the chunk whose inclusive state ends
// the sum (-1: none, the sum reaches S_0; -2: the wait ran out; -3: a summary
// it needs sits in another XCD's L2, which the sequence-per-XCD grid of the
// 16-bit kernel should never produce). The waves decide alike (the same flags,
// each read after the chunk's own flag went up) but need not agree: each sums
// its own pieces, and the exchange after the look-back poisons everything if
// any of them failed.
// lookback_sum: each wave sums its own pieces (rows i of the [DK][DV] state),
// in batches of eight tiles with every load of a batch issued before any is
// used: the fp16 (or float32) pieces of the summary, the decays of its rows
// and the summary's scale from the chunk's record.
// ---------------------------------------------------------------------------
template <class T>
__device__ __forceinline__ int lookback_base(const GlaParams& P, const T& ch, int seq, int c, unsigned xcc = 0u) {
  const unsigned* fl = P.flags + (size_t)seq * kMaxChainChunks;
  int hi = c;
  unsigned cnt = 0;
  while (hi > 0) {
    const int n = hi < 64 ? hi : 64;
    int m;  // summaries before the nearest inclusive state in this window (n if there is none)
    for (;;) {
      const unsigned f =
          ch.lane < n ? __hip_atomic_load(&fl[hi - 1 - ch.lane], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
      const uint64_t inc = __builtin_amdgcn_ballot_w64((f & kFlagInclusive) != 0);
      const uint64_t rdy = __builtin_amdgcn_ballot_w64((f & kFlagSummary) != 0);
      m = inc ? (int)__builtin_ctzll(inc) : n;
      const uint64_t need = m >= 64 ? ~0ull : (1ull << m) - 1ull;
      if ((rdy & need) == need) {
        // a summary held in the L2 of another XCD is not visible here
        const uint64_t far = __builtin_amdgcn_ballot_w64((f & kFlagLocal) != 0 && ((f >> 8) & 15u) != xcc);
        if (far & need) return -3;
        break;
      }
      if (++cnt >= P.spin) return -2;
      __builtin_amdgcn_s_sleep(1);
    }
    if (m < n) return hi - 1 - m;
    hi -= n;
  }
  return -1;
}

// Adds n look-back items to acc, nearest first, continuing the decay product
// `run` (per row i: the product of d_l[i] over the chunks already passed). Item
// k is the summary of chunk first - k, or (AGG) the aggregate of group
// first - k, which sits with its record (D_g, scale) in the state slot of the
// group's second-to-last chunk (a chunk that never stores an inclusive state).
// The tiles go in batches of B with every load of a batch issued before any is
// used; inside a batch nothing branches: a tile past the n items (and every
// tile for a thread without a piece) is read at an offset past the
// descriptors' ranges, which returns zeros, and the decay product skips it.
template <class T, bool AGG>
__device__ __forceinline__ void sum_items(const GlaParams& P, int seq, int first, int n,
                                          float (&acc)[T::SPER][8], float& run) {
  constexpr int DK = T::kDK, DV = T::kDV, SPER = T::SPER, RS = T::RS;
  constexpr bool F16 = T::F16;
  static_assert(!AGG || F16, "group aggregates are fp16 tiles");
  // tiles per batch: about T::kLookRegs registers of loads per batch
  constexpr int R = T::kLookRegs;
  constexpr int B = R / (SPER * (F16 ? 4 : 8) + 2) < 1 ? 1 : R / (SPER * (F16 ? 4 : 8) + 2);
  const int NC = P.nchunks;
  const uint32_t tile = DK * DV * (F16 ? 2 : 4);
  const uint32_t slot = DK * DV * 4;  // a state slot (bytes)
  const __amdgpu_buffer_rsrc_t ar =
      AGG ? make_rsrc(P.states + (size_t)seq * NC * (DK * DV), (uint32_t)NC * slot)
          : make_rsrc(static_cast<char*>(P.agg) + (size_t)seq * NC * tile, (uint32_t)NC * tile);
  const __amdgpu_buffer_rsrc_t rr =
      AGG ? ar : make_rsrc(P.rec + (size_t)seq * NC * RS, (uint32_t)NC * RS * 4);
  const bool mine = T::piece_ok(0);
  const uint32_t row = (uint32_t)T::piece_i(0);
  for (int k1 = 0; k1 < n; k1 += B) {
    Piece<F16> u[B][SPER];
    f2 r[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const int j = first - k1 - b;
      const bool in = k1 + b < n && mine;
      const uint32_t s = (uint32_t)(j * kGroup + kGroup - 2);  // AGG: the slot of group j
      const uint32_t roff = AGG ? s * slot + tile + row * 8 : (uint32_t)(j * RS + 2 * (int)row) * 4;
      r[b] = __builtin_bit_cast(f2, __builtin_amdgcn_raw_buffer_load_b64(rr, in ? roff : kOutOfRange, 0,
                                                                         kAgentCoherent));
      const uint32_t e0 = AGG ? s * (slot / 2) : (uint32_t)j * (DK * DV);
#pragma unroll
      for (int mm = 0; mm < SPER; ++mm)
        u[b][mm].load(ar, in ? e0 + T::piece_elem(mm) : kOutOfRange / (F16 ? 2 : 4));
    }
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const bool in = k1 + b < n;
      const float wt = run * (F16 ? r[b][1] : 1.f);  // 0 for a tile read as zeros
#pragma unroll
      for (int mm = 0; mm < SPER; ++mm) u[b][mm].fma_into(acc[mm], wt);
      run = in ? run * r[b][0] : run;
    }
  }
}

// Ends a look-back: adds the inclusive state S_[base+1] that chunk `base`
// stored (base >= 0), or S_0 (base = -1, if there is one), with the decay
// product `run` of the chunks in between.
template <class T>
__device__ __forceinline__ void add_base(const GlaParams& P, int seq, int base, float run,
                                         float (&acc)[T::SPER][8]) {
  constexpr int DK = T::kDK, DV = T::kDV, SPER = T::SPER;
  const int NC = P.nchunks;
  const bool mine = T::piece_ok(0);
  const uint32_t row = (uint32_t)T::piece_i(0);
  if (base >= 0) {
    const __amdgpu_buffer_rsrc_t sr =
        make_rsrc(P.states + (size_t)seq * NC * (DK * DV), (uint32_t)NC * DK * DV * 4);
    Piece32 st[SPER];
#pragma unroll
    for (int mm = 0; mm < SPER; ++mm)
      if (mine) st[mm].load(sr, (uint32_t)base * (DK * DV) + T::piece_elem(mm));
#pragma unroll
    for (int mm = 0; mm < SPER; ++mm)
      if (mine) st[mm].fma_into(acc[mm], run);
  } else if (P.s0 && mine) {
    // S_0 with the decay product of every chunk before c
    const int bh = seq / P.vparts, part = seq - bh * P.vparts;
    const float* s0 = P.s0 + ((size_t)bh * DK + row) * P.dvp + part * DV;
#pragma unroll
    for (int mm = 0; mm < SPER; ++mm) {
      const f4* q = reinterpret_cast<const f4*>(s0 + T::piece_n0(mm));
      const f4 lo4 = q[0], hi4 = q[1];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[mm][e] = fmaf(run, lo4[e], acc[mm][e]);
        acc[mm][e + 4] = fmaf(run, hi4[e], acc[mm][e + 4]);
      }
    }
  }
}

template <class T>
__device__ __forceinline__ void lookback_sum(const GlaParams& P, const T& ch, int seq, int c, int base,
                                             float (&acc)[T::SPER][8]) {
#pragma unroll
  for (int m = 0; m < T::SPER; ++m)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[m][e] = 0.f;
  float run = 1.f;
  sum_items<T, false>(P, seq, c - 1, c - 1 - base, acc, run);
  add_base<T>(P, seq, base, run, acc);
}

// Grouped look-back, own group: polls the summary flags of the chunks lo..c-1
// (fewer than kGroup, none with an inclusive state) until every one is set.
// Returns 0, or -2 (the wait ran out) / -3 (a summary sits in another XCD's L2).
template <class T>
__device__ __forceinline__ int wait_own_group(const GlaParams& P, const T& ch, int seq, int lo, int c, unsigned xcc) {
  const unsigned* fl = P.flags + (size_t)seq * kMaxChainChunks;
  const int n = c - lo;
  if (n <= 0) return 0;
  const uint64_t need = (1ull << n) - 1ull;
  for (unsigned cnt = 0;;) {
    const unsigned f =
        ch.lane < n ? __hip_atomic_load(&fl[c - 1 - ch.lane], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
    const uint64_t rdy = __builtin_amdgcn_ballot_w64((f & kFlagSummary) != 0);
    if ((rdy & need) == need) {
      const uint64_t far = __builtin_amdgcn_ballot_w64((f & kFlagLocal) != 0 && ((f >> 8) & 15u) != xcc);
      return (far & need) ? -3 : 0;
    }
    if (++cnt >= P.spin) return -2;
    __builtin_amdgcn_s_sleep(1);
  }
}

// Grouped look-back, earlier groups: lane l watches the end chunk of group
// gc - 1 - l and the wait lasts until every group after the nearest inclusive
// state has its aggregate. Returns the chunk whose inclusive state ends the sum
// (-1: none, S_0) with `naggs` aggregates before it, or -2 (the wait ran out).
// Aggregates and inclusive states go through memory (agent-coherent stores),
// so their placement does not matter.
template <class T>
__device__ __forceinline__ int wait_groups(const GlaParams& P, const T& ch, int seq, int gc, int& naggs) {
  const unsigned* fl = P.flags + (size_t)seq * kMaxChainChunks;
  naggs = 0;
  if (gc <= 0) return -1;
  const int n = gc;  // kMaxChainChunks / kGroup <= 64 groups
  for (unsigned cnt = 0;;) {
    const unsigned f = ch.lane < n ? __hip_atomic_load(&fl[(gc - 1 - ch.lane) * kGroup + kGroup - 1],
                                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                   : 0u;
    const uint64_t inc = __builtin_amdgcn_ballot_w64((f & kFlagInclusive) != 0);
    const uint64_t agg = __builtin_amdgcn_ballot_w64((f & kFlagGroup) != 0);
    const int m = inc ? (int)__builtin_ctzll(inc) : n;
    const uint64_t need = m >= 64 ? ~0ull : (1ull << m) - 1ull;
    if ((agg & need) == need) {
      naggs = m;
      return m < n ? (gc - 1 - m) * kGroup + kGroup - 1 : -1;
    }
    if (++cnt >= P.spin) return -2;
    __builtin_amdgcn_s_sleep(1);
  }
}

// The one-launch kernels for 16-bit inputs at chunk 64 (gla_lean.hip): the
// whole-width kernel and the value-split one (d_v / 2 columns; null unless
// d_v = 64). Returns false (both null) for every other shape or dtype.
// occ3: at most 168 registers (three work-groups per CU), look-back batches of
// about 80 registers; occ4: at most 128 (four per CU), batches of about 40.
struct LeanKernels {
  const void* whole3;
  const void* split3;
  const void* whole4;
  const void* split4;
};
bool lean_kernels(int qdt, int dk, int dv, int chunk, LeanKernels* out);

}  // namespace gtr
