// Host-side validation, workspace layout and status strings (no HIP calls).
#include <stdint.h>

#include "gtr.h"
#include "gtr_internal.h"

namespace gtr {

size_t dtype_size(int dt) {
  switch (dt) {
    case GTR_F32: return 4;
    case GTR_F16: return 2;
    case GTR_BF16: return 2;
    default: return 0;
  }
}

static bool mul_ok(int64_t a, int64_t b, int64_t* out) { return !__builtin_mul_overflow(a, b, out); }

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Range {
  uintptr_t lo, hi;  // [lo, hi)
};

static bool overlap(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

gtr_status gla_shape_from_args(const gtr_gla_args* a, GlaShape* s, bool check_pointers) {
  if (a->B <= 0 || a->heads <= 0 || a->H <= 0 || a->W <= 0 || a->dk <= 0 || a->dv <= 0 || a->chunk <= 0)
    return GTR_ERR_SHAPE;
  const bool dims_ok = (a->dk == 32 && a->dv == 32) || (a->dk == 32 && a->dv == 64) || (a->dk == 64 && a->dv == 64);
  if (!dims_ok) return GTR_ERR_UNSUPPORTED;
  if (a->chunk != 32 && a->chunk != 64 && a->chunk != 128) return GTR_ERR_UNSUPPORTED;
  const int q = a->qkv_dtype;
  if (q != GTR_F32 && q != GTR_F16 && q != GTR_BF16) return GTR_ERR_UNSUPPORTED;
  if (a->g_dtype != q && a->g_dtype != GTR_F32) return GTR_ERR_UNSUPPORTED;
  if (a->o_dtype != q && a->o_dtype != GTR_F32) return GTR_ERR_UNSUPPORTED;
  if (a->scan < GTR_SCAN_ROW || a->scan > GTR_SCAN_COL_REV) return GTR_ERR_UNSUPPORTED;
  if (a->path < GTR_PATH_AUTO || a->path > GTR_PATH_INLINE) return GTR_ERR_UNSUPPORTED;
  if (a->g_kind != GTR_GATE_LOG_DECAY && a->g_kind != GTR_GATE_LOGITS) return GTR_ERR_UNSUPPORTED;
  if (a->g_kind == GTR_GATE_LOGITS && !(a->gate_tau > 0.f && a->gate_tau <= 3.0e38f)) return GTR_ERR_UNSUPPORTED;
  if (a->out_gate) {
    if (a->out_gate_dtype != q && a->out_gate_dtype != GTR_F32) return GTR_ERR_UNSUPPORTED;
    if (!(a->norm_eps > 0.f && a->norm_eps <= 3.0e38f)) return GTR_ERR_UNSUPPORTED;
  }

  int64_t BH, L, n;
  if (!mul_ok(a->B, a->heads, &BH) || !mul_ok(a->H, a->W, &L)) return GTR_ERR_SHAPE;
  const int dmax = a->dk > a->dv ? a->dk : a->dv;
  if (!mul_ok(BH, L, &n) || !mul_ok(n, dmax, &n) || !mul_ok(n, 4, &n)) return GTR_ERR_SHAPE;
  // the kernels address one sequence's rows through a buffer descriptor with
  // a 32-bit range (and use 0x7fffff00 as their out-of-range offset)
  if (L * dmax * 4 >= 0x7fffff00LL) return GTR_ERR_SHAPE;
  const int64_t nchunks = (L + a->chunk - 1) / a->chunk;
  // launch-grid limits: staged grids are (nchunks, BH); the one-launch grid is
  // 1-D, at most (2 BH rounded up to 8) * nchunks work-groups
  int64_t chain_blocks;
  if (BH > 65535 || nchunks > 0x7fffffff) return GTR_ERR_SHAPE;
  if (!mul_ok((2 * BH + 7) / 8 * 8, nchunks, &chain_blocks) || chain_blocks > 0x7fffffff) return GTR_ERR_SHAPE;
  int64_t st;
  if (!mul_ok(BH * nchunks, (int64_t)a->dk * a->dv * 4, &st)) return GTR_ERR_SHAPE;

  s->BH = BH;
  s->L = L;
  s->nchunks = nchunks;
  s->dk = a->dk;
  s->dv = a->dv;
  s->chunk = a->chunk;
  s->qdt = q;
  s->gdt = a->g_dtype;
  s->odt = a->o_dtype;
  if (!check_pointers) return GTR_OK;

  if (!a->q || !a->k || !a->v || !a->g || !a->o) return GTR_ERR_NULL;
  // 16-byte vector loads and stores on every token row
  const uintptr_t mis = reinterpret_cast<uintptr_t>(a->q) | reinterpret_cast<uintptr_t>(a->k) |
                        reinterpret_cast<uintptr_t>(a->v) | reinterpret_cast<uintptr_t>(a->g) |
                        reinterpret_cast<uintptr_t>(a->o);
  if (mis & 15u) return GTR_ERR_UNSUPPORTED;
  if ((reinterpret_cast<uintptr_t>(a->s0) | reinterpret_cast<uintptr_t>(a->s_final)) & 3u) return GTR_ERR_UNSUPPORTED;
  // the epilogue reads 8 gate values and 8 weights of a row at a time
  if ((reinterpret_cast<uintptr_t>(a->out_gate) | reinterpret_cast<uintptr_t>(a->norm_weight)) & 15u)
    return GTR_ERR_UNSUPPORTED;

  const size_t qs = dtype_size(q), gs = dtype_size(a->g_dtype), os = dtype_size(a->o_dtype);
  const size_t ntok = (size_t)(BH * L);
  auto rng = [](const void* p, size_t bytes) {
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Range{lo, lo + bytes};
  };
  const Range rq = rng(a->q, ntok * a->dk * qs), rk = rng(a->k, ntok * a->dk * qs);
  const Range rv = rng(a->v, ntok * a->dv * qs), rg = rng(a->g, ntok * a->dk * gs);
  const Range ro = rng(a->o, ntok * a->dv * os);
  const size_t sbytes = (size_t)BH * a->dk * a->dv * 4;
  const Range rs0 = a->s0 ? rng(a->s0, sbytes) : Range{0, 0};
  const Range rsf = a->s_final ? rng(a->s_final, sbytes) : Range{0, 0};

  const WorkspaceLayout lay = gla_workspace_layout(*s);
  if (!a->workspace) return GTR_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(a->workspace) & 255u) return GTR_ERR_WORKSPACE;
  if (a->workspace_bytes < lay.total) return GTR_ERR_WORKSPACE;
  const Range rw = rng(a->workspace, lay.total);

  const Range rgate = a->out_gate ? rng(a->out_gate, ntok * a->dv * dtype_size(a->out_gate_dtype)) : Range{0, 0};
  const Range rnw = a->out_gate && a->norm_weight ? rng(a->norm_weight, (size_t)a->dv * 4) : Range{0, 0};
  const Range ins[] = {rq, rk, rv, rg, rs0, rgate, rnw};
  for (const Range& r : ins) {
    if (overlap(ro, r) || overlap(rsf, r) || overlap(rw, r)) return GTR_ERR_ALIAS;
  }
  if (overlap(ro, rsf) || overlap(ro, rw) || overlap(rsf, rw)) return GTR_ERR_ALIAS;
  return GTR_OK;
}

WorkspaceLayout gla_workspace_layout(const GlaShape& s) {
  WorkspaceLayout w;
  size_t off = 0;
  w.fault_off = off;
  off += 256;
  w.sync_off = off;
  off = align256(off + (size_t)kSyncSeqs * 4 * sizeof(uint32_t));
  w.flags_off = off;
  off = align256(off + (size_t)kSyncSeqs * kMaxChainChunks * sizeof(uint32_t));
  const size_t tiles = (size_t)s.BH * s.nchunks;  // (sequence, chunk) pairs; the value split keeps the total
  w.agg_off = off;
  off = align256(off + tiles * s.dk * s.dv * (s.qdt == GTR_F32 ? 4 : 2));
  w.rec_off = off;
  off = align256(off + 2 * tiles * (2 * s.dk) * sizeof(float));  // two records per chunk under the value split
  w.states_off = off;
  off = align256(off + tiles * s.dk * s.dv * sizeof(float));
  w.total = off;
  return w;
}

}  // namespace gtr

extern "C" const char* gtr_status_string(gtr_status st) {
  switch (st) {
    case GTR_OK: return "GTR_OK";
    case GTR_ERR_NULL: return "GTR_ERR_NULL: a required pointer is NULL";
    case GTR_ERR_SHAPE: return "GTR_ERR_SHAPE: a size is not positive or a product overflows";
    case GTR_ERR_UNSUPPORTED: return "GTR_ERR_UNSUPPORTED: dtype, head width, chunk, direction, path or alignment not supported";
    case GTR_ERR_ALIAS: return "GTR_ERR_ALIAS: an output overlaps an input or the workspace";
    case GTR_ERR_WORKSPACE: return "GTR_ERR_WORKSPACE: workspace missing, too small or misaligned";
    case GTR_ERR_HIP: return "GTR_ERR_HIP: the HIP runtime rejected a launch";
    case GTR_ERR_SCRATCH: return "GTR_ERR_SCRATCH: the call needs more workspace than the fixed scratch of gtr_gla_fwd_noalloc holds";
    default: return "unknown gtr_status";
  }
}
