// Host-side argument validation and workspace layout for libgtr.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "gtr.h"

namespace gtr {

struct GlaShape {
  int64_t BH;       // B * heads
  int64_t L;        // H * W
  int64_t nchunks;  // ceil(L / chunk)
  int dk, dv, chunk;
  int qdt, gdt, odt;
};

// The synchronisation words of the one-launch schedule (a done count per
// sequence, one flag per chunk) live in regions of fixed size right after the
// 256-byte header, for kSyncSeqs sequences of up to kMaxChainChunks chunks,
// whatever the shape of a call: the word of (sequence s, chunk c) is always at
// the same place, and every completed call leaves them zeroed, so one workspace
// serves calls of different shapes. Everything else starts behind them.
constexpr int64_t kSyncSeqs = 1024;
constexpr int64_t kMaxChainChunks = 256;

struct WorkspaceLayout {
  size_t fault_off;   // one 32-bit word: fault bits of the calls since the last init
  size_t sync_off;    // [kSyncSeqs][4] 32-bit counters
  size_t flags_off;   // [kSyncSeqs][kMaxChainChunks] 32-bit chunk flags
  size_t agg_off;     // [BH][nchunks][dk][dv] summaries: fp16 (16-bit inputs) or float32
  size_t rec_off;     // [2 BH][nchunks][dk][2] float32 chunk records (decay, summary scale)
  size_t states_off;  // [BH][nchunks][dk][dv] float32 boundary states
  size_t total;
};

// Validates everything but the workspace size (and, if check_pointers, the
// pointers, their alignment and aliasing). No HIP call.
gtr_status gla_shape_from_args(const gtr_gla_args* a, GlaShape* s, bool check_pointers);

WorkspaceLayout gla_workspace_layout(const GlaShape& s);

size_t dtype_size(int dt);

}  // namespace gtr
