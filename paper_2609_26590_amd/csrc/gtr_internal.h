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

// The per-sequence hand-off counters of the one-launch schedules live in a
// region of fixed size right after the 256-byte header, for this many
// sequences, whatever the shape of a call. Everything else of a workspace
// starts behind it, so no call of any shape ever writes where another call
// expects zeroed counters (one workspace can serve calls of different shapes).
constexpr int64_t kSyncSeqs = 1024;

struct WorkspaceLayout {
  size_t fault_off;   // one 32-bit word (fused-path wait ran out)
  size_t sync_off;    // [kSyncSeqs][4] 32-bit counters
  size_t states_off;  // [BH][nchunks][dv][dk] float32 (float32 inputs only, else size 0)
  size_t decays_off;  // [BH][nchunks][dk] float32
  size_t states16_off;  // [BH][nchunks][dv][dk] fp16 (16-bit inputs only, else 0)
  size_t total;
};

// Validates everything but the workspace size (and, if check_pointers, the
// pointers, their alignment and aliasing). No HIP call.
gtr_status gla_shape_from_args(const gtr_gla_args* a, GlaShape* s, bool check_pointers);

WorkspaceLayout gla_workspace_layout(const GlaShape& s);

size_t dtype_size(int dt);

}  // namespace gtr
