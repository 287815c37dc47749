// Internal launchers of the gfx950 kernels (not part of the public ABI).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "plan.h"

namespace hpd {

// Device views of the plan tables inside a workspace.
struct PlanDev {
  const int32_t *shared_tiles;   // paged K/V: pool row of each 64-key tile
  const int32_t *priv_tiles;
  const int32_t *branch_q_row;   // [nb] first token of branch b
  const int32_t *branch_new;     // [nb] k_b
  const int32_t *shared_items;
  const int32_t *private_items;
  const int32_t *token_slots;
  const int32_t *token_fork;
  const int32_t *token_dest;
  const int32_t *token_vis;   // [T] visible keys of token t (its position + 1)
  int32_t *counters;
  float *part_o;
  float *part_lse;
};

PlanDev plan_dev(const Plan &P, void *workspace);

// Kernel kinds of the optional benchmark timing (hpd_kernel_timing).
enum KernelKind { KK_SHARED = 0, KK_PRIVATE, KK_MERGE, KK_GEMM_QKV, KK_GEMM_O, KK_GEMM_GATE_UP,
                  KK_GEMM_DOWN, KK_NORM, KK_LM_HEAD, KK_VERIFY, KK_DRAFT_MLP, KK_DRAFT_TOKEN, KK_EMBED, KK_QK_ROPE };
// Element offset of (row, col) of a [rows][cols] 16-bit matrix in the packed
// layout (tiles of 32 rows x 64 columns, 2048 elements each, ordered by row
// tile then column tile; inside a tile, element e of 16-byte piece (j, l) is
// row l % 32, column 32 (l / 32) + 8 j + e).  Four consecutive columns
// starting at a multiple of 4 are contiguous.  cols % 64 == 0.
__device__ __forceinline__ int64_t packed_offset(int row, int col, int cols) {
  const int kk = col & 63, l = 32 * (kk >> 5) + (row & 31), j = (kk & 31) >> 3;
  return ((int64_t)(row >> 5) * (cols >> 6) + (col >> 6)) * 2048 + j * 512 + l * 8 + (kk & 7);
}

// Per-kernel timing (benchmark support).  When timing is on, timed_events
// hands out a pool pair for a launch of `kind` (else two nulls); launch()
// then binds the pair to the kernel's own dispatch (start and end of its
// execution, not markers around it).
struct TimedEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
TimedEvents timed_events(int kind);
bool attn_phase_isolation();   // hpd_attn_phase_isolation

// A roctx range (HPD_ROCTX=1) for the lifetime of the object: phases of a
// step in a profiler's marker trace.
class TraceRange {
 public:
  explicit TraceRange(const char *name);
  ~TraceRange();
  TraceRange(const TraceRange &) = delete;
  TraceRange &operator=(const TraceRange &) = delete;

 private:
  bool on_;
};
// Consecutive phases: next() closes the current range and opens another.
class TracePhase {
 public:
  explicit TracePhase(const char *name);
  void next(const char *name);
  ~TracePhase();
  TracePhase(const TracePhase &) = delete;
  TracePhase &operator=(const TracePhase &) = delete;

 private:
  bool on_;
};

template <typename... KArgs, typename... Args>
void launch(int kind, void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t stream, Args... args) {
  const TimedEvents ev = timed_events(kind);
  if (ev.start) hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, ev.start, ev.stop, 0, args...);
  else hipLaunchKernelGGL(kernel, grid, block, 0, stream, args...);
}

// One attention layer: the shared-prefix and private work (one launch for
// bf16, two for fp32), then the merge.  q/k/v in P.attn.dtype; out in
// P.attn.out_dtype, [T][Hq * 64], row-major or (out_packed, bf16 only) in
// the packed layout; lse may be NULL.
hipError_t launch_branch_attention(const Plan &P, const void *q, const void *shared_k,
                                   const void *shared_v, const void *priv_k, const void *priv_v,
                                   void *out, float *lse, void *workspace, hipStream_t stream,
                                   bool out_packed = false);

}  // namespace hpd
