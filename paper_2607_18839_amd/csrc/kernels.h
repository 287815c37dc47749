// Internal launchers of the gfx950 kernels (not part of the public ABI).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "plan.h"

namespace hpd {

// Device views of the plan tables inside a workspace.
struct PlanDev {
  const int32_t *shared_items;
  const int32_t *private_items;
  const int32_t *token_slots;
  const int32_t *token_fork;
  const int32_t *token_dest;
  int32_t *counters;
  float *part_o;
  float *part_lse;
};

PlanDev plan_dev(const Plan &P, void *workspace);

// Kernel kinds of the optional benchmark timing (hpd_kernel_timing).
enum KernelKind { KK_SHARED = 0, KK_PRIVATE, KK_MERGE, KK_GEMM_QKV, KK_GEMM_O, KK_GEMM_GATE_UP,
                  KK_GEMM_DOWN, KK_NORM };
// Per-kernel timing (benchmark support).  When timing is on, timed_events
// hands out a pool pair for a launch of `kind` (else two nulls); launch()
// then binds the pair to the kernel's own dispatch (start and end of its
// execution, not markers around it).
struct TimedEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
TimedEvents timed_events(int kind);

template <typename... KArgs, typename... Args>
void launch(int kind, void (*kernel)(KArgs...), dim3 grid, dim3 block, hipStream_t stream, Args... args) {
  const TimedEvents ev = timed_events(kind);
  if (ev.start) hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, ev.start, ev.stop, 0, args...);
  else hipLaunchKernelGGL(kernel, grid, block, 0, stream, args...);
}

// One attention layer: shared-prefix kernel, private kernel, merge kernel.
// q/k/v in P.attn.dtype; out in P.attn.out_dtype; lse may be NULL.
hipError_t launch_branch_attention(const Plan &P, const void *q, const void *shared_k,
                                   const void *shared_v, const void *priv_k, const void *priv_v,
                                   void *out, float *lse, void *workspace, hipStream_t stream);

}  // namespace hpd
