// Internal interface of the projection GEMM and RMSNorm kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"

namespace hpd {

constexpr int kGemmMaxTokenTiles = 9;      // token tiles of 16 per workgroup (144 rows)
constexpr int kGemmTokenGroup = 16 * kGemmMaxTokenTiles;
constexpr int kEpiQKV = 0, kEpiResidual = 1, kEpiSwiGLU = 2;

struct GemmArgs {
  const __bf16 *w0;         // W[N][K] (SwiGLU: gate rows)
  const __bf16 *w1;         // SwiGLU: up rows; otherwise unused
  int K;
  int N;                    // virtual output columns = 64 * n_slices
  int n_slices;             // 64-row slices of the (virtual) output
  int ksplit, k_per_wg;     // K = ksplit * k_per_wg, k_per_wg % 128 == 0
  int n_tgroups;            // token groups of kGemmTokenGroup rows
  const __bf16 *x_hi, *x_lo;   // [Tpad][K] activations (lo only when split)
  int T, Tpad;
  float *part;              // split-K partials [ksplit][Tpad][N] fp32
  // epilogues
  __bf16 *q_out; int n_q;                   // QKV: q[t][0..n_q)
  __bf16 *k_cache, *v_cache; int n_kv;      // QKV: cache rows dest[t]
  const int32_t *dest;
  __bf16 *m_hi, *m_lo; int I;               // SwiGLU output [Tpad][I]
};

// h[t] += sum over splits of part[ks][t][:] (part may be NULL), then
// x = RMSNorm(h) -> x_hi (+ x_lo) unless x_hi is NULL.
hipError_t launch_residual_norm(float *h, const float *part, int ksplit, int Tpad, int H, int T,
                                const __bf16 *gamma, float eps, __bf16 *x_hi, __bf16 *x_lo,
                                __bf16 *zero_rows, int zero_cols, hipStream_t stream);
hipError_t launch_gemm(const GemmArgs &g, bool split, int epi, int kind, hipStream_t stream);

}  // namespace hpd
