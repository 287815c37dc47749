// Internal interface of the projection GEMM and RMSNorm kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"

namespace hpd {

constexpr int kGemmTile = 32;             // weight rows and tokens of one wave's output tile
constexpr int kGemmKStep = 64;            // K per pipeline step (4 MFMAs of 16)
constexpr int kEpiQKV = 0, kEpiResidual = 1, kEpiSwiGLU = 2;

// One projection Y[t][n] = sum_k X[t][k] W[n][k].  A workgroup of 4 waves
// owns the output tile of 32 rg weight rows x 32 tokens over K range
// [ks * k_per_wg, (ks + 1) * k_per_wg): wave w takes rows 32 (w % rg) .. and
// the K quarter/half w / rg of that range (rg * kg = 4).
struct GemmArgs {
  const __bf16 *w0;         // W[N][K] (SwiGLU: gate rows [I][K])
  const __bf16 *w1;         // SwiGLU: up rows [I][K]; otherwise unused
  int K;
  int N;                    // output columns (SwiGLU: 2 I, gate and up)
  int rg;                   // row groups per workgroup: 1, 2 or 4
  int n_slices;             // N / (32 rg)
  int ksplit, k_per_wg;     // K = ksplit * k_per_wg; k_per_wg % (64 * 4 / rg) == 0
  int n_ttiles;             // Tpad / 32
  const __bf16 *x;          // [Tpad][K] activations (bf16, or fp16 for the MLP), rows >= T finite
  int T, Tpad;
  float *part;              // residual epilogue: [ksplit][Tpad][N] fp32 (rows < T written)
  // epilogues
  __bf16 *q_out; int n_q;                   // QKV: q[t][0..n_q)
  __bf16 *k_cache, *v_cache; int n_kv;      // QKV: cache rows dest[t]
  const int32_t *dest;
  __bf16 *m_out; int I;                     // SwiGLU output [Tpad][I], fp16 bits (rows >= T zero)
};

// h[t] += sum over splits of part[ks][t][:] (part may be NULL), then
// x = RMSNorm(h) -> x_out (bf16, or fp16 if out_f16) unless x_out is NULL.
hipError_t launch_residual_norm(float *h, const float *part, int ksplit, int Tpad, int H, int T,
                                const __bf16 *gamma, float eps, void *x_out, bool out_f16,
                                __bf16 *zero_rows, int zero_cols, hipStream_t stream);
// f16: fp16 GEMM (bf16 weights converted to fp16 in registers, fp16
// activations); epi: kEpi*.  The QKV and SwiGLU epilogues need ksplit == 1.
hipError_t launch_gemm(const GemmArgs &g, bool f16, int epi, int kind, hipStream_t stream);

// Tile choice for an N x K projection over Tpad tokens: rg, ksplit and the
// register ring depth, from a model of the bytes each CU has to stream.
struct GemmShape {
  int rg, ksplit;
};
GemmShape choose_gemm_shape(int N, int K, int Tpad, int epi);

}  // namespace hpd
