// Internal interface of the projection GEMM and RMSNorm kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"

namespace hpd {

constexpr int kGemmTile = 32;             // weight rows and tokens of one wave's output tile
constexpr int kGemmKStep = 64;            // K per pipeline step (4 MFMAs of 16)
constexpr int kEpiQKV = 0, kEpiResidual = 1, kEpiSwiGLU = 2;

// One projection Y[t][n] = sum_k X[t][k] W[n][k] over the full K range.  A
// workgroup of 4 waves owns the output tile of 32 rg weight rows x 32
// tokens: wave w takes rows 32 (w % rg) .. and the K quarter / half w / rg
// (rg * kg = 4; the K groups are added through LDS).
//
// RMSNorm is folded into the projections.  The residual projections (O,
// down) add their result into the fp32 residual stream h, and write the next
// norm's input unnormalised, x = h * gamma (bf16 or fp16), together with the
// sums of squares of h over each 32-column tile, ss[t][tile].  The projections
// that consume x (QKV, gate/up) scale their outputs by 1 / sqrt(sum ss / H +
// eps) per token: RMSNorm's per-token factor commutes with the product.
struct GemmArgs {
  const __bf16 *w0;         // W[N][K] (SwiGLU: gate rows [I][K])
  const __bf16 *w1;         // SwiGLU: up rows [I][K]; otherwise unused
  int K;
  int N;                    // output columns (SwiGLU: 2 I, gate and up)
  int rg;                   // row groups per workgroup: 1, 2 or 4 (K % (64 * 4 / rg) == 0)
  int n_slices;             // N / (32 rg)
  int n_ttiles;             // Tpad / 32
  const __bf16 *x;          // [Tpad][K] activations (bf16, or fp16 for the MLP), rows >= T finite
  int T, Tpad;
  // QKV / SwiGLU: per-token norm factor from ss_in [Tpad][n_ss] (sum / H + eps)
  const float *ss_in; int n_ss; float inv_H, eps;
  // fp16 norm inputs: a per-token power of two s_t [T] (pow2_scale of a norm
  // factor).  The residual epilogue writes x_out = h * gamma * s_t; the
  // SwiGLU epilogue divides its products by s_t.  NULL = no scaling.
  const float *scale_in;
  // QKV epilogue: writes s_t = pow2_scale(its RMSNorm factor) [T] (NULL = not)
  float *scale_out;
  // QKV epilogue
  __bf16 *q_out; int n_q;                   // q[t][0..n_q)
  __bf16 *k_cache, *v_cache; int n_kv;      // cache rows dest[t]
  const int32_t *dest;
  // SwiGLU epilogue
  __bf16 *m_out; int I;                     // [Tpad][I], fp16 bits (rows >= T zero)
  // residual epilogue (N = H): h += Y; then, if x_out: x_out = h * gamma, ss_out
  float *h;                                 // [T][N] fp32
  __bf16 *x_out; bool x_out_f16;            // [Tpad][N]; rows < T written
  const __bf16 *gamma;                      // [N] bf16, NULL = ones
  float *ss_out;                            // [Tpad][N / 32]
  // LM head (launch_lm_argmax): per token and 128-row slice the largest
  // logit as an ordered key (argmax_key), amax[t][N / 128]
  uint64_t *amax;
  // layouts: a_packed: w0 is packed (packed_offset; SwiGLU: the interleaved
  // gate/up pair, w1 unused); act_packed: x, x_out and m_out are packed.
  // a_packed requires act_packed; row-major weights require row-major
  // activations.
  bool a_packed, act_packed;
};

// Ordered 64-bit key of a logit and its row id: comparing keys as unsigned
// integers orders by value, and equal values by the smaller id.
__device__ __forceinline__ uint64_t argmax_key(float v, int id) {
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)id);
}
__device__ __forceinline__ int argmax_id(uint64_t key) { return (int)(0xFFFFFFFFu - (uint32_t)key); }

// The power of two s <= inv (an RMSNorm factor), clamped to [2^-100,
// 2^100].  An fp16 norm input x = h * gamma is written as x * s with s from
// the token's previous norm factor, which brings the row near unit scale so
// that a large residual stream does not overflow fp16 (65504); its consumer
// divides by the same s.  s is a power of two, so both scalings are exact.
__device__ __forceinline__ float pow2_scale(float inv) {
  if (!(inv >= 0x1p-100f)) return inv > 0x1p100f ? 0x1p100f : 0x1p-100f;   // NaN too
  if (inv > 0x1p100f) return 0x1p100f;
  return __uint_as_float(__float_as_uint(inv) & 0x7f800000u);
}

// Start of a step: h = h_in (if different), x = h * gamma, ss, and zero rows
// T..Tpad-1 of x and of `zero_rows` ([Tpad][zero_cols]).
hipError_t launch_norm_input(const float *h_in, float *h, int T, int Tpad, int H, const __bf16 *gamma,
                             __bf16 *x, float *ss, __bf16 *zero_rows, int zero_cols, bool packed,
                             hipStream_t stream);
// W[rows][cols] -> packed layout (gate_up: interleave w (gate) and w2 (up),
// each [rows / 2][cols]); to_f16: elements converted from bf16 to fp16.
hipError_t launch_pack_weight(const __bf16 *w, const __bf16 *w2, int rows, int cols, bool gate_up, bool to_f16,
                              __bf16 *out, hipStream_t stream);
// f16: fp16 GEMM (bf16 weights converted to fp16 in registers, fp16
// activations); epi: kEpiQKV, kEpiResidual or kEpiSwiGLU.
hipError_t launch_gemm(const GemmArgs &g, bool f16, int epi, int kind, hipStream_t stream);
// LM head with an argmax epilogue (bf16, packed operands): 128 rows per
// workgroup against a group of up to 5 token tiles; n_slices = N / 128,
// K a multiple of 256; writes amax[Tpad][n_slices].
hipError_t launch_lm_argmax(const GemmArgs &g, int kind, hipStream_t stream);

// Row groups per workgroup for an N x K projection over Tpad tokens, from a
// model of the bytes each CU has to stream.
int choose_gemm_rg(int N, int K, int Tpad);

}  // namespace hpd
