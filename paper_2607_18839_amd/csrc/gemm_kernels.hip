// gfx950 kernels of the decoder-stack projections (section "Overview",
// paragraph "LLM Decoder": GQA attention, RMSNorm, SwiGLU MLP).
//
// Every projection of the step is a skinny GEMM: T ~ 130 token rows against a
// bf16 weight matrix W[N][K] that is streamed from HBM once per step.  It is
// computed transposed, Y^T[N][T] = W X^T, on v_mfma_f32_16x16x32_bf16 with W
// as the A operand (16 weight rows per tile, read straight from HBM into
// registers) and the token rows X (bf16, [Tpad][K], L2-resident) as the B
// operand, Tpad = T rounded up to 16.
//
// Workgroup = 4 waves = one 64-row slice of W over one range of K; the four
// waves take consecutive quarters of that K range, each accumulating the full
// 64 x Tpad tile (every activation fragment it loads feeds 4 MFMAs), and are
// summed through LDS in a fixed order.  Large K ranges are split over several
// workgroups ("split-K"); the last workgroup of a slice to arrive (arrival
// counter) adds the partial tiles in split order and runs the epilogue, so
// results do not depend on scheduling.
//
// Activations that feed the MLP (RMSNorm output and the SwiGLU product) are
// carried as two bf16 terms hi + lo (lo = x - hi rounded to bf16) and
// multiplied with two MFMAs, which keeps them at ~16 significant bits;
// rounding them to one bf16 term costs ~1e-2 of absolute error on the
// residual stream after 18 layers.  The QKV and O projections take a single
// bf16 term (their rounding costs ~5e-4).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "gemm.h"

namespace hpd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kTT = kGemmMaxTokenTiles;   // token tiles of 16 (Tpad <= 16 * kTT)

__device__ __forceinline__ f32x4 mma16(const bf16x8 &a, const bf16x8 &b, const f32x4 &c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ------------------------------------------------------------ RMSNorm

// One workgroup per token row t < Tpad.  Rows t >= T are written as zeros
// (also `zero_rows`, the padding rows of another activation buffer).
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float *h, const __bf16 *gamma, int H, int T,
                                                      float eps, __bf16 *x_hi, __bf16 *x_lo,
                                                      __bf16 *zero_rows, int zero_cols) {
  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  if (t >= T) {
    for (int c = tid; c < H; c += 256) {
      x_hi[(int64_t)t * H + c] = (__bf16)0.f;
      if (x_lo) x_lo[(int64_t)t * H + c] = (__bf16)0.f;
    }
    if (zero_rows)
      for (int c = tid; c < zero_cols; c += 256) zero_rows[(int64_t)t * zero_cols + c] = (__bf16)0.f;
    return;
  }
  const float *row = h + (int64_t)t * H;
  float ss = 0.f;
  for (int c = tid; c < H; c += 256) ss = fmaf(row[c], row[c], ss);
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
  __shared__ float part[4];
  if ((tid & 63) == 0) part[tid >> 6] = ss;
  __syncthreads();
  const float tot = (part[0] + part[1]) + (part[2] + part[3]);
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  for (int c = tid; c < H; c += 256) {
    float x = row[c] * inv;
    if (gamma) x *= (float)gamma[c];
    const __bf16 hi = (__bf16)x;
    x_hi[(int64_t)t * H + c] = hi;
    if (x_lo) x_lo[(int64_t)t * H + c] = (__bf16)(x - (float)hi);
  }
}

// ------------------------------------------------------------ GEMM

template <bool SPLIT, int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs g) {
  __shared__ f32x4 red[2][4 * kTT][64];
  const int nwg = g.n_tgroups * g.n_slices * g.ksplit;
  const int per_xcd = gridDim.x / 8;
  // XCD-aware order: the split-K workgroups of one slice run on one XCD.
  const int logical = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (logical >= nwg) return;
  const int tile_id = logical / g.ksplit, ks = logical % g.ksplit;   // tile = (token group, slice)
  const int tg = tile_id / g.n_slices, slice = tile_id % g.n_slices;
  const int t0 = tg * kGemmTokenGroup;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ntt = min(kTT, g.Tpad / 16 - tg * kTT);
  const int kq = g.k_per_wg / 4;
  const int kbeg = ks * g.k_per_wg + wave * kq;

  // weight rows of this lane for the 4 row tiles
  const __bf16 *wrow[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    int64_t r;
    const __bf16 *base = g.w0;
    if constexpr (EPI == kEpiSwiGLU) {
      // tiles 0, 1: gate rows i0 .. i0 + 31; tiles 2, 3: up rows, same i
      r = (int64_t)slice * 32 + 16 * (nt & 1) + (lane & 15);
      if (nt >= 2) base = g.w1;
    } else {
      r = (int64_t)slice * 64 + 16 * nt + (lane & 15);
    }
    wrow[nt] = base + r * g.K + 8 * (lane >> 4);
  }
  const int64_t xoff = (int64_t)(t0 + (lane & 15)) * g.K + 8 * (lane >> 4);

  f32x4 acc[4][kTT];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int tt = 0; tt < kTT; ++tt) acc[nt][tt] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k = kbeg; k < kbeg + kq; k += 32) {
    bf16x8 a[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) a[nt] = *(const bf16x8 *)(wrow[nt] + k);
#pragma unroll
    for (int tt = 0; tt < kTT; ++tt) {
      if (tt < ntt) {
        const bf16x8 b = *(const bf16x8 *)(g.x_hi + (int64_t)tt * 16 * g.K + xoff + k);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) acc[nt][tt] = mma16(a[nt], b, acc[nt][tt]);
        if constexpr (SPLIT) {
          const bf16x8 b2 = *(const bf16x8 *)(g.x_lo + (int64_t)tt * 16 * g.K + xoff + k);
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) acc[nt][tt] = mma16(a[nt], b2, acc[nt][tt]);
        }
      }
    }
  }

  // fixed-order sum of the four waves: (w0 + w1) + (w2 + w3)
  if (wave == 1 || wave == 3) {
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int tt = 0; tt < kTT; ++tt) red[wave >> 1][nt * kTT + tt][lane] = acc[nt][tt];
  }
  __syncthreads();
  if (wave == 0 || wave == 2) {
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int tt = 0; tt < kTT; ++tt) acc[nt][tt] += red[wave >> 1][nt * kTT + tt][lane];
  }
  __syncthreads();
  if (wave == 2) {
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int tt = 0; tt < kTT; ++tt) red[0][nt * kTT + tt][lane] = acc[nt][tt];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int tt = 0; tt < kTT; ++tt) acc[nt][tt] += red[0][nt * kTT + tt][lane];

  if (g.ksplit > 1) {
    f32x4 *part = (f32x4 *)g.part + (int64_t)logical * (4 * kTT * 64);
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int tt = 0; tt < kTT; ++tt) part[(nt * kTT + tt) * 64 + lane] = acc[nt][tt];
    __threadfence();
    int old = 0;
    if (lane == 0)
      old = __hip_atomic_fetch_add(g.counters + tile_id, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    old = __shfl(old, 0);
    if (old != g.ksplit - 1) return;
    __threadfence();
    // last arrival: sum the partial tiles of this slice in split order
    const f32x4 *p0 = (const f32x4 *)g.part + (int64_t)tile_id * g.ksplit * (4 * kTT * 64);
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int tt = 0; tt < kTT; ++tt) acc[nt][tt] = p0[(nt * kTT + tt) * 64 + lane];
    for (int j = 1; j < g.ksplit; ++j) {
      const f32x4 *pj = p0 + (int64_t)j * (4 * kTT * 64);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int tt = 0; tt < kTT; ++tt) acc[nt][tt] += pj[(nt * kTT + tt) * 64 + lane];
    }
    if (lane == 0) __hip_atomic_store(g.counters + tile_id, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // epilogue: lane holds rows n = 16 nt + 4 (lane / 16) + r, token t = 16 tt + lane % 16
  const int tl = lane & 15, nq = 4 * (lane >> 4);
#pragma unroll
  for (int tt = 0; tt < kTT; ++tt) {
    const int t = t0 + 16 * tt + tl;
    if (tt >= ntt) continue;
    if constexpr (EPI == kEpiQKV) {
      if (t >= g.T) continue;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int n = slice * 64 + 16 * nt + nq;
        bf16x4 v;
        for (int r = 0; r < 4; ++r) v[r] = (__bf16)acc[nt][tt][r];
        if (n < g.n_q) {
          *(bf16x4 *)(g.q_out + (int64_t)t * g.n_q + n) = v;
        } else if (n < g.n_q + g.n_kv) {
          *(bf16x4 *)(g.k_cache + (int64_t)g.dest[t] * g.n_kv + (n - g.n_q)) = v;
        } else {
          *(bf16x4 *)(g.v_cache + (int64_t)g.dest[t] * g.n_kv + (n - g.n_q - g.n_kv)) = v;
        }
      }
    } else if constexpr (EPI == kEpiResidual) {
      if (t >= g.T) continue;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int n = slice * 64 + 16 * nt + nq;
        f32x4 *dst = (f32x4 *)(g.h + (int64_t)t * g.ldh + n);
        *dst = *dst + acc[nt][tt];
      }
    } else {   // SwiGLU: m = silu(gate) * up, written as hi + lo bf16 terms
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const int i = slice * 32 + 16 * nt + nq;
        bf16x4 hi, lo;
        for (int r = 0; r < 4; ++r) {
          const float gt = acc[nt][tt][r], up = acc[nt + 2][tt][r];
          const float m = t < g.T ? gt / (1.0f + __expf(-gt)) * up : 0.f;
          hi[r] = (__bf16)m;
          lo[r] = (__bf16)(m - (float)hi[r]);
        }
        *(bf16x4 *)(g.m_hi + (int64_t)t * g.I + i) = hi;
        *(bf16x4 *)(g.m_lo + (int64_t)t * g.I + i) = lo;
      }
    }
  }
}

}  // namespace

hipError_t launch_rmsnorm(const float *h, const __bf16 *gamma, int H, int T, int Tpad, float eps,
                          __bf16 *x_hi, __bf16 *x_lo, __bf16 *zero_rows, int zero_cols,
                          hipStream_t stream) {
  timed_begin(KK_NORM, stream);
  hipLaunchKernelGGL(rmsnorm_kernel, dim3(Tpad), dim3(256), 0, stream, h, gamma, H, T, eps, x_hi, x_lo,
                     zero_rows, zero_cols);
  timed_end(stream);
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs &g, bool split, int epi, int kind, hipStream_t stream) {
  const int nwg = g.n_tgroups * g.n_slices * g.ksplit;
  const dim3 grid((nwg + 7) / 8 * 8), block(256);
  timed_begin(kind, stream);
  if (epi == kEpiQKV && !split) hipLaunchKernelGGL((gemm_kernel<false, kEpiQKV>), grid, block, 0, stream, g);
  else if (epi == kEpiResidual && !split)
    hipLaunchKernelGGL((gemm_kernel<false, kEpiResidual>), grid, block, 0, stream, g);
  else if (epi == kEpiResidual && split)
    hipLaunchKernelGGL((gemm_kernel<true, kEpiResidual>), grid, block, 0, stream, g);
  else if (epi == kEpiSwiGLU && split)
    hipLaunchKernelGGL((gemm_kernel<true, kEpiSwiGLU>), grid, block, 0, stream, g);
  else {
    timed_end(stream);
    return hipErrorInvalidValue;
  }
  timed_end(stream);
  return hipGetLastError();
}

}  // namespace hpd
