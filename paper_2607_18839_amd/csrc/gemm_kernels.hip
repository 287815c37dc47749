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

#include <algorithm>
#include <cstdint>

#include "gemm.h"

namespace hpd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kMaxTPW = 3;   // token tiles per wave (a group of 9 tiles -> 3 waves of 3)

__device__ __forceinline__ f32x4 mma16(const bf16x8 &a, const bf16x8 &b, const f32x4 &c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ------------------------------------------------------------ GEMM

// Fragments of one 32-wide k step of one wave: the 4 weight tiles of the
// workgroup's 64 rows and the wave's TPW token tiles, x2 when the activations
// carry hi + lo terms.
template <int kTPW, bool SPLIT> struct StepFrags {
  bf16x8 a[4];
  bf16x8 b[kTPW];
  bf16x8 bl[SPLIT ? kTPW : 1];
};

template <int kTPW, bool SPLIT>
__device__ __forceinline__ void load_step(StepFrags<kTPW, SPLIT> &f, const __bf16 *const *wrow,
                                          const __bf16 *const *xh, const __bf16 *const *xl, int k) {
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) f.a[nt] = *(const bf16x8 *)(wrow[nt] + k);
#pragma unroll
  for (int j = 0; j < kTPW; ++j) {
    f.b[j] = *(const bf16x8 *)(xh[j] + k);
    if constexpr (SPLIT) f.bl[j] = *(const bf16x8 *)(xl[j] + k);
  }
}

// hi terms of every tile first, then the lo terms: consecutive MFMAs never
// update the same accumulator.  No branches: a tile beyond the group's last
// one repeats that tile and is simply not stored.
template <int kTPW, bool SPLIT>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[4][kTPW], const StepFrags<kTPW, SPLIT> &f) {
#pragma unroll
  for (int j = 0; j < kTPW; ++j)
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[nt][j] = mma16(f.a[nt], f.b[j], acc[nt][j]);
  if constexpr (SPLIT) {
#pragma unroll
    for (int j = 0; j < kTPW; ++j)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) acc[nt][j] = mma16(f.a[nt], f.bl[j], acc[nt][j]);
  }
}

// Workgroup = ceil(tiles / TPW) waves = 64 weight rows x one token group (up
// to 9 tiles of 16 tokens) x one K range.  The waves split the token tiles
// (TPW each) and each runs the whole K range, so a wave holds 4 x TPW
// accumulator tiles and nothing has to be reduced across waves; the waves
// read the same weight fragments at the same time (L1 hits after the first).
// Split-K partials: part[ks][t][n] (fp32, row-major by token), added in
// split order by the consumer.
template <int kTPW, bool SPLIT, int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs g) {
  constexpr bool SWIGLU = EPI == kEpiSwiGLU;
  const int nwg = g.n_tgroups * g.n_slices * g.ksplit;
  const int per_xcd = gridDim.x / 8;
  // XCD-aware order: consecutive logical tiles share an XCD (and its L2).
  const int logical = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (logical >= nwg) return;
  const int tile_id = logical / g.ksplit, ks = logical % g.ksplit;   // tile = (token group, slice)
  const int tg = tile_id / g.n_slices, slice = tile_id % g.n_slices;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // token tiles of this group: wave w takes tiles w TPW .. w TPW + TPW - 1
  const int ntt = min(kGemmMaxTokenTiles, g.Tpad / 16 - tg * kGemmMaxTokenTiles);
  const int tt0 = wave * kTPW;
  if (tt0 >= ntt) return;
  const int ntw = min(kTPW, ntt - tt0);            // tiles this wave stores
  const int t0 = tg * kGemmTokenGroup + 16 * tt0;   // first token of the wave's first tile
  const int kbeg = ks * g.k_per_wg, kend = kbeg + g.k_per_wg;

  const __bf16 *wrow[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    int64_t r;
    const __bf16 *base = g.w0;
    if constexpr (SWIGLU) {
      // tiles 0, 1: gate rows i0 .. i0 + 31; tiles 2, 3: up rows, same i
      r = (int64_t)slice * 32 + 16 * (nt & 1) + (lane & 15);
      if (nt >= 2) base = g.w1;
    } else {
      r = (int64_t)slice * 64 + 16 * nt + (lane & 15);
    }
    wrow[nt] = base + r * g.K + 8 * (lane >> 4);
  }
  const __bf16 *xh[kTPW], *xl[kTPW];
#pragma unroll
  for (int j = 0; j < kTPW; ++j) {
    const int jj = min(j, ntw - 1);   // absent tiles re-read the last present one
    const int64_t off = (int64_t)(t0 + 16 * jj + (lane & 15)) * g.K + 8 * (lane >> 4);
    xh[j] = g.x_hi + off;
    xl[j] = SPLIT ? g.x_lo + off : nullptr;
  }

  f32x4 acc[4][kTPW];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int j = 0; j < kTPW; ++j) acc[nt][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // two k steps in flight; scheduling barriers keep each load batch ahead of
  // the MFMAs that precede its use
  StepFrags<kTPW, SPLIT> f0, f1;
  load_step<kTPW, SPLIT>(f0, wrow, xh, xl, kbeg);
  int k = kbeg;
  for (; k + 64 <= kend; k += 64) {
    load_step<kTPW, SPLIT>(f1, wrow, xh, xl, k + 32);
    __builtin_amdgcn_sched_barrier(0);
    mma_step<kTPW, SPLIT>(acc, f0);
    __builtin_amdgcn_sched_barrier(0);
    // unconditional (clamped in range on the last pass) so that the waits
    // the compiler derives never have to cover a skipped batch
    load_step<kTPW, SPLIT>(f0, wrow, xh, xl, k + 64 < kend ? k + 64 : k);
    __builtin_amdgcn_sched_barrier(0);
    mma_step<kTPW, SPLIT>(acc, f1);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (k < kend) mma_step<kTPW, SPLIT>(acc, f0);

  // lane holds virtual columns n = 64 slice + 16 nt + 4 (lane / 16) + r of
  // token t0 + 16 j + lane % 16
  const int nq = 4 * (lane >> 4);
  if (g.ksplit > 1 || EPI == kEpiResidual) {
    float *part = g.part + (int64_t)ks * g.Tpad * g.N;
#pragma unroll
    for (int j = 0; j < kTPW; ++j) {
      if (j >= ntw) continue;
      const int t = t0 + 16 * j + (lane & 15);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
        *(f32x4 *)(part + (int64_t)t * g.N + slice * 64 + 16 * nt + nq) = acc[nt][j];
    }
    return;
  }
  // whole K in this workgroup: the epilogue runs here
#pragma unroll
  for (int j = 0; j < kTPW; ++j) {
    if (j >= ntw) continue;
    const int t = t0 + 16 * j + (lane & 15);
    if constexpr (EPI == kEpiQKV) {
      if (t >= g.T) continue;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int n = slice * 64 + 16 * nt + nq;
        bf16x4 v;
        for (int r = 0; r < 4; ++r) v[r] = (__bf16)acc[nt][j][r];
        if (n < g.n_q) *(bf16x4 *)(g.q_out + (int64_t)t * g.n_q + n) = v;
        else if (n < g.n_q + g.n_kv) *(bf16x4 *)(g.k_cache + (int64_t)g.dest[t] * g.n_kv + (n - g.n_q)) = v;
        else *(bf16x4 *)(g.v_cache + (int64_t)g.dest[t] * g.n_kv + (n - g.n_q - g.n_kv)) = v;
      }
    } else if constexpr (EPI == kEpiSwiGLU) {
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const int i = slice * 32 + 16 * nt + nq;
        bf16x4 hi, lo;
        for (int r = 0; r < 4; ++r) {
          const float gt = acc[nt][j][r], up = acc[nt + 2][j][r];
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

// ------------------------------------------------------------ consumers of the partials

// Sum over the splits of 4 consecutive partial columns; the loads of a batch
// of 8 splits are all issued before the first add (split order kept).
__device__ __forceinline__ f32x4 sum_splits(const float *part, int64_t split_stride, int ksplit) {
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < ksplit; k0 += 8) {
    f32x4 v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = *(const f32x4 *)(part + (int64_t)min(k0 + i, ksplit - 1) * split_stride);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (k0 + i < ksplit) s += v[i];
  }
  return s;
}

// QKV: y = sum of splits; q -> q_out, k/v -> cache rows dest[t] (bf16).
__global__ __launch_bounds__(256) void qkv_epilogue_kernel(GemmArgs g) {
  const int64_t i4 = (int64_t)blockIdx.x * 256 + threadIdx.x;   // one group of 4 columns
  const int N = g.N;
  if (i4 * 4 >= (int64_t)g.T * N) return;
  const int t = (int)(i4 * 4 / N), n = (int)(i4 * 4 % N);
  const f32x4 y = sum_splits(g.part + (int64_t)t * N + n, (int64_t)g.Tpad * N, g.ksplit);
  bf16x4 v;
  for (int r = 0; r < 4; ++r) v[r] = (__bf16)y[r];
  if (n < g.n_q) *(bf16x4 *)(g.q_out + (int64_t)t * g.n_q + n) = v;
  else if (n < g.n_q + g.n_kv) *(bf16x4 *)(g.k_cache + (int64_t)g.dest[t] * g.n_kv + (n - g.n_q)) = v;
  else *(bf16x4 *)(g.v_cache + (int64_t)g.dest[t] * g.n_kv + (n - g.n_q - g.n_kv)) = v;
}

// gate/up: m = silu(sum gate) * (sum up), written as hi + lo bf16 terms
// [Tpad][I] (zero rows t >= T).  Virtual column of gate i: 64 (i / 32) + i % 32,
// of up i: that + 32.
__global__ __launch_bounds__(256) void swiglu_epilogue_kernel(GemmArgs g) {
  const int64_t i4 = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int I = g.I;
  if (i4 * 4 >= (int64_t)g.Tpad * I) return;
  const int t = (int)(i4 * 4 / I), i = (int)(i4 * 4 % I);
  bf16x4 hi, lo;
  if (t < g.T) {
    const int vg = 64 * (i / 32) + i % 32;
    const f32x4 gs = sum_splits(g.part + (int64_t)t * g.N + vg, (int64_t)g.Tpad * g.N, g.ksplit);
    const f32x4 us = sum_splits(g.part + (int64_t)t * g.N + vg + 32, (int64_t)g.Tpad * g.N, g.ksplit);
    for (int r = 0; r < 4; ++r) {
      const float m = gs[r] / (1.0f + __expf(-gs[r])) * us[r];
      hi[r] = (__bf16)m;
      lo[r] = (__bf16)(m - (float)hi[r]);
    }
  } else {
    for (int r = 0; r < 4; ++r) { hi[r] = (__bf16)0.f; lo[r] = (__bf16)0.f; }
  }
  *(bf16x4 *)(g.m_hi + (int64_t)t * I + i) = hi;
  *(bf16x4 *)(g.m_lo + (int64_t)t * I + i) = lo;
}

// Residual + RMSNorm: h[t] += sum of the splits of `part` (if any), then
// x = RMSNorm(h[t]) * gamma -> x_hi (+ x_lo) unless x_hi is NULL.  One
// workgroup per row t < Tpad; rows t >= T are written as zeros (also the
// padding rows `zero_rows`).  H is a multiple of 4.
__global__ __launch_bounds__(256) void residual_norm_kernel(float *h, const float *part, int ksplit, int Tpad,
                                                            int H, int T, const __bf16 *gamma, float eps,
                                                            __bf16 *x_hi, __bf16 *x_lo, __bf16 *zero_rows,
                                                            int zero_cols) {
  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  if (t >= T) {
    if (x_hi)
      for (int c = tid; c < H; c += 256) {
        x_hi[(int64_t)t * H + c] = (__bf16)0.f;
        if (x_lo) x_lo[(int64_t)t * H + c] = (__bf16)0.f;
      }
    if (zero_rows)
      for (int c = tid; c < zero_cols; c += 256) zero_rows[(int64_t)t * zero_cols + c] = (__bf16)0.f;
    return;
  }
  float *row = h + (int64_t)t * H;
  float ss = 0.f;
  for (int c = 4 * tid; c < H; c += 1024) {
    f32x4 v = *(const f32x4 *)(row + c);
    if (part) {
      v += sum_splits(part + (int64_t)t * H + c, (int64_t)Tpad * H, ksplit);
      *(f32x4 *)(row + c) = v;
    }
    ss = fmaf(v[0], v[0], fmaf(v[1], v[1], fmaf(v[2], v[2], fmaf(v[3], v[3], ss))));
  }
  if (!x_hi) return;
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
  __shared__ float wsum[4];
  if ((tid & 63) == 0) wsum[tid >> 6] = ss;
  __syncthreads();
  const float tot = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  for (int c = 4 * tid; c < H; c += 1024) {
    const f32x4 v = *(const f32x4 *)(row + c);
    bf16x4 hi, lo;
    for (int r = 0; r < 4; ++r) {
      float x = v[r] * inv;
      if (gamma) x *= (float)gamma[c + r];
      hi[r] = (__bf16)x;
      lo[r] = (__bf16)(x - (float)hi[r]);
    }
    *(bf16x4 *)(x_hi + (int64_t)t * H + c) = hi;
    if (x_lo) *(bf16x4 *)(x_lo + (int64_t)t * H + c) = lo;
  }
}

}  // namespace

hipError_t launch_residual_norm(float *h, const float *part, int ksplit, int Tpad, int H, int T,
                                const __bf16 *gamma, float eps, __bf16 *x_hi, __bf16 *x_lo,
                                __bf16 *zero_rows, int zero_cols, hipStream_t stream) {
  timed_begin(KK_NORM, stream);
  hipLaunchKernelGGL(residual_norm_kernel, dim3(Tpad), dim3(256), 0, stream, h, part, ksplit, Tpad, H, T, gamma,
                     eps, x_hi, x_lo, zero_rows, zero_cols);
  timed_end(stream);
  return hipGetLastError();
}

// Tpad is a multiple of 16; when it exceeds one token group it must be a
// multiple of kGemmTokenGroup (every group then has the same tile count).
hipError_t launch_gemm(const GemmArgs &g, bool split, int epi, int kind, hipStream_t stream) {
  const int ntt = std::min(kGemmMaxTokenTiles, g.Tpad / 16);
  if (g.Tpad % 16 != 0 || (g.n_tgroups > 1 && g.Tpad % kGemmTokenGroup != 0) ||
      (g.n_tgroups - 1) * kGemmMaxTokenTiles + ntt != g.Tpad / 16 || g.k_per_wg % 32 != 0)
    return hipErrorInvalidValue;
  const int nwg = g.n_tgroups * g.n_slices * g.ksplit;
  const int tpw = std::min(kMaxTPW, ntt);
  const int waves = (ntt + tpw - 1) / tpw;
  const dim3 grid((nwg + 7) / 8 * 8), block(64 * waves);
  timed_begin(kind, stream);
#define HPD_GEMM_LAUNCH(TPW)                                                                                   \
  if (epi == kEpiSwiGLU) hipLaunchKernelGGL((gemm_kernel<TPW, true, kEpiSwiGLU>), grid, block, 0, stream, g);    \
  else if (epi == kEpiQKV) hipLaunchKernelGGL((gemm_kernel<TPW, false, kEpiQKV>), grid, block, 0, stream, g);    \
  else if (split) hipLaunchKernelGGL((gemm_kernel<TPW, true, kEpiResidual>), grid, block, 0, stream, g);        \
  else hipLaunchKernelGGL((gemm_kernel<TPW, false, kEpiResidual>), grid, block, 0, stream, g);
  if (tpw == 3) { HPD_GEMM_LAUNCH(3) }
  else if (tpw == 2) { HPD_GEMM_LAUNCH(2) }
  else { HPD_GEMM_LAUNCH(1) }
#undef HPD_GEMM_LAUNCH
  timed_end(stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (g.ksplit == 1) return hipSuccess;   // QKV / SwiGLU epilogues ran inside the GEMM
  if (epi == kEpiQKV) {
    timed_begin(KK_EPILOGUE, stream);
    const int64_t n4 = (int64_t)g.T * g.N / 4;
    hipLaunchKernelGGL(qkv_epilogue_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream, g);
    timed_end(stream);
  } else if (epi == kEpiSwiGLU) {
    timed_begin(KK_EPILOGUE, stream);
    const int64_t n4 = (int64_t)g.Tpad * g.I / 4;
    hipLaunchKernelGGL(swiglu_epilogue_kernel, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream, g);
    timed_end(stream);
  }
  return hipGetLastError();
}

}  // namespace hpd
