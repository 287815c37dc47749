// gfx950 kernels of the decoder-stack projections (section "Overview",
// paragraph "LLM Decoder": GQA attention, RMSNorm, SwiGLU MLP).
//
// Every projection of the step is a skinny GEMM: T ~ 130 token rows against a
// bf16 weight matrix W[N][K] that is streamed from HBM once per step.  It is
// computed transposed, Y^T[N][T] = W X^T, on v_mfma_f32_32x32x16 with W as the
// A operand and the token rows X ([Tpad][K], L2-resident) as the B operand,
// Tpad = T rounded up to 32.
//
// Work decomposition.  The cost of such a GEMM is the bytes each CU must pull
// in (its weight rows plus the token rows it multiplies them with), not the
// MFMA work, so the tiles are small: each wave owns one 32 x 32 output tile
// (32 weight rows x 32 tokens) over a K range.  The 4 waves of a workgroup
// split either the rows (rg = 4: the token tile is shared), or K (rg = 1: four
// K quarters, added through LDS at the end, in wave order), or both (rg = 2).
// Operands stream through a 4-step LDS ring filled by direct global -> LDS
// copies (8 rows x 128 bytes per instruction), 3 steps ahead of the MFMAs.
// Every output element is produced by one workgroup over the whole of K, so
// the epilogues can finish it: the QKV and SwiGLU epilogues apply the folded
// RMSNorm factor and write q / the new K/V rows / m; the residual epilogue
// adds into h and writes the next norm's input (see gemm.h).
//
// Precision: the QKV and O projections take bf16 activations (rounding them
// costs ~5e-4 of absolute error on the residual stream after 18 layers).  The
// MLP projections are sensitive (a single bf16 rounding of their inputs costs
// ~1e-2), so they run in fp16: the bf16 weights convert to fp16 exactly (all
// normal-range values; |w| < 2^-14 lose at most 2^-25 absolutely) and the
// activations carry 11 significant bits.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <type_traits>

#include "gemm.h"

namespace hpd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// ------------------------------------------------------------ GEMM

// 8 bf16 -> 8 fp16 (round to nearest even; exact for |w| >= 2^-14).
__device__ __forceinline__ u32x4 bf16x8_to_f16x8(u32x4 v) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float lo = __uint_as_float(v[i] << 16), hi = __uint_as_float(v[i] & 0xffff0000u);
    const _Float16 l16 = (_Float16)lo, h16 = (_Float16)hi;
    r[i] = (unsigned)__builtin_bit_cast(unsigned short, l16) | ((unsigned)__builtin_bit_cast(unsigned short, h16) << 16);
  }
  return r;
}

// Epilogue operands of a tile.  The token's cache row (QKV, plan data) and
// scale are loaded before the main loop; the residual row slice, the next
// norm's weights and the per-token sums of squares after the loads of the
// first pipeline steps (packed kernel, load_pre) or after the loop.
constexpr int kSsPrefetch = 32;   // sums of squares per token held in registers (hidden <= 1024)
struct EpilogueIn {
  f32x4 h[4], gamma[4];   // residual: h row slice and gamma (ones if none)
  f32x4 ss[kSsPrefetch / 4];   // QKV, SwiGLU: the token's sums of squares (load_pre)
  int dest;               // QKV: private cache row of the token
  float inv_rms;          // QKV, SwiGLU: RMSNorm factor of the token
  float scale;            // residual, SwiGLU: s_t of the fp16 norm input (scale_in), else 1
};

// Loaded before the main loop: plan data and the per-token scale, which were
// written at least two launches earlier.
template <int EPI>
__device__ __forceinline__ void load_early(const GemmArgs &g, int t, EpilogueIn &in) {
  if constexpr (EPI == kEpiQKV) in.dest = t < g.T ? g.dest[t] : 0;
  else in.scale = g.scale_in ? g.scale_in[min(t, g.T - 1)] : 1.f;
}

template <int EPI>
__device__ __forceinline__ void load_late(const GemmArgs &g, int t, int tile, int half, EpilogueIn &in) {
  if constexpr (EPI == kEpiResidual) {
    const float *hr = g.h + (int64_t)min(t, g.T - 1) * g.N + tile * kGemmTile + 4 * half;
#pragma unroll
    for (int i = 0; i < 4; ++i) in.h[i] = *(const f32x4 *)(hr + 8 * i);
    if (g.x_out && g.gamma) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bf16x4 gv = *(const bf16x4 *)(g.gamma + tile * kGemmTile + 8 * i + 4 * half);
        in.gamma[i] = f32x4{(float)gv[0], (float)gv[1], (float)gv[2], (float)gv[3]};
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) in.gamma[i] = f32x4{1.f, 1.f, 1.f, 1.f};
    }
  } else {
    // per-token RMSNorm factor from the partial sums of squares
    const float *sr = g.ss_in + (int64_t)t * g.n_ss;
    float sum = 0.f;
    for (int i = 0; i < g.n_ss; i += 4) {
      const f32x4 v = *(const f32x4 *)(sr + i);
      sum += (v[0] + v[1]) + (v[2] + v[3]);
    }
    in.inv_rms = 1.0f / sqrtf(sum * g.inv_H + g.eps);
  }
}

// The packed kernel's epilogue loads, split around its main loop: load_pre
// issues them right after the loads of the first pipeline steps, so that the
// waits for those steps do not cover them and their latency overlaps the
// loop; load_post reduces them.  (Issued before the first steps' loads they
// delayed the loop: loads retire in order.)  Every buffer they read was
// written at least two launches earlier (h by the residual projection
// before the previous kernel, the sums of squares and gamma earlier still).
// Sums of squares beyond kSsPrefetch values per token are loaded late.
template <int EPI>
__device__ __forceinline__ void load_pre(const GemmArgs &g, int t, int tile, int half, EpilogueIn &in) {
  if constexpr (EPI == kEpiResidual) {
    load_late<EPI>(g, t, tile, half, in);
  } else if (g.n_ss <= kSsPrefetch) {
    const float *sr = g.ss_in + (int64_t)t * g.n_ss;
    // unconditional loads (an index past the row repeats its last four
    // values, unused): a load under a condition would be followed by a wait
#pragma unroll
    for (int i = 0; i < kSsPrefetch / 4; ++i) in.ss[i] = *(const f32x4 *)(sr + min(4 * i, g.n_ss - 4));
  }
}
template <int EPI>
__device__ __forceinline__ void load_post(const GemmArgs &g, int t, int tile, int half, EpilogueIn &in) {
  if constexpr (EPI != kEpiResidual) {
    if (g.n_ss <= kSsPrefetch) {   // the sum in load_late's order
      float sum = 0.f;
#pragma unroll
      for (int i = 0; i < kSsPrefetch / 4; ++i)
        if (4 * i < g.n_ss) sum += (in.ss[i][0] + in.ss[i][1]) + (in.ss[i][2] + in.ss[i][3]);
      in.inv_rms = 1.0f / sqrtf(sum * g.inv_H + g.eps);
    } else {
      load_late<EPI>(g, t, tile, half, in);
    }
  }
}

// Writes the finished 32 x 32 tile `tile` for token t (this lane: rows
// 8 (r / 4) + 4 half + r % 4 of the tile, see below) through epilogue EPI.
template <int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs &g, const f32x16 &acc, EpilogueIn &in, int t, int tile,
                                         int half) {
  if constexpr (EPI == kEpiResidual) {
    // h += Y; x_out = h * gamma (the next norm's input, unnormalised) and the
    // sum of squares of h over this 32-column tile
    if (t >= g.T) return;
    float *hr = g.h + (int64_t)t * g.N + tile * kGemmTile + 4 * half;
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        in.h[i][r] += acc[4 * i + r];
        ss = fmaf(in.h[i][r], in.h[i][r], ss);
      }
      *(f32x4 *)(hr + 8 * i) = in.h[i];
    }
    if (!g.x_out) return;
    ss += __shfl_xor(ss, 32);
    if (half == 0) g.ss_out[(int64_t)t * (g.N / kGemmTile) + tile] = ss;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int n = tile * kGemmTile + 8 * i + 4 * half;
      const f32x4 v = in.h[i] * in.gamma[i] * in.scale;
      const int64_t off = g.act_packed ? packed_offset(t, n, g.N) : (int64_t)t * g.N + n;
      if (g.x_out_f16) {
        f16x4 o;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = (_Float16)v[r];
        *(f16x4 *)((_Float16 *)g.x_out + off) = o;
      } else {
        bf16x4 o;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[r] = (__bf16)v[r];
        *(bf16x4 *)(g.x_out + off) = o;
      }
    }
  } else {
    const float inv_rms = in.inv_rms;
    if constexpr (EPI == kEpiQKV) {
      if (t >= g.T) return;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int n = tile * kGemmTile + 8 * i + 4 * half;   // 4-runs never straddle q / k / v
        bf16x4 v;
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = (__bf16)(acc[4 * i + r] * inv_rms);
        if (n < g.n_q) *(bf16x4 *)(g.q_out + (int64_t)t * g.n_q + n) = v;
        else if (n < g.n_q + g.n_kv) *(bf16x4 *)(g.k_cache + (int64_t)in.dest * g.n_kv + (n - g.n_q)) = v;
        else *(bf16x4 *)(g.v_cache + (int64_t)in.dest * g.n_kv + (n - g.n_q - g.n_kv)) = v;
      }
      if (g.scale_out && tile == 0 && half == 0) g.scale_out[t] = pow2_scale(inv_rms);
    } else {   // SwiGLU: m = silu(gate) * up, fp16; rows t >= T are written as zeros
      const float f = inv_rms / in.scale;   // exact: s_t is a power of two
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        f16x4 mv;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float gt = acc[4 * i + r] * f, up = acc[4 * i + 8 + r] * f;
          mv[r] = (_Float16)(t < g.T ? gt / (1.0f + __expf(-gt)) * up : 0.f);
        }
        const int col = tile * 16 + 8 * i + 4 * half;
        const int64_t off = g.act_packed ? packed_offset(t, col, g.I) : (int64_t)t * g.I + col;
        *(f16x4 *)((_Float16 *)g.m_out + off) = mv;
      }
    }
  }
}

// LDS rows are 128 bytes (64 K values); 16-byte piece q of row r is stored at
// piece q ^ ((r >> 1) & 7), so the 16 lanes of one LDS cycle (16 consecutive
// rows, same logical piece) cover all 64 banks.
__device__ __forceinline__ int swz(int row, int q) { return q ^ ((row >> 1) & 7); }

// Direct global -> LDS copy of 16 bytes per lane: lane i of the wave writes
// lds_base + 16 i (the LDS address must be wave-uniform).
__device__ __forceinline__ void dma16(const void *src, void *lds_base) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)lds_base, 16, 0, 0);
}

// s_waitcnt vmcnt(n) with expcnt and lgkmcnt left free.
template <int N> __device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier of the LDS ring: completes this wave's LDS reads but not
// its in-flight global -> LDS copies (those are waited for by count).
__device__ __forceinline__ void ring_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// LDS ring depth in pipeline steps (measured: 2 to 7 steps stream equally
// fast or slower; the per-step cost, not the bytes in flight, sets the pace).
constexpr int kRing = 4;

// Each step (64 K) of a K group lands in LDS as RG weight tiles and one token
// tile of [32 rows][128 bytes].  The copies are spread over the group's waves
// with 8 rows x 128 bytes per instruction (8 cache lines), S - 1 steps ahead
// of the MFMAs; each wave then reads its fragments from LDS.
//
// Fragments: lane l reads row l % 32, K values 32 (l / 32) + 8 j .. + 7 for
// MFMA j of the step.  MFMA j thus contracts, in lane half h, the K values
// 32 h + 8 j .. of the step: a permutation of the step's 64 K values that the
// A (weight) and B (token) operands share, leaving the dot products unchanged.
//
// Output layout (v_mfma_f32_32x32x16): lane l holds, for token 32 tt + l % 32,
// the weight rows 8 (r / 4) + 4 (l / 32) + r % 4 of the tile, r = 0..15.
// SwiGLU tiles put 16 gate rows i0..i0+15 in tile rows 0..15 and the matching
// up rows in tile rows 16..31, so gate register r pairs with up register
// r + 8 of the same lane.
template <int RG, bool F16, int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs g) {
  // the arguments in one round trip to the argument segment
  asm volatile("" ::"s"(g.n_slices), "s"(g.n_ttiles), "s"(g.K), "s"(g.w0), "s"(g.w1), "s"(g.x), "s"(g.T), "s"(g.dest),
               "s"(g.scale_in), "s"(g.ss_in), "s"(g.n_ss), "s"((int)g.act_packed), "s"(gridDim.x));
  constexpr int KG = 4 / RG, S = kRing;
  constexpr int kTileBytes = kGemmTile * 128;
  constexpr int kGroupBytes = (RG + 1) * kTileBytes;
  constexpr int kStageBytes = KG * kGroupBytes;
  constexpr int kInstr = (RG + 1) * 4 / RG;   // copy instructions per wave per step
  __shared__ __attribute__((aligned(16))) unsigned char lds[S * kStageBytes];

  const int nwg = g.n_slices * g.n_ttiles;
  const int per_xcd = gridDim.x / 8;
  // XCD-aware order: consecutive logical tiles share an XCD (and its L2); the
  // token tiles of one weight slice are consecutive, so the slice is fetched
  // from HBM once per XCD.
  const int logical = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (logical >= nwg) return;
  const int tt = logical % g.n_ttiles, slice = logical / g.n_ttiles;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rg = wave % RG, kgi = wave / RG;
  const int kw = g.K / KG;   // K per wave
  const int nsteps = kw / kGemmKStep;
  const int64_t kbase = (int64_t)kgi * kw;
  const int frow = lane & 31, half = lane >> 5;
  const int t = tt * kGemmTile + frow;   // this lane's token in the epilogue
  const int tile = slice * RG + rg;      // 32-row tile of the output columns
  // each token tile walks K from its own starting step (as gemm_packed_kernel)
  // when the waves split K; with rg > 1 (row-major rows shared by the token
  // tiles' copies) the rotated walk measured slower (gate/up 12.7 -> 13.3 us)
  const int rot = RG == 1 ? tt * nsteps / g.n_ttiles : 0;

  EpilogueIn ein;
  load_early<EPI>(g, t, ein);

  // copy sources: instruction q of the K group covers tile q / 4 (row group
  // q / 4 < RG, else the token tile), rows 8 (q % 4) + lane / 8
  const __bf16 *src[kInstr];
  int dst[kInstr];
#pragma unroll
  for (int j = 0; j < kInstr; ++j) {
    const int q = rg * kInstr + j, ti = q / 4;
    const int row = 8 * (q % 4) + (lane >> 3), piece = swz(row, lane & 7);
    const __bf16 *p;
    if (ti < RG) {
      const int tile = slice * RG + ti;
      if constexpr (EPI == kEpiSwiGLU) p = (row < 16 ? g.w0 : g.w1) + (int64_t)(tile * 16 + (row & 15)) * g.K;
      else p = g.w0 + (int64_t)(tile * kGemmTile + row) * g.K;
    } else {
      p = g.x + (int64_t)(tt * kGemmTile + row) * g.K;
    }
    src[j] = p + kbase + 8 * piece;
    dst[j] = kgi * kGroupBytes + q * 1024;
  }
  auto issue = [&](int c) {
    unsigned char *st = lds + (c % S) * kStageBytes;
    const int p = c + rot < nsteps ? c + rot : c + rot - nsteps;   // c < nsteps
#pragma unroll
    for (int j = 0; j < kInstr; ++j) dma16(src[j] + p * kGemmKStep, st + dst[j]);
  };
  // wait until this wave's copies of the current step have landed, with
  // `ahead` (<= S - 2) later steps still in flight
  auto wait_step = [&](int ahead) {
    static_assert(S <= 7 && (S - 2) * kInstr < 64, "vmcnt range");
    switch (ahead) {
      case 0: wait_vm<0>(); break;
      case 1: wait_vm<kInstr>(); break;
      case 2: wait_vm<2 * kInstr>(); break;
      case 3: wait_vm<3 * kInstr>(); break;
      case 4: wait_vm<4 * kInstr>(); break;
      default: wait_vm<5 * kInstr>(); break;
    }
  };

  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  const int a_off = kgi * kGroupBytes + rg * kTileBytes + frow * 128;
  const int b_off = kgi * kGroupBytes + RG * kTileBytes + frow * 128;
#pragma unroll
  for (int c = 0; c < S - 1; ++c)
    if (c < nsteps) issue(c);
  for (int c = 0; c < nsteps; ++c) {
    wait_step(min(nsteps - 1 - c, S - 2));
    // step c visible to every wave, the slot of step c - 1 free: with rg = 1
    // each wave reads only the tiles it copied itself, so its own waits and
    // LDS-completion suffice; otherwise the waves share the token tile
    if constexpr (RG > 1) ring_barrier();
    else asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (c + S - 1 < nsteps) issue(c + S - 1);
    const unsigned char *st = lds + (c % S) * kStageBytes;
    u32x4 av[4], bv[4];   // all fragments of the step are read before the first MFMA
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      av[j] = *(const u32x4 *)(st + a_off + 16 * swz(frow, 4 * half + j));
      bv[j] = *(const u32x4 *)(st + b_off + 16 * swz(frow, 4 * half + j));
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if constexpr (F16)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, bf16x8_to_f16x8(av[j])),
                                                     __builtin_bit_cast(f16x8, bv[j]), acc, 0, 0, 0);
      else
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, av[j]),
                                                      __builtin_bit_cast(bf16x8, bv[j]), acc, 0, 0, 0);
    }
  }

  if constexpr (KG > 1) {
    // K groups 1.. hand their tiles to K group 0, which adds them in order
    // (through the ring's LDS, once every wave is done with it).
    float *red = (float *)lds;
    ring_barrier();
    if (kgi > 0) {
#pragma unroll
      for (int r = 0; r < 16; ++r) red[(((kgi - 1) * RG + rg) * 16 + r) * 64 + lane] = acc[r];
    }
    __syncthreads();
    if (kgi > 0) return;
#pragma unroll
    for (int k = 0; k < KG - 1; ++k)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] += red[((k * RG + rg) * 16 + r) * 64 + lane];
  }

  load_late<EPI>(g, t, tile, half, ein);
  epilogue<EPI>(g, acc, ein, t, tile, half);
}

// The same projection with both operands in the packed layout (packed_offset:
// weights packed once by hpd_pack_weight / hpd_pack_gate_up, activations
// written packed by their producers).  A wave's fragments for one step are
// then 4 whole contiguous 1 KB pieces per operand, loaded straight into a
// register ring of kPackedRing steps (kPackedRing - 1 ahead of the MFMAs);
// no LDS is used until the K groups are added.  Measured on the c4 step:
// rings of 6 and 8 steps are slower than 4 (gate/up 9.0 -> 15.7 us at 6,
// down 8.3 -> 16.6 us at 8): past 256 VGPRs the ring spills into
// accumulator registers and a SIMD holds one wave instead of two.
constexpr int kPackedRing = 4;

// f(integral_constant<int, rem>) for the runtime value rem in 1..N.
template <int N, typename F>
__device__ __forceinline__ void with_rem(int rem, F &&f) {
  if constexpr (N >= 1) {
    if (rem == N) f(std::integral_constant<int, N>{});
    else with_rem<N - 1>(rem, f);
  }
}

template <int RG, bool F16, int EPI>
__global__ __launch_bounds__(256) void gemm_packed_kernel(GemmArgs g) {
  // The arguments that the first loads depend on, in one round trip to the
  // argument segment (the compiler would otherwise fetch them in three,
  // each behind the branch that first needs them; measured: the c4 step
  // 0.761 -> 0.754 ms).
  asm volatile("" ::"s"(g.n_slices), "s"(g.n_ttiles), "s"(g.K), "s"(g.w0), "s"(g.x), "s"(g.T), "s"(g.dest),
               "s"(g.scale_in), "s"(g.ss_in), "s"(g.n_ss), "s"((int)g.act_packed), "s"((int)g.x_out_f16),
               "s"(gridDim.x));
  constexpr int KG = 4 / RG, S = kPackedRing;
  const int nwg = g.n_slices * g.n_ttiles;
  const int per_xcd = gridDim.x / 8;
  const int logical = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;   // XCD-aware, as gemm_kernel
  if (logical >= nwg) return;
  const int tt = logical % g.n_ttiles, slice = logical / g.n_ttiles;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rg = wave % RG, kgi = wave / RG;
  const int frow = lane & 31, half = lane >> 5;
  const int t = tt * kGemmTile + frow;
  const int tile = slice * RG + rg;
  const int ksteps = g.K / kGemmKStep, nsteps = ksteps / KG, ks0 = kgi * nsteps;
  // The n_ttiles workgroups of one weight slice run at the same time on one
  // XCD.  Walking K in the same order, they would all ask for the same bytes
  // at once, and the slice's HBM requests in flight would be those of one
  // workgroup.  Each token tile starts instead at its own fraction of the K
  // range and wraps around: the group's first requests cover the whole slice,
  // and each workgroup later finds the others' parts in the XCD's L2
  // (measured on the c4 step: down 8.4 -> 7.1 us, QKV 5.2 -> 4.8 us).
  const int rot = tt * nsteps / g.n_ttiles;

  EpilogueIn ein;
  load_early<EPI>(g, t, ein);

  const __bf16 *arow = g.w0 + ((int64_t)tile * ksteps + ks0) * 2048 + lane * 8;
  const __bf16 *brow = g.x + ((int64_t)tt * ksteps + ks0) * 2048 + lane * 8;
  u32x4 a[S][4], b[S][4];   // step c lives in slot c % S
  // The scheduling barriers keep each step's loads where they are issued (the
  // scheduler would otherwise sink them next to their MFMAs, emptying the ring).
  auto load = [&](int step, int slot) {
    const int p = step + rot < nsteps ? step + rot : step + rot - nsteps;   // step < nsteps
#pragma unroll
    for (int j = 0; j < 4; ++j) a[slot][j] = *(const u32x4 *)(arow + (int64_t)p * 2048 + 512 * j);
#pragma unroll
    for (int j = 0; j < 4; ++j) b[slot][j] = *(const u32x4 *)(brow + (int64_t)p * 2048 + 512 * j);
    __builtin_amdgcn_sched_barrier(0);
  };
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  // F16: the packed MLP weights are stored in fp16 already
  auto compute = [&](int slot) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if constexpr (F16)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a[slot][j]),
                                                     __builtin_bit_cast(f16x8, b[slot][j]), acc, 0, 0, 0);
      else
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[slot][j]),
                                                      __builtin_bit_cast(bf16x8, b[slot][j]), acc, 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Steps 0..S-2 are loaded up front; step c + S - 1 goes into the slot freed
  // by step c - 1 just before step c computes.  The main loop takes whole
  // groups of S steps whose loads are all in range; the remaining REM steps
  // (at most 2 S - 2; all of them when nsteps < 2 S - 1) run as a straight-
  // line tail specialised on REM.  No load sits under a runtime condition, so
  // the compiler waits for exactly the slot being consumed.
  auto tail = [&](int base, auto rem) {
    constexpr int REM = decltype(rem)::value;
#pragma unroll
    for (int u = 0; u < REM; ++u) {
      if (u + S - 1 < REM) load(base + u + S - 1, (u + S - 1) % S);
      compute(u % S);
    }
  };
  // unconditional (a step index past the end repeats the last step, unused),
  // so that no load sits under a runtime condition
#pragma unroll
  for (int u = 0; u < S - 1; ++u) load(min(u, nsteps - 1), u);
  if (kgi == 0) load_pre<EPI>(g, t, tile, half, ein);   // behind the first steps' loads
  if (nsteps >= 2 * S - 1) {
    const int n_main = (nsteps - (2 * S - 1)) / S + 1;
    for (int gi = 0; gi < n_main; ++gi) {
#pragma unroll
      for (int u = 0; u < S; ++u) {
        load(gi * S + u + S - 1, (u + S - 1) % S);
        compute(u);
      }
    }
    const int base = n_main * S;
    with_rem<2 * S - 2>(nsteps - base, [&](auto rem) { tail(base, rem); });   // S - 1 .. 2 S - 2
  } else {
    with_rem<2 * S - 2>(nsteps, [&](auto rem) { tail(0, rem); });            // 1 .. 2 S - 2
  }

  if (kgi == 0) load_post<EPI>(g, t, tile, half, ein);
  if constexpr (KG > 1) {
    // K groups 1.. hand their tiles to K group 0, which adds them in order
    __shared__ float red[(KG - 1) * RG * 16 * 64];
    if (kgi > 0) {
#pragma unroll
      for (int r = 0; r < 16; ++r) red[(((kgi - 1) * RG + rg) * 16 + r) * 64 + lane] = acc[r];
    }
    __syncthreads();
    if (kgi > 0) return;
#pragma unroll
    for (int k = 0; k < KG - 1; ++k)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] += red[((k * RG + rg) * 16 + r) * 64 + lane];
  }
  epilogue<EPI>(g, acc, ein, t, tile, half);
}

// LM head with an argmax epilogue: a workgroup of 4 waves owns 128
// vocabulary rows (32 per wave) against a group of up to 5 token tiles at
// once, so its weight rows are streamed once per group (the generic kernel
// re-reads them once per token tile).  With more than 5 token tiles the
// groups of one weight slice are consecutive workgroups of one XCD, so the
// later groups find the slice in that XCD's L2.  A wave's own weight tile
// (4 KB per K step, the packed layout: 4 whole 1 KB loads) goes straight into
// a register ring of 4 steps; the group's token tiles, which all 4 waves
// multiply, go through an LDS ring of 4 steps (direct global -> LDS copies,
// 1 KB per wave and tile).  Both are issued 3 steps ahead; a wave issues 4 +
// NTT loads per step (a group's padding tiles re-read the last token tile,
// so the count is fixed).  Requires K a multiple of 256 (4 steps of 64).
template <int NTT>
__global__ __launch_bounds__(256) void lm_argmax_kernel(GemmArgs g, int groups) {
  // the arguments in one round trip to the argument segment
  asm volatile("" ::"s"(g.n_slices), "s"(g.n_ttiles), "s"(g.K), "s"(g.w0), "s"(g.x), "s"(g.T), "s"(groups),
               "s"(gridDim.x));
  constexpr int SB = 4, kStage = NTT * 4096;
  __shared__ __attribute__((aligned(16))) unsigned char lds[SB * kStage];
  const int per_xcd = gridDim.x / 8;
  const int item = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (item >= g.n_slices * groups) return;
  const int slice = item / groups, tt0 = (item % groups) * NTT;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int frow = lane & 31, half = lane >> 5;
  const int tile = slice * 4 + wave, ksteps = g.K / kGemmKStep;
  const __bf16 *asrc = g.w0 + (int64_t)tile * ksteps * 2048 + lane * 8;
  u32x4 a[4][4];   // weight fragments of step s in a[s % 4]
  auto issue = [&](int step, u32x4 (&slot)[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) slot[j] = *(const u32x4 *)(asrc + (int64_t)step * 2048 + 512 * j);
    unsigned char *st = lds + (step % SB) * kStage;
#pragma unroll
    for (int i = 0; i < NTT; ++i) {
      const int q = wave + 4 * i, j = q & 3;                    // group tile q / 4, piece j
      const int tt = min(tt0 + (q >> 2), g.n_ttiles - 1);       // token tile (padding: the last one)
      dma16(g.x + ((int64_t)tt * ksteps + step) * 2048 + 512 * j + lane * 8, st + 1024 * q);
    }
  };
  f32x16 acc[NTT];
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[tt][r] = 0.f;
  auto step = [&](int c, u32x4 (&cur)[4], u32x4 (&next)[4]) {
    // step c landed (this wave's loads; the steps after it may stay in
    // flight), the token tiles visible to every wave; the slot of c - 1 is free
    const int pending = min(2, ksteps - 1 - c);
    if (pending >= 2) wait_vm<2 * (4 + NTT)>();
    else if (pending == 1) wait_vm<4 + NTT>();
    else wait_vm<0>();
    ring_barrier();
    if (c + 3 < ksteps) issue(c + 3, next);
    const unsigned char *st = lds + (c % SB) * kStage;
#pragma unroll
    for (int tt = 0; tt < NTT; ++tt) {
      u32x4 b[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = *(const u32x4 *)(st + 1024 * (4 * tt + j) + 16 * lane);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, cur[j]),
                                                          __builtin_bit_cast(bf16x8, b[j]), acc[tt], 0, 0, 0);
    }
  };
  issue(0, a[0]);
  issue(1, a[1]);
  issue(2, a[2]);
  for (int c = 0; c < ksteps; c += 4) {   // the ring slot of each step is a compile-time index
    step(c, a[0], a[3]);
    step(c + 1, a[1], a[0]);
    step(c + 2, a[2], a[1]);
    step(c + 3, a[3], a[2]);
  }
  // argmax epilogue: per token, the largest logit of the slice's 128 rows as
  // an ordered key (ties to the smaller row).  A lane holds rows
  // 8 (r / 4) + 4 half + r % 4 of its wave's tile for token frow; lanes l and
  // l ^ 32 combine, then the 4 waves through LDS (the ring is free once every
  // wave is past its last step).
  __syncthreads();
  uint64_t *red = (uint64_t *)lds;   // [NTT][4 waves][32 tokens]
#pragma unroll
  for (int tt = 0; tt < NTT; ++tt) {
    uint64_t best = 0;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const uint64_t k = argmax_key(acc[tt][r], tile * kGemmTile + 8 * (r >> 2) + 4 * half + (r & 3));
      best = k > best ? k : best;
    }
    const uint64_t other = ((uint64_t)(uint32_t)__shfl_xor((int)(best >> 32), 32) << 32) |
                           (uint32_t)__shfl_xor((int)(uint32_t)best, 32);
    best = other > best ? other : best;
    if (half == 0) red[(tt * 4 + wave) * 32 + frow] = best;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < NTT * 32; i += 256) {
    const int tt = i >> 5, tok = i & 31;
    if (tt0 + tt >= g.n_ttiles) continue;
    const uint64_t *v = red + tt * 128 + tok;
    const uint64_t m01 = v[0] > v[32] ? v[0] : v[32], m23 = v[64] > v[96] ? v[64] : v[96];
    g.amax[(int64_t)((tt0 + tt) * kGemmTile + tok) * g.n_slices + slice] = m01 > m23 ? m01 : m23;
  }
}

// Packs W[rows][cols] (bf16) into the packed layout: one thread per 16-byte
// piece of the output.  gate_up: rows are the pair's interleaved rows (row tile
// r = gate rows 16 r .. 16 r + 15, then up rows 16 r .. 16 r + 15) read from
// w (gate) and w2 (up), each [rows / 2][cols].  to_f16: the elements are
// converted to fp16 (as the torch-layout kernels convert them on the fly).
__global__ __launch_bounds__(256) void pack_weight_kernel(const __bf16 *w, const __bf16 *w2, int rows, int cols,
                                                          int gate_up, int to_f16, __bf16 *out) {
  const int64_t piece = (int64_t)blockIdx.x * 256 + threadIdx.x;   // 8 elements each
  if (piece * 8 >= (int64_t)rows * cols) return;
  const int64_t tile_id = piece / 256;
  const int in_tile = (int)(piece % 256), j = in_tile / 64, l = in_tile % 64;
  const int ctiles = cols / 64;
  const int r = (int)(tile_id / ctiles) * 32 + (l & 31);
  const int c = (int)(tile_id % ctiles) * 64 + 32 * (l >> 5) + 8 * j;
  const __bf16 *src;
  if (gate_up) {
    const int src_row = (r >> 5) * 16 + (r & 15);
    src = ((r & 31) < 16 ? w : w2) + (int64_t)src_row * cols + c;
  } else {
    src = w + (int64_t)r * cols + c;
  }
  const u32x4 v = *(const u32x4 *)src;
  *(u32x4 *)(out + piece * 8) = to_f16 ? bf16x8_to_f16x8(v) : v;
}

// Start of a step: h = h_in, x = h * gamma (bf16), sums of squares of h over
// 32-column tiles; rows T..Tpad-1 of x and zero_rows are zeroed.  x and
// zero_rows are row-major or, if packed, in the packed layout.  One workgroup
// per row; H and zero_cols are multiples of 128.
__global__ __launch_bounds__(256) void norm_input_kernel(const float *h_in, float *h, int T, int H,
                                                         const __bf16 *gamma, __bf16 *x, float *ss,
                                                         __bf16 *zero_rows, int zero_cols, int packed) {
  // the arguments in one round trip to the argument segment
  asm volatile("" ::"s"(h_in), "s"(h), "s"(T), "s"(H), "s"(gamma), "s"(x), "s"(ss), "s"(zero_rows), "s"(zero_cols),
               "s"(packed));
  const int t = blockIdx.x, tid = threadIdx.x;
  auto at = [&](int c, int cols) { return packed ? packed_offset(t, c, cols) : (int64_t)t * cols + c; };
  if (t >= T) {
    const bf16x4 z = {(__bf16)0.f, (__bf16)0.f, (__bf16)0.f, (__bf16)0.f};   // 0 in bf16 and fp16
    for (int c = 4 * tid; c < H; c += 1024) *(bf16x4 *)(x + at(c, H)) = z;
    if (zero_rows)
      for (int c = 4 * tid; c < zero_cols; c += 1024) *(bf16x4 *)(zero_rows + at(c, zero_cols)) = z;
    return;
  }
  for (int c = 4 * tid; c < H; c += 1024) {
    const f32x4 v = *(const f32x4 *)(h_in + (int64_t)t * H + c);
    if (h != h_in) *(f32x4 *)(h + (int64_t)t * H + c) = v;
    float sq = fmaf(v[0], v[0], fmaf(v[1], v[1], fmaf(v[2], v[2], v[3] * v[3])));
    // 8 consecutive threads cover one 32-column tile
    sq += __shfl_xor(sq, 1);
    sq += __shfl_xor(sq, 2);
    sq += __shfl_xor(sq, 4);
    if ((tid & 7) == 0) ss[(int64_t)t * (H / kGemmTile) + c / kGemmTile] = sq;
    bf16x4 o;
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = (__bf16)(v[r] * (gamma ? (float)gamma[c + r] : 1.f));
    *(bf16x4 *)(x + at(c, H)) = o;
  }
}

}  // namespace

hipError_t launch_norm_input(const float *h_in, float *h, int T, int Tpad, int H, const __bf16 *gamma,
                             __bf16 *x, float *ss, __bf16 *zero_rows, int zero_cols, bool packed,
                             hipStream_t stream) {
  if (H % 128 != 0 || zero_cols % 128 != 0 || T < 1 || Tpad < T || Tpad % kGemmTile != 0) return hipErrorInvalidValue;
  launch(KK_NORM, norm_input_kernel, dim3(Tpad), dim3(256), stream, h_in, h, T, H, gamma, x, ss, zero_rows, zero_cols,
         packed ? 1 : 0);
  return hipGetLastError();
}

namespace {

template <bool F16, int EPI>
void launch_epi(const GemmArgs &g, int kind, dim3 grid, hipStream_t stream) {
  if (g.rg == 4) launch(kind, gemm_kernel<4, F16, EPI>, grid, dim3(256), stream, g);
  else if (g.rg == 2) launch(kind, gemm_kernel<2, F16, EPI>, grid, dim3(256), stream, g);
  else launch(kind, gemm_kernel<1, F16, EPI>, grid, dim3(256), stream, g);
}

template <bool F16, int EPI>
void launch_packed(const GemmArgs &g, int kind, dim3 grid, hipStream_t stream) {
  if (g.rg == 4) launch(kind, gemm_packed_kernel<4, F16, EPI>, grid, dim3(256), stream, g);
  else if (g.rg == 2) launch(kind, gemm_packed_kernel<2, F16, EPI>, grid, dim3(256), stream, g);
  else launch(kind, gemm_packed_kernel<1, F16, EPI>, grid, dim3(256), stream, g);
}

}  // namespace

hipError_t launch_pack_weight(const __bf16 *w, const __bf16 *w2, int rows, int cols, bool gate_up, bool to_f16,
                              __bf16 *out, hipStream_t stream) {
  if (!w || !out || (gate_up && !w2) || rows <= 0 || cols <= 0 || rows % kGemmTile != 0 || cols % kGemmKStep != 0)
    return hipErrorInvalidValue;
  const int64_t pieces = (int64_t)rows * cols / 8;
  hipLaunchKernelGGL(pack_weight_kernel, dim3((unsigned)((pieces + 255) / 256)), dim3(256), 0, stream, w, w2, rows,
                     cols, gate_up ? 1 : 0, to_f16 ? 1 : 0, out);
  return hipGetLastError();
}

hipError_t launch_lm_argmax(const GemmArgs &g, int kind, hipStream_t stream) {
  const int ntt = g.Tpad / kGemmTile;
  if (ntt < 1 || g.n_ttiles != ntt || g.Tpad % kGemmTile || g.N % (4 * kGemmTile) || g.K % (4 * kGemmKStep) ||
      !g.amax || !g.a_packed || !g.act_packed || g.n_slices != g.N / (4 * kGemmTile))
    return hipErrorInvalidValue;
  const int groups = (ntt + 4) / 5, per = (ntt + groups - 1) / groups;   // per <= 5 token tiles per group
  const dim3 grid(((int64_t)g.n_slices * groups + 7) / 8 * 8), block(256);
  switch (per) {
    case 1: launch(kind, lm_argmax_kernel<1>, grid, block, stream, g, groups); break;
    case 2: launch(kind, lm_argmax_kernel<2>, grid, block, stream, g, groups); break;
    case 3: launch(kind, lm_argmax_kernel<3>, grid, block, stream, g, groups); break;
    case 4: launch(kind, lm_argmax_kernel<4>, grid, block, stream, g, groups); break;
    default: launch(kind, lm_argmax_kernel<5>, grid, block, stream, g, groups); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs &g, bool f16, int epi, int kind, hipStream_t stream) {
  const int kg = g.rg == 4 ? 1 : g.rg == 2 ? 2 : g.rg == 1 ? 4 : 0;
  if (kg == 0 || g.K <= 0 || g.K % (kGemmKStep * kg) != 0 || g.Tpad % kGemmTile != 0 ||
      g.n_ttiles * kGemmTile != g.Tpad || g.T < 1 || g.T > g.Tpad || g.N != g.n_slices * kGemmTile * g.rg ||
      (epi == kEpiSwiGLU && (g.N != 2 * g.I || !f16)) || (epi == kEpiQKV && f16))
    return hipErrorInvalidValue;
  if (epi < kEpiQKV || epi > kEpiSwiGLU ||
      (epi == kEpiResidual ? (!g.h || (g.x_out && !g.ss_out)) : (!g.ss_in || g.n_ss < 4 || g.n_ss % 4 != 0)))
    return hipErrorInvalidValue;
  const int nwg = g.n_slices * g.n_ttiles;
  const dim3 grid((nwg + 7) / 8 * 8);
  if (g.a_packed) {
    if (!g.act_packed) return hipErrorInvalidValue;
    if (epi == kEpiSwiGLU) launch_packed<true, kEpiSwiGLU>(g, kind, grid, stream);
    else if (epi == kEpiQKV) launch_packed<false, kEpiQKV>(g, kind, grid, stream);
    else if (f16) launch_packed<true, kEpiResidual>(g, kind, grid, stream);
    else launch_packed<false, kEpiResidual>(g, kind, grid, stream);
    return hipGetLastError();
  }
  if (g.act_packed) return hipErrorInvalidValue;   // the LDS-ring kernel reads row-major activations
  if (epi == kEpiSwiGLU) launch_epi<true, kEpiSwiGLU>(g, kind, grid, stream);
  else if (epi == kEpiQKV) launch_epi<false, kEpiQKV>(g, kind, grid, stream);
  else if (f16) launch_epi<true, kEpiResidual>(g, kind, grid, stream);
  else launch_epi<false, kEpiResidual>(g, kind, grid, stream);
  return hipGetLastError();
}

// Bytes one CU streams for a choice of rg: per workgroup (32 rg + 32) rows of
// K values (2 bytes each), times the workgroups per CU (256 CUs).  The
// cheapest shape wins (fewer workgroups on ties).
int choose_gemm_rg(int N, int K, int Tpad) {
  int best = 0;
  double best_cost = 0;
  const int tiles = Tpad / kGemmTile;
  for (int rg : {1, 2, 4}) {
    const int kg = 4 / rg;
    if (N % (kGemmTile * rg) != 0 || K % (kGemmKStep * kg) != 0) continue;
    const double nwg = (double)(N / (kGemmTile * rg)) * tiles;
    const double cost = (double)(kGemmTile * rg + kGemmTile) * K * 2 * std::max(1.0, nwg / 256.0);
    if (best == 0 || cost < best_cost * 0.999) {
      best = rg;
      best_cost = cost;
    }
  }
  return best;
}

}  // namespace hpd
