// gfx950 kernels of one branch-parallel attention layer.
//
// Every branch attends over its page's shared prefix and its own private rows
// (section "Layout-Coordinated Parallel Decoding", paragraph "Dynamic Branch
// Forking and Efficient Context Isolation"); the k drafts of a branch are
// causal among themselves (section "Integration with P-MTP").  The layer is
// computed in split form:
//
//   shared items    for each (page, kv head): the query rows of ALL branches
//                   of the page that use this kv head are stacked into 32-row
//                   MFMA tiles (row r = token r / G, head g * G + r % G), so a
//                   prefix K/V tile is fetched once and used by every branch.
//                   An item = 128 stacked rows over one key range; it writes
//                   a partial (O, log2-sum-exp) per row.
//   private items   for each (branch, kv head, key chunk of <= 128 keys): the
//                   branch's ragged private rows with the bottom-right causal
//                   mask (draft j sees private keys 0 .. L_b + j).
//   merge kernel    per (token, query head): log-sum-exp merge of all
//                   partials into the output row and its natural-log lse.
//
// bf16: one launch (shared_prefix_ring_kernel, or its fork-offset twin) runs
// both kinds of item: a shared item on a workgroup of 8 waves (4 row groups x
// the even and the odd key tiles) fed by an LDS ring of direct global -> LDS
// copies, a private item on one wave.  fp32: attn_f32_kernel, also one
// launch, register-staged (a shared item on 4 waves, a private item on one).
//
// MFMA formulation (v_mfma_f32_32x32x16_bf16; fp32 inputs use eight
// v_mfma_f32_32x32x2_f32 per step): scores are computed transposed,
// S^T = K Q^T, so each lane owns one query (lane % 32) and 16 keys of every
// 32-key block.  The row max then needs a single cross-lane exchange (lane ^
// 32), the row sum none until the end, and the P^T registers are directly the
// B operand of O^T += V^T P^T.  The contraction index of QK^T is permuted
// (lane half h, step s -> dims 32h + 8s .. +7, identical for K and Q).  The
// PV operand is one contiguous 16-byte LDS read: the fp32 tiles store V^T
// with key bits 2 and 3 swapped; the bf16 ring stores V as loaded and reads
// it transposed (ds_read_b64_tr_b16).
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"

namespace hpd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int D = HPD_HEAD_DIM;

// ------------------------------------------------------------ MFMA operands

template <typename T> struct Frag;                     // 8 contraction elements per lane
template <> struct Frag<__bf16> { bf16x8 v; };
template <> struct Frag<float> { f32x4 lo, hi; };

__device__ __forceinline__ void mma(f32x16 &acc, const Frag<__bf16> &a, const Frag<__bf16> &b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v, b.v, acc, 0, 0, 0);
}
// fp32: lane half h holds contraction index 8h + e in element e; eight
// 32x32x2 steps each take element e of both halves (indices e and 8 + e).
__device__ __forceinline__ void mma(f32x16 &acc, const Frag<float> &a, const Frag<float> &b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[0], b.lo[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[1], b.lo[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[2], b.lo[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[3], b.lo[3], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[0], b.hi[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[1], b.hi[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[2], b.hi[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[3], b.hi[3], acc, 0, 0, 0);
}

__device__ __forceinline__ void ld16(Frag<__bf16> &f, const __bf16 *p) { f.v = *(const bf16x8 *)p; }
__device__ __forceinline__ void ld16(Frag<float> &f, const float *p) {
  f.lo = *(const f32x4 *)p;
  f.hi = *(const f32x4 *)(p + 4);
}

__device__ __forceinline__ void zero(Frag<__bf16> &f) {
  for (int e = 0; e < 8; ++e) f.v[e] = (__bf16)0.f;
}
__device__ __forceinline__ void zero(Frag<float> &f) {
  f.lo = f32x4{0.f, 0.f, 0.f, 0.f};
  f.hi = f.lo;
}

// Eight fp32 probabilities -> B operand.
__device__ __forceinline__ void from_f32(Frag<__bf16> &f, const float *x) {
  for (int e = 0; e < 8; ++e) f.v[e] = (__bf16)x[e];
}
__device__ __forceinline__ void from_f32(Frag<float> &f, const float *x) {
  f.lo = f32x4{x[0], x[1], x[2], x[3]};
  f.hi = f32x4{x[4], x[5], x[6], x[7]};
}

// ------------------------------------------------------------ LDS tiles
//
// K tile: [64 keys][64 dims], 16-byte chunks XOR-swizzled per row so that the
// 16 lanes of one LDS cycle (16 keys, same logical chunk) hit 64 banks.
// V^T tile: [64 dims][64 keys + 16 B pad], keys stored at swap23(key).

template <typename T> struct Tile {
  static constexpr int kRowBytes = D * (int)sizeof(T);           // K row
  static constexpr int kChunks = kRowBytes / 16;                 // 16-B chunks per K row
  static constexpr int kVRowBytes = 64 * (int)sizeof(T) + 16;    // V^T row (one dim)
  static constexpr int kKBytes = 64 * kRowBytes;
  static constexpr int kVBytes = D * kVRowBytes;
  static constexpr int kBytes = kKBytes + kVBytes;
  __device__ static __forceinline__ int kchunk(int key, int q) {
    if constexpr (sizeof(T) == 2) return q ^ ((key >> 1) & 7);
    else return q ^ (key & 15);
  }
};

__device__ __forceinline__ int swap23(int k) { return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1); }

// Cooperative global -> register -> LDS staging of one 64-key K/V tile by NT
// threads.  Keys at or beyond `nkeys` (relative to the tile) are zero-filled
// and never read from memory.
template <typename T, int NT> struct TileLoader {
  using Tl = Tile<T>;
  static constexpr int kKTasks = 64 * Tl::kChunks / NT;   // K chunks per thread
  static constexpr int kVTasks = 32 * Tl::kChunks / NT;   // V key-pair chunks per thread
  static_assert(kKTasks >= 1 && kVTasks >= 1, "tile loader thread count");
  u32x4 kr[kKTasks];
  u32x4 vr[kVTasks][2];

  // rows: pointer to element [key 0][0] of this kv head; row stride in elements.
  __device__ __forceinline__ void load(const T *rows, int64_t stride, int nkeys, int tid) {
#pragma unroll
    for (int i = 0; i < kKTasks; ++i) {
      const int idx = tid + i * NT, key = idx / Tl::kChunks, q = idx % Tl::kChunks;
      kr[i] = key < nkeys ? *(const u32x4 *)((const char *)(rows + key * stride) + 16 * q)
                          : u32x4{0u, 0u, 0u, 0u};
    }
  }
  __device__ __forceinline__ void load_v(const T *rows, int64_t stride, int nkeys, int tid) {
#pragma unroll
    for (int i = 0; i < kVTasks; ++i) {
      const int idx = tid + i * NT, m = idx / Tl::kChunks, q = idx % Tl::kChunks;
      const int k0 = 2 * m, k1 = 2 * m + 1;
      vr[i][0] = k0 < nkeys ? *(const u32x4 *)((const char *)(rows + k0 * stride) + 16 * q)
                            : u32x4{0u, 0u, 0u, 0u};
      vr[i][1] = k1 < nkeys ? *(const u32x4 *)((const char *)(rows + k1 * stride) + 16 * q)
                            : u32x4{0u, 0u, 0u, 0u};
    }
  }
  __device__ __forceinline__ void store(unsigned char *lds, int tid) const {
#pragma unroll
    for (int i = 0; i < kKTasks; ++i) {
      const int idx = tid + i * NT, key = idx / Tl::kChunks, q = idx % Tl::kChunks;
      *(u32x4 *)(lds + key * Tl::kRowBytes + 16 * Tl::kchunk(key, q)) = kr[i];
    }
    unsigned char *vt = lds + Tl::kKBytes;
#pragma unroll
    for (int i = 0; i < kVTasks; ++i) {
      const int idx = tid + i * NT, m = idx / Tl::kChunks, q = idx % Tl::kChunks;
      const int pos = swap23(2 * m);
      if constexpr (sizeof(T) == 2) {
        // chunk = 8 bf16 dims of key 2m (vr[i][0]) and of key 2m+1 (vr[i][1])
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const unsigned w0 = vr[i][0][e / 2], w1 = vr[i][1][e / 2];
          const unsigned lo = (e & 1) ? (w0 >> 16) : (w0 & 0xffffu);
          const unsigned hi = (e & 1) ? (w1 & 0xffff0000u) : (w1 << 16);
          *(unsigned *)(vt + (q * 8 + e) * Tl::kVRowBytes + pos * 2) = lo | hi;
        }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          *(u32x2 *)(vt + (q * 4 + e) * Tl::kVRowBytes + pos * 4) = u32x2{vr[i][0][e], vr[i][1][e]};
      }
    }
  }
};

// ------------------------------------------------------------ bf16 LDS ring
//
// The bf16 shared-prefix kernel streams K and V tiles (64 keys x 128 bytes
// each) through an LDS ring filled by direct global -> LDS copies, several
// tiles ahead of the MFMAs.  K keeps the swizzle of Tile<bf16>.  V is stored
// untransposed, [key][dims], with 16-byte chunk q of key row r at chunk
// q ^ (4 ((r >> 1) & 1)), and the V^T operand of the PV product is read with
// ds_read_b64_tr_b16: in each group of 16 lanes, lane i receives element
// i % 4 of the 4 elements addressed by lane 4 j + i / 4, for j = 0..3.
// Lane s of a group addresses V[K0 + s / 4][D0 + 4 (s % 4) .. + 3], so lane i
// gets dims D0 + i of keys K0 .. K0 + 3: one half of an MFMA operand.  A
// 32-lane half of the wave reads 4 key rows x 64 bytes (dims 0..31 or
// 32..63 of a block): key bit 0 selects a 32-bank half (rows are 128 bytes)
// and the swizzle's key bit 1 a 16-bank quarter within it, so the 32 lanes
// cover the 64 banks once.  Measured with SQ_LDS_BANK_CONFLICT on an LDS
// microbenchmark of this read: 2 cycles per instruction and no conflicts,
// against 4 cycles and half the cycles in conflicts for q ^ (2 ((r >> 1) & 3)).
// The swizzle depends on key bit 1 only, so whole 8-row offsets keep it.


__device__ __forceinline__ int vchunk(int key, int q) { return q ^ (4 * ((key >> 1) & 1)); }

// The transpose read is issued as inline assembly: the compiler's own
// ds_read_tr builtin makes it wait for every in-flight global -> LDS copy
// (vmcnt(0)) before the read, which would drain the ring.  The caller waits
// for the results with lds_wait_tr (lgkmcnt(0), tied to the result registers).
typedef unsigned int u32x2t __attribute__((ext_vector_type(2)));
template <int OFF>
__device__ __forceinline__ u32x2t ds_read_tr16(const unsigned char *p) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset field");
  u32x2t v;
  const unsigned addr = (unsigned)(uintptr_t)(const __attribute__((address_space(3))) unsigned char *)p;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF) : "memory");
  return v;
}

// The 16 transpose reads of one V tile for a lane, [b][st][hh], from the
// lane's two block bases (vt + voff[b]).
template <int I>
__device__ __forceinline__ void ds_read_tr16_tile(u32x2t (&vr)[16], const unsigned char *vb0, const unsigned char *vb1) {
  if constexpr (I < 16) {
    constexpr int b = I / 8, st = (I / 2) % 4, hh = I % 2;
    constexpr int off = 128 * (32 * (st >> 1) + 16 * (st & 1) + 8 * hh);
    vr[I] = ds_read_tr16<off>(b == 0 ? vb0 : vb1);
    ds_read_tr16_tile<I + 1>(vr, vb0, vb1);
  }
}
__device__ __forceinline__ void lds_wait_tr(u32x2t (&v)[16]) {
  asm volatile("s_waitcnt lgkmcnt(0)"
               : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]),
                 "+v"(v[7]), "+v"(v[8]), "+v"(v[9]), "+v"(v[10]), "+v"(v[11]), "+v"(v[12]), "+v"(v[13]),
                 "+v"(v[14]), "+v"(v[15])
               :
               : "memory");
}

// 16 bytes per lane, global -> LDS: lane i writes lds_base + 16 i (the LDS
// address must be wave-uniform).
__device__ __forceinline__ void dma16(const void *src, void *lds_base) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void *)lds_base, 16, 0, 0);
}

// s_waitcnt vmcnt(n) with expcnt and lgkmcnt left free.
template <int N> __device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier of an LDS ring: completes this wave's LDS reads but not
// its in-flight global -> LDS copies (those are waited for by count).
__device__ __forceinline__ void ring_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// ------------------------------------------------------------ wave state

// One wave: 32 query rows (lane % 32) against the keys of successive tiles.
template <typename T> struct WaveAttn {
  Frag<T> qf[4];      // Q^T operand for the 4 contraction steps of D = 64
  f32x16 o[2];        // O^T accumulators: dims 0..31 and 32..63
  f32x16 lsum;        // step_ring: row sums of P on the matrix core (every register = l)
  float m;            // running max of the scaled log2 scores of this query
  float l;            // this lane's share of the running sum (tile())
  int half;           // lane / 32

  __device__ __forceinline__ void init(const T *qrow, bool valid, int lane) {
    half = lane >> 5;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (valid) ld16(qf[s], qrow + 32 * half + 8 * s);
      else zero(qf[s]);
    }
    for (int r = 0; r < 16; ++r) { o[0][r] = 0.f; o[1][r] = 0.f; lsum[r] = 0.f; }
    m = -INFINITY;
    l = 0.f;
  }

  // Processes one LDS tile whose first key has index key0; keys with index
  // >= limit are masked for this lane's query.  `masked` is wave-uniform:
  // false when every key of the tile is visible to every row of the wave.
  __device__ __forceinline__ void tile(const unsigned char *lds, int key0, int limit, bool masked,
                                       float c, int lane) {
    using Tl = Tile<T>;
    const int kr = lane & 31;
    f32x16 s[2];
    for (int r = 0; r < 16; ++r) { s[0][r] = 0.f; s[1][r] = 0.f; }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int key = 32 * kb + kr;
      const unsigned char *row = lds + key * Tl::kRowBytes;
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        Frag<T> a;
        if constexpr (sizeof(T) == 2) {
          ld16(a, (const T *)(row + 16 * Tl::kchunk(key, 4 * half + st)));
        } else {
          a.lo = *(const f32x4 *)(row + 16 * Tl::kchunk(key, 8 * half + 2 * st));
          a.hi = *(const f32x4 *)(row + 16 * Tl::kchunk(key, 8 * half + 2 * st + 1));
        }
        mma(s[kb], a, qf[st]);
      }
    }
    if (masked) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = key0 + 32 * kb + (r >> 2) * 8 + 4 * half + (r & 3);
          if (key >= limit) s[kb][r] = -INFINITY;
        }
    }
    float mx = s[0][0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[0][r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[1][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m, mx * c);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m - m_use);
    m = m_new;
    float p[32];
    float sum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      p[r] = __builtin_amdgcn_exp2f(fmaf(s[0][r], c, -m_use));
      p[16 + r] = __builtin_amdgcn_exp2f(fmaf(s[1][r], c, -m_use));
    }
#pragma unroll
    for (int r = 0; r < 32; ++r) sum += p[r];
    l = fmaf(l, alpha, sum);
#pragma unroll
    for (int r = 0; r < 16; ++r) { o[0][r] *= alpha; o[1][r] *= alpha; }
    Frag<T> pf[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) from_f32(pf[st], p + 8 * st);
    const unsigned char *vt = lds + Tl::kKBytes;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const unsigned char *vrow = vt + (32 * b + kr) * Tl::kVRowBytes;
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        Frag<T> a;
        ld16(a, (const T *)(vrow + (16 * st + 8 * half) * (int)sizeof(T)));
        mma(o[b], a, pf[st]);
      }
    }
  }

  // Byte offsets, within a K tile of the ring (Tile<bf16> swizzle), of this
  // lane's operand for contraction step st of key block 0 (key lane % 32).
  // Key block 1 (32 keys on) is 32 rows further with the same swizzle, so it
  // is a constant offset from these.
  __device__ static __forceinline__ void k_offsets(int lane, int (&koff)[4]) {
    using Tl = Tile<T>;
    const int kr = lane & 31;
#pragma unroll
    for (int st = 0; st < 4; ++st) koff[st] = kr * Tl::kRowBytes + 16 * Tl::kchunk(kr, 4 * (lane >> 5) + st);
  }

  // Raw scores S^T of a K tile in the ring (Tile<bf16> swizzle): the two
  // 32-key blocks' MFMA chains are interleaved.
  __device__ __forceinline__ void qk_ring(const unsigned char *kt, const int (&koff)[4], f32x16 (&s)[2]) {
    static_assert(sizeof(T) == 2, "bf16 only");
    using Tl = Tile<T>;
    for (int r = 0; r < 16; ++r) { s[0][r] = 0.f; s[1][r] = 0.f; }
    Frag<T> a[2][4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int st = 0; st < 4; ++st) ld16(a[kb][st], (const T *)(kt + koff[st] + 32 * kb * Tl::kRowBytes));
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) mma(s[kb], a[kb][st], qf[st]);
  }

  // One software-pipelined step of the ring kernel: the LDS reads of the
  // next tile's K (kt_next, or none) and of this tile's V^T are issued first,
  // then the next tile's QK^T MFMAs (into s_next), which need only the K
  // reads and run while the VALU does the softmax of this tile's raw scores
  // s_cur, then this tile's PV and row-sum MFMAs.  (Measured: giving the
  // two waves of a SIMD opposite orders, QK^T last on one of them, is
  // slower.)  The running max is raised only when a score exceeds it by
  // more than 2^8 (log2 units): the probabilities then stay <= 256, and the
  // O / row-sum rescale is skipped for the (common) tiles that do not raise
  // it.  The row sums are taken on the matrix core (an all-ones A operand
  // makes every output row of lsum the sum over the tile's keys).  FSUM: they
  // are instead taken in fp32 on the VALU into l (this lane's half of the
  // keys), which keeps the exported log-sum-exp exact to fp32 rounding when a
  // row sees only a few keys (the matrix-core sum adds bf16-rounded
  // probabilities).
  template <bool FSUM = false>
  __device__ __forceinline__ void step_ring(const unsigned char *kt_next, const int (&koff)[4], const unsigned char *vt,
                                            const int (&voff)[2], f32x16 (&s_cur)[2], f32x16 (&s_next)[2], int key0,
                                            int limit, bool masked, float c) {
    static_assert(sizeof(T) == 2, "bf16 only");
    using Tl = Tile<T>;
    Frag<T> ka[2][4];
    if (kt_next) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int st = 0; st < 4; ++st)
          ld16(ka[kb][st], (const T *)(kt_next + koff[st] + 32 * kb * Tl::kRowBytes));
    }
    step_frags<FSUM>(kt_next != nullptr, ka, vt, voff, s_cur, s_next, key0, limit, masked, c);
  }

  // Raw scores S^T of a K tile held in registers: ka[kb][st] is the K
  // operand of key block kb (32 keys) and contraction step st, as qk_ring
  // reads it from LDS.
  __device__ __forceinline__ void qk_frags(const Frag<T> (&ka)[2][4], f32x16 (&s)[2]) {
    for (int r = 0; r < 16; ++r) { s[0][r] = 0.f; s[1][r] = 0.f; }
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) mma(s[kb], ka[kb][st], qf[st]);
  }

  // step_ring with the next tile's K operand already in registers (ka, used
  // if has_next).
  template <bool FSUM = false>
  __device__ __forceinline__ void step_frags(bool has_next, const Frag<T> (&ka)[2][4], const unsigned char *vt,
                                             const int (&voff)[2], f32x16 (&s_cur)[2], f32x16 (&s_next)[2], int key0,
                                             int limit, bool masked, float c) {
    static_assert(sizeof(T) == 2, "bf16 only");
    u32x2t vr[16];   // [b][st][hh]
    ds_read_tr16_tile<0>(vr, vt + voff[0], vt + voff[1]);
    // matrix core first: the next tile's scores need only the K reads, and
    // run while the VALU does this tile's softmax
    if (has_next) {
      for (int r = 0; r < 16; ++r) { s_next[0][r] = 0.f; s_next[1][r] = 0.f; }
#pragma unroll
      for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) mma(s_next[kb], ka[kb][st], qf[st]);
    }
    // softmax of this tile (VALU)
    if (masked) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = key0 + 32 * kb + (r >> 2) * 8 + 4 * half + (r & 3);
          if (key >= limit) s_cur[kb][r] = -INFINITY;
        }
    }
    float mx = s_cur[0][0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s_cur[0][r]);
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s_cur[1][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32)) * c;
    if (__ballot(mx > m + 8.f)) {   // wave-uniform: some query's max grew by > 2^8
      const float m_new = fmaxf(m, mx);
      const float alpha = __builtin_amdgcn_exp2f(m - (m_new == -INFINITY ? 0.f : m_new));
      m = m_new;
#pragma unroll
      for (int r = 0; r < 16; ++r) { o[0][r] *= alpha; o[1][r] *= alpha; lsum[r] *= alpha; }
      l *= alpha;
    }
    const float m_use = m == -INFINITY ? 0.f : m;
    float p[32];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      p[r] = __builtin_amdgcn_exp2f(fmaf(s_cur[0][r], c, -m_use));
      p[16 + r] = __builtin_amdgcn_exp2f(fmaf(s_cur[1][r], c, -m_use));
    }
    if constexpr (FSUM) {
      float ps = 0.f;
#pragma unroll
      for (int r = 0; r < 32; ++r) ps += p[r];
      l += ps;
    }
    Frag<T> pf[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) from_f32(pf[st], p + 8 * st);
    lds_wait_tr(vr);   // (lgkmcnt(0))
    // matrix core: this tile's PV and row sums
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        Frag<T> va;
        va.v = __builtin_bit_cast(bf16x8, u32x4{vr[(b * 4 + st) * 2][0], vr[(b * 4 + st) * 2][1],
                                                vr[(b * 4 + st) * 2 + 1][0], vr[(b * 4 + st) * 2 + 1][1]});
        mma(o[b], va, pf[st]);
      }
    if constexpr (!FSUM) {
      Frag<T> ones;
#pragma unroll
      for (int e = 0; e < 8; ++e) ones.v[e] = (__bf16)1.f;
#pragma unroll
      for (int st = 0; st < 4; ++st) mma(lsum, ones, pf[st]);
    }
  }

  // Transpose-read offsets (bytes, within a V tile) of this lane for dims
  // blocks 0 and 1 at key offset 0: the lane addresses key 4 h + (lane % 16) / 4
  // and dims 32 b + 16 ((lane / 16) % 2) + 4 (lane % 4).  Adding 8, 16 or 32
  // keys leaves the vchunk swizzle unchanged, so the 8 reads of a block are
  // constant offsets from these.
  __device__ static __forceinline__ void vt_offsets(int lane, int (&voff)[2]) {
    const int grp = lane >> 4, s16 = lane & 15, key = 4 * (lane >> 5) + (s16 >> 2);
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int dim = 32 * b + 16 * (grp & 1) + 4 * (s16 & 3);
      voff[b] = key * 128 + 16 * vchunk(key, dim >> 3) + 2 * (dim & 7);
    }
  }

  // Epilogue of the ring kernels, per wave.  The even-tile (P = 0) and
  // odd-tile (P = 1) waves of a row group saw disjoint key tiles of the same
  // 32 rows; wave P finishes head dims 32 P .. 32 P + 31.  It merges its own
  // accumulators of that half with its partner's (ob2, with the partner's
  // m2 and l2), taking the two states in the same order in both waves (the
  // even one first) so that both normalise by the same sum, and writes the
  // half rows as fp16 through its 2 KB of LDS scratch ([32 rows][32 dims],
  // 16-byte chunk q of row r at q ^ ((r / 4) % 4)), 16 whole 64-byte half
  // rows per store instruction.  The even wave also writes the lse.
  // prow_of(r): as for write_f16.
  template <int P, typename RowFn>
  __device__ __forceinline__ void finish_half(float m2, float l2, const f32x16 &ob2, unsigned char *scratch,
                                              _Float16 *part_o, float *part_lse, RowFn prow_of, int lane) {
    typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
    const float me = P ? m2 : m, mo = P ? m : m2, le = P ? l2 : l, lo = P ? l : l2;
    const float m_new = fmaxf(me, mo), m_use = m_new == -INFINITY ? 0.f : m_new;
    const float ae = __builtin_amdgcn_exp2f(me - m_use), ao = __builtin_amdgcn_exp2f(mo - m_use);
    const float l_tot = le * ae + lo * ao;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const float a_own = (P ? ao : ae) * inv, a_other = (P ? ae : ao) * inv;
    const int qr = lane & 31;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f16x4 v;
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = (_Float16)(o[P][4 * j + e] * a_own + ob2[4 * j + e] * a_other);
      *(f16x4 *)(scratch + qr * 64 + 16 * (j ^ ((qr >> 2) & 3)) + 8 * half) = v;
    }
    if constexpr (P == 0) {
      const int64_t pr_self = prow_of(qr);   // every lane calls prow_of (it may use cross-lane reads)
      if (half == 0 && pr_self >= 0)
        part_lse[pr_self] = l_tot > 0.f ? m_new + __builtin_amdgcn_logf(l_tot) : -INFINITY;
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the wave's LDS writes precede its reads
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int row = 16 * k + (lane >> 2), c = lane & 3;
      const u32x4 v = *(const u32x4 *)(scratch + row * 64 + 16 * (c ^ ((row >> 2) & 3)));
      const int64_t pr = prow_of(row);
      if (pr >= 0) *(u32x4 *)(part_o + pr * D + 32 * P + 8 * c) = v;
    }
  }

  // Normalises the wave's 32 partial rows and writes them as fp16 (bf16
  // path): the O^T registers go to this wave's 4 KB of LDS as [32 rows][64
  // dims] (16-byte chunk q of row r at q ^ (r & 7)), and are stored back 8
  // whole 128-byte rows per instruction.  prow_of(r) gives the partial row of
  // the wave's row r (lane % 32 order), or -1 for a row without a query.
  // l_total: l already holds the query's whole sum (step_ring), rather than
  // this lane's share of it (tile()).
  template <typename RowFn>
  __device__ __forceinline__ void write_f16(unsigned char *scratch, _Float16 *part_o, float *part_lse,
                                            RowFn prow_of, int lane, bool l_total) {
    typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
    const float l_other = __shfl_xor(l, 32);
    const float l_tot = l_total ? l : l + l_other;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const int qr = lane & 31;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        f16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = (_Float16)(o[b][4 * j + e] * inv);
        *(f16x4 *)(scratch + qr * 128 + 16 * ((4 * b + j) ^ (qr & 7)) + 8 * half) = v;
      }
    const int64_t pr_self = prow_of(qr);   // every lane calls prow_of (it may use cross-lane reads)
    if (half == 0 && pr_self >= 0) part_lse[pr_self] = l_tot > 0.f ? m + __builtin_amdgcn_logf(l_tot) : -INFINITY;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the wave's LDS writes precede its reads
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int row = 8 * k + (lane >> 3), c = lane & 7;
      const u32x4 v = *(const u32x4 *)(scratch + row * 128 + 16 * (c ^ (row & 7)));
      const int64_t pr = prow_of(row);
      if (pr >= 0) *(u32x4 *)(part_o + pr * D + 8 * c) = v;
    }
  }

  // Normalises and writes this lane's half of the partial row.
  __device__ __forceinline__ void write(float *part_o, float *part_lse, int64_t prow, bool valid) {
    const float l_tot = l + __shfl_xor(l, 32);
    if (!valid) return;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    float *dst = part_o + prow * D;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int d = 32 * b + 8 * j + 4 * half;
        *(f32x4 *)(dst + d) = f32x4{o[b][4 * j] * inv, o[b][4 * j + 1] * inv,
                                    o[b][4 * j + 2] * inv, o[b][4 * j + 3] * inv};
      }
    if (half == 0) part_lse[prow] = l_tot > 0.f ? m + __builtin_amdgcn_logf(l_tot) : -INFINITY;
  }
};

__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = min(v, __shfl_xor(v, off));
  return v;
}

__device__ __forceinline__ int wave_max(int v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = max(v, __shfl_xor(v, off));
  return v;
}

// ------------------------------------------------------------ shared kernel

struct AttnArgs {
  const void *q, *shared_k, *shared_v, *priv_k, *priv_v;
  PlanDev dev;
  int n_shared, n_private;
  int Hq, Hkv, G;
  float c;   // softmax scale * log2(e)
  Plan::RegularShared reg;
  int priv_first;   // bf16 kernel: private workgroups take the first grid slots
  int priv_per_wg;  // bf16 kernel: private items per workgroup (1..kPrivMaxPerWG)
  int priv_slots;   // bf16 kernel: private workgroups, rounded up to a multiple of 8
  int paged;        // K/V rows through the plan's tile tables
};

// K/V row of key i of a sequence (a page's prefix or a branch's private
// rows) whose item field `base` is its first row, or with paged K/V its first
// tile-table entry; i0 is the first key of i's 64-key tile (a multiple of 64),
// so the table entry is wave-uniform.
__device__ __forceinline__ int64_t kv_row(const AttnArgs &a, const int32_t *tiles, int base, int i0, int i) {
  return a.paged ? (int64_t)tiles[base + (i0 >> 6)] + (i - i0) : (int64_t)base + i;
}

// Fields of shared work item `item`: computed from its index for a regular
// plan (one page, no fork offsets: items ordered kv head, split, row group),
// else read from the plan's table (a dependent load at the head of every
// workgroup's chain, which the regular form avoids).
struct SharedItem {
  int g, row0, nrows, key0, key1, slot, flags, prefix_row, page_q_row, pos;
};
__device__ __forceinline__ SharedItem shared_item(const AttnArgs &a, int item) {
  SharedItem si;
  if (a.reg.on) {
    const int rgi = item % a.reg.groups, rest = item / a.reg.groups;
    const int s = rest % a.reg.splits;
    si.g = rest / a.reg.splits;
    si.row0 = rgi * kSharedWaves * kTileRows;
    si.nrows = min(kSharedWaves * kTileRows, a.reg.rows - si.row0);
    si.key0 = s * a.reg.split_keys;
    si.key1 = min(a.reg.prefix_len, si.key0 + a.reg.split_keys);
    si.slot = s;
    si.flags = 0;
    si.prefix_row = a.reg.prefix_row;
    si.page_q_row = a.reg.page_q_row;
    si.pos = 0;
  } else {
    const int32_t *it = a.dev.shared_items + (int64_t)item * SI_NFIELDS;
    si.g = it[SI_KVH]; si.row0 = it[SI_ROW0]; si.nrows = it[SI_NROWS];
    si.key0 = it[SI_KEY0]; si.key1 = it[SI_KEY1]; si.slot = it[SI_SLOT]; si.flags = it[SI_FLAGS];
    si.prefix_row = it[SI_PREFIX_ROW]; si.page_q_row = it[SI_PAGE_Q_ROW]; si.pos = it[SI_POS];
  }
  return si;
}

// Token of stacked position pos of a shared item's page, and with fork
// offsets the row's key limit (min of limit and the token's visible
// prefix).  Sorted pages (fork offsets) map positions through the plan's
// pos_token table (the item's pos field locates the page's entries from
// token_fork), whose entries also carry the visible prefix.
__device__ __forceinline__ void row_token(const AttnArgs &a, const SharedItem &si, int pos, bool valid, int &t,
                                          int &limit) {
  const int flags = si.flags, page_q_row = si.page_q_row;
  if (flags & SI_FLAG_SORTED) {
    const int2 e = *(const int2 *)(a.dev.token_fork + si.pos + 2 * (int64_t)pos);
    t = e.x;
    if (valid) limit = min(limit, e.y);
  } else {
    t = page_q_row + pos;
    if ((flags & SI_FLAG_FORK) && valid) limit = min(limit, a.dev.token_fork[t]);
  }
}

// One shared-prefix item of the register-staged form (fp32) on a 256-thread
// workgroup: K/V tiles through two LDS buffers of Tile<T>::kBytes at lds.
template <typename T>
__device__ __forceinline__ void shared_item_staged(const AttnArgs &a, int item, unsigned char *lds) {
  constexpr int NT = 256;
  using Tl = Tile<T>;
  const SharedItem si = shared_item(a, item);
  const int g = si.g, row0 = si.row0, nrows = si.nrows;
  const int key0 = si.key0, key1 = si.key1, slot = si.slot, flags = si.flags;
  const int prefix_row = si.prefix_row, page_q_row = si.page_q_row;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rloc = wave * 32 + (lane & 31);
  const bool valid = rloc < nrows;
  const int R = row0 + rloc;                           // stacked row of (page, g)
  int t, limit = key1;
  row_token(a, si, valid ? R / a.G : 0, valid, t, limit);
  const int hq = g * a.G + (valid ? R % a.G : 0);
  const bool wave_active = wave * 32 < nrows;
  const int wmin = wave_min(valid ? limit : key1);
  // keys past it: no row of the wave sees them
  const int wmax = (flags & SI_FLAG_FORK) ? __builtin_amdgcn_readfirstlane(wave_max(valid ? limit : key0)) : key1;

  const int64_t stride = (int64_t)a.Hkv * D;
  const T *kbase = (const T *)a.shared_k + (int64_t)g * D;
  const T *vbase = (const T *)a.shared_v + (int64_t)g * D;
  auto row = [&](int k0) { return kv_row(a, a.dev.shared_tiles, prefix_row, k0, k0) * stride; };

  WaveAttn<T> w;
  w.init((const T *)a.q + ((int64_t)t * a.Hq + hq) * D, valid, lane);

  TileLoader<T, NT> ld;
  const int ntiles = (key1 - key0 + 63) / 64;
  ld.load(kbase + row(key0), stride, key1 - key0, tid);
  ld.load_v(vbase + row(key0), stride, key1 - key0, tid);
  ld.store(lds, tid);
  __syncthreads();
  for (int i = 0; i < ntiles; ++i) {
    const int k0 = key0 + 64 * i;
    if (i + 1 < ntiles) {
      ld.load(kbase + row(k0 + 64), stride, key1 - k0 - 64, tid);
      ld.load_v(vbase + row(k0 + 64), stride, key1 - k0 - 64, tid);
    }
    if (wave_active && k0 < wmax) w.tile(lds + (i & 1) * Tl::kBytes, k0, limit, k0 + 64 > wmin, a.c, lane);
    if (i + 1 < ntiles) ld.store(lds + ((i + 1) & 1) * Tl::kBytes, tid);
    __syncthreads();
  }
  // a row writes its partial of this split only if it sees the split's first
  // key (fork offsets: the planner gives it no slot otherwise)
  const bool writes = valid && limit > key0;
  const int64_t prow = writes ? ((int64_t)a.dev.token_slots[2 * t] + slot) * a.Hq + hq : 0;
  if (wave_active) w.write(a.dev.part_o, a.dev.part_lse, prow, writes);
}

// bf16 shared-prefix kernel: same items and arithmetic as shared_item_staged,
// on 8 waves: waves w and w + 4 own the same 32 rows and take the even and
// odd key tiles of the item, so two waves share each SIMD; at the end they
// exchange their states through LDS and each merges and writes one half of
// the head dims (ring_epilogue).  K and V stream through an LDS ring of
// kPairRing tile pairs filled by direct global -> LDS copies, up to three pairs
// ahead.  Each wave is software-pipelined by one tile: the QK^T MFMAs of its
// next tile are issued before the softmax of the current one, so they run on
// the matrix core while the VALU works.  Each tile is 16 copy instructions of
// 8 key rows x 128 bytes (4 per wave and pair).  Key rows past the item's
// range are clamped to its last key (their scores are masked; a pair's
// missing odd tile is loaded clamped and not used), which keeps every wave's
// copy count the same.
constexpr int kPairRing = 4;

// Private work items of the bf16 kernel: one per wave on the first
// priv_per_wg (at most kPrivMaxPerWG = all 8) waves of a workgroup, each wave
// with kPrivWaveBytes of LDS for the item's V tiles (an item has at most
// kPrivateChunkKeys = 128 keys: two tiles; its K tiles go to registers).
constexpr int kPrivMaxPerWG = 8;
constexpr int kPrivWaveBytes = 2 * 64 * 128;
static_assert(kPrivateChunkKeys <= 128, "a private item fits two tiles");
__device__ __forceinline__ void private_item_ring(const AttnArgs &a, int item, int lane, unsigned char *lds);

// The ring kernels' epilogue (after the ring's last barrier, its LDS free):
// the two waves of row group rw hand each other (m, l) and their
// accumulators of the partner's half of the head dims (18 x 64 floats per
// wave), then each finishes its half (WaveAttn::finish_half).  my_prow: the
// partial row of this lane's query (lanes 0..31), or -1.
__device__ __forceinline__ void ring_epilogue(WaveAttn<__bf16> &w, unsigned char *lds, const AttnArgs &a, int rw,
                                              int par, int lane, bool wave_active, int my_prow) {
  constexpr int kXch = 18 * 64;   // floats handed over per wave
  static_assert(8 * kXch * 4 + 8 * 2048 <= kPairRing * 4 * 64 * 128, "epilogue scratch within the ring's LDS");
  float *mine = (float *)lds + (2 * rw + par) * kXch;
  const float *theirs = (const float *)lds + (2 * rw + (par ^ 1)) * kXch;
  if (wave_active) {
    mine[lane] = w.m;
    mine[64 + lane] = w.l;
#pragma unroll
    for (int r = 0; r < 16; ++r) mine[(2 + r) * 64 + lane] = par ? w.o[0][r] : w.o[1][r];
  }
  __syncthreads();
  if (!wave_active) return;
  f32x16 ob2;
#pragma unroll
  for (int r = 0; r < 16; ++r) ob2[r] = theirs[(2 + r) * 64 + lane];
  auto prow_of = [&](int r) -> int64_t { return __shfl(my_prow, r); };
  unsigned char *scratch = lds + 8 * kXch * 4 + (2 * rw + par) * 2048;
  if (par == 0)
    w.finish_half<0>(theirs[lane], theirs[64 + lane], ob2, scratch, (_Float16 *)a.dev.part_o, a.dev.part_lse, prow_of,
                     lane);
  else
    w.finish_half<1>(theirs[lane], theirs[64 + lane], ob2, scratch, (_Float16 *)a.dev.part_o, a.dev.part_lse, prow_of,
                     lane);
}

__global__ __launch_bounds__(512) void shared_prefix_ring_kernel(AttnArgs a) {
  using T = __bf16;
  using Tl = Tile<T>;
  constexpr int S = kPairRing, kTileBytes = 64 * 128, kTile = 2 * kTileBytes, kPair = 2 * kTile;
  constexpr int kRingBytes = S * kPair, kPrivBytes = kPrivMaxPerWG * kPrivWaveBytes;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kRingBytes > kPrivBytes ? kRingBytes : kPrivBytes];

  // Workgroups run either priv_per_wg private items or one shared item.  Both
  // ranges are rounded up to multiples of 8 so that the shared items keep
  // the XCD-aware order of the other kernels.  priv_first (the grid fits the
  // chip in one round): the private range comes first, so the longer
  // dependency chain of a private item starts first; otherwise the shared
  // items, the larger work, are dispatched first and the private items fill
  // in behind them.
  // (the private slot count comes from the host: a division by the runtime
  // items per workgroup would delay every workgroup's start)
  const int n_priv_slots = a.priv_slots, n_shared_slots = (a.n_shared + 7) / 8 * 8;
  const int priv0 = a.priv_first ? 0 : n_shared_slots, shared0 = a.priv_first ? n_priv_slots : 0;
  const int bid = blockIdx.x;
  if (bid >= priv0 && bid < priv0 + n_priv_slots) {
    // wave-uniform (scalar loads of the item's fields)
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), pi = (bid - priv0) * a.priv_per_wg + wave;
    if (wave < a.priv_per_wg && pi < a.n_private)
      private_item_ring(a, pi, threadIdx.x & 63, lds + wave * kPrivWaveBytes);
    return;
  }
  const int b = bid - shared0, per_xcd = n_shared_slots / 8;
  if (b < 0 || b >= n_shared_slots) return;
  const int item = (b % 8) * per_xcd + b / 8;
  if (item >= a.n_shared) return;
  const SharedItem si = shared_item(a, item);
  const int g = si.g, row0 = si.row0, nrows = si.nrows;
  const int key0 = si.key0, key1 = si.key1, slot = si.slot, flags = si.flags;
  const int prefix_row = si.prefix_row, page_q_row = si.page_q_row;

  // (wave-uniform, so that the ring's slot and copy addresses stay scalar)
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rw = wave & 3, par = wave >> 2;             // row group, key-tile parity
  const int rloc = rw * 32 + (lane & 31);
  const bool valid = rloc < nrows;
  const int R = row0 + rloc;                           // stacked row of (page, g)
  const int t = page_q_row + (valid ? R / a.G : 0);
  const int hq = g * a.G + (valid ? R % a.G : 0);
  int limit = key1;
  if ((flags & SI_FLAG_FORK) && valid) limit = min(limit, a.dev.token_fork[t]);
  const bool wave_active = rw * 32 < nrows;
  const int wmin = wave_min(valid ? limit : key1);

  const T *kbase = (const T *)a.shared_k + (int64_t)g * D;
  const T *vbase = (const T *)a.shared_v + (int64_t)g * D;
  int voff[2], koff[4];
  WaveAttn<T>::vt_offsets(lane, voff);
  WaveAttn<T>::k_offsets(lane, koff);

  // copy instructions of this wave for a pair: its parity's tile, K and V
  // rows 16 rw + lane / 8 and 16 rw + 8 + lane / 8, physical chunk lane % 8.
  // A tile's first row is a scalar address; each lane adds its 32-bit byte
  // offset within the tile (the copies' scalar-base + vector-offset form),
  // so the copies of a tile that lies wholly inside the item take no vector
  // arithmetic.
  const int crow = 16 * rw + (lane >> 3), pch = lane & 7;
  const int kq0 = Tl::kchunk(crow, pch), kq1 = Tl::kchunk(crow + 8, pch);
  const int vq0 = vchunk(crow, pch), vq1 = vchunk(crow + 8, pch);
  const unsigned rowb = (unsigned)(a.Hkv * D * (int)sizeof(T));   // bytes per K/V row
  const unsigned ko0 = crow * rowb + 16 * kq0, ko1 = (crow + 8) * rowb + 16 * kq1;
  const unsigned vo0 = crow * rowb + 16 * vq0, vo1 = (crow + 8) * rowb + 16 * vq1;
  const int ntiles = (key1 - key0 + 63) / 64, npairs = (ntiles + 1) / 2;
  // paged K/V: lane l holds the pool row of the item's tile l (at most 64
  // tiles per item), read with a uniform lane index when a tile is issued
  const int tile_row = a.paged && lane < ntiles ? a.dev.shared_tiles[prefix_row + (key0 >> 6) + lane] : 0;
  auto issue = [&](int j) {
    unsigned char *st = lds + (j % S) * kPair + par * kTile + 2048 * rw;
    const int tj = 2 * j + par;
    // the last pair's missing odd tile re-reads the item's last tile
    const int ti = min(tj, ntiles - 1), kt = key0 + 64 * ti;
    const int64_t base = a.paged ? (int64_t)__builtin_amdgcn_readlane(tile_row, ti) : (int64_t)prefix_row + kt;
    const unsigned char *kr = (const unsigned char *)kbase + base * rowb;
    const unsigned char *vr = (const unsigned char *)vbase + base * rowb;
    unsigned k0o = ko0, k1o = ko1, v0o = vo0, v1o = vo1;
    if (key0 + 64 * tj + 64 > key1) {
      // rows past the item's last key (key1 - 1) are clamped to it
      const int last = key1 - 1 - kt, r = key0 + 64 * tj - kt + crow;
      const unsigned r0 = (unsigned)min(r, last) * rowb, r1 = (unsigned)min(r + 8, last) * rowb;
      k0o = r0 + 16 * kq0; k1o = r1 + 16 * kq1; v0o = r0 + 16 * vq0; v1o = r1 + 16 * vq1;
    }
    dma16(kr + k0o, st);
    dma16(kr + k1o, st + 1024);
    dma16(vr + v0o, st + kTileBytes);
    dma16(vr + v1o, st + kTileBytes + 1024);
  };
  // wait until pair j's copies (this wave's 4) have landed, with `ahead`
  // later pairs still in flight
  auto wait_pair = [&](int ahead) {
    if (ahead >= 2) wait_vm<8>();
    else if (ahead == 1) wait_vm<4>();
    else wait_vm<0>();
  };
  static_assert(kPairRing == 4, "the ring holds pairs j - 1 .. j + 2 at iteration j");
  // Pair 0, then this lane's Q fragments and partial-row index, then pairs 1
  // and 2.  Pair 0 and the loads behind it are retired here, so the loop
  // never waits for the Q loads.
  if (npairs > 0) issue(0);
  WaveAttn<T> w;
  w.init((const T *)a.q + ((int64_t)t * a.Hq + hq) * D, valid, lane);
  const int my_slots = valid ? a.dev.token_slots[2 * t] : 0;
  if (npairs > 1) issue(1);
  if (npairs > 2) issue(2);
  wait_pair(min(npairs - 1, 2));
  // a row writes its partial of this split only if it sees the split's first
  // key (fork offsets: the planner gives it no slot otherwise)
  const int my_prow = valid && limit > key0 ? (my_slots + slot) * a.Hq + hq : -1;
  ring_barrier();   // pair 0 visible to every wave
  // the raw scores of this wave's current tile and of its next one; the
  // loop is unrolled twice so that the two swap roles without copies
  f32x16 s_a[2], s_b[2];
  if (wave_active && par < ntiles) w.qk_ring(lds + par * kTile, koff, s_a);
  auto pair = [&](int j, f32x16 (&s_cur)[2], f32x16 (&s_next)[2]) {
    // pair j + 1 visible; the slot of pair j - 1 (read in iteration j - 1) is free
    if (j + 1 < npairs) {
      wait_pair(min(npairs - 1, j + 2) - (j + 1));
      ring_barrier();
      if (j + 3 < npairs) issue(j + 3);
    }
    const int ti = 2 * j + par;
    if (wave_active && ti < ntiles) {
      const unsigned char *kt_next = ti + 2 < ntiles ? lds + ((j + 1) % S) * kPair + par * kTile : nullptr;
      const int k0 = key0 + 64 * ti;
      w.step_ring(kt_next, koff, lds + (j % S) * kPair + par * kTile + kTileBytes, voff, s_cur, s_next, k0, limit,
                  k0 + 64 > wmin, a.c);
    }
  };
  for (int j = 0; j < npairs; j += 2) {
    pair(j, s_a, s_b);
    if (j + 1 < npairs) pair(j + 1, s_b, s_a);
  }
  ring_barrier();   // every wave is done with the ring; its LDS becomes scratch
  w.l = w.lsum[0];  // the query's whole sum (the row-sum MFMAs of step_ring)
  ring_epilogue(w, lds, a, rw, par, lane, wave_active, my_prow);
}

// The bf16 kernel for plans with fork offsets: the same work as
// shared_prefix_ring_kernel, with each page's stacked positions mapped to
// tokens through the plan's pos_token table (items with SI_FLAG_SORTED) and
// each wave skipping the compute of the key tiles none of its rows sees.  It
// is a kernel of its own because folding these steps into
// shared_prefix_ring_kernel, even behind a compile-time switch, measured
// 0.1 - 0.3 us slower per launch on plans without fork offsets (same-box A/B
// of the 18-layer step: 0.760 -> 0.765 ms).
__global__ __launch_bounds__(512) void shared_prefix_ring_fork_kernel(AttnArgs a) {
  using T = __bf16;
  using Tl = Tile<T>;
  constexpr int S = kPairRing, kTileBytes = 64 * 128, kTile = 2 * kTileBytes, kPair = 2 * kTile;
  constexpr int kRingBytes = S * kPair, kPrivBytes = kPrivMaxPerWG * kPrivWaveBytes;
  __shared__ __attribute__((aligned(16))) unsigned char lds[kRingBytes > kPrivBytes ? kRingBytes : kPrivBytes];

  // Workgroups run either priv_per_wg private items or one shared item.  Both
  // ranges are rounded up to multiples of 8 so that the shared items keep
  // the XCD-aware order of the other kernels.  priv_first (the grid fits the
  // chip in one round): the private range comes first, so the longer
  // dependency chain of a private item starts first; otherwise the shared
  // items, the larger work, are dispatched first and the private items fill
  // in behind them.
  // (the private slot count comes from the host: a division by the runtime
  // items per workgroup would delay every workgroup's start)
  const int n_priv_slots = a.priv_slots, n_shared_slots = (a.n_shared + 7) / 8 * 8;
  const int priv0 = a.priv_first ? 0 : n_shared_slots, shared0 = a.priv_first ? n_priv_slots : 0;
  const int bid = blockIdx.x;
  if (bid >= priv0 && bid < priv0 + n_priv_slots) {
    // wave-uniform (scalar loads of the item's fields)
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), pi = (bid - priv0) * a.priv_per_wg + wave;
    if (wave < a.priv_per_wg && pi < a.n_private)
      private_item_ring(a, pi, threadIdx.x & 63, lds + wave * kPrivWaveBytes);
    return;
  }
  const int b = bid - shared0, per_xcd = n_shared_slots / 8;
  if (b < 0 || b >= n_shared_slots) return;
  const int item = (b % 8) * per_xcd + b / 8;
  if (item >= a.n_shared) return;
  const SharedItem si = shared_item(a, item);
  const int g = si.g, row0 = si.row0, nrows = si.nrows;
  const int key0 = si.key0, key1 = si.key1, slot = si.slot, flags = si.flags;
  const int prefix_row = si.prefix_row, page_q_row = si.page_q_row;

  // (wave-uniform, so that the ring's slot and copy addresses stay scalar)
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rw = wave & 3, par = wave >> 2;             // row group, key-tile parity
  const int rloc = rw * 32 + (lane & 31);
  const bool valid = rloc < nrows;
  const int R = row0 + rloc;                           // stacked row of (page, g)
  int t, limit = key1;
  row_token(a, si, valid ? R / a.G : 0, valid, t, limit);
  const int hq = g * a.G + (valid ? R % a.G : 0);
  const bool wave_active = rw * 32 < nrows;
  const int wmin = wave_min(valid ? limit : key1);
  // key tiles of the item that some row of this wave sees (fork offsets:
  // the rest are skipped; their copies are still issued for the others)
  // (wave-uniform, in a scalar register, so the loop's tests stay scalar branches)
  int ntw = (key1 - key0 + 63) / 64;
  if (flags & SI_FLAG_FORK)
    ntw = __builtin_amdgcn_readfirstlane(max(0, (min(key1, wave_max(valid ? limit : key0)) - key0 + 63) / 64));

  const T *kbase = (const T *)a.shared_k + (int64_t)g * D;
  const T *vbase = (const T *)a.shared_v + (int64_t)g * D;
  int voff[2], koff[4];
  WaveAttn<T>::vt_offsets(lane, voff);
  WaveAttn<T>::k_offsets(lane, koff);

  // copy instructions of this wave for a pair: its parity's tile, K and V
  // rows 16 rw + lane / 8 and 16 rw + 8 + lane / 8, physical chunk lane % 8.
  // A tile's first row is a scalar address; each lane adds its 32-bit byte
  // offset within the tile (the copies' scalar-base + vector-offset form),
  // so the copies of a tile that lies wholly inside the item take no vector
  // arithmetic.
  const int crow = 16 * rw + (lane >> 3), pch = lane & 7;
  const int kq0 = Tl::kchunk(crow, pch), kq1 = Tl::kchunk(crow + 8, pch);
  const int vq0 = vchunk(crow, pch), vq1 = vchunk(crow + 8, pch);
  const unsigned rowb = (unsigned)(a.Hkv * D * (int)sizeof(T));   // bytes per K/V row
  const unsigned ko0 = crow * rowb + 16 * kq0, ko1 = (crow + 8) * rowb + 16 * kq1;
  const unsigned vo0 = crow * rowb + 16 * vq0, vo1 = (crow + 8) * rowb + 16 * vq1;
  const int ntiles = (key1 - key0 + 63) / 64, npairs = (ntiles + 1) / 2;
  // paged K/V: lane l holds the pool row of the item's tile l (at most 64
  // tiles per item), read with a uniform lane index when a tile is issued
  const int tile_row = a.paged && lane < ntiles ? a.dev.shared_tiles[prefix_row + (key0 >> 6) + lane] : 0;
  auto issue = [&](int j) {
    unsigned char *st = lds + (j % S) * kPair + par * kTile + 2048 * rw;
    const int tj = 2 * j + par;
    // the last pair's missing odd tile re-reads the item's last tile
    const int ti = min(tj, ntiles - 1), kt = key0 + 64 * ti;
    const int64_t base = a.paged ? (int64_t)__builtin_amdgcn_readlane(tile_row, ti) : (int64_t)prefix_row + kt;
    const unsigned char *kr = (const unsigned char *)kbase + base * rowb;
    const unsigned char *vr = (const unsigned char *)vbase + base * rowb;
    unsigned k0o = ko0, k1o = ko1, v0o = vo0, v1o = vo1;
    if (key0 + 64 * tj + 64 > key1) {
      // rows past the item's last key (key1 - 1) are clamped to it
      const int last = key1 - 1 - kt, r = key0 + 64 * tj - kt + crow;
      const unsigned r0 = (unsigned)min(r, last) * rowb, r1 = (unsigned)min(r + 8, last) * rowb;
      k0o = r0 + 16 * kq0; k1o = r1 + 16 * kq1; v0o = r0 + 16 * vq0; v1o = r1 + 16 * vq1;
    }
    dma16(kr + k0o, st);
    dma16(kr + k1o, st + 1024);
    dma16(vr + v0o, st + kTileBytes);
    dma16(vr + v1o, st + kTileBytes + 1024);
  };
  // wait until pair j's copies (this wave's 4) have landed, with `ahead`
  // later pairs still in flight
  auto wait_pair = [&](int ahead) {
    if (ahead >= 2) wait_vm<8>();
    else if (ahead == 1) wait_vm<4>();
    else wait_vm<0>();
  };
  static_assert(kPairRing == 4, "the ring holds pairs j - 1 .. j + 2 at iteration j");
  // Pair 0, then this lane's Q fragments and partial-row index, then pairs 1
  // and 2.  Pair 0 and the loads behind it are retired here, so the loop
  // never waits for the Q loads.
  if (npairs > 0) issue(0);
  WaveAttn<T> w;
  w.init((const T *)a.q + ((int64_t)t * a.Hq + hq) * D, valid, lane);
  const int my_slots = valid ? a.dev.token_slots[2 * t] : 0;
  if (npairs > 1) issue(1);
  if (npairs > 2) issue(2);
  wait_pair(min(npairs - 1, 2));
  // a row writes its partial of this split only if it sees the split's first
  // key (fork offsets: the planner gives it no slot otherwise)
  const int my_prow = valid && limit > key0 ? (my_slots + slot) * a.Hq + hq : -1;
  ring_barrier();   // pair 0 visible to every wave
  // the raw scores of this wave's current tile and of its next one; the
  // loop is unrolled twice so that the two swap roles without copies
  f32x16 s_a[2], s_b[2];
  if (wave_active && par < ntw) w.qk_ring(lds + par * kTile, koff, s_a);
  auto pair = [&](int j, f32x16 (&s_cur)[2], f32x16 (&s_next)[2]) {
    // pair j + 1 visible; the slot of pair j - 1 (read in iteration j - 1) is free
    if (j + 1 < npairs) {
      wait_pair(min(npairs - 1, j + 2) - (j + 1));
      ring_barrier();
      if (j + 3 < npairs) issue(j + 3);
    }
    const int ti = 2 * j + par;
    if (wave_active && ti < ntw) {
      const unsigned char *kt_next = ti + 2 < ntw ? lds + ((j + 1) % S) * kPair + par * kTile : nullptr;
      const int k0 = key0 + 64 * ti;
      w.step_ring(kt_next, koff, lds + (j % S) * kPair + par * kTile + kTileBytes, voff, s_cur, s_next, k0, limit,
                  k0 + 64 > wmin, a.c);
    }
  };
  for (int j = 0; j < npairs; j += 2) {
    pair(j, s_a, s_b);
    if (j + 1 < npairs) pair(j + 1, s_b, s_a);
  }
  ring_barrier();   // every wave is done with the ring; its LDS becomes scratch
  w.l = w.lsum[0];  // the query's whole sum (the row-sum MFMAs of step_ring)
  ring_epilogue(w, lds, a, rw, par, lane, wave_active, my_prow);
}

// One private work item on one wave of the bf16 kernel.  Every load of the
// item is issued at once: its K rows straight into the registers of the
// QK^T operand (per MFMA a lane needs 16 contiguous bytes of one key row),
// its V rows into the wave's own kPrivWaveBytes of LDS in the ring layout
// (the PV operand is read transposed from there; no other wave touches the
// region), its Q fragments and the partial-row indices of its rows.  Key
// rows past the item's range are clamped to its last key and masked; an
// item of one tile loads its second tile clamped as well (not used), so
// that no load depends on the item's length.
__device__ __forceinline__ void private_item_ring(const AttnArgs &a, int item, int lane, unsigned char *lds) {
  using T = __bf16;
  constexpr int kTileBytes = 64 * 128;
  const int32_t *it = a.dev.private_items + (int64_t)item * PI_NFIELDS;
  const int g = it[PI_KVH], row0 = it[PI_ROW0], nrows = it[PI_NROWS];
  const int key0 = it[PI_KEY0], key1 = it[PI_KEY1], slot = it[PI_SLOT], past = it[PI_PAST];
  const int priv_row = it[PI_PRIV_ROW], q_row = it[PI_Q_ROW];

  const int rloc = lane & 31, half = lane >> 5;
  const bool valid = rloc < nrows;
  const int R = row0 + rloc;                            // stacked row of (branch, g)
  const int j = valid ? R / a.G : 0;                    // draft index within the branch
  const int t = q_row + j;
  const int hq = g * a.G + (valid ? R % a.G : 0);
  const int limit = valid ? min(key1, past + j + 1) : key1;   // bottom-right causal
  const int wmin = wave_min(limit);
  const int ntiles = (key1 - key0 + 63) / 64;           // 1 or 2

  const int64_t stride = (int64_t)a.Hkv * D;
  const T *kbase = (const T *)a.priv_k + (int64_t)g * D;
  const T *vbase = (const T *)a.priv_v + (int64_t)g * D;
  // K/V row of key k (clamped into the item's range) loaded for tile c is
  // base[c] + k - first key of tile min(c, ntiles - 1): with one tile, tile
  // 1's keys are all the item's last key, in tile 0.  Paged K/V: the pool
  // rows of the item's tiles, read before any copy is issued (a wait for
  // them behind the copies would wait for the copies too).
  int64_t base[2];
  if (a.paged) {
    const int tile_row = a.dev.priv_tiles[priv_row + (key0 >> 6) + min(lane & 1, ntiles - 1)];
    base[0] = __builtin_amdgcn_readlane(tile_row, 0);
    base[1] = __builtin_amdgcn_readlane(tile_row, 1);
  } else {
    base[0] = (int64_t)priv_row + key0;
    base[1] = (int64_t)priv_row + key0 + 64 * (ntiles - 1);
  }
  auto row_of = [&](int c, int k) -> int64_t { return base[c] + (k - key0 - 64 * min(c, ntiles - 1)); };
  // first partial slot of the token of the wave's row `lane` (lanes 0..31
  // with a query), loaded with the tiles
  const int tr = q_row + (row0 + (lane & 31)) / a.G;
  const int tslot = a.dev.token_slots[2 * (lane < nrows ? tr : q_row)];
  // V tile c: 8 copies of rows 8 i + lane / 8 (physical chunk lane % 8)
  const int rsub = lane >> 3, pch = lane & 7;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int kt = key0 + 64 * c;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int row = 8 * i + rsub;
      const int64_t r = row_of(c, min(kt + row, key1 - 1));
      dma16(vbase + r * stride + 8 * vchunk(row, pch), lds + c * kTileBytes + 1024 * i);
    }
  }
  // K tile c: key block kb, contraction step st holds dims 32 half + 8 st ..
  // + 8 of key 32 kb + lane % 32 (the order of the Q fragments)
  Frag<T> ka[2][2][4];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int kt = key0 + 64 * c;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const T *kr = kbase + row_of(c, min(kt + 32 * kb + rloc, key1 - 1)) * stride + 32 * half;
#pragma unroll
      for (int st = 0; st < 4; ++st) ld16(ka[c][kb][st], kr + 8 * st);
    }
  }
  WaveAttn<T> w;
  w.init((const T *)a.q + ((int64_t)t * a.Hq + hq) * D, valid, lane);
  wait_vm<0>();   // the V copies into LDS (the register loads are waited for by the compiler)
  int voff[2];
  WaveAttn<T>::vt_offsets(lane, voff);
  f32x16 s_cur[2], s_next[2];
  w.qk_frags(ka[0], s_cur);
  w.step_frags<true>(ntiles > 1, ka[1], lds, voff, s_cur, s_next, key0, limit, key0 + 64 > wmin, a.c);
  if (ntiles > 1) {
#pragma unroll
    for (int r = 0; r < 16; ++r) { s_cur[0][r] = s_next[0][r]; s_cur[1][r] = s_next[1][r]; }
    w.step_frags<true>(false, ka[1], lds + kTileBytes, voff, s_cur, s_next, key0 + 64, limit, key0 + 128 > wmin,
                       a.c);
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the V tiles are consumed; tile 0 becomes write scratch
  // partial row of the wave's row `lane` (the planner keeps partial rows below 2^31)
  const int my_prow = lane < nrows ? (tslot + slot) * a.Hq + g * a.G + (row0 + lane) % a.G : -1;
  auto prow_of = [&](int r) -> int64_t { return __shfl(my_prow, r); };
  w.write_f16(lds, (_Float16 *)a.dev.part_o, a.dev.part_lse, prow_of, lane, false);
}

// ------------------------------------------------------------ private kernel

// One fp32 private work item on one wave, staged through the wave's own
// LDS tile `lds` (Tile<float>::kBytes).
__device__ __forceinline__ void private_item_f32(const AttnArgs &a, int item, int lane, unsigned char *lds) {
  using T = float;
  constexpr int NT = 64;
  const int32_t *it = a.dev.private_items + (int64_t)item * PI_NFIELDS;
  const int g = it[PI_KVH], row0 = it[PI_ROW0], nrows = it[PI_NROWS];
  const int key0 = it[PI_KEY0], key1 = it[PI_KEY1], slot = it[PI_SLOT], past = it[PI_PAST];
  const int priv_row = it[PI_PRIV_ROW], q_row = it[PI_Q_ROW];

  const int rloc = lane & 31;
  const bool valid = rloc < nrows;
  const int R = row0 + rloc;                            // stacked row of (branch, g)
  const int j = valid ? R / a.G : 0;                    // draft index within the branch
  const int t = q_row + j;
  const int hq = g * a.G + (valid ? R % a.G : 0);
  const int limit = valid ? min(key1, past + j + 1) : key1;   // bottom-right causal
  const int wmin = wave_min(limit);

  const int64_t stride = (int64_t)a.Hkv * D;
  const T *kbase = (const T *)a.priv_k + (int64_t)g * D;
  const T *vbase = (const T *)a.priv_v + (int64_t)g * D;

  WaveAttn<T> w;
  w.init((const T *)a.q + ((int64_t)t * a.Hq + hq) * D, valid, lane);
  TileLoader<T, NT> ld;
  for (int k0 = key0; k0 < key1; k0 += 64) {
    const int64_t r = kv_row(a, a.dev.priv_tiles, priv_row, k0, k0) * stride;
    ld.load(kbase + r, stride, key1 - k0, lane);
    ld.load_v(vbase + r, stride, key1 - k0, lane);
    // the wave's own LDS tile: its reads of the previous tile are done before
    // the stores, and the stores before the reads (one wave, so no barrier)
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    ld.store(lds, lane);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    w.tile(lds, k0, limit, k0 + 64 > wmin, a.c, lane);
  }
  const int64_t prow = valid ? ((int64_t)a.dev.token_slots[2 * t] + slot) * a.Hq + hq : 0;
  w.write(a.dev.part_o, a.dev.part_lse, prow, valid);
}

// fp32 attention in one launch: the shared items on the first workgroups
// (XCD-aware order: consecutive workgroup ids go round-robin over the 8
// XCDs, so each XCD gets a contiguous run of items and items that read the
// same key range share one L2), then the private items, one per wave and 4
// per workgroup, each wave with its own LDS tile.
__global__ __launch_bounds__(256) void attn_f32_kernel(AttnArgs a) {
  using Tl = Tile<float>;
  __shared__ __attribute__((aligned(16))) unsigned char lds[4 * Tl::kBytes];
  const int n_shared_slots = (a.n_shared + 7) / 8 * 8, bid = blockIdx.x;
  if (bid < n_shared_slots) {
    const int per_xcd = n_shared_slots / 8;
    const int item = (bid % 8) * per_xcd + bid / 8;
    if (item < a.n_shared) shared_item_staged<float>(a, item, lds);
    return;
  }
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pi = (bid - n_shared_slots) * 4 + wave;
  if (pi < a.n_private) private_item_f32(a, pi, threadIdx.x & 63, lds + wave * Tl::kBytes);
}

// ------------------------------------------------------------ merge kernel

// TPR threads per (token, head) row, D / TPR dims each, 128-thread
// workgroups.  Partial lse values are in log2 units; the exported lse is
// natural-log.  One pass over the partials in batches of 16 (every load of
// a batch issued before its first use), with a running max:
// sum_i 2^(lse_i - m) O_i / sum_i 2^(lse_i - m), partials in slot order.
// The host takes TPR = 16 for up to kMergeWideRows rows (the launch is
// latency-bound: more, smaller workgroups) and TPR = 8 above (throughput-
// bound: half the loads, each twice as wide).  Measured: 16 threads per row
// in 128-thread workgroups against 256-thread ones, the c4 step 0.749 ->
// 0.747 ms (32 and 64 rows per workgroup slower, 4 no faster); 8 threads per
// row: the 16-page merge (21,312 rows) 6.4 -> 4.6 us, while at 2,064 rows
// (c4) the narrow form stays the faster.
constexpr int kMergeWideRows = 4096;
template <typename TO, typename TP, int TPR>
__global__ __launch_bounds__(128) void merge_kernel(PlanDev dev, TO *out, float *lse, int T, int Hq,
                                                    int out_packed) {
  // every argument in one round trip to the argument segment
  asm volatile("" ::"s"(T), "s"(Hq), "s"(dev.token_slots), "s"(dev.part_o), "s"(dev.part_lse), "s"(out), "s"(lse),
               "s"(out_packed));
  static_assert(TPR == 8 || TPR == 16, "threads per row");
  constexpr int B = 16, DPT = D / TPR, NV = DPT / 4;   // dims per thread, in 4-wide vectors
  const int row = blockIdx.x * (128 / TPR) + (int)threadIdx.x / TPR;
  if (row >= T * Hq) return;
  const int sub = threadIdx.x % TPR;
  const int t = row / Hq, h = row % Hq;
  const int first = dev.token_slots[2 * t], cnt = dev.token_slots[2 * t + 1];
  const float *lse_p = dev.part_lse + (int64_t)first * Hq + h;
  const TP *o_p = (const TP *)dev.part_o + ((int64_t)first * Hq + h) * D + DPT * sub;
  float m = -INFINITY, wsum = 0.f;
  f32x4 acc[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) acc[v] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int i0 = 0; i0 < cnt; i0 += B) {
    float lb[B];
    f32x4 ob[B][NV];
#pragma unroll
    for (int i = 0; i < B; ++i) {
      const int64_t j = min(i0 + i, cnt - 1);
      lb[i] = lse_p[j * Hq];
      if constexpr (sizeof(TP) == 2) {
        typedef _Float16 f16xN __attribute__((ext_vector_type(DPT)));
        const f16xN hv = *(const f16xN *)(o_p + j * Hq * D);
#pragma unroll
        for (int v = 0; v < NV; ++v)
          ob[i][v] = f32x4{(float)hv[4 * v], (float)hv[4 * v + 1], (float)hv[4 * v + 2], (float)hv[4 * v + 3]};
      } else {
#pragma unroll
        for (int v = 0; v < NV; ++v) ob[i][v] = *(const f32x4 *)(o_p + j * Hq * D + 4 * v);
      }
    }
    float mb = m;
#pragma unroll
    for (int i = 0; i < B; ++i)
      if (i0 + i < cnt) mb = fmaxf(mb, lb[i]);
    const float mu = mb == -INFINITY ? 0.f : mb;
    const float alpha = __builtin_amdgcn_exp2f(m - mu);   // 0 on the first batch (m = -inf)
    wsum *= alpha;
#pragma unroll
    for (int v = 0; v < NV; ++v) acc[v] *= alpha;
#pragma unroll
    for (int i = 0; i < B; ++i) {
      if (i0 + i < cnt) {
        const float wgt = __builtin_amdgcn_exp2f(lb[i] - mu);
        wsum += wgt;
#pragma unroll
        for (int v = 0; v < NV; ++v) acc[v] += wgt * ob[i][v];
      }
    }
    m = mb;
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  // out is [T][Hq * D], row-major or (16-bit outputs only) packed; a
  // thread's DPT (4 or 8) columns start at a multiple of DPT, so they are
  // contiguous in the packed layout too
  TO *dst = out + (out_packed ? packed_offset(t, h * D + DPT * sub, Hq * D) : (int64_t)row * D + DPT * sub);
  if constexpr (sizeof(TO) == 2) {
    typedef __bf16 bf16xN __attribute__((ext_vector_type(DPT)));
    bf16xN r;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 4; ++e) r[4 * v + e] = (__bf16)(acc[v][e] * inv);
    *(bf16xN *)dst = r;
  } else {
#pragma unroll
    for (int v = 0; v < NV; ++v) *(f32x4 *)(dst + 4 * v) = acc[v] * inv;
  }
  if (lse && sub == 0) lse[row] = wsum > 0.f ? (m + __builtin_amdgcn_logf(wsum)) * kLn2 : -INFINITY;
}

}  // namespace

// Compute units of the current device (cached per device).
int num_cus() {
  static int cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    cus[dev] = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0 ? n : 256;
  }
  return cus[dev];
}

PlanDev plan_dev(const Plan &P, void *workspace) {
  unsigned char *ws = (unsigned char *)workspace;
  PlanDev d;
  d.shared_tiles = (const int32_t *)(ws + P.off_shared_tiles);
  d.priv_tiles = (const int32_t *)(ws + P.off_priv_tiles);
  d.branch_q_row = (const int32_t *)(ws + P.off_branch_q_row);
  d.branch_new = (const int32_t *)(ws + P.off_branch_new);
  d.shared_items = (const int32_t *)(ws + P.off_shared_items);
  d.private_items = (const int32_t *)(ws + P.off_private_items);
  d.token_slots = (const int32_t *)(ws + P.off_token_slots);
  d.token_fork = (const int32_t *)(ws + P.off_token_fork);
  d.token_dest = (const int32_t *)(ws + P.off_token_dest);
  d.token_vis = (const int32_t *)(ws + P.off_token_vis);
  d.counters = (int32_t *)(ws + P.off_counters);
  d.part_o = (float *)(ws + P.off_part_o);
  d.part_lse = (float *)(ws + P.off_part_lse);
  return d;
}

hipError_t launch_branch_attention(const Plan &P, const void *q, const void *shared_k,
                                   const void *shared_v, const void *priv_k, const void *priv_v,
                                   void *out, float *lse, void *workspace, hipStream_t stream, bool out_packed) {
  AttnArgs a{};
  a.q = q; a.shared_k = shared_k; a.shared_v = shared_v; a.priv_k = priv_k; a.priv_v = priv_v;
  a.dev = plan_dev(P, workspace);
  a.n_shared = P.num_shared_items();
  a.n_private = P.num_private_items();
  a.Hq = P.attn.num_q_heads;
  a.Hkv = P.attn.num_kv_heads;
  a.G = P.G;
  a.c = P.scale * kLog2e;
  a.reg = P.regular;
  a.paged = P.paged ? 1 : 0;
  const bool bf16 = P.attn.dtype == HPD_BF16;
  if (bf16) {
    // one launch: the private items and the shared-prefix items; phase
    // isolation: the shared items, then the private items, in launches of
    // their own
    auto priv_slots = [](const AttnArgs &x) {
      const int n_priv_wg = (x.n_private + x.priv_per_wg - 1) / x.priv_per_wg;
      return (n_priv_wg + 7) / 8 * 8;
    };
    auto grid = [&](const AttnArgs &x) { return priv_slots(x) + (x.n_shared + 7) / 8 * 8; };
    // Private items per workgroup: the fewest that still fit the grid on
    // the chip in one round (one workgroup per CU: the launch's LDS), so
    // that the items spread over the CUs the shared items leave free.  When
    // the grid takes more than one round anyway, the private workgroups
    // follow the shared ones and fill the CUs those free, 4 items each
    // (measured on the 16-page workload, 252 shared items and 1,422 private
    // ones: 46.4 us per launch; 8 per workgroup 47.6 us, 2 per workgroup
    // 51.6 us, the private workgroups first 51.4 us).
    auto fit = [&](AttnArgs &x) {
      for (x.priv_per_wg = 1; x.priv_per_wg < kPrivMaxPerWG; ++x.priv_per_wg)
        if (grid(x) <= num_cus()) break;
      x.priv_first = grid(x) <= num_cus() ? 1 : 0;
      if (!x.priv_first) x.priv_per_wg = 4;
      x.priv_slots = priv_slots(x);
    };
    fit(a);
    auto ring = P.has_fork ? shared_prefix_ring_fork_kernel : shared_prefix_ring_kernel;
    if (attn_phase_isolation()) {
      AttnArgs sh = a, pr = a;
      sh.n_private = 0;
      pr.n_shared = 0;
      fit(sh);
      fit(pr);
      if (sh.n_shared > 0) launch(KK_SHARED, ring, dim3(grid(sh)), dim3(512), stream, sh);
      if (pr.n_private > 0) launch(KK_PRIVATE, ring, dim3(grid(pr)), dim3(512), stream, pr);
    } else if (grid(a) > 0) {
      launch(KK_SHARED, ring, dim3(grid(a)), dim3(512), stream, a);
    }
  } else {
    // one launch, as for bf16; phase isolation: the shared items, then the
    // private items, in launches of their own
    auto grid = [](const AttnArgs &x) { return (x.n_shared + 7) / 8 * 8 + (x.n_private + 3) / 4; };
    if (attn_phase_isolation()) {
      AttnArgs sh = a, pr = a;
      sh.n_private = 0;
      pr.n_shared = 0;
      if (sh.n_shared > 0) launch(KK_SHARED, attn_f32_kernel, dim3(grid(sh)), dim3(256), stream, sh);
      if (pr.n_private > 0) launch(KK_PRIVATE, attn_f32_kernel, dim3(grid(pr)), dim3(256), stream, pr);
    } else if (grid(a) > 0) {
      launch(KK_SHARED, attn_f32_kernel, dim3(grid(a)), dim3(256), stream, a);
    }
  }
  const int rows = P.T * P.attn.num_q_heads;
  const int T = P.T, Hq = P.attn.num_q_heads;
  const bool wide = rows > kMergeWideRows;
  const dim3 mgrid(wide ? (rows + 15) / 16 : (rows + 7) / 8), mblock(128);
  // bf16 inputs: fp16 partials; fp32 inputs: fp32 partials
  // The narrow instances are named first, so that they are emitted first,
  // right behind the attention kernels.  (Measured: with the wide ones
  // first, the c4 step ran 0.747 -> 0.750 ms, the narrow merge itself no
  // slower: the code's placement in the library moves the step by that much.)
  auto merge = [&](auto k16, auto k8, auto *o, int packed) {
    if (wide) launch(KK_MERGE, k8, mgrid, mblock, stream, a.dev, o, lse, T, Hq, packed);
    else launch(KK_MERGE, k16, mgrid, mblock, stream, a.dev, o, lse, T, Hq, packed);
  };
  if (P.attn.out_dtype == HPD_BF16) {
    if (bf16) merge(merge_kernel<__bf16, _Float16, 16>, merge_kernel<__bf16, _Float16, 8>, (__bf16 *)out, out_packed ? 1 : 0);
    else merge(merge_kernel<__bf16, float, 16>, merge_kernel<__bf16, float, 8>, (__bf16 *)out, out_packed ? 1 : 0);
  } else {
    if (bf16) merge(merge_kernel<float, _Float16, 16>, merge_kernel<float, _Float16, 8>, (float *)out, 0);
    else merge(merge_kernel<float, float, 16>, merge_kernel<float, float, 8>, (float *)out, 0);
  }
  return hipGetLastError();
}

}  // namespace hpd
