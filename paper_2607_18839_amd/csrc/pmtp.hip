// P-MTP verification and drafting (C ABI entry points hpd_pmtp_workspace_bytes
// and hpd_verify_draft_step; section "Integration with P-MTP", Algorithm 1's
// speculative decoding and verification).
//
// Per call: the final-norm input of the T decoder outputs, the LM head with an
// argmax epilogue (per token and 128-row slice the largest logit as an
// ordered key), then one workgroup per branch reduces the keys to y* at each
// of its positions (one wave per position), verifies its drafts, writes n_acc and the bonus token and seeds
// the draft state f = h at the last verified position.  Each draft iteration:
// the draft input [f ; embed(token)] with its sums of squares, the draft
// MLP's gate/up (SwiGLU epilogue, RMSNorm folded) and down projection
// (residual epilogue: f += ..., x = f * g_final), and the LM head on x.  The
// draft input kernel of the next iteration (or the final token kernel)
// reduces that iteration's keys to the drafted token.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <string>

#include "gemm.h"
#include "hpd.h"
#include "kernels.h"
#include "plan.h"

namespace hpd {

void set_last_error(const std::string &msg);

namespace {

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
int round32(int x) { return (x + kGemmTile - 1) / kGemmTile * kGemmTile; }

struct PmtpLayout {
  int T, Tpad, nb, nbpad, H, V, Id, kmax, ntile;
  size_t off_x_lm, off_ss_lm, off_amax_v, off_f, off_x_d, off_ss_d, off_scale_d, off_m_d, off_x_f, off_ss_f,
      off_amax_d, off_tok, bytes;
};

PmtpLayout pmtp_layout(const hpd_model_desc &m, const hpd_pmtp_desc &d, const Plan &P) {
  PmtpLayout L;
  L.T = P.T;
  L.Tpad = round32(P.T);
  L.nb = P.num_branches;
  L.nbpad = round32(P.num_branches);
  L.H = m.hidden;
  L.V = d.vocab;
  L.Id = d.draft_inner;
  L.kmax = d.window > 0 ? d.window : *std::max_element(P.num_new.begin(), P.num_new.end());
  L.ntile = d.vocab / (4 * kGemmTile);   // argmax keys per token: one per 128-row slice
  size_t off = align256(P.workspace_bytes);
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  L.off_x_lm = take((size_t)L.Tpad * L.H * 2);
  L.off_ss_lm = take((size_t)L.Tpad * (L.H / kGemmTile) * 4);
  L.off_amax_v = take((size_t)L.Tpad * L.ntile * 8);
  L.off_f = take((size_t)L.nbpad * L.H * 4);
  L.off_x_d = take((size_t)L.nbpad * 2 * L.H * 2);
  L.off_ss_d = take((size_t)L.nbpad * (2 * L.H / kGemmTile) * 4);
  L.off_scale_d = take((size_t)L.nbpad * 4);
  L.off_m_d = take((size_t)L.nbpad * L.Id * 2);
  L.off_x_f = take((size_t)L.nbpad * L.H * 2);
  L.off_ss_f = take((size_t)L.nbpad * (L.H / kGemmTile) * 4);
  L.off_amax_d = take((size_t)L.nbpad * L.ntile * 8);
  L.off_tok = take((size_t)L.nbpad * 4);
  L.bytes = off;
  return L;
}

// Largest of keys[0..n), reduced over the 64 lanes of the calling wave:
// thread t of the STRIDE threads that share the work issues its loads U at a
// time into independent registers (one round trip per U loads, not per load).
template <int STRIDE, int U>
__device__ uint64_t wave_max_key(const uint64_t *keys, int n, int t) {
  uint64_t best = 0;
  for (int i0 = t; i0 < n; i0 += STRIDE * U) {
    uint64_t v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + STRIDE * u;
      v[u] = i < n ? keys[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) best = max(best, v[u]);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const uint64_t o = ((uint64_t)(uint32_t)__shfl_xor((int)(best >> 32), off) << 32) |
                       (uint32_t)__shfl_xor((int)(uint32_t)best, off);
    best = max(best, o);
  }
  return best;
}

// Largest key of keys[0..n) over the workgroup (256 threads); every thread
// gets the result.
__device__ uint64_t wg_max_key(const uint64_t *keys, int n, uint64_t *sh) {
  const uint64_t best = wave_max_key<256, 8>(keys, n, threadIdx.x);
  __syncthreads();   // sh is free (previous readers are done)
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = best;
  __syncthreads();
  return max(max(sh[0], sh[1]), max(sh[2], sh[3]));
}

// One workgroup per (padded) branch: y* at each position, verification,
// n_acc, bonus token, draft seed f = h at position n_acc.
__global__ __launch_bounds__(256) void verify_kernel(PlanDev dev, int nb, int ntile, const uint64_t *amax,
                                                     const int32_t *tokens_in, const float *hidden, int H,
                                                     int32_t *verified, int32_t *n_acc, int32_t *draft_out,
                                                     float *f, int32_t *cur_tok) {
  __shared__ int ystar[HPD_MAX_K];
  __shared__ int acc_n;
  // the arguments in one round trip to the argument segment
  asm volatile("" ::"s"(dev.branch_q_row), "s"(dev.branch_new), "s"(nb), "s"(ntile), "s"(amax), "s"(tokens_in),
               "s"(hidden), "s"(H), "s"(f), "s"(cur_tok));
  const int b = blockIdx.x;
  float *fr = f + (int64_t)b * H;
  if (b >= nb) {   // padding rows of the draft state stay finite
    for (int c = threadIdx.x; c < H; c += 256) fr[c] = 0.f;
    if (threadIdx.x == 0) cur_tok[b] = 0;
    return;
  }
  const int q0 = dev.branch_q_row[b], k = dev.branch_new[b];
  // one wave per position (all of a position's keys loaded at once)
  const int lane = threadIdx.x & 63;
  for (int j = threadIdx.x >> 6; j < k; j += 4) {
    const uint64_t key = wave_max_key<64, 24>(amax + (int64_t)(q0 + j) * ntile, ntile, lane);
    if (lane == 0) {
      ystar[j] = argmax_id(key);
      verified[q0 + j] = ystar[j];
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int n = 0;
    while (n < k - 1 && ystar[n] == tokens_in[q0 + n + 1]) ++n;
    acc_n = n;
    n_acc[b] = n;
    draft_out[(int64_t)b * HPD_MAX_K] = ystar[n];
    cur_tok[b] = ystar[n];
  }
  __syncthreads();
  const float *hr = hidden + (int64_t)(q0 + acc_n) * H;
  for (int c = threadIdx.x; c < H; c += 256) fr[c] = hr[c];
}

// Draft input of iteration `it` for (padded) branch b: its token (it > 1: the
// argmax of the previous iteration, recorded as draft entry it - 1), then
// D = [f ; embed(token)] (2H values) as the packed fp16 norm input x_d of the
// fp16 draft MLP, with the sums of squares over each 32 columns.  Padding
// rows are zero.
__global__ __launch_bounds__(256) void draft_input_kernel(int it, int nb, int ntile, const uint64_t *amax,
                                                          const __bf16 *embed, const float *f, int H, float eps,
                                                          __bf16 *x_d, float *ss_d, float *scale_d,
                                                          int32_t *cur_tok, int32_t *draft_out) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  __shared__ uint64_t sh[4];
  __shared__ int tok_sh;
  const int b = blockIdx.x;
  const bool real = b < nb;
  if (it > 1 && real) {
    const uint64_t key = wg_max_key(amax + (int64_t)b * ntile, ntile, sh);
    if (threadIdx.x == 0) {
      const int tok = argmax_id(key);
      draft_out[(int64_t)b * HPD_MAX_K + it - 1] = tok;
      cur_tok[b] = tok;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) tok_sh = real ? cur_tok[b] : 0;
  __syncthreads();
  const int tok = tok_sh, W = 2 * H, n_ss = W / kGemmTile;
  auto value = [&](int c) -> f32x4 {
    if (!real) return f32x4{0.f, 0.f, 0.f, 0.f};
    if (c < H) return *(const f32x4 *)(f + (int64_t)b * H + c);
    const bf16x4 e = *(const bf16x4 *)(embed + (int64_t)tok * H + (c - H));
    return f32x4{(float)e[0], (float)e[1], (float)e[2], (float)e[3]};
  };
  // pass 1: sums of squares per 32-column tile (for the SwiGLU GEMM's norm
  // factor) and of the whole row, reduced in registers and LDS; the row's
  // first kCache chunks per thread stay in registers for pass 2
  constexpr int kCache = 4;
  __shared__ float wsum[4];
  f32x4 vals[kCache];
  float part = 0.f;
  auto tile_sum = [&](int c, const f32x4 &v) {
    float sq = fmaf(v[0], v[0], fmaf(v[1], v[1], fmaf(v[2], v[2], v[3] * v[3])));
    part += sq;
    sq += __shfl_xor(sq, 1);   // 8 consecutive threads cover one 32-column tile
    sq += __shfl_xor(sq, 2);
    sq += __shfl_xor(sq, 4);
    if ((threadIdx.x & 7) == 0) ss_d[(int64_t)b * n_ss + c / kGemmTile] = sq;
  };
#pragma unroll
  for (int i = 0; i < kCache; ++i) {
    const int c = 4 * threadIdx.x + 1024 * i;
    vals[i] = c < W ? value(c) : f32x4{0.f, 0.f, 0.f, 0.f};
    if (c < W) tile_sum(c, vals[i]);
  }
  for (int c = 4 * threadIdx.x + 1024 * kCache; c < W; c += 1024) tile_sum(c, value(c));
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) part += __shfl_xor(part, off);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = part;
  __syncthreads();
  // pass 2: the row as fp16, scaled by the power of two of its norm factor,
  // which the SwiGLU GEMM divides back out
  const float sum = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
  const float s = pow2_scale(1.0f / sqrtf(sum / (float)W + eps));
  if (threadIdx.x == 0) scale_d[b] = s;
  typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
  auto put = [&](int c, const f32x4 &v) {
    f16x4 o;
#pragma unroll
    for (int r = 0; r < 4; ++r) o[r] = (_Float16)(v[r] * s);
    *(f16x4 *)((_Float16 *)x_d + packed_offset(b, c, W)) = o;
  };
#pragma unroll
  for (int i = 0; i < kCache; ++i) {
    const int c = 4 * threadIdx.x + 1024 * i;
    if (c < W) put(c, vals[i]);
  }
  for (int c = 4 * threadIdx.x + 1024 * kCache; c < W; c += 1024) put(c, value(c));
}

// Embedding rows of the tokens a step feeds, as fp32 (one workgroup per token).
__global__ __launch_bounds__(256) void embed_kernel(const __bf16 *embed, int V, int H, const int32_t *tokens,
                                                    float *out) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  // the arguments in one round trip to the argument segment
  asm volatile("" ::"s"(embed), "s"(V), "s"(H), "s"(tokens), "s"(out));
  const int t = blockIdx.x, tok = tokens[t];
  const bool ok = tok >= 0 && tok < V;
  for (int c = 4 * threadIdx.x; c < H; c += 1024) {
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    if (ok) {
      const bf16x4 e = *(const bf16x4 *)(embed + (int64_t)tok * H + c);
      v = f32x4{(float)e[0], (float)e[1], (float)e[2], (float)e[3]};
    }
    *(f32x4 *)(out + (int64_t)t * H + c) = v;
  }
}

// The last drafted token of each branch.
__global__ __launch_bounds__(256) void draft_token_kernel(int it, int ntile, const uint64_t *amax,
                                                          int32_t *draft_out) {
  __shared__ uint64_t sh[4];
  const int b = blockIdx.x;
  const uint64_t key = wg_max_key(amax + (int64_t)b * ntile, ntile, sh);
  if (threadIdx.x == 0) draft_out[(int64_t)b * HPD_MAX_K + it] = argmax_id(key);
}

hpd_status validate(const hpd_model_desc *m, const hpd_pmtp_desc *d, const hpd_plan *plan, std::string *err) {
  if (!m || !d || !plan) { *err = "NULL model, pmtp or plan"; return HPD_ERR_INVALID_ARGUMENT; }
  if (plan->p.attn.dtype != HPD_BF16) { *err = "the plan must be HPD_BF16"; return HPD_ERR_UNSUPPORTED; }
  if (m->hidden < 256 || m->hidden % 256) { *err = "hidden must be a positive multiple of 256"; return HPD_ERR_UNSUPPORTED; }
  if (d->vocab < 128 || d->vocab % 128 || d->draft_inner < 128 || d->draft_inner % 128) {
    *err = "vocab and draft_inner must be positive multiples of 128";
    return HPD_ERR_UNSUPPORTED;
  }
  if (!(m->rms_eps >= 0.f) || m->rms_eps > 1.f) { *err = "rms_eps out of range"; return HPD_ERR_INVALID_ARGUMENT; }
  if (d->window < 0 || d->window > HPD_MAX_K) { *err = "window must be in 0..HPD_MAX_K"; return HPD_ERR_INVALID_ARGUMENT; }
  auto bad = [](const void *p) { return !p || ((uintptr_t)p & 15); };
  if (bad(d->lm_head) || bad(d->embed) || bad(d->w_draft_gate_up) || bad(d->w_draft_down) ||
      (d->g_final && ((uintptr_t)d->g_final & 15))) {
    *err = "NULL or misaligned P-MTP weight";
    return HPD_ERR_INVALID_ARGUMENT;
  }
  return HPD_OK;
}

}  // namespace
}  // namespace hpd

extern "C" {

hpd_status hpd_embed_tokens(const void *embed, int32_t vocab, int32_t hidden, const int32_t *tokens, int32_t T,
                            float *out, void *stream) {
  if (!embed || !tokens || !out || vocab < 1 || hidden < 4 || hidden % 4 || T < 0 || ((uintptr_t)embed & 7) ||
      ((uintptr_t)out & 15)) {
    hpd::set_last_error("hpd_embed_tokens: NULL or misaligned pointer, or bad sizes");
    return HPD_ERR_INVALID_ARGUMENT;
  }
  if (T == 0) return HPD_OK;
  hpd::launch(hpd::KK_EMBED, hpd::embed_kernel, dim3(T), dim3(256), (hipStream_t)stream, (const __bf16 *)embed,
              (int)vocab, (int)hidden, tokens, out);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    hpd::set_last_error(std::string("hpd_embed_tokens: ") + hipGetErrorString(e));
    return HPD_ERR_HIP;
  }
  return HPD_OK;
}

size_t hpd_pmtp_workspace_bytes(const hpd_model_desc *model, const hpd_pmtp_desc *pmtp, const hpd_plan *plan) {
  std::string err;
  if (hpd::validate(model, pmtp, plan, &err) != HPD_OK) return 0;
  const hpd::PmtpLayout L = hpd::pmtp_layout(*model, *pmtp, plan->p);
  return L.bytes - hpd::align256(plan->p.workspace_bytes);
}

hpd_status hpd_verify_draft_step(const hpd_model_desc *model, const hpd_pmtp_desc *pmtp, const hpd_plan *plan,
                                 const float *hidden, const int32_t *tokens_in, int32_t *verified,
                                 int32_t *n_acc, int32_t *draft_out, void *workspace, size_t workspace_bytes,
                                 void *stream_) {
  std::string err;
  hpd_status st = hpd::validate(model, pmtp, plan, &err);
  if (st == HPD_OK && (!hidden || !tokens_in || !verified || !n_acc || !draft_out || !workspace)) {
    err = "NULL tensor or workspace";
    st = HPD_ERR_INVALID_ARGUMENT;
  }
  if (st == HPD_OK && (((uintptr_t)hidden & 15) || ((uintptr_t)workspace & 255))) {
    err = "hidden must be 16-byte and workspace 256-byte aligned";
    st = HPD_ERR_INVALID_ARGUMENT;
  }
  if (st != HPD_OK) {
    hpd::set_last_error("hpd_verify_draft_step: " + err);
    return st;
  }
  const hpd::Plan &P = plan->p;
  const hpd::PmtpLayout L = hpd::pmtp_layout(*model, *pmtp, P);
  if (workspace_bytes < L.bytes) {
    hpd::set_last_error("hpd_verify_draft_step: workspace too small");
    return HPD_ERR_WORKSPACE_TOO_SMALL;
  }
  hipStream_t stream = (hipStream_t)stream_;
  const hpd::TraceRange range("hpd_verify_draft_step");
  unsigned char *ws = (unsigned char *)workspace;
  const hpd::PlanDev dev = hpd::plan_dev(P, workspace);
  __bf16 *x_lm = (__bf16 *)(ws + L.off_x_lm);
  float *ss_lm = (float *)(ws + L.off_ss_lm);
  uint64_t *amax_v = (uint64_t *)(ws + L.off_amax_v), *amax_d = (uint64_t *)(ws + L.off_amax_d);
  float *f = (float *)(ws + L.off_f);
  __bf16 *x_d = (__bf16 *)(ws + L.off_x_d), *m_d = (__bf16 *)(ws + L.off_m_d), *x_f = (__bf16 *)(ws + L.off_x_f);
  float *ss_d = (float *)(ws + L.off_ss_d), *ss_f = (float *)(ws + L.off_ss_f);
  float *scale_d = (float *)(ws + L.off_scale_d);   // per branch: the draft input's power-of-two prescale
  int32_t *tok = (int32_t *)(ws + L.off_tok);
  const __bf16 *g_final = (const __bf16 *)pmtp->g_final;

  auto lm_head = [&](const __bf16 *x, int T, int Tpad, uint64_t *amax) {
    hpd::GemmArgs g{};
    g.w0 = (const __bf16 *)pmtp->lm_head;
    g.K = L.H;
    g.N = L.V;
    g.rg = 4;
    g.n_slices = L.V / (4 * hpd::kGemmTile);
    g.n_ttiles = Tpad / hpd::kGemmTile;
    g.x = x;
    g.T = T;
    g.Tpad = Tpad;
    g.amax = amax;
    g.a_packed = g.act_packed = true;
    return hpd::launch_lm_argmax(g, hpd::KK_LM_HEAD, stream);
  };

  // verification: x = bf16(h * g_final) (the norm factor does not move the argmax)
  hipError_t e = hpd::launch_norm_input(hidden, const_cast<float *>(hidden), L.T, L.Tpad, L.H, g_final, x_lm, ss_lm,
                                        nullptr, 0, true, stream);
  if (e == hipSuccess) e = lm_head(x_lm, L.T, L.Tpad, amax_v);
  if (e == hipSuccess) {
    hpd::launch(hpd::KK_VERIFY, hpd::verify_kernel, dim3(L.nbpad), dim3(256), stream, dev, L.nb, L.ntile, amax_v,
                tokens_in, hidden, L.H, verified, n_acc, draft_out, f, tok);
    e = hipGetLastError();
  }
  // drafting: iterations 1 .. W - 1 (W = the window)
  for (int it = 1; it < L.kmax && e == hipSuccess; ++it) {
    hpd::launch(hpd::KK_DRAFT_MLP, hpd::draft_input_kernel, dim3(L.nbpad), dim3(256), stream, it, L.nb, L.ntile,
                amax_d, (const __bf16 *)pmtp->embed, f, L.H, model->rms_eps, x_d, ss_d, scale_d, tok,
                draft_out);
    e = hipGetLastError();
    if (e != hipSuccess) break;
    hpd::GemmArgs g{};   // gate/up over [f ; e], SwiGLU, RMSNorm folded
    g.w0 = (const __bf16 *)pmtp->w_draft_gate_up;
    g.K = 2 * L.H;
    g.N = 2 * L.Id;
    g.rg = hpd::choose_gemm_rg(g.N, g.K, L.nbpad);
    g.n_slices = g.N / (hpd::kGemmTile * g.rg);
    g.n_ttiles = L.nbpad / hpd::kGemmTile;
    g.x = x_d;
    g.T = L.nb;
    g.Tpad = L.nbpad;
    g.ss_in = ss_d;
    g.scale_in = scale_d;   // the draft input's power-of-two prescale
    g.n_ss = 2 * L.H / hpd::kGemmTile;
    g.inv_H = 1.0f / (float)(2 * L.H);
    g.eps = model->rms_eps;
    g.m_out = m_d;
    g.I = L.Id;
    g.a_packed = g.act_packed = true;
    e = hpd::launch_gemm(g, true, hpd::kEpiSwiGLU, hpd::KK_DRAFT_MLP, stream);
    if (e != hipSuccess) break;
    hpd::GemmArgs r{};   // down: f += m W^T; x_f = f * g_final
    r.w0 = (const __bf16 *)pmtp->w_draft_down;
    r.K = L.Id;
    r.N = L.H;
    r.rg = hpd::choose_gemm_rg(r.N, r.K, L.nbpad);
    r.n_slices = r.N / (hpd::kGemmTile * r.rg);
    r.n_ttiles = L.nbpad / hpd::kGemmTile;
    r.x = m_d;
    r.T = L.nb;
    r.Tpad = L.nbpad;
    r.h = f;
    r.x_out = x_f;
    r.x_out_f16 = false;
    r.gamma = g_final;
    r.ss_out = ss_f;
    r.a_packed = r.act_packed = true;
    e = hpd::launch_gemm(r, true, hpd::kEpiResidual, hpd::KK_DRAFT_MLP, stream);
    if (e == hipSuccess) e = lm_head(x_f, L.nb, L.nbpad, amax_d);
  }
  if (e == hipSuccess && L.kmax > 1) {
    hpd::launch(hpd::KK_DRAFT_TOKEN, hpd::draft_token_kernel, dim3(L.nb), dim3(256), stream, L.kmax - 1, L.ntile,
                (const uint64_t *)amax_d, draft_out);
    e = hipGetLastError();
  }
  if (e != hipSuccess) {
    hpd::set_last_error(std::string("hpd_verify_draft_step: ") + hipGetErrorString(e));
    return HPD_ERR_HIP;
  }
  return HPD_OK;
}

}  // extern "C"
