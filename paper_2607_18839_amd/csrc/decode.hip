// One branch-parallel decode step of the decoder stack (C ABI entry points).
//
// The step runs every new token of every branch through all layers at once
// (Algorithm 1, the parallel draft over the active pool).  Per layer, with
// the residual stream h [T][hidden] kept in fp32 in hidden_out:
//   1 [h += previous down projection] RMSNorm(h) -> x (bf16)
//   2 QKV GEMM (split-K partials), epilogue kernel -> q (bf16) and the new
//     K/V rows, written into the layer's private cache at row priv_row + L + j
//   3 branch attention (shared-prefix, private, merge kernels) -> a (bf16)
//   4 O GEMM (partials)
//   5 h += a W_o^T, RMSNorm(h) -> x as hi + lo bf16 terms (one kernel)
//   6 gate/up GEMM (partials), SwiGLU epilogue kernel -> m, hi + lo terms
//   7 down GEMM (partials), added to h by the next layer's step 1 (or by a
//     final residual kernel after the last layer)
// (section "Overview", paragraph "LLM Decoder": GQA, RMSNorm, SwiGLU).
// Split-K partials are summed by the consuming kernel in split order, so the
// result does not depend on scheduling and needs no cross-workgroup sync.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <string>

#include "gemm.h"
#include "hpd.h"
#include "kernels.h"
#include "plan.h"

namespace hpd {

void set_last_error(const std::string &msg);

namespace {

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct GemmShape {
  int n_slices, ksplit, k_per_wg, n_tgroups;
};

// Split-K factor of one projection: the largest divisor of K / 32 that keeps
// the grid within `max_wg` workgroups (default 512, two per CU) and leaves
// each split at least `min_k` (default 256) of K, so that a split's fp32
// partial tile (64 x Tpad) stays about as large as the weight slice it comes
// from.  With one split the QKV and SwiGLU epilogues run inside the GEMM;
// otherwise a consumer kernel adds the splits in order.
GemmShape gemm_shape(int N_virtual, int K, int Tpad, bool allow_split) {
  GemmShape s;
  s.n_slices = N_virtual / 64;
  s.n_tgroups = (Tpad + kGemmTokenGroup - 1) / kGemmTokenGroup;
  const int steps = K / 32;
  int max_wg = 512, min_k = 256;
  if (const char *e = std::getenv("HPD_GEMM_MAX_WG")) max_wg = std::max(1, std::atoi(e));
  if (const char *e = std::getenv("HPD_GEMM_MIN_K")) min_k = std::max(32, std::atoi(e));
  s.ksplit = 1;
  if (allow_split)
    for (int d = 1; d <= steps; ++d)
      if (steps % d == 0 && s.n_tgroups * s.n_slices * d <= max_wg && K / d >= min_k) s.ksplit = d;
  s.k_per_wg = K / s.ksplit;
  return s;
}

struct DecodeLayout {
  int T, Tpad, H, I, nq, nkv;
  GemmShape qkv, o, gu, down;
  size_t off_x_hi, off_x_lo, off_q, off_attn, off_m_hi, off_m_lo, off_part, bytes;
};

DecodeLayout decode_layout(const hpd_model_desc &m, const Plan &P) {
  DecodeLayout L;
  L.T = P.T;
  // one token group of up to 144 rows; beyond that whole groups of 144
  L.Tpad = P.T <= kGemmTokenGroup ? (P.T + 15) / 16 * 16
                                  : (P.T + kGemmTokenGroup - 1) / kGemmTokenGroup * kGemmTokenGroup;
  L.H = m.hidden;
  L.I = m.intermediate;
  L.nq = P.attn.num_q_heads * HPD_HEAD_DIM;
  L.nkv = P.attn.num_kv_heads * HPD_HEAD_DIM;
  const bool split_wide = std::getenv("HPD_GEMM_NO_SPLIT_WIDE") == nullptr;
  L.qkv = gemm_shape(L.nq + 2 * L.nkv, L.H, L.Tpad, split_wide);
  L.o = gemm_shape(L.H, L.nq, L.Tpad, true);
  L.gu = gemm_shape(2 * L.I, L.H, L.Tpad, split_wide);
  L.down = gemm_shape(L.H, L.I, L.Tpad, true);
  size_t off = align256(P.workspace_bytes);
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  L.off_x_hi = take((size_t)L.Tpad * L.H * 2);
  L.off_x_lo = take((size_t)L.Tpad * L.H * 2);
  L.off_q = take((size_t)L.T * L.nq * 2);
  L.off_attn = take((size_t)L.Tpad * L.nq * 2);
  L.off_m_hi = take((size_t)L.Tpad * L.I * 2);
  L.off_m_lo = take((size_t)L.Tpad * L.I * 2);
  size_t part = 0;
  for (const GemmShape &s : {L.qkv, L.o, L.gu, L.down})
    part = std::max(part, (size_t)s.ksplit * L.Tpad * s.n_slices * 64 * sizeof(float));
  L.off_part = take(part);
  L.bytes = off;
  return L;
}

hpd_status validate(const hpd_model_desc *m, const hpd_plan *plan, std::string *err) {
  if (!m || !plan) { *err = "NULL model or plan"; return HPD_ERR_INVALID_ARGUMENT; }
  const Plan &P = plan->p;
  if (P.attn.dtype != HPD_BF16 || P.attn.out_dtype != HPD_BF16) {
    *err = "the plan of a decode step must have dtype and out_dtype HPD_BF16";
    return HPD_ERR_UNSUPPORTED;
  }
  if (m->num_layers < 1) { *err = "num_layers must be >= 1"; return HPD_ERR_INVALID_ARGUMENT; }
  if (m->hidden < 128 || m->hidden % 128 || m->intermediate < 128 || m->intermediate % 128 ||
      (P.attn.num_q_heads * HPD_HEAD_DIM) % 128) {
    *err = "hidden, intermediate and num_q_heads * 64 must be positive multiples of 128";
    return HPD_ERR_UNSUPPORTED;
  }
  if (!(m->rms_eps >= 0.f) || m->rms_eps > 1.f) { *err = "rms_eps out of range"; return HPD_ERR_INVALID_ARGUMENT; }
  if (!m->w_qkv || !m->w_o || !m->w_gate || !m->w_up || !m->w_down) {
    *err = "NULL weight array";
    return HPD_ERR_INVALID_ARGUMENT;
  }
  for (int l = 0; l < m->num_layers; ++l) {
    if (!m->w_qkv[l] || !m->w_o[l] || !m->w_gate[l] || !m->w_up[l] || !m->w_down[l]) {
      *err = "NULL weight of layer " + std::to_string(l);
      return HPD_ERR_INVALID_ARGUMENT;
    }
  }
  return HPD_OK;
}

}  // namespace
}  // namespace hpd

extern "C" {

size_t hpd_decode_workspace_bytes(const hpd_model_desc *model, const hpd_plan *plan) {
  if (!model || !plan) return 0;
  const hpd::DecodeLayout L = hpd::decode_layout(*model, plan->p);
  return L.bytes - hpd::align256(plan->p.workspace_bytes);
}

hpd_status hpd_decode_step(const hpd_model_desc *model, const hpd_plan *plan, const float *hidden_in,
                           float *hidden_out, const void *const *shared_k, const void *const *shared_v,
                           void *const *priv_k, void *const *priv_v, void *workspace,
                           size_t workspace_bytes, void *stream_) {
  std::string err;
  hpd_status st = hpd::validate(model, plan, &err);
  if (st != HPD_OK) {
    hpd::set_last_error("hpd_decode_step: " + err);
    return st;
  }
  const hpd::Plan &P = plan->p;
  const hpd_model_desc &m = *model;
  if (!hidden_in || !hidden_out || !priv_k || !priv_v || !workspace ||
      (P.shared_rows > 0 && (!shared_k || !shared_v))) {
    hpd::set_last_error("hpd_decode_step: NULL tensor, cache array or workspace");
    return HPD_ERR_INVALID_ARGUMENT;
  }
  for (int l = 0; l < m.num_layers; ++l) {
    if (!priv_k[l] || !priv_v[l] || (P.shared_rows > 0 && (!shared_k[l] || !shared_v[l])) ||
        ((uintptr_t)priv_k[l] | (uintptr_t)priv_v[l]) % 16 ||
        (P.shared_rows > 0 && ((uintptr_t)shared_k[l] | (uintptr_t)shared_v[l]) % 16)) {
      hpd::set_last_error("hpd_decode_step: NULL or misaligned cache pointer of layer " + std::to_string(l));
      return HPD_ERR_INVALID_ARGUMENT;
    }
  }
  if (((uintptr_t)hidden_in | (uintptr_t)hidden_out) % 16 || (uintptr_t)workspace % 256) {
    hpd::set_last_error("hpd_decode_step: hidden_in/out must be 16-byte and workspace 256-byte aligned");
    return HPD_ERR_INVALID_ARGUMENT;
  }
  const hpd::DecodeLayout L = hpd::decode_layout(m, P);
  if (workspace_bytes < L.bytes) {
    hpd::set_last_error("hpd_decode_step: workspace too small");
    return HPD_ERR_WORKSPACE_TOO_SMALL;
  }
  hipStream_t stream = (hipStream_t)stream_;
  unsigned char *ws = (unsigned char *)workspace;
  __bf16 *x_hi = (__bf16 *)(ws + L.off_x_hi), *x_lo = (__bf16 *)(ws + L.off_x_lo);
  __bf16 *q = (__bf16 *)(ws + L.off_q), *attn = (__bf16 *)(ws + L.off_attn);
  __bf16 *m_hi = (__bf16 *)(ws + L.off_m_hi), *m_lo = (__bf16 *)(ws + L.off_m_lo);
  float *part = (float *)(ws + L.off_part);
  const hpd::PlanDev dev = hpd::plan_dev(P, workspace);

  hipError_t e = hipSuccess;
  if (hidden_out != hidden_in)
    e = hipMemcpyAsync(hidden_out, hidden_in, (size_t)L.T * L.H * sizeof(float), hipMemcpyDeviceToDevice,
                       stream);
  float *h = hidden_out;
  auto base = [&](const hpd::GemmShape &s, const __bf16 *xh, const __bf16 *xl, int K) {
    hpd::GemmArgs g{};
    g.K = K;
    g.N = 64 * s.n_slices;
    g.n_slices = s.n_slices;
    g.ksplit = s.ksplit;
    g.k_per_wg = s.k_per_wg;
    g.n_tgroups = s.n_tgroups;
    g.x_hi = xh;
    g.x_lo = xl;
    g.T = L.T;
    g.Tpad = L.Tpad;
    g.part = part;
    return g;
  };
  int pending_ksplit = 0;   // down-projection partials not yet added to h
  for (int l = 0; l < m.num_layers && e == hipSuccess; ++l) {
    const __bf16 *g1 = m.g_attn_norm ? (const __bf16 *)m.g_attn_norm[l] : nullptr;
    const __bf16 *g2 = m.g_mlp_norm ? (const __bf16 *)m.g_mlp_norm[l] : nullptr;
    // 1: previous layer's down projection into h, attention-input norm
    e = hpd::launch_residual_norm(h, pending_ksplit ? part : nullptr, pending_ksplit, L.Tpad, L.H, L.T, g1,
                                  m.rms_eps, x_hi, nullptr, attn, L.nq, stream);
    if (e != hipSuccess) break;
    // 2: QKV projection; the epilogue appends the new K/V rows to the cache
    hpd::GemmArgs g = base(L.qkv, x_hi, nullptr, L.H);
    g.w0 = (const __bf16 *)m.w_qkv[l];
    g.q_out = q;
    g.n_q = L.nq;
    g.k_cache = (__bf16 *)priv_k[l];
    g.v_cache = (__bf16 *)priv_v[l];
    g.n_kv = L.nkv;
    g.dest = dev.token_dest;
    e = hpd::launch_gemm(g, false, hpd::kEpiQKV, hpd::KK_GEMM_QKV, stream);
    if (e != hipSuccess) break;
    // 3: attention over the shared prefix and the private rows
    e = hpd::launch_branch_attention(P, q, shared_k ? shared_k[l] : nullptr, shared_v ? shared_v[l] : nullptr,
                                     priv_k[l], priv_v[l], attn, nullptr, workspace, stream);
    if (e != hipSuccess) break;
    // 4 + 5: O projection, residual add and MLP-input norm
    g = base(L.o, attn, nullptr, L.nq);
    g.w0 = (const __bf16 *)m.w_o[l];
    e = hpd::launch_gemm(g, false, hpd::kEpiResidual, hpd::KK_GEMM_O, stream);
    if (e != hipSuccess) break;
    e = hpd::launch_residual_norm(h, part, L.o.ksplit, L.Tpad, L.H, L.T, g2, m.rms_eps, x_hi, x_lo, nullptr, 0,
                                  stream);
    if (e != hipSuccess) break;
    // 6: gate/up projection, SwiGLU
    g = base(L.gu, x_hi, x_lo, L.H);
    g.w0 = (const __bf16 *)m.w_gate[l];
    g.w1 = (const __bf16 *)m.w_up[l];
    g.m_hi = m_hi;
    g.m_lo = m_lo;
    g.I = L.I;
    e = hpd::launch_gemm(g, true, hpd::kEpiSwiGLU, hpd::KK_GEMM_GATE_UP, stream);
    if (e != hipSuccess) break;
    // 7: down projection (added to h by the next layer's first kernel)
    g = base(L.down, m_hi, m_lo, L.I);
    g.w0 = (const __bf16 *)m.w_down[l];
    e = hpd::launch_gemm(g, true, hpd::kEpiResidual, hpd::KK_GEMM_DOWN, stream);
    pending_ksplit = L.down.ksplit;
  }
  if (e == hipSuccess)
    e = hpd::launch_residual_norm(h, part, pending_ksplit, L.Tpad, L.H, L.T, nullptr, m.rms_eps, nullptr, nullptr,
                                  nullptr, 0, stream);
  if (e != hipSuccess) {
    hpd::set_last_error(std::string("hpd_decode_step: ") + hipGetErrorString(e));
    return HPD_ERR_HIP;
  }
  return HPD_OK;
}

}  // extern "C"
