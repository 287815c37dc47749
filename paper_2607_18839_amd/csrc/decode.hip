// One branch-parallel decode step of the decoder stack (C ABI entry points).
//
// The step runs every new token of every branch through all layers at once
// (Algorithm 1, the parallel draft over the active pool).  Per layer, with
// the residual stream h [T][hidden] kept in fp32 in hidden_out:
//   1 [h += previous down projection] RMSNorm(h) -> x (bf16)
//   2 QKV GEMM -> q (bf16) and the new K/V rows (bf16), written into the
//     layer's private cache at row priv_row + L + j
//   3 branch attention (shared-prefix, private, merge kernels) -> a (bf16)
//   4 O GEMM (split-K partials)
//   5 h += a W_o^T, RMSNorm(h) -> x (fp16) (one kernel)
//   6 gate/up GEMM (fp16), SwiGLU -> m (fp16)
//   7 down GEMM (fp16, partials), added to h by the next layer's step 1 (or
//     by a final residual kernel after the last layer)
// (section "Overview", paragraph "LLM Decoder": GQA, RMSNorm, SwiGLU).
// Split-K partials are summed by the consuming kernel in split order, so the
// result does not depend on scheduling and needs no cross-workgroup sync.
// Buffers: x, q, attn, m and the partials live in the workspace after the
// attention plan's tables; rows T..Tpad-1 of x, attn and m are kept zero.
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

struct DecodeLayout {
  int T, Tpad, H, I, nq, nkv;
  GemmShape qkv, o, gu, down;
  size_t off_x, off_q, off_attn, off_m, off_part, bytes;
};

DecodeLayout decode_layout(const hpd_model_desc &m, const Plan &P) {
  DecodeLayout L;
  L.T = P.T;
  L.Tpad = (P.T + kGemmTile - 1) / kGemmTile * kGemmTile;
  L.H = m.hidden;
  L.I = m.intermediate;
  L.nq = P.attn.num_q_heads * HPD_HEAD_DIM;
  L.nkv = P.attn.num_kv_heads * HPD_HEAD_DIM;
  L.qkv = choose_gemm_shape(L.nq + 2 * L.nkv, L.H, L.Tpad, kEpiQKV);
  L.o = choose_gemm_shape(L.H, L.nq, L.Tpad, kEpiResidual);
  L.gu = choose_gemm_shape(2 * L.I, L.H, L.Tpad, kEpiSwiGLU);
  L.down = choose_gemm_shape(L.H, L.I, L.Tpad, kEpiResidual);
  size_t off = align256(P.workspace_bytes);
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  L.off_x = take((size_t)L.Tpad * L.H * 2);
  L.off_q = take((size_t)L.T * L.nq * 2);
  L.off_attn = take((size_t)L.Tpad * L.nq * 2);
  L.off_m = take((size_t)L.Tpad * L.I * 2);
  // partials of the residual projections (O, down); N = hidden for both
  const size_t part = (size_t)std::max(L.o.ksplit, L.down.ksplit) * L.Tpad * L.H * sizeof(float);
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
  __bf16 *x = (__bf16 *)(ws + L.off_x);   // bf16 (attention input) or fp16 (MLP input)
  __bf16 *q = (__bf16 *)(ws + L.off_q), *attn = (__bf16 *)(ws + L.off_attn);
  __bf16 *mlp = (__bf16 *)(ws + L.off_m);   // SwiGLU product, fp16 bits
  float *part = (float *)(ws + L.off_part);
  const hpd::PlanDev dev = hpd::plan_dev(P, workspace);

  hipError_t e = hipSuccess;
  if (hidden_out != hidden_in)
    e = hipMemcpyAsync(hidden_out, hidden_in, (size_t)L.T * L.H * sizeof(float), hipMemcpyDeviceToDevice,
                       stream);
  float *h = hidden_out;
  auto base = [&](const hpd::GemmShape &s, const __bf16 *xh, int N, int K) {
    hpd::GemmArgs g{};
    g.K = K;
    g.N = N;
    g.rg = s.rg;
    g.n_slices = N / (hpd::kGemmTile * s.rg);
    g.ksplit = s.ksplit;
    g.k_per_wg = K / s.ksplit;
    g.n_ttiles = L.Tpad / hpd::kGemmTile;
    g.x = xh;
    g.T = L.T;
    g.Tpad = L.Tpad;
    g.part = part;
    return g;
  };
  int pending_ksplit = 0;   // down-projection partials not yet added to h
  for (int l = 0; l < m.num_layers && e == hipSuccess; ++l) {
    const __bf16 *g1 = m.g_attn_norm ? (const __bf16 *)m.g_attn_norm[l] : nullptr;
    const __bf16 *g2 = m.g_mlp_norm ? (const __bf16 *)m.g_mlp_norm[l] : nullptr;
    // 1: previous layer's down projection into h, attention-input norm (bf16)
    e = hpd::launch_residual_norm(h, pending_ksplit ? part : nullptr, pending_ksplit, L.Tpad, L.H, L.T, g1,
                                  m.rms_eps, x, false, attn, L.nq, stream);
    if (e != hipSuccess) break;
    // 2: QKV projection; the epilogue appends the new K/V rows to the cache
    hpd::GemmArgs g = base(L.qkv, x, L.nq + 2 * L.nkv, L.H);
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
    // 4 + 5: O projection, residual add and MLP-input norm (fp16)
    g = base(L.o, attn, L.H, L.nq);
    g.w0 = (const __bf16 *)m.w_o[l];
    e = hpd::launch_gemm(g, false, hpd::kEpiResidual, hpd::KK_GEMM_O, stream);
    if (e != hipSuccess) break;
    e = hpd::launch_residual_norm(h, part, L.o.ksplit, L.Tpad, L.H, L.T, g2, m.rms_eps, x, true, nullptr, 0,
                                  stream);
    if (e != hipSuccess) break;
    // 6: gate/up projection, SwiGLU (fp16)
    g = base(L.gu, x, 2 * L.I, L.H);
    g.w0 = (const __bf16 *)m.w_gate[l];
    g.w1 = (const __bf16 *)m.w_up[l];
    g.m_out = mlp;
    g.I = L.I;
    e = hpd::launch_gemm(g, true, hpd::kEpiSwiGLU, hpd::KK_GEMM_GATE_UP, stream);
    if (e != hipSuccess) break;
    // 7: down projection (fp16; added to h by the next layer's first kernel)
    g = base(L.down, mlp, L.H, L.I);
    g.w0 = (const __bf16 *)m.w_down[l];
    e = hpd::launch_gemm(g, true, hpd::kEpiResidual, hpd::KK_GEMM_DOWN, stream);
    pending_ksplit = L.down.ksplit;
  }
  if (e == hipSuccess)
    e = hpd::launch_residual_norm(h, part, pending_ksplit, L.Tpad, L.H, L.T, nullptr, m.rms_eps, nullptr, false,
                                  nullptr, 0, stream);
  if (e != hipSuccess) {
    hpd::set_last_error(std::string("hpd_decode_step: ") + hipGetErrorString(e));
    return HPD_ERR_HIP;
  }
  return HPD_OK;
}

}  // extern "C"
