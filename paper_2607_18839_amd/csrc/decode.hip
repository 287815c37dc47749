// One branch-parallel decode step of the decoder stack (C ABI entry points).
//
// The step runs every new token of every branch through all layers at once
// (Algorithm 1, the parallel draft over the active pool).  The residual
// stream h [T][hidden] stays in fp32 in hidden_out.  RMSNorm is folded into
// the projections (see gemm.h): a norm's input x = h * gamma is written by
// whatever last updated h, with per-token sums of squares, and the next
// projection scales its outputs by the per-token factor.  Per step:
//   0 h = hidden_in; x = h * gamma_attn[0] (bf16), sums of squares
// and per layer:
//   1 QKV GEMM -> q (bf16) and the new K/V rows (bf16), written into the
//     layer's private cache at row priv_row + L + j (optionally followed by
//     the Qwen3-style QK norm and rotary embedding of q and the new k rows)
//   2 branch attention (one launch for the shared-prefix and private work
//     items, then the merge) -> a (bf16)
//   3 O GEMM: h += a W_o^T; x = h * gamma_mlp * s (fp16, s the power of two
//     of the attention norm's factor of the token, undone by the next GEMM),
//     sums of squares
//   4 gate/up GEMM (fp16), SwiGLU -> m (fp16)
//   5 down GEMM (fp16): h += m W_down^T; x = h * gamma_attn[l + 1] (bf16),
//     sums of squares (not after the last layer)
// (section "Overview", paragraph "LLM Decoder": GQA, RMSNorm, SwiGLU).
// Every output element is written by one workgroup, so the result does not
// depend on scheduling.  With HPD_WEIGHTS_PACKED weights the activations x,
// attn and m are kept in the same packed layout as the weights.  Buffers x, q, attn, m and the sums of squares live
// in the workspace after the attention plan's tables; rows T..Tpad-1 of x,
// attn and m are kept zero.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
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
  int rg_qkv, rg_o, rg_gu, rg_down;
  size_t off_x, off_q, off_attn, off_m, off_ss, off_ss_mlp, off_scale, bytes;
};

DecodeLayout decode_layout(const hpd_model_desc &m, const Plan &P) {
  DecodeLayout L;
  L.T = P.T;
  L.Tpad = (P.T + kGemmTile - 1) / kGemmTile * kGemmTile;
  L.H = m.hidden;
  L.I = m.intermediate;
  L.nq = P.attn.num_q_heads * HPD_HEAD_DIM;
  L.nkv = P.attn.num_kv_heads * HPD_HEAD_DIM;
  L.rg_qkv = choose_gemm_rg(L.nq + 2 * L.nkv, L.H, L.Tpad);
  L.rg_o = choose_gemm_rg(L.H, L.nq, L.Tpad);
  L.rg_gu = choose_gemm_rg(2 * L.I, L.H, L.Tpad);
  L.rg_down = choose_gemm_rg(L.H, L.I, L.Tpad);
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
  L.off_ss = take((size_t)L.Tpad * (L.H / kGemmTile) * sizeof(float));
  L.off_ss_mlp = take((size_t)L.Tpad * (L.H / kGemmTile) * sizeof(float));
  L.off_scale = take((size_t)L.Tpad * sizeof(float));
  L.bytes = off;
  return L;
}

// Qwen3-style q / k after the QKV projection (hpd_model_desc q_norm, k_norm,
// rope_theta): per (token, head) an RMSNorm over the head's 64 values with
// its gain, then the rotary position embedding at the token's position in
// its branch's sequence (visible keys - 1).  q is rewritten in place, k in
// the cache row the projection appended.  One wave per (token, head); lane i
// (and i + 32, which computes the same values) owns dims i and i + 32.  The
// angle and its sine and cosine are taken in fp64 (positions reach the
// thousands), the rest in fp32; results are rounded to bf16 once.
__global__ __launch_bounds__(256) void qk_norm_rope_kernel(PlanDev dev, __bf16 *q, __bf16 *k_cache, int T, int Hq,
                                                           int Hkv, const __bf16 *gq, const __bf16 *gk, float eps,
                                                           float theta) {
  // the arguments in one round trip to the argument segment
  asm volatile("" ::"s"(dev.token_dest), "s"(dev.token_vis), "s"(q), "s"(k_cache), "s"(T), "s"(Hq), "s"(Hkv), "s"(gq),
               "s"(gk), "s"(eps), "s"(theta));
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, nh = Hq + Hkv;
  const int64_t item = (int64_t)blockIdx.x * 4 + wave;   // (token, head)
  if (item >= (int64_t)T * nh) return;
  const int t = (int)(item / nh), hh = (int)(item % nh);
  __bf16 *row;
  const __bf16 *g;
  if (hh < Hq) {
    row = q + ((int64_t)t * Hq + hh) * HPD_HEAD_DIM;
    g = gq;
  } else {
    row = k_cache + ((int64_t)dev.token_dest[t] * Hkv + (hh - Hq)) * HPD_HEAD_DIM;
    g = gk;
  }
  const int i = lane & 31;
  float x0 = (float)row[i], x1 = (float)row[i + 32];
  if (g) {
    float ss = fmaf(x0, x0, x1 * x1);
#pragma unroll
    for (int off = 16; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
    const float r = 1.0f / sqrtf(ss * (1.0f / HPD_HEAD_DIM) + eps);
    x0 = x0 * r * (float)g[i];
    x1 = x1 * r * (float)g[i + 32];
  }
  if (theta > 0.f) {
    const double ang = (double)(dev.token_vis[t] - 1) * pow((double)theta, -(double)i / 32.0);
    double s, c;
    sincos(ang, &s, &c);
    const float cf = (float)c, sf = (float)s;
    const float y0 = x0 * cf - x1 * sf, y1 = x1 * cf + x0 * sf;
    x0 = y0;
    x1 = y1;
  }
  if (lane < 32) {
    row[i] = (__bf16)x0;
    row[i + 32] = (__bf16)x1;
  }
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
  if (m->weight_format != HPD_WEIGHTS_TORCH && m->weight_format != HPD_WEIGHTS_PACKED) {
    *err = "unknown weight_format";
    return HPD_ERR_INVALID_ARGUMENT;
  }
  const bool packed = m->weight_format == HPD_WEIGHTS_PACKED;   // w_up unused when packed
  if (!m->w_qkv || !m->w_o || !m->w_gate || (!packed && !m->w_up) || !m->w_down) {
    *err = "NULL weight array";
    return HPD_ERR_INVALID_ARGUMENT;
  }
  if (!(m->rope_theta >= 0.f) || m->rope_theta > 3.0e38f) {
    *err = "rope_theta must be finite and >= 0";
    return HPD_ERR_INVALID_ARGUMENT;
  }
  auto misaligned = [](const void *p) { return ((uintptr_t)p & 15) != 0; };
  for (int l = 0; l < m->num_layers; ++l) {
    if ((m->q_norm && (!m->q_norm[l] || misaligned(m->q_norm[l]))) ||
        (m->k_norm && (!m->k_norm[l] || misaligned(m->k_norm[l])))) {
      *err = "NULL or misaligned q_norm / k_norm gain of layer " + std::to_string(l);
      return HPD_ERR_INVALID_ARGUMENT;
    }
    if (!m->w_qkv[l] || !m->w_o[l] || !m->w_gate[l] || (!packed && !m->w_up[l]) || !m->w_down[l]) {
      *err = "NULL weight of layer " + std::to_string(l);
      return HPD_ERR_INVALID_ARGUMENT;
    }
    if (misaligned(m->w_qkv[l]) || misaligned(m->w_o[l]) || misaligned(m->w_gate[l]) ||
        (!packed && misaligned(m->w_up[l])) || misaligned(m->w_down[l]) ||
        (m->g_attn_norm && misaligned(m->g_attn_norm[l])) || (m->g_mlp_norm && misaligned(m->g_mlp_norm[l]))) {
      *err = "weight or gain of layer " + std::to_string(l) + " not 16-byte aligned";
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
  __bf16 *x = (__bf16 *)(ws + L.off_x);   // x = h * gamma: bf16 (attention input) or fp16 (MLP input)
  __bf16 *q = (__bf16 *)(ws + L.off_q), *attn = (__bf16 *)(ws + L.off_attn);
  __bf16 *mlp = (__bf16 *)(ws + L.off_m);   // SwiGLU product, fp16 bits
  // sums of squares of h per 32 columns: at the attention norm's input and at
  // the MLP norm's input
  float *ss = (float *)(ws + L.off_ss), *ss_mlp = (float *)(ws + L.off_ss_mlp);
  float *scale = (float *)(ws + L.off_scale);   // per token: power of two of the attention norm factor
  const hpd::PlanDev dev = hpd::plan_dev(P, workspace);
  float *h = hidden_out;
  // packed weights: every activation buffer (x, attn, m) is kept in the packed
  // layout too, and the projections stream both operands with whole 1 KB loads
  const bool packed = m.weight_format == HPD_WEIGHTS_PACKED;
  auto gamma = [&](const void *const *arr, int l) { return arr ? (const __bf16 *)arr[l] : nullptr; };
  auto base = [&](int rg, const __bf16 *xin, int N, int K) {
    hpd::GemmArgs g{};
    g.K = K;
    g.N = N;
    g.rg = rg;
    g.n_slices = N / (hpd::kGemmTile * rg);
    g.n_ttiles = L.Tpad / hpd::kGemmTile;
    g.x = xin;
    g.T = L.T;
    g.Tpad = L.Tpad;
    g.ss_in = ss;
    g.n_ss = L.H / hpd::kGemmTile;
    g.inv_H = 1.0f / (float)L.H;
    g.eps = m.rms_eps;
    g.a_packed = packed;
    g.act_packed = packed;
    return g;
  };

  const hpd::TraceRange step_range("hpd_decode_step");
  const bool qwen3 = m.q_norm || m.k_norm || m.rope_theta > 0.f;
  const int Hq = P.attn.num_q_heads, Hkv = P.attn.num_kv_heads;
  hipError_t e = hpd::launch_norm_input(hidden_in, h, L.T, L.Tpad, L.H, gamma(m.g_attn_norm, 0), x, ss, attn,
                                         L.nq, packed, stream);
  for (int l = 0; l < m.num_layers && e == hipSuccess; ++l) {
    char layer_name[32];
    std::snprintf(layer_name, sizeof layer_name, "layer %d", l);
    const hpd::TraceRange layer_range(layer_name);
    hpd::TracePhase phase("qkv");
    // 1: QKV projection; the epilogue appends the new K/V rows to the cache
    hpd::GemmArgs g = base(L.rg_qkv, x, L.nq + 2 * L.nkv, L.H);
    g.w0 = (const __bf16 *)m.w_qkv[l];
    g.q_out = q;
    g.n_q = L.nq;
    g.k_cache = (__bf16 *)priv_k[l];
    g.v_cache = (__bf16 *)priv_v[l];
    g.n_kv = L.nkv;
    g.dest = dev.token_dest;
    g.scale_out = scale;
    e = hpd::launch_gemm(g, false, hpd::kEpiQKV, hpd::KK_GEMM_QKV, stream);
    if (e != hipSuccess) break;
    if (qwen3) {   // 1b: QK norm and rotary embedding of q and the new k rows
      const int64_t items = (int64_t)L.T * (Hq + Hkv);
      hpd::launch(hpd::KK_QK_ROPE, hpd::qk_norm_rope_kernel, dim3((unsigned)((items + 3) / 4)), dim3(256), stream,
                  dev, q, (__bf16 *)priv_k[l], L.T, Hq, Hkv, gamma(m.q_norm, l), gamma(m.k_norm, l), m.rms_eps,
                  m.rope_theta);
      if ((e = hipGetLastError()) != hipSuccess) break;
    }
    // 2: attention over the shared prefix and the private rows
    phase.next("attention");
    e = hpd::launch_branch_attention(P, q, shared_k ? shared_k[l] : nullptr, shared_v ? shared_v[l] : nullptr,
                                     priv_k[l], priv_v[l], attn, nullptr, workspace, stream, packed);
    if (e != hipSuccess) break;
    phase.next("o_proj");
    // 3: O projection into h; MLP norm input (fp16), scaled by the power of
    // two of the attention norm's factor so that it stays in fp16's range
    g = base(L.rg_o, attn, L.H, L.nq);
    g.w0 = (const __bf16 *)m.w_o[l];
    g.h = h;
    g.x_out = x;
    g.x_out_f16 = true;
    g.gamma = gamma(m.g_mlp_norm, l);
    g.ss_out = ss_mlp;
    g.scale_in = scale;
    e = hpd::launch_gemm(g, false, hpd::kEpiResidual, hpd::KK_GEMM_O, stream);
    if (e != hipSuccess) break;
    phase.next("mlp");
    // 4: gate/up projection, SwiGLU (fp16)
    g = base(L.rg_gu, x, 2 * L.I, L.H);
    g.ss_in = ss_mlp;
    g.scale_in = scale;
    g.w0 = (const __bf16 *)m.w_gate[l];   // packed: the interleaved gate/up pair
    g.w1 = packed ? nullptr : (const __bf16 *)m.w_up[l];
    g.m_out = mlp;
    g.I = L.I;
    e = hpd::launch_gemm(g, true, hpd::kEpiSwiGLU, hpd::KK_GEMM_GATE_UP, stream);
    if (e != hipSuccess) break;
    // 5: down projection into h (fp16); next layer's attention norm input
    g = base(L.rg_down, mlp, L.H, L.I);
    g.w0 = (const __bf16 *)m.w_down[l];
    g.h = h;
    if (l + 1 < m.num_layers) {
      g.x_out = x;
      g.x_out_f16 = false;
      g.gamma = gamma(m.g_attn_norm, l + 1);
      g.ss_out = ss;
    }
    e = hpd::launch_gemm(g, true, hpd::kEpiResidual, hpd::KK_GEMM_DOWN, stream);
  }
  if (e != hipSuccess) {
    hpd::set_last_error(std::string("hpd_decode_step: ") + hipGetErrorString(e));
    return HPD_ERR_HIP;
  }
  return HPD_OK;
}

}  // extern "C"
