// C ABI entry points (declared in include/hpd.h).  Validation happens here,
// before any launch; nothing below throws across the boundary.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <string>

#include "gemm.h"
#include "hpd.h"
#include "kernels.h"
#include "plan.h"

namespace {

thread_local std::string g_last_error;

hpd_status set_err(hpd_status st, const std::string &msg) {
  g_last_error = msg;
  return st;
}

hpd_status hip_err(hipError_t e, const char *where) {
  return set_err(HPD_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
}

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

}  // namespace

// Scratch memory of hpd_branch_attn_step_noalloc: plan tables, then the
// partial softmax results.  Each GPU holds its own copy until the process
// ends.  In host code this name is only a stand-in for the symbol: the
// device address comes from hipGetSymbolAddress, once per device.
__device__ __align__(256) unsigned char scratch[HPD_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch` (looked up on the first call on
// that device, with that device current).
hpd_status scratch_address(const char *fn, void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_err(e, fn);
  if (dev < 0 || dev >= kMaxDevices)
    return set_err(HPD_ERR_UNSUPPORTED, std::string(fn) + ": device id out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_err(e, "hipGetSymbolAddress(scratch)");
    if (!p || !aligned(p, 256))
      return set_err(HPD_ERR_HIP, std::string(fn) + ": scratch symbol has no usable device address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return HPD_OK;
}

// Checks shared by both attention entry points; nothing is launched before
// they pass.
hpd_status check_attn_tensors(const char *fn, const hpd_plan *plan, const void *q, const void *shared_k,
                              const void *shared_v, const void *priv_k, const void *priv_v, const void *out,
                              const float *lse) {
  const std::string f(fn);
  if (!plan) return set_err(HPD_ERR_INVALID_ARGUMENT, f + ": plan is NULL");
  if (!q || !priv_k || !priv_v || !out) return set_err(HPD_ERR_INVALID_ARGUMENT, f + ": NULL tensor");
  if (plan->p.shared_rows > 0 && (!shared_k || !shared_v))
    return set_err(HPD_ERR_INVALID_ARGUMENT, f + ": shared_k/v NULL with a non-empty prefix");
  if (!aligned(q, 16) || !aligned(priv_k, 16) || !aligned(priv_v, 16) || !aligned(out, 16) ||
      (shared_k && !aligned(shared_k, 16)) || (shared_v && !aligned(shared_v, 16)) || (lse && !aligned(lse, 4)))
    return set_err(HPD_ERR_INVALID_ARGUMENT, f + ": tensors must be 16-byte aligned");
  return HPD_OK;
}

}  // namespace

namespace hpd {
void set_last_error(const std::string &msg) { g_last_error = msg; }
}  // namespace hpd

extern "C" {

const char *hpd_status_string(hpd_status s) {
  switch (s) {
    case HPD_OK: return "HPD_OK";
    case HPD_ERR_INVALID_ARGUMENT: return "HPD_ERR_INVALID_ARGUMENT";
    case HPD_ERR_UNSUPPORTED: return "HPD_ERR_UNSUPPORTED";
    case HPD_ERR_WORKSPACE_TOO_SMALL: return "HPD_ERR_WORKSPACE_TOO_SMALL";
    case HPD_ERR_HIP: return "HPD_ERR_HIP";
    case HPD_ERR_HOST_ALLOC: return "HPD_ERR_HOST_ALLOC";
    case HPD_ERR_OUT_OF_BLOCKS: return "HPD_ERR_OUT_OF_BLOCKS";
  }
  return "HPD_ERR_UNKNOWN";
}

const char *hpd_last_error_message(void) { return g_last_error.c_str(); }

hpd_status hpd_plan_create(const hpd_attn_desc *attn, const hpd_batch_desc *batch, hpd_plan **out) {
  if (!out) return set_err(HPD_ERR_INVALID_ARGUMENT, "hpd_plan_create: out is NULL");
  *out = nullptr;
  hpd_plan *p = new (std::nothrow) hpd_plan;
  if (!p) return set_err(HPD_ERR_HOST_ALLOC, "hpd_plan_create: out of host memory");
  std::string err;
  hpd_status st;
  try {
    st = hpd::build_plan(attn, batch, &p->p, &err);
  } catch (const std::bad_alloc &) {
    delete p;
    return set_err(HPD_ERR_HOST_ALLOC, "hpd_plan_create: out of host memory");
  }
  if (st != HPD_OK) {
    delete p;
    return set_err(st, "hpd_plan_create: " + err);
  }
  *out = p;
  return HPD_OK;
}

void hpd_plan_destroy(hpd_plan *plan) { delete plan; }

size_t hpd_plan_workspace_bytes(const hpd_plan *plan) { return plan ? plan->p.workspace_bytes : 0; }

hpd_status hpd_plan_query(const hpd_plan *plan, hpd_plan_info *o) {
  if (!plan || !o) return set_err(HPD_ERR_INVALID_ARGUMENT, "hpd_plan_query: NULL argument");
  const hpd::Plan &P = plan->p;
  o->num_tokens = P.T;
  o->num_pages = P.num_pages;
  o->num_branches = P.num_branches;
  o->q_row = P.q_row.data();
  o->priv_row = P.priv_row.data();
  o->prefix_row = P.prefix_row.data();
  o->page_q_row = P.page_q_row.data();
  o->page_T = P.page_T.data();
  o->visible = P.visible.data();
  o->shared_rows = P.shared_rows;
  o->priv_rows = P.priv_rows;
  o->num_shared_items = P.num_shared_items();
  o->num_private_items = P.num_private_items();
  o->shared_items = P.shared_items.data();
  o->private_items = P.private_items.data();
  o->token_slots = P.token_slots.data();
  o->num_partial_slots = P.num_slots;
  o->pos_token = P.pos_token.data();
  return HPD_OK;
}

hpd_status hpd_plan_upload(const hpd_plan *plan, void *workspace, size_t bytes, void *stream) {
  if (!plan || !workspace) return set_err(HPD_ERR_INVALID_ARGUMENT, "hpd_plan_upload: NULL argument");
  if (!aligned(workspace, 256))
    return set_err(HPD_ERR_INVALID_ARGUMENT, "hpd_plan_upload: workspace must be 256-byte aligned");
  if (bytes < plan->p.workspace_bytes)
    return set_err(HPD_ERR_WORKSPACE_TOO_SMALL, "hpd_plan_upload: workspace too small");
  if (plan->p.table_bytes == 0) return HPD_OK;
  hipError_t e = hipMemcpyAsync(workspace, plan->p.table_image.data(), plan->p.table_bytes,
                                hipMemcpyHostToDevice, (hipStream_t)stream);
  if (e != hipSuccess) return hip_err(e, "hpd_plan_upload");
  return HPD_OK;
}

hpd_status hpd_branch_attn_step(const hpd_plan *plan, const void *q, const void *shared_k,
                                const void *shared_v, const void *priv_k, const void *priv_v,
                                void *out, float *lse, void *workspace, size_t workspace_bytes,
                                void *stream) {
  hpd_status st = check_attn_tensors("hpd_branch_attn_step", plan, q, shared_k, shared_v, priv_k, priv_v, out, lse);
  if (st != HPD_OK) return st;
  const hpd::Plan &P = plan->p;
  if (!workspace) return set_err(HPD_ERR_INVALID_ARGUMENT, "hpd_branch_attn_step: NULL workspace");
  if (!aligned(workspace, 256))
    return set_err(HPD_ERR_INVALID_ARGUMENT, "hpd_branch_attn_step: workspace must be 256-byte aligned");
  if (workspace_bytes < P.workspace_bytes)
    return set_err(HPD_ERR_WORKSPACE_TOO_SMALL, "hpd_branch_attn_step: workspace too small");
  const hpd::TraceRange range("hpd_branch_attn_step");
  hipError_t e = hpd::launch_branch_attention(P, q, shared_k, shared_v, priv_k, priv_v, out, lse,
                                              workspace, (hipStream_t)stream);
  if (e != hipSuccess) return hip_err(e, "hpd_branch_attn_step");
  return HPD_OK;
}

hpd_status hpd_branch_attn_step_noalloc(const hpd_plan *plan, const void *q, const void *shared_k,
                                        const void *shared_v, const void *priv_k, const void *priv_v,
                                        void *out, float *lse, void *stream) {
  static const char *fn = "hpd_branch_attn_step_noalloc";
  hpd_status st = check_attn_tensors(fn, plan, q, shared_k, shared_v, priv_k, priv_v, out, lse);
  if (st != HPD_OK) return st;
  const hpd::Plan &P = plan->p;
  if (P.workspace_bytes > (size_t)HPD_NOALLOC_SCRATCH_BYTES)
    return set_err(HPD_ERR_WORKSPACE_TOO_SMALL,
                   std::string(fn) + ": the plan needs " + std::to_string(P.workspace_bytes) +
                       " bytes of scratch, more than the library's static " +
                       std::to_string((size_t)HPD_NOALLOC_SCRATCH_BYTES) + " (use hpd_branch_attn_step)");
  void *ws = nullptr;
  st = scratch_address(fn, &ws);
  if (st != HPD_OK) return st;
  // The plan's tables go into this device's scratch first (stream-ordered
  // before the kernels that read them); the partials behind them are written
  // by the kernels before they are read, so nothing needs clearing.
  hipError_t e = hipSuccess;
  if (P.table_bytes > 0)
    e = hipMemcpyAsync(ws, P.table_image.data(), P.table_bytes, hipMemcpyHostToDevice, (hipStream_t)stream);
  if (e == hipSuccess)
    e = hpd::launch_branch_attention(P, q, shared_k, shared_v, priv_k, priv_v, out, lse, ws, (hipStream_t)stream);
  if (e != hipSuccess) return hip_err(e, fn);
  return HPD_OK;
}

size_t hpd_packed_weight_bytes(int32_t rows, int32_t cols) {
  if (rows <= 0 || cols <= 0) return 0;
  return (size_t)rows * (size_t)cols * 2;
}

static hpd_status pack_weight(const char *name, const void *w, int32_t rows, int32_t cols, bool to_f16, void *out,
                              void *stream) {
  const std::string fn(name);
  if (!w || !out) return set_err(HPD_ERR_INVALID_ARGUMENT, fn + ": NULL pointer");
  if (rows <= 0 || cols <= 0 || rows % 32 != 0 || cols % 64 != 0)
    return set_err(HPD_ERR_INVALID_ARGUMENT, fn + ": rows must be a positive multiple of 32, cols of 64");
  if (!aligned(w, 16) || !aligned(out, 16))
    return set_err(HPD_ERR_INVALID_ARGUMENT, fn + ": pointers must be 16-byte aligned");
  hipError_t e = hpd::launch_pack_weight((const __bf16 *)w, nullptr, rows, cols, false, to_f16, (__bf16 *)out,
                                         (hipStream_t)stream);
  if (e != hipSuccess) return hip_err(e, name);
  return HPD_OK;
}

hpd_status hpd_pack_weight(const void *w, int32_t rows, int32_t cols, void *out, void *stream) {
  return pack_weight("hpd_pack_weight", w, rows, cols, false, out, stream);
}

hpd_status hpd_pack_weight_f16(const void *w, int32_t rows, int32_t cols, void *out, void *stream) {
  return pack_weight("hpd_pack_weight_f16", w, rows, cols, true, out, stream);
}

hpd_status hpd_pack_gate_up(const void *w_gate, const void *w_up, int32_t intermediate, int32_t hidden, void *out,
                            void *stream) {
  if (!w_gate || !w_up || !out) return set_err(HPD_ERR_INVALID_ARGUMENT, "hpd_pack_gate_up: NULL pointer");
  if (intermediate <= 0 || hidden <= 0 || intermediate % 16 != 0 || hidden % 64 != 0)
    return set_err(HPD_ERR_INVALID_ARGUMENT,
                   "hpd_pack_gate_up: intermediate must be a positive multiple of 16, hidden of 64");
  if (!aligned(w_gate, 16) || !aligned(w_up, 16) || !aligned(out, 16))
    return set_err(HPD_ERR_INVALID_ARGUMENT, "hpd_pack_gate_up: pointers must be 16-byte aligned");
  hipError_t e = hpd::launch_pack_weight((const __bf16 *)w_gate, (const __bf16 *)w_up, 2 * intermediate, hidden,
                                         true, true, (__bf16 *)out, (hipStream_t)stream);
  if (e != hipSuccess) return hip_err(e, "hpd_pack_gate_up");
  return HPD_OK;
}

}  // extern "C"
