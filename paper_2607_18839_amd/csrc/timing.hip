// Optional per-kernel timing with HIP events, for benchmarks.
//
// When enabled, every launch gets a pair of events bound to its dispatch
// (hipExtLaunchKernel: the kernel's own start and end).  Events come from a
// pool created when timing is switched on, so the timed region creates
// nothing.
#include <hip/hip_runtime.h>

#include <dlfcn.h>

#include <atomic>
#include <cstdlib>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"

namespace hpd {

void set_last_error(const std::string &msg);

namespace {

struct Pair {
  hipEvent_t start, stop;
  int kind;
};

std::mutex g_mu;
bool g_enabled = false;
std::atomic<bool> g_phase_isolation{false};
std::vector<Pair> g_pool;
size_t g_used = 0;
double g_total_ms[HPD_NUM_KERNEL_KINDS] = {};
int64_t g_count[HPD_NUM_KERNEL_KINDS] = {};
int64_t g_dropped = 0;

const char *kKindNames[HPD_NUM_KERNEL_KINDS] = {
    "shared_prefix", "private", "merge", "gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down",
    "norm_input", "lm_head", "verify", "draft_mlp", "draft_token", "embed", "qk_norm_rope"};

}  // namespace

TimedEvents timed_events(int kind) {
  TimedEvents ev;
  if (!g_enabled) return ev;
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_used >= g_pool.size()) {
    ++g_dropped;
    return ev;
  }
  Pair &p = g_pool[g_used++];
  p.kind = kind;
  ev.start = p.start;
  ev.stop = p.stop;
  return ev;
}

bool attn_phase_isolation() { return g_phase_isolation.load(std::memory_order_relaxed); }

// roctx ranges around the phases of a step (HPD_ROCTX=1 in the environment):
// the rocprofiler-sdk roctx library is opened on first use; without it, or
// with the variable unset, ranges cost one branch.  The ranges mark the host
// enqueueing the phases, so they bracket kernels when the step runs eagerly;
// a captured graph replays the kernels without them.
namespace {
struct Roctx {
  int (*push)(const char *) = nullptr;
  int (*pop)() = nullptr;
};
const Roctx &roctx() {
  static const Roctx r = [] {
    Roctx x;
    const char *env = std::getenv("HPD_ROCTX");
    if (!env || std::string(env) != "1") return x;
    void *h = dlopen("librocprofiler-sdk-roctx.so.1", RTLD_NOW | RTLD_LOCAL);
    if (!h) h = dlopen("librocprofiler-sdk-roctx.so", RTLD_NOW | RTLD_LOCAL);
    if (!h) return x;
    x.push = (int (*)(const char *))dlsym(h, "roctxRangePushA");
    x.pop = (int (*)())dlsym(h, "roctxRangePop");
    if (!x.push || !x.pop) x.push = nullptr, x.pop = nullptr;
    return x;
  }();
  return r;
}
}  // namespace

TraceRange::TraceRange(const char *name) : on_(roctx().push != nullptr) {
  if (on_) roctx().push(name);
}
TraceRange::~TraceRange() {
  if (on_) roctx().pop();
}
TracePhase::TracePhase(const char *name) : on_(roctx().push != nullptr) {
  if (on_) roctx().push(name);
}
void TracePhase::next(const char *name) {
  if (!on_) return;
  roctx().pop();
  roctx().push(name);
}
TracePhase::~TracePhase() {
  if (on_) roctx().pop();
}

}  // namespace hpd

extern "C" {

hpd_status hpd_attn_phase_isolation(int enable) {
  hpd::g_phase_isolation.store(enable != 0, std::memory_order_relaxed);
  return HPD_OK;
}

hpd_status hpd_kernel_timing(int enable, int max_launches) {
  std::lock_guard<std::mutex> lk(hpd::g_mu);
  if (enable) {
    if (max_launches < 1) {
      hpd::set_last_error("hpd_kernel_timing: max_launches must be >= 1");
      return HPD_ERR_INVALID_ARGUMENT;
    }
    for (auto &p : hpd::g_pool) {   // events of a previous enable (a failed one may have left NULLs)
      if (p.start) (void)hipEventDestroy(p.start);
      if (p.stop) (void)hipEventDestroy(p.stop);
    }
    hpd::g_pool.assign(max_launches, hpd::Pair{});
    for (auto &p : hpd::g_pool) {
      if (hipEventCreate(&p.start) != hipSuccess || hipEventCreate(&p.stop) != hipSuccess) {
        hpd::g_enabled = false;
        hpd::set_last_error("hpd_kernel_timing: hipEventCreate failed");
        return HPD_ERR_HIP;
      }
    }
    hpd::g_used = 0;
    hpd::g_enabled = true;
  } else {
    hpd::g_enabled = false;
  }
  return HPD_OK;
}

hpd_status hpd_kernel_times_read(hpd_kernel_times *out, int keep_pairs) {
  if (!out) return HPD_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lk(hpd::g_mu);
  for (size_t i = 0; i < hpd::g_used; ++i) {
    hpd::Pair &p = hpd::g_pool[i];
    if (hipEventSynchronize(p.stop) != hipSuccess) return HPD_ERR_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p.start, p.stop) != hipSuccess) return HPD_ERR_HIP;
    hpd::g_total_ms[p.kind] += ms;
    hpd::g_count[p.kind] += 1;
  }
  if (!keep_pairs) hpd::g_used = 0;
  for (int k = 0; k < HPD_NUM_KERNEL_KINDS; ++k) {
    out->total_ms[k] = hpd::g_total_ms[k];
    out->count[k] = hpd::g_count[k];
    hpd::g_total_ms[k] = 0.0;
    hpd::g_count[k] = 0;
  }
  out->dropped = hpd::g_dropped;
  hpd::g_dropped = 0;
  return HPD_OK;
}

const char *hpd_kernel_kind_name(int kind) {
  return (kind >= 0 && kind < HPD_NUM_KERNEL_KINDS) ? hpd::kKindNames[kind] : "unknown";
}

}  // extern "C"
