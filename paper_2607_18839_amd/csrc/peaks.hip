// Microbenchmarks of the GPU this runs on, for the roofline denominators and
// for calibrating hardware byte counters: streaming read and copy bandwidth,
// dense bf16 MFMA rate, v_exp_f32 rate and dependent-load latency.
//
//   peaks [copy_mib]      prints one JSON object
//   peaks copy N          N MiB copies only (the reference for scaling
//                         memory-traffic counters)
//   peaks read K1 K2 ...  streaming-read rate of a single launch that reads
//                         K KiB, from buffers rotated over 512 MiB (beyond the
//                         Infinity Cache), each launch timed by its own
//                         dispatch events: the rate a kernel of that size can
//                         reach at all
//   peaks mfma M1 M2 ...  the same for bf16 MFMA work: one launch of one
//                         256-thread workgroup per CU doing about M MFLOP of
//                         v_mfma_f32_32x32x16_bf16 (4 independent chains per
//                         wave), timed by its dispatch events
//
// Every kernel has a fixed trip count and touches only its own buffers.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#define CHECK(x)                                                                      \
  do {                                                                                \
    hipError_t e_ = (x);                                                              \
    if (e_ != hipSuccess) {                                                           \
      std::fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));             \
      std::exit(1);                                                                   \
    }                                                                                 \
  } while (0)

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// n4 float4 elements, grid-stride
__global__ __launch_bounds__(256) void copy_kernel(const f32x4 *src, f32x4 *dst, size_t n4) {
  for (size_t i = blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) dst[i] = src[i];
}

__global__ __launch_bounds__(256) void read_kernel(const f32x4 *src, size_t n4, float *sink) {
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (size_t i = blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) acc += src[i];
  if (acc[0] + acc[1] + acc[2] + acc[3] == 123.456f) sink[0] = 1.f;   // keeps the loads alive
}

// 8 independent accumulators per wave, `iters` rounds of 8 MFMAs each.
__global__ __launch_bounds__(256) void mfma_kernel(int iters, float *sink) {
  bf16x8 a, b;
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(0.001f * (threadIdx.x + e));
    b[e] = (__bf16)(0.002f * e);
  }
  f32x4 c[8];
  for (int j = 0; j < 8; ++j) c[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) c[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c[j], 0, 0, 0);
  }
  float s = 0.f;
  for (int j = 0; j < 8; ++j) s += c[j][0] + c[j][1] + c[j][2] + c[j][3];
  if (s == 123.456f) sink[0] = s;
}

// 4 independent 32x32 accumulators per wave, `iters` rounds of 4 MFMAs.
typedef float f32x16 __attribute__((ext_vector_type(16)));
__global__ __launch_bounds__(256) void mfma32_kernel(int iters, float *sink) {
  bf16x8 a, b;
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(0.001f * (threadIdx.x + e));
    b[e] = (__bf16)(0.002f * e);
  }
  f32x16 c[4];
  for (int j = 0; j < 4; ++j)
    for (int r = 0; r < 16; ++r) c[j][r] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 4; ++j) c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[j], 0, 0, 0);
  }
  float s = 0.f;
  for (int j = 0; j < 4; ++j)
    for (int r = 0; r < 16; ++r) s += c[j][r];
  if (s == 123.456f) sink[0] = s;
}

// 8 independent exp2 chains per lane
__global__ __launch_bounds__(256) void exp_kernel(int iters, float *sink) {
  float x[8];
  for (int j = 0; j < 8; ++j) x[j] = -0.001f * (threadIdx.x + j);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = __builtin_amdgcn_exp2f(x[j]) - 1.0f;
  }
  float s = 0.f;
  for (int j = 0; j < 8; ++j) s += x[j];
  if (s == 123.456f) sink[0] = s;
}

// one lane follows a pointer chain of `steps` hops through a permutation
__global__ void chase_kernel(const unsigned *next, int steps, unsigned *out) {
  unsigned p = 0;
  for (int i = 0; i < steps; ++i) p = next[p];
  out[0] = p;
}

// Each workgroup writes its 4 KB tile; with `fence`, it then publishes it with
// an agent-scope release + arrival counter and the last arriving workgroup
// reads a tile back after an acquire -- the synchronisation cost of an
// in-kernel cross-workgroup reduction.  The counter is reset by the last
// arrival.
__global__ __launch_bounds__(256) void arrive_kernel(float *tiles, int *counter, float *sink, int fence) {
  float *my = tiles + (size_t)blockIdx.x * 1024;
  for (int i = threadIdx.x; i < 1024; i += 256) my[i] = (float)(blockIdx.x + i);
  if (!fence) return;
  __threadfence();
  __shared__ int last;
  if (threadIdx.x == 0) {
    const int old = __hip_atomic_fetch_add(counter, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    last = old == (int)gridDim.x - 1;
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  float s = 0.f;
  for (int i = threadIdx.x; i < 1024; i += 256) s += tiles[i];   // one tile back
  if (s == 123.456f) sink[0] = s;
  if (threadIdx.x == 0) __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ void empty_kernel(float *sink) {
  if (threadIdx.x == 1023) sink[0] = 0.f;
}

template <typename F> float time_ms(F launch, int reps) {
  hipEvent_t a, b;
  CHECK(hipEventCreate(&a));
  CHECK(hipEventCreate(&b));
  launch();
  CHECK(hipDeviceSynchronize());
  CHECK(hipEventRecord(a));
  for (int i = 0; i < reps; ++i) launch();
  CHECK(hipEventRecord(b));
  CHECK(hipEventSynchronize(b));
  float ms = 0.f;
  CHECK(hipEventElapsedTime(&ms, a, b));
  return ms / reps;
}

int main(int argc, char **argv) {
  // "peaks copy N": only N MiB copies (3 launches), the reference for
  // scaling memory-traffic counters; otherwise "peaks [N]" runs everything.
  if (argc > 1 && std::string(argv[1]) == "read") {
    const size_t pool = (size_t)512 << 20;
    f32x4 *buf;
    float *sk;
    CHECK(hipMalloc(&buf, pool));
    CHECK(hipMalloc(&sk, 64));
    CHECK(hipMemset(buf, 0, pool));
    hipDeviceProp_t pr;
    CHECK(hipGetDeviceProperties(&pr, 0));
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    std::string kib_s, gbs_s, us_s;
    for (int i = 2; i < argc; ++i) {
      const size_t kib = std::strtoul(argv[i], nullptr, 10), bytes = kib << 10, n4 = bytes / 16;
      if (bytes == 0 || bytes > pool / 2) continue;
      const size_t nbuf = pool / bytes;   // the launches rotate over every slice of the pool
      const int reps = 64;
      double total_ms = 0.0;
      for (int r = -8; r < reps; ++r) {   // 8 untimed launches first
        const f32x4 *src = buf + (size_t)((r + 8) % nbuf) * (bytes / 16);
        hipExtLaunchKernelGGL(read_kernel, dim3(pr.multiProcessorCount * 8), dim3(256), 0, 0, e0, e1, 0, src, n4, sk);
        CHECK(hipGetLastError());
        CHECK(hipEventSynchronize(e1));
        float ms = 0.f;
        CHECK(hipEventElapsedTime(&ms, e0, e1));
        if (r >= 0) total_ms += ms;
      }
      const double us = total_ms * 1e3 / reps;
      char b[64];
      std::snprintf(b, sizeof b, "%s%zu", kib_s.empty() ? "" : ", ", kib); kib_s += b;
      std::snprintf(b, sizeof b, "%s%.1f", gbs_s.empty() ? "" : ", ", bytes / (us * 1e3)); gbs_s += b;
      std::snprintf(b, sizeof b, "%s%.2f", us_s.empty() ? "" : ", ", us); us_s += b;
    }
    std::printf("{\"read_kib\": [%s], \"read_gbs\": [%s], \"read_us\": [%s]}\n", kib_s.c_str(), gbs_s.c_str(),
                us_s.c_str());
    return 0;
  }
  if (argc > 1 && std::string(argv[1]) == "mfma") {
    float *sk;
    CHECK(hipMalloc(&sk, 64));
    hipDeviceProp_t pr;
    CHECK(hipGetDeviceProperties(&pr, 0));
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    const int cus = pr.multiProcessorCount;
    const double per_iter = (double)cus * 4 /*waves*/ * 4 /*MFMAs*/ * (32.0 * 32 * 16 * 2);
    std::string m_s, t_s, us_s;
    for (int i = 2; i < argc; ++i) {
      const double mflop = std::strtod(argv[i], nullptr);
      const int iters = (int)(mflop * 1e6 / per_iter + 0.5);
      if (iters < 1 || iters > (1 << 20)) continue;
      const int reps = 64;
      double total_ms = 0.0;
      for (int r = -8; r < reps; ++r) {
        hipExtLaunchKernelGGL(mfma32_kernel, dim3(cus), dim3(256), 0, 0, e0, e1, 0, iters, sk);
        CHECK(hipGetLastError());
        CHECK(hipEventSynchronize(e1));
        float ms = 0.f;
        CHECK(hipEventElapsedTime(&ms, e0, e1));
        if (r >= 0) total_ms += ms;
      }
      const double us = total_ms * 1e3 / reps, flop = iters * per_iter;
      char b[64];
      std::snprintf(b, sizeof b, "%s%.0f", m_s.empty() ? "" : ", ", flop / 1e6); m_s += b;
      std::snprintf(b, sizeof b, "%s%.1f", t_s.empty() ? "" : ", ", flop / (us * 1e6)); t_s += b;
      std::snprintf(b, sizeof b, "%s%.2f", us_s.empty() ? "" : ", ", us); us_s += b;
    }
    std::printf("{\"mfma_mflop\": [%s], \"mfma_tflops\": [%s], \"mfma_us\": [%s]}\n", m_s.c_str(), t_s.c_str(),
                us_s.c_str());
    return 0;
  }
  const bool copy_only = argc > 1 && std::string(argv[1]) == "copy";
  const int size_arg = copy_only ? 2 : 1;
  const size_t mib = argc > size_arg ? std::strtoul(argv[size_arg], nullptr, 10) : 1024;
  const size_t bytes = mib << 20, n4 = bytes / 16;
  hipDeviceProp_t prop;
  CHECK(hipGetDeviceProperties(&prop, 0));
  f32x4 *src, *dst;
  float *sink;
  CHECK(hipMalloc(&src, bytes));
  CHECK(hipMalloc(&dst, bytes));
  CHECK(hipMalloc(&sink, 64));
  CHECK(hipMemset(src, 0, bytes));
  const int cus = prop.multiProcessorCount;
  const int grid = cus * 8;
  if (copy_only) {
    for (int i = 0; i < 3; ++i) hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(256), 0, 0, src, dst, n4);
    CHECK(hipDeviceSynchronize());
    std::printf("{\"copy_mib\": %zu, \"launches\": 3}\n", mib);
    return 0;
  }

  const float copy_ms = time_ms([&] { hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(256), 0, 0, src, dst, n4); }, 10);
  const float read_ms = time_ms([&] { hipLaunchKernelGGL(read_kernel, dim3(grid), dim3(256), 0, 0, src, n4, sink); }, 10);
  const int miters = 4096;
  const float mfma_ms = time_ms([&] { hipLaunchKernelGGL(mfma_kernel, dim3(cus * 8), dim3(256), 0, 0, miters, sink); }, 5);
  const double mfma_flop = (double)cus * 8 * 4 /*waves*/ * miters * 8 * (16.0 * 16 * 32 * 2);
  const float mfma32_ms = time_ms([&] { hipLaunchKernelGGL(mfma32_kernel, dim3(cus * 8), dim3(256), 0, 0, miters, sink); }, 5);
  const double mfma32_flop = (double)cus * 8 * 4 * miters * 4 * (32.0 * 32 * 16 * 2);
  const int eiters = 4096;
  const float exp_ms = time_ms([&] { hipLaunchKernelGGL(exp_kernel, dim3(cus * 8), dim3(256), 0, 0, eiters, sink); }, 5);
  const double exps = (double)cus * 8 * 256 * eiters * 8;

  // pointer chase over 64 MiB (beyond L2), stride pattern via a permutation
  const unsigned nelem = 16u << 20;
  std::vector<unsigned> h(nelem);
  unsigned x = 1;
  std::vector<unsigned> perm(nelem);
  for (unsigned i = 0; i < nelem; ++i) perm[i] = i;
  for (unsigned i = nelem - 1; i > 0; --i) {   // xorshift Fisher-Yates
    x ^= x << 13; x ^= x >> 17; x ^= x << 5;
    const unsigned j = x % (i + 1);
    const unsigned t = perm[i]; perm[i] = perm[j]; perm[j] = t;
  }
  for (unsigned i = 0; i < nelem; ++i) h[perm[i]] = perm[(i + 1) % nelem];
  unsigned *d_next, *d_out;
  CHECK(hipMalloc(&d_next, nelem * 4ull));
  CHECK(hipMalloc(&d_out, 64));
  CHECK(hipMemcpy(d_next, h.data(), nelem * 4ull, hipMemcpyHostToDevice));
  const int steps = 20000;
  const float chase_ms = time_ms([&] { hipLaunchKernelGGL(chase_kernel, dim3(1), dim3(1), 0, 0, d_next, steps, d_out); }, 3);

  // dispatch floor: back-to-back empty launches (256 workgroups) on a stream and in a graph
  const float empty_ms = time_ms([&] { hipLaunchKernelGGL(empty_kernel, dim3(256), dim3(256), 0, 0, sink); }, 200);
  hipStream_t gs;
  CHECK(hipStreamCreate(&gs));
  hipGraph_t graph;
  hipGraphExec_t exec;
  CHECK(hipStreamBeginCapture(gs, hipStreamCaptureModeGlobal));
  for (int i = 0; i < 100; ++i) hipLaunchKernelGGL(empty_kernel, dim3(256), dim3(256), 0, gs, sink);
  CHECK(hipStreamEndCapture(gs, &graph));
  CHECK(hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0));
  const float graph_ms = time_ms([&] { hipGraphLaunch(exec, 0); }, 10) / 100.f;

  float *tiles;
  int *counter;
  CHECK(hipMalloc(&tiles, (size_t)512 * 1024 * 4));
  CHECK(hipMalloc(&counter, 64));
  CHECK(hipMemset(counter, 0, 64));
  const float nofence_ms = time_ms([&] { hipLaunchKernelGGL(arrive_kernel, dim3(512), dim3(256), 0, 0, tiles, counter, sink, 0); }, 50);
  const float fence_ms = time_ms([&] { hipLaunchKernelGGL(arrive_kernel, dim3(512), dim3(256), 0, 0, tiles, counter, sink, 1); }, 50);

  std::printf("{\"device\": \"%s\", \"cus\": %d, \"clock_mhz\": %d, \"copy_mib\": %zu, "
              "\"copy_gbs\": %.1f, \"read_gbs\": %.1f, \"mfma_bf16_tflops\": %.1f, "
              "\"mfma32_bf16_tflops\": %.1f, \"exp2_gops\": %.1f, \"exp2_per_cu_per_clk\": %.2f, \"load_latency_ns\": %.0f, "
              "\"copy_us\": %.2f, \"empty_kernel_stream_us\": %.2f, \"empty_kernel_graph_us\": %.2f, \"arrive512_nofence_us\": %.2f, \"arrive512_fence_us\": %.2f}\n",
              prop.gcnArchName, cus, prop.clockRate / 1000, mib, 2.0 * bytes / copy_ms / 1e6,
              bytes / read_ms / 1e6, mfma_flop / mfma_ms / 1e9, mfma32_flop / mfma32_ms / 1e9, exps / exp_ms / 1e6,
              exps / (exp_ms * 1e-3) / cus / (prop.clockRate * 1e3), chase_ms * 1e6 / steps, copy_ms * 1e3,
              empty_ms * 1e3, graph_ms * 1e3, nofence_ms * 1e3, fence_ms * 1e3);
  return 0;
}
