// f3c_drive: a torch-free command-line driver of the cached sampler through
// the C ABI (include/f3c.h). It runs whole trajectories of Algorithm 1 on one
// GPU with the HIP runtime of the ROCm installation, for hardware-counter runs
// (rocprofv3 --pmc) and for timing without Python.
//
//   f3c_drive [--grid G] [--width D] [--depth L] [--heads H] [--cond NC]
//             [--cond-width DC] [--f32] [--batch B] [--steps T] [--eta E]
//             [--quotas c1,c2,...] [--repeat R] [--copy-mib M] [--graph]
//   f3c_drive --peaks
//
// Defaults: the 24-block, width-1024 bf16 model on a 16^3 grid with 1374 x
// 1024 condition tokens, 25 steps with the eta = 3 time shift (Eq. S1), every
// step full. --quotas gives the cached-token count of each step (0 = full
// step), the same for every sample. Each trajectory starts from zeroed caches,
// the same x_T and a recomputed condition K/V, like the Python benchmark.
//
// Weights (N(0, 0.02)), noise and condition tokens (N(0, 1)) come from a
// fixed-seed generator of this driver; they are not the seeded arrays of the
// Python workloads, and the work done does not depend on the values.
//
// --copy-mib M first runs one plain float4 copy of M MiB (k_copy_ref): a
// known-size reference for hardware byte counters.
//
// --graph captures the T steps of a trajectory once into a HIP graph and
// replays it; the per-trajectory cache reset, the copy of x_T, the condition
// K/V and the modulation plan stay eager launches before each replay.
//
// --peaks measures what the chip sustains, for the rooflines, and exits: the
// dense bf16 matrix-core rate (every wave issues independent
// v_mfma_f32_32x32x16_bf16 on register operands, four waves per SIMD) and the
// HBM bandwidth of a plain 1 GiB float4 copy (bytes read plus written).
#include <hip/hip_runtime.h>

#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "f3c.h"

namespace {

__global__ void k_copy_ref(const float4* __restrict__ src, float4* __restrict__ dst, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256) void k_mfma_peak(float* __restrict__ out, int iters, float seed) {
  bf16x8_t a, b;
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(seed * (float)(threadIdx.x + e));
    b[e] = (__bf16)(seed - (float)e);
  }
  f32x16_t acc[8];
  for (int i = 0; i < 8; ++i)
    for (int e = 0; e < 16; ++e) acc[i][e] = 0.0f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i], 0, 0, 0);
  }
  float sum = 0.0f;
  for (int i = 0; i < 8; ++i)
    for (int e = 0; e < 16; ++e) sum += acc[i][e];
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = sum;
}

[[noreturn]] void die(const char* what) {
  std::fprintf(stderr, "f3c_drive: %s\n", what);
  std::exit(1);
}

void check(int rc, const char* call) {
  if (rc != F3C_OK) {
    std::fprintf(stderr, "f3c_drive: %s failed (%d): %s\n", call, rc, f3c_last_error());
    std::exit(1);
  }
}

void hip_check(hipError_t e, const char* call) {
  if (e != hipSuccess) {
    std::fprintf(stderr, "f3c_drive: %s: %s\n", call, hipGetErrorString(e));
    std::exit(1);
  }
}

// splitmix64 stream with Box-Muller normals.
struct Rng {
  uint64_t s;
  explicit Rng(uint64_t seed) : s(seed) {}
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  double uniform() { return ((next() >> 11) + 0.5) * (1.0 / 9007199254740992.0); }
  void normals(float* out, size_t n, float scale) {
    for (size_t i = 0; i < n; i += 2) {
      const double r = std::sqrt(-2.0 * std::log(uniform())), a = 6.283185307179586 * uniform();
      out[i] = (float)(scale * r * std::cos(a));
      if (i + 1 < n) out[i + 1] = (float)(scale * r * std::sin(a));
    }
  }
};

std::vector<int> parse_list(const char* s) {
  std::vector<int> v;
  while (*s) {
    char* end = nullptr;
    const long x = std::strtol(s, &end, 10);
    if (end == s) die("bad --quotas list");
    v.push_back((int)x);
    s = *end == ',' ? end + 1 : end;
  }
  return v;
}

}  // namespace

int main(int argc, char** argv) {
  f3c_model_cfg cfg{};
  cfg.grid = 16;
  cfg.in_ch = 8;
  cfg.width = 1024;
  cfg.depth = 24;
  cfg.heads = 16;
  cfg.mlp_ratio = 4;
  cfg.cond_tokens = 1374;
  cfg.cond_width = 1024;
  cfg.dtype = F3C_BF16;
  int batch = 1, steps = 25, repeat = 1, copy_mib = 0;
  bool use_graph = false, peaks = false;
  double eta = 3.0;
  std::vector<int> quotas;
  for (int i = 1; i < argc; ++i) {
    const std::string a = argv[i];
    auto val = [&]() -> const char* {
      if (i + 1 >= argc) die(("missing value for " + a).c_str());
      return argv[++i];
    };
    if (a == "--grid") cfg.grid = std::atoi(val());
    else if (a == "--width") cfg.width = std::atoi(val());
    else if (a == "--depth") cfg.depth = std::atoi(val());
    else if (a == "--heads") cfg.heads = std::atoi(val());
    else if (a == "--cond") cfg.cond_tokens = std::atoi(val());
    else if (a == "--cond-width") cfg.cond_width = std::atoi(val());
    else if (a == "--f32") cfg.dtype = F3C_F32;
    else if (a == "--batch") batch = std::atoi(val());
    else if (a == "--steps") steps = std::atoi(val());
    else if (a == "--eta") eta = std::atof(val());
    else if (a == "--quotas") quotas = parse_list(val());
    else if (a == "--repeat") repeat = std::atoi(val());
    else if (a == "--copy-mib") copy_mib = std::atoi(val());
    else if (a == "--graph") use_graph = true;
    else if (a == "--peaks") peaks = true;
    else die(("unknown argument " + a).c_str());
  }
  if (quotas.empty()) quotas.assign(steps, 0);
  if ((int)quotas.size() != steps) die("--quotas needs one count per step");
  if (repeat < 1 || batch < 1) die("--repeat and --batch must be positive");
  const size_t N = (size_t)cfg.grid * cfg.grid * cfg.grid;
  for (int q : quotas)
    if (q < 0 || (size_t)q > N) die("quota outside [0, N]");

  hip_check(hipSetDevice(0), "hipSetDevice");
  hipStream_t st;
  hip_check(hipStreamCreate(&st), "hipStreamCreate");

  if (peaks) {
    hipEvent_t p0, p1;
    hip_check(hipEventCreate(&p0), "hipEventCreate");
    hip_check(hipEventCreate(&p1), "hipEventCreate");
    int cus = 0;
    hip_check(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0), "hipDeviceGetAttribute");
    // Matrix cores: four 4-wave workgroups per CU, 4096 x 8 MFMAs per wave.
    const int blocks = 4 * cus, iters = 4096;
    float* out = nullptr;
    hip_check(hipMalloc(&out, (size_t)blocks * 256 * sizeof(float)), "hipMalloc");
    hipLaunchKernelGGL(k_mfma_peak, dim3(blocks), dim3(256), 0, st, out, 16, 1.0f);
    hip_check(hipGetLastError(), "k_mfma_peak");
    float best = 1e30f;
    for (int r = 0; r < 3; ++r) {
      hip_check(hipEventRecord(p0, st), "hipEventRecord");
      hipLaunchKernelGGL(k_mfma_peak, dim3(blocks), dim3(256), 0, st, out, iters, 1.0f);
      hip_check(hipEventRecord(p1, st), "hipEventRecord");
      hip_check(hipEventSynchronize(p1), "k_mfma_peak");
      float ms = 0.0f;
      hip_check(hipEventElapsedTime(&ms, p0, p1), "hipEventElapsedTime");
      best = std::fmin(best, ms);
    }
    const double flops = (double)blocks * 4 * iters * 8 * 32768.0;
    std::printf("peak: bf16 matrix cores %.1f TFLOP/s on %d CUs (%.1f%% of 2500)\n", flops / best * 1e-9, cus,
                flops / best * 1e-9 / 25.0);
    hip_check(hipFree(out), "hipFree");
    // HBM: a 1 GiB float4 copy, best of 10 (bytes read plus written).
    const size_t n4 = ((size_t)1 << 30) / sizeof(float4);
    float4 *src, *dst;
    hip_check(hipMalloc(&src, n4 * sizeof(float4)), "hipMalloc");
    hip_check(hipMalloc(&dst, n4 * sizeof(float4)), "hipMalloc");
    hip_check(hipMemsetAsync(src, 0, n4 * sizeof(float4), st), "hipMemsetAsync");
    hipLaunchKernelGGL(k_copy_ref, dim3(4096), dim3(256), 0, st, src, dst, n4);
    best = 1e30f;
    for (int r = 0; r < 10; ++r) {
      hip_check(hipEventRecord(p0, st), "hipEventRecord");
      hipLaunchKernelGGL(k_copy_ref, dim3(4096), dim3(256), 0, st, src, dst, n4);
      hip_check(hipEventRecord(p1, st), "hipEventRecord");
      hip_check(hipEventSynchronize(p1), "k_copy_ref");
      float ms = 0.0f;
      hip_check(hipEventElapsedTime(&ms, p0, p1), "hipEventElapsedTime");
      best = std::fmin(best, ms);
    }
    const double bytes = 2.0 * n4 * sizeof(float4);
    std::printf("peak: HBM copy %.0f GB/s (%.1f%% of 8000)\n", bytes / best * 1e-6, bytes / best * 1e-6 / 80.0);
    hip_check(hipFree(src), "hipFree");
    hip_check(hipFree(dst), "hipFree");
    return 0;
  }

  if (copy_mib > 0) {
    const size_t n4 = ((size_t)copy_mib << 20) / sizeof(float4);
    float4 *src, *dst;
    hip_check(hipMalloc(&src, n4 * sizeof(float4)), "hipMalloc");
    hip_check(hipMalloc(&dst, n4 * sizeof(float4)), "hipMalloc");
    hip_check(hipMemsetAsync(src, 0, n4 * sizeof(float4), st), "hipMemsetAsync");
    hipLaunchKernelGGL(k_copy_ref, dim3(4096), dim3(256), 0, st, src, dst, n4);
    hip_check(hipGetLastError(), "k_copy_ref");
    hip_check(hipStreamSynchronize(st), "copy");
    hip_check(hipFree(src), "hipFree");
    hip_check(hipFree(dst), "hipFree");
    std::printf("copy reference: %d MiB read, %d MiB written\n", copy_mib, copy_mib);
  }

  f3c_model* m = nullptr;
  check(f3c_model_create(&cfg, &m), "f3c_model_create");
  int32_t nw = 0;
  check(f3c_weight_count(m, &nw), "f3c_weight_count");
  Rng rng(20251128);
  std::vector<std::vector<float>> host(nw);
  std::vector<const float*> ptrs(nw);
  for (int i = 0; i < nw; ++i) {
    const char* name = nullptr;
    int64_t numel = 0;
    check(f3c_weight_info(m, i, &name, &numel), "f3c_weight_info");
    host[i].resize((size_t)numel);
    rng.normals(host[i].data(), host[i].size(), 0.02f);
    ptrs[i] = host[i].data();
  }
  size_t wbytes = 0;
  check(f3c_model_weights_bytes(m, &wbytes), "f3c_model_weights_bytes");
  void* wdev = nullptr;
  hip_check(hipMalloc(&wdev, wbytes), "hipMalloc weights");
  check(f3c_model_load_weights(m, wdev, wbytes, ptrs.data(), nw), "f3c_model_load_weights");
  host.clear();

  size_t sbytes = 0;
  check(f3c_state_bytes(m, batch, &sbytes), "f3c_state_bytes");
  void* sdev = nullptr;
  hip_check(hipMalloc(&sdev, sbytes), "hipMalloc state");
  f3c_state* s = nullptr;
  check(f3c_state_create(m, batch, sdev, sbytes, st, &s), "f3c_state_create");

  const size_t nx = (size_t)batch * N * cfg.in_ch, nc = (size_t)batch * cfg.cond_tokens * cfg.cond_width;
  std::vector<float> hx(nx), hc(nc);
  rng.normals(hx.data(), nx, 1.0f);
  rng.normals(hc.data(), nc, 1.0f);
  float *x0, *x, *cond;
  hip_check(hipMalloc(&x0, nx * 4), "hipMalloc");
  hip_check(hipMalloc(&x, nx * 4), "hipMalloc");
  hip_check(hipMalloc(&cond, nc * 4), "hipMalloc");
  hip_check(hipMemcpy(x0, hx.data(), nx * 4, hipMemcpyHostToDevice), "hipMemcpy");
  hip_check(hipMemcpy(cond, hc.data(), nc * 4, hipMemcpyHostToDevice), "hipMemcpy");

  std::vector<double> times(steps + 1);
  check(f3c_time_grid(steps, eta, times.data()), "f3c_time_grid");
  std::vector<int32_t> qb(batch);
  // The modulation of every step time, planned at each trajectory start.
  size_t pbytes = 0;
  check(f3c_plan_bytes(m, steps, &pbytes), "f3c_plan_bytes");
  void* plan = nullptr;
  hip_check(hipMalloc(&plan, pbytes), "hipMalloc plan");

  auto run_steps = [&]() {
    for (int k = 0; k < steps; ++k) {
      if (quotas[k] == 0) {
        check(f3c_full_step(s, x, times[k], times[k + 1], st), "f3c_full_step");
      } else {
        for (int b = 0; b < batch; ++b) qb[b] = quotas[k];
        check(f3c_cached_step(s, x, times[k], times[k + 1], qb.data(), st), "f3c_cached_step");
      }
    }
  };
  hipGraphExec_t gexec = nullptr;
  if (use_graph) {
    check(f3c_set_cond(s, cond, st), "f3c_set_cond");    // the steps check that a condition is set
    check(f3c_state_plan_times(s, times.data(), steps, plan, pbytes, st), "f3c_state_plan_times");
    hip_check(hipStreamSynchronize(st), "hipStreamSynchronize");
    hipGraph_t graph;
    hip_check(hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal), "hipStreamBeginCapture");
    run_steps();
    hip_check(hipStreamEndCapture(st, &graph), "hipStreamEndCapture");
    hip_check(hipGraphInstantiate(&gexec, graph, nullptr, nullptr, 0), "hipGraphInstantiate");
    hip_check(hipGraphDestroy(graph), "hipGraphDestroy");
  }

  hipEvent_t e0, e1;
  hip_check(hipEventCreate(&e0), "hipEventCreate");
  hip_check(hipEventCreate(&e1), "hipEventCreate");
  hip_check(hipEventRecord(e0, st), "hipEventRecord");
  const auto w0 = std::chrono::steady_clock::now();
  for (int r = 0; r < repeat; ++r) {
    check(f3c_state_reset(s, st), "f3c_state_reset");
    hip_check(hipMemcpyAsync(x, x0, nx * 4, hipMemcpyDeviceToDevice, st), "hipMemcpyAsync");
    check(f3c_set_cond(s, cond, st), "f3c_set_cond");
    check(f3c_state_plan_times(s, times.data(), steps, plan, pbytes, st), "f3c_state_plan_times");
    if (use_graph) hip_check(hipGraphLaunch(gexec, st), "hipGraphLaunch");
    else run_steps();
  }
  hip_check(hipEventRecord(e1, st), "hipEventRecord");
  hip_check(hipEventSynchronize(e1), "hipEventSynchronize");
  const double wall = std::chrono::duration<double>(std::chrono::steady_clock::now() - w0).count();
  float ms = 0.0f;
  hip_check(hipEventElapsedTime(&ms, e0, e1), "hipEventElapsedTime");
  std::printf("f3c_drive: %d trajectories x %d steps, batch %d%s: %.3f ms per step (GPU), %.3f ms per step (wall)\n",
              repeat, steps, batch, use_graph ? ", graph replay" : "", ms / (repeat * steps),
              wall * 1e3 / (repeat * steps));
  if (gexec) hip_check(hipGraphExecDestroy(gexec), "hipGraphExecDestroy");

  f3c_state_destroy(s);
  f3c_model_destroy(m);
  hip_check(hipFree(x0), "hipFree");
  hip_check(hipFree(x), "hipFree");
  hip_check(hipFree(cond), "hipFree");
  hip_check(hipFree(plan), "hipFree");
  hip_check(hipFree(sdev), "hipFree");
  hip_check(hipFree(wdev), "hipFree");
  hip_check(hipStreamDestroy(st), "hipStreamDestroy");
  return 0;
}
