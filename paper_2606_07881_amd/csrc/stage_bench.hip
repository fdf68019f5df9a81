// Native driver of the stage library, for profiling without Python.
//
// Replays the canonical asynchronous 1F1B schedule of M micro-batches through
// paci_stage_run on synthetic inputs resident in HBM (by default the
// GPT-2-medium-shaped bf16 middle stage: 6 blocks, d 1024, 16 heads of 64,
// FFN 4096, seq 1024, micro-batch 8, K 8, delay 3, M 64) and prints the
// replay time and, optionally, the per-family kernel times. Hardware counter
// collection (rocprofv3 --pmc) wants a process with a single HIP runtime,
// which a Python process that also loads torch is not.
//
// Inputs: stage inputs N(0, 1) and output gradients N(0, 0.01^2), weight
// matrices N(0, 0.02^2), biases 0, LayerNorm gains 1; drawn on the device from
// a counter-based hash (splitmix64) with the Box-Muller transform, rounded to
// bf16 (round to nearest even) for bf16 stages.
//
// usage: stage_bench [--layers L] [--d D] [--heads H] [--ff F] [--seq S] [--mu U]
//                    [--K K] [--delay N] [--M M] [--steps n] [--warmup n] [--fp32] [--timing]
//                    [--window] [--copy-probe] [--hbm-probe]
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "paci_stage.h"

#define CHECK_HIP(x)                                                                        \
  do {                                                                                      \
    hipError_t e_ = (x);                                                                    \
    if (e_ != hipSuccess) {                                                                 \
      fprintf(stderr, "%s:%d: %s: %s\n", __FILE__, __LINE__, #x, hipGetErrorString(e_));    \
      exit(1);                                                                              \
    }                                                                                       \
  } while (0)
#define CHECK_PACI(x)                                                                       \
  do {                                                                                      \
    int r_ = (x);                                                                           \
    if (r_ < 0) {                                                                           \
      fprintf(stderr, "%s:%d: %s: %s\n", __FILE__, __LINE__, #x, paci_strerror(r_));        \
      exit(1);                                                                              \
    }                                                                                       \
  } while (0)

__device__ __forceinline__ uint64_t splitmix64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// element i: N(0, std^2) by Box-Muller from two 24-bit uniforms of splitmix64(seed, i)
__device__ __forceinline__ float normal_at(uint64_t seed, int64_t i, float std) {
  const uint64_t h = splitmix64(seed * 0x100000001B3ull + (uint64_t)i);
  const float u1 = ((float)(h >> 40) + 1.0f) * (1.0f / 16777217.0f);   // (0, 1]
  const float u2 = (float)((h >> 16) & 0xFFFFFF) * (1.0f / 16777216.0f);
  return std * sqrtf(-2.0f * logf(u1)) * cosf(6.283185307179586f * u2);
}

__global__ void fill_normal(void* p, int64_t n, uint64_t seed, float std, int bf16) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const float v = normal_at(seed, i, std);
    if (bf16) {
      uint32_t u = __float_as_uint(v);
      u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest even
      reinterpret_cast<uint16_t*>(p)[i] = (uint16_t)(u >> 16);
    } else {
      reinterpret_cast<float*>(p)[i] = v;
    }
  }
}

// plain copy, 16 bytes per thread per iteration: a kernel of known traffic for scaling byte counters
__global__ void copy16(const uint4* src, uint4* dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}
// the same copy with non-temporal loads and stores (each byte is touched once)
typedef unsigned int u32v4 __attribute__((ext_vector_type(4)));
__global__ void copy16_nt(const uint4* src, uint4* dst, int64_t n) {
  const u32v4* s = reinterpret_cast<const u32v4*>(src);
  u32v4* d = reinterpret_cast<u32v4*>(dst);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    __builtin_nontemporal_store(__builtin_nontemporal_load(s + i), d + i);
}

__global__ void fill_const(float* p, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

static int arg_int(int argc, char** argv, const char* name, int dflt) {
  for (int i = 1; i + 1 < argc; ++i)
    if (!strcmp(argv[i], name)) return atoi(argv[i + 1]);
  return dflt;
}
static bool arg_flag(int argc, char** argv, const char* name) {
  for (int i = 1; i < argc; ++i)
    if (!strcmp(argv[i], name)) return true;
  return false;
}

int main(int argc, char** argv) {
  paci_shapes s;
  memset(&s, 0, sizeof(s));
  s.n_layers = arg_int(argc, argv, "--layers", 6);
  s.d_model = arg_int(argc, argv, "--d", 1024);
  s.n_heads = arg_int(argc, argv, "--heads", 16);
  s.head_dim = s.d_model / s.n_heads;
  s.d_ff = arg_int(argc, argv, "--ff", 4 * s.d_model);
  s.seq = arg_int(argc, argv, "--seq", 1024);
  s.micro_batch = arg_int(argc, argv, "--mu", 8);
  s.kind = PACI_MIDDLE;
  s.dtype = arg_flag(argc, argv, "--fp32") ? PACI_FP32 : PACI_BF16;
  s.lr = 1e-3f;
  s.beta1 = 0.9f;
  s.beta2 = 0.95f;
  s.eps = 1e-8f;
  s.weight_decay = 0.1f;
  s.ln_eps = 1e-5f;
  s.window = arg_flag(argc, argv, "--window") ? 1 : 0;
  const int K = arg_int(argc, argv, "--K", 8), delay = arg_int(argc, argv, "--delay", 3);
  const int M = arg_int(argc, argv, "--M", 64);
  const int steps = arg_int(argc, argv, "--steps", 2), warmup = arg_int(argc, argv, "--warmup", 1);
  const bool timing = arg_flag(argc, argv, "--timing");
  const bool bf16 = s.dtype == PACI_BF16;
  const int64_t T = (int64_t)s.micro_batch * s.seq, d = s.d_model;
  printf("stage_bench: layers %d d %d heads %dx%d ff %d seq %d mu %d K %d delay %d M %d %s%s\n", s.n_layers,
         s.d_model, s.n_heads, s.head_dim, s.d_ff, s.seq, s.micro_batch, K, delay, M, bf16 ? "bf16" : "fp32",
         s.window ? " windowed" : "");
  fflush(stdout);

  size_t bytes = 0;
  CHECK_PACI(paci_stage_arena_bytes(&s, K, delay, &bytes));
  void* arena = nullptr;
  CHECK_HIP(hipMalloc(&arena, bytes));
  hipStream_t st;
  CHECK_HIP(hipStreamCreate(&st));
  paci_stage* h = nullptr;
  CHECK_PACI(paci_stage_init(&s, K, delay, arena, bytes, st, &h));

  // parameters: matrices N(0, 0.02^2), LayerNorm gains 1, biases and shifts 0
  int n_tensors = 0;
  int64_t n_params = 0;
  CHECK_PACI(paci_param_count(&s, &n_tensors, &n_params));
  float* theta = nullptr;
  CHECK_HIP(hipMalloc(&theta, n_params * sizeof(float)));
  for (int i = 0; i < n_tensors; ++i) {
    paci_param_info info;
    CHECK_PACI(paci_param_info_at(&s, i, &info));
    float* p = theta + info.offset;
    const char* tail = strrchr(info.name, '.');
    tail = tail ? tail + 1 : info.name;
    if (info.cols > 1)
      hipLaunchKernelGGL(fill_normal, dim3(1024), dim3(256), 0, st, (void*)p, info.numel, (uint64_t)(1000 + i), 0.02f, 0);
    else
      hipLaunchKernelGGL(fill_const, dim3(256), dim3(256), 0, st, p, info.numel,
                         (tail[strlen(tail) - 1] == 'g') ? 1.0f : 0.0f);
    CHECK_HIP(hipGetLastError());
  }
  CHECK_PACI(paci_stage_load(h, PACI_PARAMS, theta, n_params, 1));

  const size_t esz = bf16 ? 2 : 4;
  const int64_t n_act = (int64_t)M * T * d;
  void *x_all = nullptr, *dy_all = nullptr;
  CHECK_HIP(hipMalloc(&x_all, n_act * esz));
  CHECK_HIP(hipMalloc(&dy_all, n_act * esz));
  hipLaunchKernelGGL(fill_normal, dim3(4096), dim3(256), 0, st, x_all, n_act, (uint64_t)1, 1.0f, (int)bf16);
  hipLaunchKernelGGL(fill_normal, dim3(4096), dim3(256), 0, st, dy_all, n_act, (uint64_t)2, 0.01f, (int)bf16);
  CHECK_HIP(hipGetLastError());
  CHECK_HIP(hipStreamSynchronize(st));
  printf("stage_bench: inputs resident (%.2f GiB arena)\n", bytes / 1073741824.0);
  fflush(stdout);

  if (arg_flag(argc, argv, "--copy-probe")) {   // 3 copies of 256 MiB
    const int64_t n16 = (256ll << 20) / 16;
    uint4 *a = nullptr, *b = nullptr;
    CHECK_HIP(hipMalloc(&a, n16 * 16));
    CHECK_HIP(hipMalloc(&b, n16 * 16));
    CHECK_HIP(hipMemsetAsync(a, 0, n16 * 16, st));
    for (int i = 0; i < 3; ++i) hipLaunchKernelGGL(copy16, dim3(8192), dim3(256), 0, st, a, b, n16);
    CHECK_HIP(hipGetLastError());
    CHECK_HIP(hipStreamSynchronize(st));
    CHECK_HIP(hipFree(a));
    CHECK_HIP(hipFree(b));
    printf("stage_bench: copy probe done (3 x 256 MiB, kernel copy16)\n");
    fflush(stdout);
  }

  if (arg_flag(argc, argv, "--hbm-probe")) {   // attainable HBM bandwidth: copies of 1 GiB, timed
    const int64_t n16 = (1ll << 30) / 16;
    uint4 *a = nullptr, *b = nullptr;
    CHECK_HIP(hipMalloc(&a, n16 * 16));
    CHECK_HIP(hipMalloc(&b, n16 * 16));
    CHECK_HIP(hipMemsetAsync(a, 0, n16 * 16, st));
    hipEvent_t e0, e1;
    CHECK_HIP(hipEventCreate(&e0));
    CHECK_HIP(hipEventCreate(&e1));
    for (int nt = 0; nt < 2; ++nt) {
      for (int grid : {2048, 8192, 32768}) {
        auto launch = [&] {
          if (nt) hipLaunchKernelGGL(copy16_nt, dim3(grid), dim3(256), 0, st, a, b, n16);
          else hipLaunchKernelGGL(copy16, dim3(grid), dim3(256), 0, st, a, b, n16);
        };
        launch();
        CHECK_HIP(hipEventRecord(e0, st));
        for (int i = 0; i < 10; ++i) launch();
        CHECK_HIP(hipEventRecord(e1, st));
        CHECK_HIP(hipEventSynchronize(e1));
        float ms = 0.f;
        CHECK_HIP(hipEventElapsedTime(&ms, e0, e1));
        printf("stage_bench: hbm probe %s grid %5d: %.0f GB/s (1 GiB read + 1 GiB written per copy)\n",
               nt ? "copy16_nt" : "copy16   ", grid, 10.0 * 2.0 * n16 * 16 / (ms * 1e-3) / 1e9);
      }
    }
    fflush(stdout);
    CHECK_HIP(hipEventDestroy(e0));
    CHECK_HIP(hipEventDestroy(e1));
    CHECK_HIP(hipFree(a));
    CHECK_HIP(hipFree(b));
  }

  std::vector<int32_t> stamps((size_t)M * 3);
  auto replay = [&]() {
    CHECK_PACI(paci_stage_reset_counters(h));
    CHECK_PACI(paci_stage_run(h, M, x_all, nullptr, dy_all, nullptr, nullptr, stamps.data()));
  };
  for (int i = 0; i < warmup; ++i) {
    replay();
    CHECK_PACI(paci_stage_sync(h));
    printf("stage_bench: warmup %d/%d done\n", i + 1, warmup);
    fflush(stdout);
  }
  hipEvent_t e0, e1;
  CHECK_HIP(hipEventCreate(&e0));
  CHECK_HIP(hipEventCreate(&e1));
  if (timing) CHECK_PACI(paci_stage_set_timing(h, 1));
  CHECK_HIP(hipEventRecord(e0, st));
  for (int i = 0; i < steps; ++i) replay();
  CHECK_HIP(hipEventRecord(e1, st));
  CHECK_HIP(hipEventSynchronize(e1));
  float ms = 0.f;
  CHECK_HIP(hipEventElapsedTime(&ms, e0, e1));
  const double ms_step = ms / steps;
  printf("stage_bench: %d replays, %.3f ms per replay, %.1f tokens/s\n", steps, ms_step,
         (double)M * T / (ms_step / 1e3));
  if (timing) {
    CHECK_PACI(paci_stage_set_timing(h, 0));
    for (int f = 0; f < paci_kernel_family_count(); ++f) {
      int64_t n = 0;
      double fms = 0, work = 0;
      CHECK_PACI(paci_stage_kernel_times(h, f, &n, &fms, &work));
      if (n) printf("  %-16s launches %8lld  ms/replay %9.3f  avg us %8.2f\n", paci_kernel_family_name(f),
                    (long long)n, fms / steps, 1e3 * fms / n);
    }
  }
  fflush(stdout);
  CHECK_PACI(paci_stage_destroy(h));
  CHECK_HIP(hipFree(x_all));
  CHECK_HIP(hipFree(dy_all));
  CHECK_HIP(hipFree(theta));
  CHECK_HIP(hipFree(arena));
  CHECK_HIP(hipStreamDestroy(st));
  return 0;
}
