// ffbench: native driver of the C ABI for timing and hardware-counter runs.
//
//   ffbench [m n N iters dtype(bf16|f32) damping]   (default 4096 4096 128 10 bf16 0)
//
// Before the job it runs one plain device-to-device copy of 1 GiB, a
// reference of known size for scaling the FETCH_SIZE / WRITE_SIZE counters.
// Fills G on the device with a counter-based hash (uniform entries; timing
// does not depend on the values), allocates the workspace, and times
// ff_iterate(iters) after one untimed iteration on the same handle, with HIP
// events on one stream.  Prints the
// job time, iterations per second and the per-kernel measurement hook.
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ff.h"

#define CHECK(x)                                                                     \
  do {                                                                               \
    hipError_t e_ = (x);                                                             \
    if (e_ != hipSuccess) {                                                          \
      fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));                 \
      return 1;                                                                      \
    }                                                                                \
  } while (0)

__device__ __forceinline__ uint64_t mix64(uint64_t z) {  // splitmix64 finaliser
  z += 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

__global__ void fill(void* G, int64_t count, int bf16) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) {
    const float u = (float)(mix64((uint64_t)i) >> 40) * (1.0f / 16777216.0f) * 2.0f - 1.0f;
    if (bf16) ((__bf16*)G)[i] = (__bf16)u;
    else ((float*)G)[i] = u;
  }
}

int main(int argc, char** argv) {
  int64_t m = 4096, n = 4096, N = 128;
  int iters = 10, bf16 = 1;
  if (argc > 1) m = atoll(argv[1]);
  if (argc > 2) n = atoll(argv[2]);
  if (argc > 3) N = atoll(argv[3]);
  if (argc > 4) iters = atoi(argv[4]);
  if (argc > 5) bf16 = strcmp(argv[5], "f32") != 0;
  double damping = 0.0;
  if (argc > 6) damping = atof(argv[6]);
  const size_t elem = bf16 ? 2 : 4;
  void* G = nullptr;
  CHECK(hipMalloc(&G, (size_t)N * m * n * elem));
  hipStream_t s;
  CHECK(hipStreamCreate(&s));
  hipLaunchKernelGGL(fill, dim3(4096), dim3(256), 0, s, G, N * m * n, bf16);
  CHECK(hipGetLastError());
  ff_config cfg;
  memset(&cfg, 0, sizeof cfg);
  cfg.m = m;
  cfg.n = n;
  cfg.N = N;
  cfg.dtype = bf16 ? FF_BF16 : FF_F32;
  cfg.G = G;
  cfg.stream = s;
  cfg.order = FF_ORDER_B_FIRST;
  cfg.whiten_split = 0;  // the library's default (automatic)
  cfg.damping = damping;
  size_t ws = 0;
  if (ff_workspace_size(&cfg, &ws) != FF_OK) {
    fprintf(stderr, "ff_workspace_size: %s\n", ff_last_error());
    return 1;
  }
  CHECK(hipMalloc(&cfg.workspace, ws));
  cfg.workspace_bytes = ws;
  {
    const size_t ref = (size_t)1 << 30;  // counter reference: copy 1 GiB
    if (ws >= 2 * ref) {
      CHECK(hipMemcpyAsync((char*)cfg.workspace + ref, cfg.workspace, ref, hipMemcpyDeviceToDevice, s));
      printf("reference copy: %zu bytes read, %zu bytes written\n", ref, ref);
    }
  }
  CHECK(hipStreamSynchronize(s));
  // warm-up job
  ff_handle h;
  int done = 0;
  if (ff_init(&cfg, &h) != FF_OK || ff_iterate(h, 1, &done, nullptr) != FF_OK) {
    fprintf(stderr, "warm-up failed: %s\n", ff_last_error());
    return 1;
  }
  ff_destroy(h);
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  // the timed job: iterations after one untimed iteration on the same handle
  if (ff_init(&cfg, &h) != FF_OK || ff_iterate(h, 1, &done, nullptr) != FF_OK) return 1;
  ff_set_timing(h, 1);
  CHECK(hipEventRecord(e0, s));
  const ff_status rc = ff_iterate(h, iters, &done, nullptr);
  CHECK(hipEventRecord(e1, s));
  CHECK(hipEventSynchronize(e1));
  float ms = 0;
  CHECK(hipEventElapsedTime(&ms, e0, e1));
  const double dm = (double)m, dn = (double)n, dN = (double)N;
  const double flop = 2.0 * dN * dm * dn * (dm + dn) + (dm * dm * dm + dn * dn * dn) / 3.0;
  printf("ffbench m=%lld n=%lld N=%lld %s: status %s, %d iterations in %.3f ms: %.3f iter/s, "
         "%.1f TFLOP/s\n",
         (long long)m, (long long)n, (long long)N, bf16 ? "bf16" : "f32", ff_status_string(rc), done,
         ms, 1000.0 * done / ms, flop * done / (ms * 1e-3) / 1e12);
  const char* names[4] = {"whiten", "syrk", "reduce", "cholinv"};
  for (int k = 0; k < 4; ++k) {
    int64_t nl = 0;
    double t = 0, fl = 0;
    ff_kernel_timing(h, k, &nl, &t, &fl);
    printf("  %-8s %4lld launches  %9.3f ms  avg %8.3f ms  %8.1f TFLOP/s\n", names[k],
           (long long)nl, t, nl ? t / nl : 0.0, t > 0 ? fl / (t * 1e-3) / 1e12 : 0.0);
  }
  ff_destroy(h);
  CHECK(hipFree(cfg.workspace));
  CHECK(hipFree(G));
  return rc == FF_OK ? 0 : 1;
}
