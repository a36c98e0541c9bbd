// HBM read probe (gfx950): each workgroup streams a contiguous share of 5 GiB with
// 16-byte loads, eight in flight per lane; an xor of the data keeps the loads.
// Two forms of the load: ordinary, and non-temporal (the data need not stay in
// the caches), which is what the decoding kernel uses for the K/V cache.
// Build: hipcc --offload-arch=gfx950 -O3 hbm_read.hip -o hbm_read
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdint.h>
typedef unsigned v4u __attribute__((ext_vector_type(4)));
template <int UNROLL, bool NT>
__global__ void __launch_bounds__(256) rd(const v4u* __restrict__ src, size_t n16_per_wg, unsigned* out) {
  const v4u* p = src + (size_t)blockIdx.x * n16_per_wg;
  unsigned acc = 0;
  for (size_t i = threadIdx.x; i < n16_per_wg; i += 256 * UNROLL) {
    v4u v[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const size_t j = i + (size_t)u * 256;
      if (j < n16_per_wg) {
        if constexpr (NT)
          v[u] = __builtin_nontemporal_load(p + j);
        else
          v[u] = p[j];
      } else {
        v[u] = v4u{0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) acc ^= v[u].x ^ v[u].w;
  }
  if (acc == 0x9e3779b9u) out[blockIdx.x] = acc;
}
template <bool NT>
static bool sweep(const v4u* src, unsigned* out, size_t bytes, const char* name) {
  hipEvent_t e0, e1;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return false;
  for (int wgs : {1024, 2048, 4096, 8192}) {
    const size_t n16 = bytes / 16 / wgs;
    for (int rep = 0; rep < 2; ++rep) {
      if (hipEventRecord(e0) != hipSuccess) return false;
      for (int it = 0; it < 5; ++it) hipLaunchKernelGGL((rd<8, NT>), dim3(wgs), dim3(256), 0, 0, src, n16, out);
      if (hipEventRecord(e1) != hipSuccess || hipEventSynchronize(e1) != hipSuccess) return false;
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, e0, e1) != hipSuccess) return false;
      ms /= 5;
      if (rep) printf("%s workgroups %5d unroll 8: %.3f ms  %.1f GB/s\n", name, wgs, ms, (double)n16 * 16 * wgs / (ms * 1e-3) / 1e9);
    }
  }
  return true;
}
int main() {
  const size_t bytes = (size_t)5 << 30;  // 5 GiB, like one decoding step
  v4u* src;
  unsigned* out;
  if (hipMalloc(&src, bytes) != hipSuccess || hipMalloc(&out, 65536 * 4) != hipSuccess) return 1;
  if (hipMemset(src, 1, bytes) != hipSuccess) return 1;
  if (!sweep<false>(src, out, bytes, "ordinary    ") || !sweep<true>(src, out, bytes, "non-temporal")) return 1;
  hipError_t err = hipDeviceSynchronize();
  printf("status %s\n", hipGetErrorString(err));
  return err == hipSuccess ? 0 : 1;
}
