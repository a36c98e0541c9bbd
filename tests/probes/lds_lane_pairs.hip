// LDS lane-group probe (gfx950): only lanes a and b are active; lane a reads byte
// address 0 and lane b address 256 (the same banks with 64 four-byte banks),
// so a bank conflict shows iff the hardware serves a and b in the same cycle.
// Build: hipcc --offload-arch=gfx950 -O3 lds_lane_pairs.hip -o lds_lane_pairs
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdint.h>

constexpr int ITERS = 400;

__global__ void __launch_bounds__(256) pair(int a, int b, int mode, int sep, int* __restrict__ out) {
  __shared__ __align__(16) unsigned char smem[4096];
  for (int x = threadIdx.x; x < 4096 / 16; x += 256) reinterpret_cast<uint4*>(smem)[x] = uint4{(unsigned)x, 1u, 2u, 3u};
  __syncthreads();
  const int lane = threadIdx.x & 63;
  unsigned acc = 0;
  if (lane == a || lane == b) {
    const uint32_t la = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)(smem + (lane == b ? sep : 0));
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    if (mode == 0) {
      for (int it = 0; it < ITERS; ++it) {
        u32x4 v0;
        asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v0) : "v"(la) : "memory");
        acc += v0.x;
      }
    } else if (mode == 1) {
      for (int it = 0; it < ITERS; ++it) {
        u32x2 v0;
        asm volatile("ds_read_b64 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v0) : "v"(la) : "memory");
        acc += v0.x;
      }
    } else {
      for (int it = 0; it < ITERS; ++it) {
        u32x2 v0;
        asm volatile("ds_read_b64_tr_b16 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v0) : "v"(la) : "memory");
        acc += v0.x;
      }
    }
  }
  if (acc == 0x12345678u) out[threadIdx.x] = acc;
}

int main() {
  int* d_out;
  if (hipMalloc(&d_out, 256 * sizeof(int)) != hipSuccess) return 1;
  const int anchors[] = {0, 5, 8, 16, 32};
  int n = 0;
  for (int mode = 0; mode < 3; ++mode)
    for (int a : anchors)
      for (int b = 0; b < 64; ++b) {
        if (b == a) continue;
        hipLaunchKernelGGL(pair, dim3(256), dim3(64), 0, 0, a, b, mode, 256, d_out);
        printf("%d mode %d a %d b %d\n", n++, mode, a, b);
      }
  hipError_t err = hipDeviceSynchronize();
  printf("status %s\n", hipGetErrorString(err));
  return err == hipSuccess ? 0 : 1;
}
