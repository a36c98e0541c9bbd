// LDS bank-conflict probe (gfx950): each launch reads LDS with a per-lane
// byte-address table (every address inside the 64 KB array, aligned to the
// access size), so the SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE counters per
// dispatch tell which lane patterns the hardware serves without conflicts.
// Patterns: plain strides, and the read patterns of the attention kernels on
// tiles laid out with the earlier chunk swizzle ("old") and the current one
// ("new", the swz of mfma_tiles.h).
// Build: hipcc --offload-arch=gfx950 -O3 lds_patterns.hip -o lds_patterns
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <vector>
#include <string>

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int ITERS = 2000;
constexpr int LDS_BYTES = 65536;

// mode 0: ds_read_b128, 1: ds_read_b64, 2: ds_read_b64_tr_b16, 3: ds_write_b128
__global__ void __launch_bounds__(256) probe(const int* __restrict__ addr_tab, int mode, int* __restrict__ out) {
  __shared__ __align__(16) unsigned char smem[LDS_BYTES];
  const int lane = threadIdx.x & 63;
  for (int x = threadIdx.x; x < LDS_BYTES / 16; x += 256) reinterpret_cast<uint4*>(smem)[x] = uint4{(unsigned)x, 1u, 2u, 3u};
  __syncthreads();
  const int a = addr_tab[lane];
  unsigned acc = 0;
  const uint32_t la = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)(smem + a);
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
  if (mode == 0) {
    for (int it = 0; it < ITERS / 4; ++it) {
      u32x4 v0, v1, v2, v3;
      asm volatile("ds_read_b128 %0, %4\n\tds_read_b128 %1, %4\n\tds_read_b128 %2, %4\n\tds_read_b128 %3, %4\n\ts_waitcnt lgkmcnt(0)"
                   : "=v"(v0), "=v"(v1), "=v"(v2), "=v"(v3) : "v"(la) : "memory");
      acc += v0.x ^ v1.y ^ v2.z ^ v3.w;
    }
  } else if (mode == 1) {
    for (int it = 0; it < ITERS / 4; ++it) {
      u32x2 v0, v1, v2, v3;
      asm volatile("ds_read_b64 %0, %4\n\tds_read_b64 %1, %4\n\tds_read_b64 %2, %4\n\tds_read_b64 %3, %4\n\ts_waitcnt lgkmcnt(0)"
                   : "=v"(v0), "=v"(v1), "=v"(v2), "=v"(v3) : "v"(la) : "memory");
      acc += v0.x ^ v1.y ^ v2.x ^ v3.y;
    }
  } else if (mode == 2) {
    for (int it = 0; it < ITERS / 4; ++it) {
      u32x2 v0, v1, v2, v3;
      asm volatile("ds_read_b64_tr_b16 %0, %4\n\tds_read_b64_tr_b16 %1, %4\n\tds_read_b64_tr_b16 %2, %4\n\tds_read_b64_tr_b16 %3, %4\n\ts_waitcnt lgkmcnt(0)"
                   : "=v"(v0), "=v"(v1), "=v"(v2), "=v"(v3) : "v"(la) : "memory");
      acc += v0.x ^ v1.y ^ v2.x ^ v3.y;
    }
  } else {
    u32x4 w = {acc, 1u, 2u, 3u};
    for (int it = 0; it < ITERS / 4; ++it) {
      w.x += it;
      asm volatile("ds_write_b128 %0, %1\n\tds_write_b128 %0, %1\n\tds_write_b128 %0, %1\n\tds_write_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)"
                   : : "v"(la), "v"(w) : "memory");
    }
    acc = w.x;
  }
  if (acc == 0x12345678u) out[threadIdx.x] = acc;
}

// 16-byte chunk XOR by row (D = 128: 16 chunks per row, 256-byte rows)
static int swz_old(int row) { return ((row & 7) << 1) | (((row >> 2) ^ (row >> 3)) & 1); }
static int swz_new(int row) { return ((row & 3) << 2) | ((((row >> 2) ^ (row >> 3)) & 1) << 1) | ((row >> 3) & 1); }
static bool g_new = false;
static int off128(int row, int chunk) { return row * 256 + ((chunk ^ (g_new ? swz_new : swz_old)(row & 15)) << 4); }
static int offcol128(int row, int col) { return off128(row, col >> 3) + ((col & 7) << 1); }

int main() {
  std::vector<std::pair<std::string, std::pair<int, std::vector<int>>>> pats;
  auto add = [&](const char* name, int mode, auto f) {
    std::vector<int> t(64);
    for (int l = 0; l < 64; ++l) t[l] = f(l);
    pats.push_back({name, {mode, t}});
  };
  // plain strides
  add("b128_linear", 0, [](int l) { return 16 * l; });
  add("b128_bcast", 0, [](int l) { return 0; });
  add("b128_8x256", 0, [](int l) { return 16 * (l % 8) + 256 * (l / 8); });     // 8 lanes per 128 B, 256 B apart
  add("b128_16x256", 0, [](int l) { return 16 * (l % 16) + 512 * (l / 16); });  // 16 lanes per 256 B
  add("b128_rowpitch", 0, [](int l) { return 256 * (l % 16) + 16 * (l / 16); }); // unswizzled column read
  add("b64_linear", 1, [](int l) { return 8 * l; });
  add("b64_16x256", 1, [](int l) { return 8 * (l % 16) + 256 * (l / 16); });
  add("b64_32x512", 1, [](int l) { return 8 * (l % 32) + 512 * (l / 32); });
  add("tr_linear", 2, [](int l) { return 8 * l; });
  add("tr_16x256", 2, [](int l) { return 8 * (l % 16) + 256 * (l / 16); });
  add("tr_32x512", 2, [](int l) { return 8 * (l % 32) + 512 * (l / 32); });
  add("w128_linear", 3, [](int l) { return 16 * l; });
  add("w128_8x256", 3, [](int l) { return 16 * (l % 8) + 256 * (l / 8); });
  // the kernels' read patterns on 128-column bf16 tiles, old and new swizzle
  for (int nw = 0; nw < 2; ++nw) {
    const char* tag = nw ? "new" : "old";
    char nm[64];
    // row fragments of the backward / dQ pass: lane (lr, lg) reads row lr, chunk 4 ks + lg
    for (int ks = 0; ks < 4; ++ks) {
      snprintf(nm, 64, "%s_b128_bwd_row8_ks%d", tag, ks);
      add(strdup(nm), 0, [ks, nw](int l) { g_new = nw; return off128(l & 15, 4 * ks + (l >> 4)); });
    }
    // forward K rows: row l % 32, chunk 2 ks + l / 32
    for (int ks = 0; ks < 8; ks += 3) {
      snprintf(nm, 64, "%s_b128_fwd_k_ks%d", tag, ks);
      add(strdup(nm), 0, [ks, nw](int l) { g_new = nw; return off128(l & 31, 2 * ks + (l >> 5)); });
    }
    // transposing reads of the backward / dQ pass: row 4 lg + lr / 4, column 16 md + 4 (lr % 4)
    for (int md = 0; md < 8; md += 3) {
      snprintf(nm, 64, "%s_tr_bwd_md%d", tag, md);
      add(strdup(nm), 2, [md, nw](int l) {
        const int lr = l & 15, lg = l >> 4;
        g_new = nw;
        return offcol128(4 * lg + (lr >> 2), 16 * md + 4 * (lr & 3));
      });
    }
    // forward V^T reads: rows 4 (l / 32) + (l % 16) / 4 (+ 8 hf), columns 32 md + 16 ((l / 16) % 2) + 4 (l % 4)
    for (int md = 0; md < 4; md += 3)
      for (int hf = 0; hf < 2; ++hf) {
        snprintf(nm, 64, "%s_tr_fwd_v_md%d_hf%d", tag, md, hf);
        add(strdup(nm), 2, [md, hf, nw](int l) {
          g_new = nw;
          return offcol128(4 * (l >> 5) + ((l & 15) >> 2) + 8 * hf, 32 * md + 16 * ((l >> 4) & 1) + 4 * (l & 3));
        });
      }
  }

  int *d_tab, *d_out;
  if (hipMalloc(&d_tab, 64 * sizeof(int)) != hipSuccess || hipMalloc(&d_out, 256 * sizeof(int)) != hipSuccess) return 1;
  printf("dispatch order:\n");
  for (size_t i = 0; i < pats.size(); ++i) {
    auto& p = pats[i];
    for (int a : p.second.second)
      if (a < 0 || a + 16 > LDS_BYTES) { printf("bad address in %s\n", p.first.c_str()); return 1; }
    if (hipMemcpy(d_tab, p.second.second.data(), 64 * sizeof(int), hipMemcpyHostToDevice) != hipSuccess) return 1;
    hipEvent_t e0, e1;
    hipEventCreate(&e0); hipEventCreate(&e1);
    hipEventRecord(e0);
    hipLaunchKernelGGL(probe, dim3(1024), dim3(256), 0, 0, d_tab, p.second.first, d_out);
    hipEventRecord(e1);
    hipEventSynchronize(e1);
    float ms = 0; hipEventElapsedTime(&ms, e0, e1);
    // 1024 workgroups x 4 waves x ITERS instructions over 256 CUs
    double per_inst_ns = ms * 1e6 / (1024.0 / 256.0 * ITERS);
    printf("%2zu %-22s mode %d  %.3f ms  %.2f ns per instruction per CU (4 waves)\n", i, p.first.c_str(),
           p.second.first, ms, per_inst_ns);
    fflush(stdout);
  }
  hipError_t err = hipDeviceSynchronize();
  printf("status %s\n", hipGetErrorString(err));
  return err == hipSuccess ? 0 : 1;
}
