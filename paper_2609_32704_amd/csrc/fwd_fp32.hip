// CoWA forward in float32 (Alg. 1) on the vector ALUs.
//
// One workgroup per (QO block i, QO head h, sequence b) with 8 lanes per query
// row: lane (row, sub) keeps the d/8-wide slice `sub` of its query and of its
// output accumulator in registers.  The KV blocks of J_{h_k}(i) are visited in
// the schedule's (descending) order, staged through LDS 32 keys at a time;
// a score is the sum of the 8 slice dot products (butterfly over the 8 lanes).
// The online softmax (running max m, running sum l, rescaled O) follows Alg. 1
// in base 2: scores are pre-multiplied by scale * log2(e) and the final
// LSE = (m + log2 l) * ln 2 is the natural-log value the backward expects.
#include "internal.h"
#include "window_rule.h"
#include "work_item.h"

namespace cowa {
namespace {

constexpr int kChunk = 32;  // keys staged per LDS pass

template <int D>
__global__ void __launch_bounds__(1024) fwd_fp32_kernel(cowa_params p, SchedView sv, const float* __restrict__ q,
                                                        const float* __restrict__ k, const float* __restrict__ v,
                                                        float* __restrict__ o, float* __restrict__ lse) {
  constexpr int SL = D / 8;  // slice width per lane
  __shared__ float ks[kChunk][D];
  __shared__ float vs[kChunk][D];

  const int tq = p.tile_q, tk = p.tile_k;
  const int h = blockIdx.y;
  const int hk_h = (int)(((int64_t)h * p.h_k) / p.h_q);
  int hk;
  const SeqCtx sc = seq_ctx(p, sv, blockIdx.x, sv.ragged ? hk_h : (int)blockIdx.z * p.h_k + hk_h, true, hk);
  const int i = sc.tile;
  const int n_q = sc.n_q, n_k = sc.n_k;

  const int tid = threadIdx.x;
  const int row = tid >> 3, sub = tid & 7;
  const int64_t qpos = (int64_t)i * tq + row;
  const bool row_ok = qpos < n_q;
  const int64_t row_base = sc.q0 + (int64_t)h * sc.qh;

  const float* qrow = q + (row_base + (row_ok ? qpos : 0)) * D + sub * SL;
  const float* kbase = k + (sc.k0 + (int64_t)hk * sc.kh) * D;
  const float* vbase = v + (sc.k0 + (int64_t)hk * sc.kh) * D;

  const float c = p.softmax_scale * 1.4426950408889634f;  // log2(e)
  float qr[SL], acc[SL];
#pragma unroll
  for (int t = 0; t < SL; ++t) { qr[t] = row_ok ? qrow[t] : 0.f; acc[t] = 0.f; }
  float m = -INFINITY, l = 0.f;

  const int r = sc.sched;
  const int e0 = sv.fwd_row_ptr[r], e1 = sv.fwd_row_ptr[r + 1];
  const int nthreads = blockDim.x;
  for (int e = e0; e < e1; ++e) {
    const uint32_t ent = sv.fwd_ent[e];
    const int j = (int)(ent >> 1);
    const bool partial = ent & 1u;
    for (int c0 = 0; c0 < tk; c0 += kChunk) {
      const int64_t kfirst = (int64_t)j * tk + c0;
      __syncthreads();
      for (int x = tid; x < kChunk * D; x += nthreads) {
        const int kk = x / D, dd = x % D;
        const int64_t kp = kfirst + kk;
        const bool ok = kp < n_k;
        ks[kk][dd] = ok ? kbase[kp * D + dd] : 0.f;
        vs[kk][dd] = ok ? vbase[kp * D + dd] : 0.f;
      }
      __syncthreads();
      for (int k8 = 0; k8 < kChunk; k8 += 8) {
        float s[8];
        float mx = -INFINITY;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int kk = k8 + u;
          float part = 0.f;
#pragma unroll
          for (int t = 0; t < SL; ++t) part = fmaf(qr[t], ks[kk][sub * SL + t], part);
          part += __shfl_xor(part, 1, 8);
          part += __shfl_xor(part, 2, 8);
          part += __shfl_xor(part, 4, 8);
          float sv2 = part * c;
          const int64_t kp = kfirst + kk;
          if (kp >= n_k || (partial && !legal32(sc.g, (int)qpos, (int)kp))) sv2 = -INFINITY;
          s[u] = sv2;
          mx = fmaxf(mx, sv2);
        }
        const float m_new = fmaxf(m, mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2f(m - m_use);
        float psum = 0.f;
#pragma unroll
        for (int t = 0; t < SL; ++t) acc[t] *= alpha;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const float pu = exp2f(s[u] - m_use);
          psum += pu;
#pragma unroll
          for (int t = 0; t < SL; ++t) acc[t] = fmaf(pu, vs[k8 + u][sub * SL + t], acc[t]);
        }
        l = l * alpha + psum;
        m = m_new;
      }
    }
  }
  if (!row_ok) return;
  float* orow = o + (row_base + qpos) * D + sub * SL;
  const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
  for (int t = 0; t < SL; ++t) orow[t] = acc[t] * inv;
  if (sub == 0)
    lse[row_base + qpos] = l > 0.f ? (m + log2f(l)) * 0.6931471805599453f : -INFINITY;
}

}  // namespace

hipError_t launch_fwd_fp32(const cowa_params& p, const SchedView& sv, const float* q, const float* k,
                           const float* v, float* o, float* lse, hipStream_t stream) {
  dim3 grid(sv.n_qt, p.h_q, sv.ragged ? 1 : p.batch), block(p.tile_q * 8);
  if (p.head_dim == 64)
    hipLaunchKernelGGL(fwd_fp32_kernel<64>, grid, block, 0, stream, p, sv, q, k, v, o, lse);
  else
    hipLaunchKernelGGL(fwd_fp32_kernel<128>, grid, block, 0, stream, p, sv, q, k, v, o, lse);
  return hipGetLastError();
}

}  // namespace cowa
