// Block-schedule builder (Sec. 2.3): J_h(i) per (local KV head, QO block) with
// KV blocks descending (the order of Alg. 1) and the inverse I_h(j) per (local
// KV head, KV block) with QO blocks ascending (the order of Alg. 2), each entry
// flagged FULL or partial (only partial blocks need the element mask).
//
// Three launches on the caller's stream: per-row counts, an in-place prefix
// sum of the counts (one workgroup per array), and the entry fill (one wave
// per row or column, lanes writing consecutive entries).
#include "internal.h"
#include "window_rule.h"

namespace cowa {
namespace {

struct SchedArgs {
  int32_t n_q, n_k, w_sink, w_near, tile_q, tile_k, h_k, h_total, h_offset, n_qt, n_kt;
  int32_t* fwd_row_ptr;
  int32_t* bwd_col_ptr;
  uint32_t* fwd_ent;
  uint32_t* bwd_ent;
};

__device__ inline HeadGeo geo_of(const SchedArgs& a, int32_t h) {
  return make_geo(a.n_q, a.n_k, a.w_sink, a.w_near, a.tile_q, a.tile_k, a.h_offset + h, a.h_total);
}

// Counts go to ptr[r + 1]; ptr[0] = 0.
__global__ void sched_count(SchedArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nf = (int64_t)a.h_k * a.n_qt, nb = (int64_t)a.h_k * a.n_kt;
  if (t < nf) {
    const int32_t h = (int32_t)(t / a.n_qt), i = (int32_t)(t % a.n_qt);
    a.fwd_row_ptr[t + 1] = ranges_count(fwd_block_ranges(geo_of(a, h), i));
    if (t == 0) a.fwd_row_ptr[0] = 0;
  } else if (t < nf + nb) {
    const int64_t c = t - nf;
    const int32_t h = (int32_t)(c / a.n_kt), j = (int32_t)(c % a.n_kt);
    a.bwd_col_ptr[c + 1] = ranges_count(bwd_block_ranges(geo_of(a, h), j));
    if (c == 0) a.bwd_col_ptr[0] = 0;
  }
}

// Inclusive scan of ptr[1..n] in place; block 0 scans the forward rows,
// block 1 the backward columns.  Chunks of 1024 with a running carry.
__global__ void __launch_bounds__(1024) sched_scan(SchedArgs a) {
  __shared__ int32_t buf[1024];
  __shared__ int32_t carry;
  int32_t* p = blockIdx.x == 0 ? a.fwd_row_ptr : a.bwd_col_ptr;
  const int64_t n = (int64_t)a.h_k * (blockIdx.x == 0 ? a.n_qt : a.n_kt);
  const int tid = threadIdx.x;
  if (tid == 0) carry = 0;
  __syncthreads();
  for (int64_t base = 0; base < n; base += 1024) {
    const int64_t idx = base + tid;
    buf[tid] = idx < n ? p[idx + 1] : 0;
    __syncthreads();
    for (int off = 1; off < 1024; off <<= 1) {
      const int32_t add = tid >= off ? buf[tid - off] : 0;
      __syncthreads();
      buf[tid] += add;
      __syncthreads();
    }
    if (idx < n) p[idx + 1] = buf[tid] + carry;
    __syncthreads();
    if (tid == 1023) carry += buf[1023];
    __syncthreads();
  }
}

// One 64-lane wave per forward row or backward column.
__global__ void sched_fill(SchedArgs a) {
  const int64_t w = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t nf = (int64_t)a.h_k * a.n_qt, nb = (int64_t)a.h_k * a.n_kt;
  if (w < nf) {
    const int32_t h = (int32_t)(w / a.n_qt), i = (int32_t)(w % a.n_qt);
    const HeadGeo g = geo_of(a, h);
    const Ranges r = fwd_block_ranges(g, i);
    const int32_t cnt = ranges_count(r);
    uint32_t* out = a.fwd_ent + a.fwd_row_ptr[w];
    for (int32_t t = lane; t < cnt; t += 64) {
      int32_t rem = t, j = 0;
      for (int x = r.n - 1; x >= 0; --x) {  // descending over the merged ranges
        const int32_t sz = r.b[x] - r.a[x] + 1;
        if (rem < sz) { j = r.b[x] - rem; break; }
        rem -= sz;
      }
      out[t] = ((uint32_t)j << 1) | (tile_full(g, i, j) ? 0u : 1u);
    }
  } else if (w < nf + nb) {
    const int64_t c = w - nf;
    const int32_t h = (int32_t)(c / a.n_kt), j = (int32_t)(c % a.n_kt);
    const HeadGeo g = geo_of(a, h);
    const Ranges r = bwd_block_ranges(g, j);
    const int32_t cnt = ranges_count(r);
    uint32_t* out = a.bwd_ent + a.bwd_col_ptr[c];
    for (int32_t t = lane; t < cnt; t += 64) {
      int32_t rem = t, i = 0;
      for (int x = 0; x < r.n; ++x) {  // ascending
        const int32_t sz = r.b[x] - r.a[x] + 1;
        if (rem < sz) { i = r.a[x] + rem; break; }
        rem -= sz;
      }
      out[t] = ((uint32_t)i << 1) | (tile_full(g, i, j) ? 0u : 1u);
    }
  }
}

}  // namespace

hipError_t launch_schedule(const cowa_schedule_t* s, hipStream_t stream) {
  char* b = static_cast<char*>(s->buf);
  SchedArgs a;
  a.n_q = s->p.n_q; a.n_k = s->p.n_k; a.w_sink = s->p.w_sink; a.w_near = s->p.w_near;
  a.tile_q = s->p.tile_q; a.tile_k = s->p.tile_k; a.h_k = s->p.h_k; a.h_total = s->p.h_k_total;
  a.h_offset = s->p.h_k_offset; a.n_qt = s->n_qt; a.n_kt = s->n_kt;
  a.fwd_row_ptr = reinterpret_cast<int32_t*>(b + s->off_fwd_row_ptr);
  a.bwd_col_ptr = reinterpret_cast<int32_t*>(b + s->off_bwd_col_ptr);
  a.fwd_ent = reinterpret_cast<uint32_t*>(b + s->off_fwd_ent);
  a.bwd_ent = reinterpret_cast<uint32_t*>(b + s->off_bwd_ent);
  const int64_t rows = (int64_t)a.h_k * (a.n_qt + a.n_kt);
  hipLaunchKernelGGL(sched_count, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, stream, a);
  hipLaunchKernelGGL(sched_scan, dim3(2), dim3(1024), 0, stream, a);
  hipLaunchKernelGGL(sched_fill, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace cowa
