// Block-schedule builder (Sec. 2.3): J_h(i) per (local KV head, QO block) with
// KV blocks descending (the order of Alg. 1) and the inverse I_h(j) per (local
// KV head, KV block) with QO blocks ascending (the order of Alg. 2), each entry
// flagged FULL or partial (only partial blocks need the element mask).
//
// Launches on the caller's stream: the host-resolved window table (and, for a
// ragged batch, the sequence table) copied in through kernel arguments; for a
// ragged batch the block-to-sequence maps; then per-row counts, an in-place
// prefix sum of the counts (one workgroup per array), and the entry fill (one
// wave per row or column, lanes writing consecutive entries).
#include <algorithm>
#include <cstring>

#include "internal.h"
#include "window_rule.h"

namespace cowa {
namespace {

// Words copied per launch through the kernel arguments.
constexpr int kPutWords = 480;
struct PutArgs {
  uint32_t* dst;
  int32_t n;
  uint32_t w[kPutWords];
};

__global__ void __launch_bounds__(512) put_words(PutArgs a) {
  const int t = threadIdx.x;
  if (t < a.n) a.dst[t] = a.w[t];
}

struct SchedArgs {
  cowa_params p;
  SchedView sv;  // read-only view of the tables
  int32_t* fwd_row_ptr;
  int32_t* bwd_col_ptr;
  uint32_t* fwd_ent;
  uint32_t* bwd_ent;
  int32_t* qt_seq;
  int32_t* kt_seq;
};

// Block-to-sequence maps of a ragged batch: the last sequence whose first
// block is at or before the block (binary search over the sequence table;
// sequences without blocks share their first block index with the next one
// and are skipped by taking the last match).
__global__ void sched_tile_map(SchedArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int nq = a.sv.n_qt, nk = a.sv.n_kt, nb = a.p.batch;
  if (t >= (int64_t)nq + nk) return;
  const bool qside = t < nq;
  const int tile = qside ? (int)t : (int)(t - nq);
  int lo = 0, hi = nb - 1;  // answer in [lo, hi]
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    const int off = qside ? a.sv.seq[mid].qt_off : a.sv.seq[mid].kt_off;
    if (off <= tile) lo = mid; else hi = mid - 1;
  }
  (qside ? a.qt_seq : a.kt_seq)[tile] = lo;
}

// Geometry of (local KV head h, block row) on the QO (qside) or KV side.
__device__ inline HeadGeo row_geo(const SchedArgs& a, int h, int row, bool qside, int* tile) {
  const SchedView& sv = a.sv;
  int32_t n_q = a.p.n_q, n_k = a.p.n_k, b = 0;
  *tile = row;
  if (sv.ragged) {
    b = (qside ? sv.qt_seq : sv.kt_seq)[row];
    const SeqDesc sd = sv.seq[b];
    n_q = sd.n_q;
    n_k = sd.n_k;
    *tile = row - (qside ? sd.qt_off : sd.kt_off);
  }
  const WinDesc w = sv.win[(sv.per_seq_win ? b * a.p.h_k : 0) + h];
  return make_geo_bounds(n_q, n_k, w.sink, w.near, w.lo, w.hi, a.p.tile_q, a.p.tile_k);
}

// Counts go to ptr[r + 1]; ptr[0] = 0.
__global__ void sched_count(SchedArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t nf = (int64_t)a.p.h_k * a.sv.n_qt, nb = (int64_t)a.p.h_k * a.sv.n_kt;
  int tile;
  if (t < nf) {
    const int32_t h = (int32_t)(t / a.sv.n_qt), row = (int32_t)(t % a.sv.n_qt);
    const HeadGeo g = row_geo(a, h, row, true, &tile);
    a.fwd_row_ptr[t + 1] = ranges_count(fwd_block_ranges(g, tile));
    if (t == 0) a.fwd_row_ptr[0] = 0;
  } else if (t < nf + nb) {
    const int64_t c = t - nf;
    const int32_t h = (int32_t)(c / a.sv.n_kt), row = (int32_t)(c % a.sv.n_kt);
    const HeadGeo g = row_geo(a, h, row, false, &tile);
    a.bwd_col_ptr[c + 1] = ranges_count(bwd_block_ranges(g, tile));
    if (c == 0) a.bwd_col_ptr[0] = 0;
  }
}

// Inclusive scan of ptr[1..n] in place; block 0 scans the forward rows,
// block 1 the backward columns.  Chunks of 1024 with a running carry.
__global__ void __launch_bounds__(1024) sched_scan(SchedArgs a) {
  __shared__ int32_t buf[1024];
  __shared__ int32_t carry;
  int32_t* p = blockIdx.x == 0 ? a.fwd_row_ptr : a.bwd_col_ptr;
  const int64_t n = (int64_t)a.p.h_k * (blockIdx.x == 0 ? a.sv.n_qt : a.sv.n_kt);
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
  const int64_t nf = (int64_t)a.p.h_k * a.sv.n_qt, nb = (int64_t)a.p.h_k * a.sv.n_kt;
  int tile;
  if (w < nf) {
    const int32_t h = (int32_t)(w / a.sv.n_qt), row = (int32_t)(w % a.sv.n_qt);
    const HeadGeo g = row_geo(a, h, row, true, &tile);
    const int32_t i = tile;
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
    const int32_t h = (int32_t)(c / a.sv.n_kt), row = (int32_t)(c % a.sv.n_kt);
    const HeadGeo g = row_geo(a, h, row, false, &tile);
    const int32_t j = tile;
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

hipError_t launch_schedule(const cowa_schedule_t* s, const void* tables, size_t table_bytes, hipStream_t stream) {
  char* b = static_cast<char*>(s->buf);
  // the tables: words [off_windows, off_windows + table_bytes) of the buffer
  const uint32_t* words = static_cast<const uint32_t*>(tables);
  const size_t n_words = table_bytes / 4;
  uint32_t* dst = reinterpret_cast<uint32_t*>(b + s->off_windows);
  for (size_t w0 = 0; w0 < n_words; w0 += kPutWords) {
    PutArgs pa;
    pa.dst = dst + w0;
    pa.n = (int32_t)std::min<size_t>(kPutWords, n_words - w0);
    std::memcpy(pa.w, words + w0, 4 * (size_t)pa.n);
    hipLaunchKernelGGL(put_words, dim3(1), dim3(512), 0, stream, pa);
  }
  SchedArgs a;
  a.p = s->p;
  a.sv = sched_view(s);
  a.fwd_row_ptr = reinterpret_cast<int32_t*>(b + s->off_fwd_row_ptr);
  a.bwd_col_ptr = reinterpret_cast<int32_t*>(b + s->off_bwd_col_ptr);
  a.fwd_ent = reinterpret_cast<uint32_t*>(b + s->off_fwd_ent);
  a.bwd_ent = reinterpret_cast<uint32_t*>(b + s->off_bwd_ent);
  a.qt_seq = reinterpret_cast<int32_t*>(b + s->off_qt_seq);
  a.kt_seq = reinterpret_cast<int32_t*>(b + s->off_kt_seq);
  if (a.sv.ragged) {
    const int64_t tiles = (int64_t)s->n_qt + s->n_kt;
    if (tiles > 0)
      hipLaunchKernelGGL(sched_tile_map, dim3((unsigned)((tiles + 255) / 256)), dim3(256), 0, stream, a);
  }
  const int64_t rows = (int64_t)s->p.h_k * (s->n_qt + s->n_kt);
  if (rows > 0) {
    hipLaunchKernelGGL(sched_count, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, stream, a);
    hipLaunchKernelGGL(sched_scan, dim3(2), dim3(1024), 0, stream, a);
    hipLaunchKernelGGL(sched_fill, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, stream, a);
  } else {
    // no blocks at all: the two row-pointer arrays are the single word 0
    PutArgs pa;
    pa.n = 1;
    pa.w[0] = 0;
    pa.dst = reinterpret_cast<uint32_t*>(a.fwd_row_ptr);
    hipLaunchKernelGGL(put_words, dim3(1), dim3(512), 0, stream, pa);
    pa.dst = reinterpret_cast<uint32_t*>(a.bwd_col_ptr);
    hipLaunchKernelGGL(put_words, dim3(1), dim3(512), 0, stream, pa);
  }
  return hipGetLastError();
}

}  // namespace cowa
