// Internal launchers of the CoWA library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cowa.h"

namespace cowa {

// One sequence of a ragged batch (a table in the schedule buffer).
struct SeqDesc {
  int32_t q_start, k_start;  // first query / key position in the packed [H, N_total, d] tensors
  int32_t n_q, n_k;          // its lengths
  int32_t qt_off, kt_off;    // its first QO / KV block over the batch
  int32_t pad0, pad1;
};

// Resolved window of one KV head (a table in the schedule buffer): sink and
// near widths and the long-range distance bounds [lo, hi), clamped to 2^30
// (a causal distance is always below N_k < 2^30).
struct WinDesc {
  int32_t sink, near, lo, hi;
};

// Device view of a built schedule.
struct SchedView {
  const int32_t* fwd_row_ptr;
  const int32_t* bwd_col_ptr;
  const uint32_t* fwd_ent;
  const uint32_t* bwd_ent;
  const WinDesc* win;     // [n_win][h_k]: n_win = batch for a ragged batch under the default rule, else 1
  const SeqDesc* seq;     // [batch], ragged batches only
  const int32_t* qt_seq;  // [n_qt]: sequence of each QO block, ragged batches only
  const int32_t* kt_seq;  // [n_kt]: sequence of each KV block, ragged batches only
  int32_t n_qt, n_kt;     // QO / KV blocks: of one sequence (fixed lengths) or of the whole batch (ragged)
  int32_t max_qt, max_kt; // QO / KV blocks of the longest sequence
  int32_t ragged, per_seq_win;
};

inline SchedView sched_view(const cowa_schedule_t* s) {
  const char* b = static_cast<const char*>(s->buf);
  const bool ragged = s->p.cu_seqlens_q != nullptr;
  SchedView v;
  v.fwd_row_ptr = reinterpret_cast<const int32_t*>(b + s->off_fwd_row_ptr);
  v.bwd_col_ptr = reinterpret_cast<const int32_t*>(b + s->off_bwd_col_ptr);
  v.fwd_ent = reinterpret_cast<const uint32_t*>(b + s->off_fwd_ent);
  v.bwd_ent = reinterpret_cast<const uint32_t*>(b + s->off_bwd_ent);
  v.win = reinterpret_cast<const WinDesc*>(b + s->off_windows);
  v.seq = ragged ? reinterpret_cast<const SeqDesc*>(b + s->off_seqs) : nullptr;
  v.qt_seq = ragged ? reinterpret_cast<const int32_t*>(b + s->off_qt_seq) : nullptr;
  v.kt_seq = ragged ? reinterpret_cast<const int32_t*>(b + s->off_kt_seq) : nullptr;
  v.n_qt = s->n_qt;
  v.n_kt = s->n_kt;
  v.max_qt = s->max_qt;
  v.max_kt = s->max_kt;
  v.ragged = ragged ? 1 : 0;
  v.per_seq_win = (ragged && s->p.windows == nullptr) ? 1 : 0;
  return v;
}

// Query rows (of d elements) in Q, O and dO: B H_q N_q, or H_q N_total when ragged.
inline int64_t q_rows(const cowa_params& p) {
  return (p.cu_seqlens_q ? 1 : (int64_t)p.batch) * p.h_q * p.n_q;
}

// Raise a kernel's dynamic LDS limit to `bytes`, once per (kernel, device);
// thread-safe.  Called by the launchers before their first launch on a device.
hipError_t allow_lds(const void* kernel, int bytes);

// Each launcher enqueues on `stream` and returns hipGetLastError() of its launches.
// Builds the schedule: uploads the host tables (windows, then the sequence
// table of a ragged batch; `tables` holds their bytes laid out as in the
// buffer from off_windows on), then counts, scans and fills the block lists.
hipError_t launch_schedule(const cowa_schedule_t* s, const void* tables, size_t table_bytes, hipStream_t stream);

hipError_t launch_fwd_fp32(const cowa_params& p, const SchedView& sv, const float* q, const float* k,
                           const float* v, float* o, float* lse, hipStream_t stream);

// the bf16 forward keeps one row's block list in LDS: at most this many key blocks
int fwd_bf16_max_kblocks(int head_dim, int tile_k);
bool fwd_bf16_supported(int head_dim, int tile_q, int tile_k);
bool bwd_bf16_supported(int head_dim, int tile_q, int tile_k);
// the dK/dV pass keeps one column's block list in LDS: at most this many query blocks
int bwd_main_max_qblocks(int head_dim, int tile_k);
// the dQ pass keeps one row's block list in LDS: at most this many key blocks
int bwd_dq_max_kblocks(int head_dim, int tile_k);

hipError_t launch_fwd_bf16(const cowa_params& p, const SchedView& sv, const void* q, const void* k,
                           const void* v, void* o, float* lse, hipStream_t stream);

// Split of the dK/dV pass's heaviest columns.  Every query that reaches a sink
// key sees it, so the sink KV blocks have query lists as long as the sequence
// while every other column holds only its near and long-range runs; walked by
// one workgroup, a sink column would set the pass's length whenever the other
// columns do not fill the device for longer (one KV head per device, short or
// few sequences).  The first S KV blocks of every (sequence, KV head) are
// therefore walked by P workgroups, each taking a contiguous share of the
// column's steps and writing float32 partial dK and dV; a reduction kernel
// sums the P partials of a column in a fixed order (deterministic) and writes
// bf16.  P = 1: no split.
struct BwdSplit {
  int32_t S = 0, P = 1;  // leading KV blocks split per (sequence, KV head); parts per column
  int64_t n_cols = 0;    // split columns: sequences x KV heads x S
};
// float32 partial bytes of a column part: dK and dV of one KV block
inline size_t bwd_part_floats(const cowa_params& p) { return (size_t)2 * p.tile_k * p.head_dim; }

// Backward workspace: per query row (layout of LSE), nd = -D with
// D = rowsum(O * dO) (the term of Alg. 2), then nl = -LSE log2(e); then the
// float32 partials of the split dK/dV columns; each array 256-byte aligned.
struct BwdWork {
  float* nd;
  float* nl;
  float* part;  // [n_cols][P][2][tile_k * head_dim], or null when P = 1
  BwdSplit split;
};
inline size_t bwd_array_bytes(const cowa_params& p) { return ((size_t)q_rows(p) * sizeof(float) + 255) & ~size_t(255); }
inline size_t bwd_split_bytes(const cowa_params& p, const BwdSplit& s) {
  return s.P > 1 ? (((size_t)s.n_cols * s.P * bwd_part_floats(p) * sizeof(float) + 255) & ~size_t(255)) : 0;
}
inline size_t bwd_workspace_bytes(const cowa_params& p, const BwdSplit& s) {
  return 2 * bwd_array_bytes(p) + bwd_split_bytes(p, s);
}
inline BwdWork bwd_work(const cowa_params& p, const BwdSplit& s, void* ws) {
  BwdWork w;
  w.nd = static_cast<float*>(ws);
  w.nl = reinterpret_cast<float*>(static_cast<char*>(ws) + bwd_array_bytes(p));
  w.part = s.P > 1 ? reinterpret_cast<float*>(static_cast<char*>(ws) + 2 * bwd_array_bytes(p)) : nullptr;
  w.split = s;
  return w;
}

// Backward stages (Alg. 2): the row values; the dK/dV pass; the dQ pass.
hipError_t launch_bwd_prepare(const cowa_params& p, const void* o, const void* d_o, const float* lse,
                              const BwdWork& w, hipStream_t stream);
hipError_t launch_bwd_main(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                           const void* d_o, void* dk, void* dv, const BwdWork& w, hipStream_t stream);
hipError_t launch_bwd_dq(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                         const void* d_o, void* dq, const BwdWork& w, hipStream_t stream);
// the pipelined dQ pass on 32x32 products (128-key blocks, four-wave
// workgroups); launch_bwd_dq uses it where supported
bool bwd_dq32_supported(const cowa_params& p);
hipError_t launch_bwd_dq32(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                           const void* d_o, void* dq, const BwdWork& w, hipStream_t stream);

bool decode_supported(int head_dim, int group);
size_t decode_workspace_bytes(const cowa_decode_params& p);
int32_t decode_num_splits(const cowa_decode_params& p);
int32_t decode_split_keys(const cowa_decode_params& p);

// decode with explicit windows: at most this many local KV heads
constexpr int kDecodeMaxExplicitHeads = 256;

// The allocation-free decoding entry point keeps its split partials in a
// device array of this many bytes (per GPU); decode_scratch() gives the
// current device's address of it (looked up once per device).
constexpr size_t kDecodeScratchBytes = size_t(32) << 20;
hipError_t decode_scratch(void** ptr);

hipError_t launch_decode(const cowa_decode_params& p, const void* q, const void* k_cache,
                         const void* v_cache, const int32_t* seqlens, void* o, float* lse, void* ws,
                         hipStream_t stream);

}  // namespace cowa
