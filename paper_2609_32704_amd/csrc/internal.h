// Internal launchers of the CoWA library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cowa.h"

namespace cowa {

// Device view of a built schedule.
struct SchedView {
  const int32_t* fwd_row_ptr;
  const int32_t* bwd_col_ptr;
  const uint32_t* fwd_ent;
  const uint32_t* bwd_ent;
  int32_t n_qt, n_kt;
};

inline SchedView sched_view(const cowa_schedule_t* s) {
  const char* b = static_cast<const char*>(s->buf);
  SchedView v;
  v.fwd_row_ptr = reinterpret_cast<const int32_t*>(b + s->off_fwd_row_ptr);
  v.bwd_col_ptr = reinterpret_cast<const int32_t*>(b + s->off_bwd_col_ptr);
  v.fwd_ent = reinterpret_cast<const uint32_t*>(b + s->off_fwd_ent);
  v.bwd_ent = reinterpret_cast<const uint32_t*>(b + s->off_bwd_ent);
  v.n_qt = s->n_qt;
  v.n_kt = s->n_kt;
  return v;
}

// Raise a kernel's dynamic LDS limit to `bytes`, once per (kernel, device);
// thread-safe.  Called by the launchers before their first launch on a device.
hipError_t allow_lds(const void* kernel, int bytes);

// Each launcher enqueues on `stream` and returns hipGetLastError() of its launches.
hipError_t launch_schedule(const cowa_schedule_t* s, hipStream_t stream);

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

// Backward stages (Alg. 2): D = rowsum(O * dO); the dK/dV pass; the dQ pass.
hipError_t launch_bwd_prepare(const cowa_params& p, const void* o, const void* d_o, float* dsum,
                              hipStream_t stream);
hipError_t launch_bwd_main(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                           const float* lse, const void* d_o, void* dk, void* dv, const float* dsum,
                           hipStream_t stream);
hipError_t launch_bwd_dq(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                         const float* lse, const void* d_o, void* dq, const float* dsum, hipStream_t stream);

bool decode_supported(int head_dim, int group);
size_t decode_workspace_bytes(const cowa_decode_params& p);
int32_t decode_num_splits(const cowa_decode_params& p);
int32_t decode_split_keys(const cowa_decode_params& p);

hipError_t launch_decode(const cowa_decode_params& p, const void* q, const void* k_cache,
                         const void* v_cache, const int32_t* seqlens, void* o, float* lse, void* ws,
                         hipStream_t stream);

}  // namespace cowa
