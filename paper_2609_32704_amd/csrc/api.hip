// C ABI of the CoWA library: argument validation, sizing, and launches on the
// caller's stream.  Every check runs before the first launch, so a failing call
// writes nothing.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <set>
#include <utility>

#include "internal.h"
#include "window_rule.h"

namespace {

thread_local char g_err[512] = "";

cowa_status fail(cowa_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

bool aligned(const void* ptr, size_t a) { return (reinterpret_cast<uintptr_t>(ptr) % a) == 0; }

cowa_status check_params(const cowa_params* p) {
  if (!p) return fail(COWA_ERR_INVALID_ARG, "params is NULL");
  if (p->batch < 0) return fail(COWA_ERR_INVALID_ARG, "batch must be >= 0 (got %d)", p->batch);
  if (p->n_q < 1 || p->n_k < 1) return fail(COWA_ERR_INVALID_ARG, "n_q and n_k must be >= 1");
  if (p->n_q > p->n_k) return fail(COWA_ERR_INVALID_ARG, "n_q (%d) must not exceed n_k (%d)", p->n_q, p->n_k);
  if (p->n_k >= (1 << 30)) return fail(COWA_ERR_INVALID_ARG, "n_k must be < 2^30");
  if (p->h_q < 1 || p->h_k < 1) return fail(COWA_ERR_INVALID_ARG, "h_q and h_k must be >= 1");
  if (p->h_q % p->h_k != 0) return fail(COWA_ERR_INVALID_ARG, "h_q (%d) must be a multiple of h_k (%d)", p->h_q, p->h_k);
  if (p->w_sink < 0 || p->w_near < 0) return fail(COWA_ERR_INVALID_ARG, "window widths must be >= 0");
  if (p->h_k_total < 1 || p->h_k_offset < 0 || (int64_t)p->h_k_offset + p->h_k > p->h_k_total)
    return fail(COWA_ERR_INVALID_ARG, "need 0 <= h_k_offset and h_k_offset + h_k <= h_k_total (%d + %d > %d)",
                p->h_k_offset, p->h_k, p->h_k_total);
  if (p->tile_q != 32 && p->tile_q != 64 && p->tile_q != 128)
    return fail(COWA_ERR_INVALID_ARG, "tile_q must be 32, 64 or 128 (got %d)", p->tile_q);
  if (p->tile_k != 32 && p->tile_k != 64 && p->tile_k != 128)
    return fail(COWA_ERR_INVALID_ARG, "tile_k must be 32, 64 or 128 (got %d)", p->tile_k);
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(COWA_ERR_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", p->head_dim);
  if (p->dtype != COWA_BF16 && p->dtype != COWA_FP32) return fail(COWA_ERR_INVALID_ARG, "unknown dtype %d", p->dtype);
  if (!std::isfinite(p->softmax_scale) || !(p->softmax_scale > 0.f))
    return fail(COWA_ERR_INVALID_ARG, "softmax_scale must be finite and > 0");
  return COWA_OK;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Every schedule-relevant field must match.
bool same_schedule(const cowa_params* a, const cowa_params* b) {
  return a->n_q == b->n_q && a->n_k == b->n_k && a->h_k == b->h_k && a->w_sink == b->w_sink &&
         a->w_near == b->w_near && a->h_k_total == b->h_k_total && a->h_k_offset == b->h_k_offset &&
         a->tile_q == b->tile_q && a->tile_k == b->tile_k;
}

cowa_status check_schedule(const cowa_params* p, const cowa_schedule_t* s) {
  if (!s) return fail(COWA_ERR_INVALID_ARG, "schedule is NULL");
  if (!same_schedule(p, &s->p)) return fail(COWA_ERR_SCHEDULE_MISMATCH, "schedule was sized for other shapes or windows");
  // the sized fields must be the ones cowa_schedule_size produces
  if (s->n_qt != (p->n_q + p->tile_q - 1) / p->tile_q || s->n_kt != (p->n_k + p->tile_k - 1) / p->tile_k)
    return fail(COWA_ERR_SCHEDULE_MISMATCH, "schedule block counts do not match the params");
  if (!s->buf || !aligned(s->buf, 256)) return fail(COWA_ERR_INVALID_ARG, "schedule buffer is NULL or not 256-byte aligned");
  return COWA_OK;
}

// Device present and gfx950; cached per device id.
cowa_status check_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    (void)hipGetLastError();
    return fail(COWA_ERR_NO_DEVICE, "no HIP device");
  }
  static std::atomic<int> ok_cache[64];  // 0 unknown, 1 ok, -1 not gfx950 (zero-initialised statics)
  const int known = dev < 64 ? ok_cache[dev].load(std::memory_order_acquire) : 0;
  if (known != 0) return known > 0 ? COWA_OK : fail(COWA_ERR_NO_DEVICE, "device %d is not gfx950", dev);
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
    (void)hipGetLastError();
    return fail(COWA_ERR_NO_DEVICE, "cannot query device %d", dev);
  }
  const bool ok = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
  if (dev < 64) ok_cache[dev].store(ok ? 1 : -1, std::memory_order_release);
  return ok ? COWA_OK : fail(COWA_ERR_NO_DEVICE, "device %d is %s, the library is built for gfx950", dev, prop.gcnArchName);
}

cowa_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return COWA_OK;
  return fail(COWA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

cowa_status check_tensor(const void* ptr, const char* name, size_t align) {
  if (!ptr) return fail(COWA_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned(ptr, align)) return fail(COWA_ERR_INVALID_ARG, "%s is not %zu-byte aligned", name, align);
  return COWA_OK;
}

#define COWA_TRY(expr)                     \
  do {                                     \
    cowa_status st_ = (expr);              \
    if (st_ != COWA_OK) return st_;        \
  } while (0)

}  // namespace

namespace cowa {

hipError_t allow_lds(const void* kernel, int bytes) {
  int dev = -1;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  static std::mutex mu;
  static std::set<std::pair<const void*, int>> done;
  std::lock_guard<std::mutex> lock(mu);
  if (done.count({kernel, dev})) return hipSuccess;
  err = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (err == hipSuccess) done.insert({kernel, dev});
  return err;
}

}  // namespace cowa

extern "C" {

const char* cowa_version(void) { return "cowa-mi355x 0.1 (gfx950)"; }

const char* cowa_last_error(void) { return g_err; }

cowa_status cowa_windows(const cowa_params* p, cowa_window* out_host) {
  COWA_TRY(check_params(p));
  if (!out_host) return fail(COWA_ERR_INVALID_ARG, "out_host is NULL");
  for (int h = 0; h < p->h_k; ++h) {
    int64_t lo, hi;
    cowa::long_bounds(p->n_k, p->w_sink, p->w_near, (int64_t)p->h_k_offset + h, p->h_k_total, &lo, &hi);
    out_host[h].sink = p->w_sink;
    out_host[h].near = p->w_near;
    out_host[h].gap = (int32_t)(lo - p->w_near);
    out_host[h].width = (int32_t)(hi - lo);
  }
  return COWA_OK;
}

cowa_status cowa_schedule_size(const cowa_params* p, cowa_schedule_t* out) {
  COWA_TRY(check_params(p));
  if (!out) return fail(COWA_ERR_INVALID_ARG, "out is NULL");
  const int32_t n_qt = (p->n_q + p->tile_q - 1) / p->tile_q;
  const int32_t n_kt = (p->n_k + p->tile_k - 1) / p->tile_k;
  int64_t nnz = 0, nnz_b = 0;
  int32_t max_row = 0, max_col = 0;
  for (int h = 0; h < p->h_k; ++h) {
    const cowa::HeadGeo g = cowa::make_geo(p->n_q, p->n_k, p->w_sink, p->w_near, p->tile_q, p->tile_k,
                                           p->h_k_offset + h, p->h_k_total);
    for (int32_t i = 0; i < n_qt; ++i) {
      const int32_t c = cowa::ranges_count(cowa::fwd_block_ranges(g, i));
      nnz += c;
      if (c > max_row) max_row = c;
    }
    for (int32_t j = 0; j < n_kt; ++j) {
      const int32_t c = cowa::ranges_count(cowa::bwd_block_ranges(g, j));
      nnz_b += c;
      if (c > max_col) max_col = c;
    }
  }
  if (nnz != nnz_b) return fail(COWA_ERR_INVALID_ARG, "internal: block-set sizes disagree (%lld vs %lld)",
                                (long long)nnz, (long long)nnz_b);
  if (nnz >= (int64_t(1) << 31)) return fail(COWA_ERR_UNSUPPORTED, "schedule has more than 2^31 entries");
  std::memset(out, 0, sizeof(*out));
  out->p = *p;
  out->n_qt = n_qt;
  out->n_kt = n_kt;
  out->max_row = max_row;
  out->max_col = max_col;
  out->nnz = nnz;
  size_t off = 0;
  out->off_fwd_row_ptr = off;
  off = align256(off + 4 * ((size_t)p->h_k * n_qt + 1));
  out->off_bwd_col_ptr = off;
  off = align256(off + 4 * ((size_t)p->h_k * n_kt + 1));
  out->off_fwd_ent = off;
  off = align256(off + 4 * (size_t)nnz);
  out->off_bwd_ent = off;
  off = align256(off + 4 * (size_t)nnz);
  out->bytes = off;
  out->buf = nullptr;
  return COWA_OK;
}

cowa_status cowa_legal_pairs(const cowa_params* p, int64_t* pairs) {
  COWA_TRY(check_params(p));
  if (!pairs) return fail(COWA_ERR_INVALID_ARG, "pairs is NULL");
  const int64_t off = (int64_t)p->n_k - p->n_q;
  int64_t total = 0;
  for (int h = 0; h < p->h_k; ++h) {
    int64_t lo, hi;
    cowa::long_bounds(p->n_k, p->w_sink, p->w_near, (int64_t)p->h_k_offset + h, p->h_k_total, &lo, &hi);
    for (int64_t iq = 0; iq < p->n_q; ++iq)  // runs of the query whose distance-0 key is iq + off
      total += cowa::ranges_count(cowa::decode_key_runs(iq + off + 1, p->w_sink, p->w_near, lo, hi));
  }
  *pairs = total * (p->h_q / p->h_k) * (int64_t)p->batch;
  return COWA_OK;
}

cowa_status cowa_decode_visible_keys(const cowa_decode_params* p, const int32_t* seqlens_host, int64_t* keys) {
  if (!p || !seqlens_host || !keys) return fail(COWA_ERR_INVALID_ARG, "NULL argument");
  if (p->batch < 0 || p->h_k < 1 || p->h_k_total < 1 || p->h_k_offset < 0 ||
      (int64_t)p->h_k_offset + p->h_k > p->h_k_total || p->w_sink < 0 || p->w_near < 0)
    return fail(COWA_ERR_INVALID_ARG, "invalid decode parameters");
  int64_t total = 0;
  for (int b = 0; b < p->batch; ++b) {
    const int64_t n_k = seqlens_host[b];
    if (n_k < 1 || n_k > p->n_max) continue;
    for (int h = 0; h < p->h_k; ++h) {
      int64_t lo, hi;
      cowa::long_bounds(n_k, p->w_sink, p->w_near, (int64_t)p->h_k_offset + h, p->h_k_total, &lo, &hi);
      total += cowa::ranges_count(cowa::decode_key_runs(n_k, p->w_sink, p->w_near, lo, hi));
    }
  }
  *keys = total;
  return COWA_OK;
}

cowa_status cowa_schedule(const cowa_schedule_t* s, void* stream) {
  if (!s) return fail(COWA_ERR_INVALID_ARG, "schedule is NULL");
  COWA_TRY(check_params(&s->p));
  cowa_schedule_t ref;
  COWA_TRY(cowa_schedule_size(&s->p, &ref));
  if (ref.nnz != s->nnz || ref.bytes != s->bytes || ref.n_qt != s->n_qt || ref.n_kt != s->n_kt ||
      ref.off_fwd_ent != s->off_fwd_ent || ref.off_bwd_ent != s->off_bwd_ent ||
      ref.off_bwd_col_ptr != s->off_bwd_col_ptr)
    return fail(COWA_ERR_SCHEDULE_MISMATCH, "schedule fields were not produced by cowa_schedule_size for its params");
  if (!s->buf || !aligned(s->buf, 256)) return fail(COWA_ERR_INVALID_ARG, "schedule buffer is NULL or not 256-byte aligned");
  COWA_TRY(check_device());
  return hip_status(cowa::launch_schedule(s, static_cast<hipStream_t>(stream)), "schedule launch");
}

cowa_status cowa_fwd(const cowa_params* p, const cowa_schedule_t* s, const void* q, const void* k, const void* v,
                     void* o, float* lse, void* stream) {
  COWA_TRY(check_params(p));
  COWA_TRY(check_schedule(p, s));
  if (p->batch == 0) return COWA_OK;
  COWA_TRY(check_tensor(q, "q", 16));
  COWA_TRY(check_tensor(k, "k", 16));
  COWA_TRY(check_tensor(v, "v", 16));
  COWA_TRY(check_tensor(o, "o", 16));
  COWA_TRY(check_tensor(lse, "lse", 4));
  if ((int64_t)s->n_qt * p->h_q * p->batch >= (int64_t(1) << 31))
    return fail(COWA_ERR_UNSUPPORTED, "too many query blocks for one launch");
  if (p->dtype == COWA_BF16 && !cowa::fwd_bf16_supported(p->head_dim, p->tile_q, p->tile_k))
    return fail(COWA_ERR_UNSUPPORTED, "bf16 forward is built for tile_q and tile_k in {64, 128} (got %d x %d)", p->tile_q, p->tile_k);
  if (p->dtype == COWA_BF16 && s->n_kt > cowa::fwd_bf16_max_kblocks(p->head_dim, p->tile_k))
    return fail(COWA_ERR_UNSUPPORTED, "bf16 forward supports at most %d key blocks (got %d)",
                cowa::fwd_bf16_max_kblocks(p->head_dim, p->tile_k), s->n_kt);
  COWA_TRY(check_device());
  const cowa::SchedView sv = cowa::sched_view(s);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (p->dtype == COWA_FP32)
    return hip_status(cowa::launch_fwd_fp32(*p, sv, static_cast<const float*>(q), static_cast<const float*>(k),
                                            static_cast<const float*>(v), static_cast<float*>(o), lse, st),
                      "fp32 forward launch");
  return hip_status(cowa::launch_fwd_bf16(*p, sv, q, k, v, o, lse, st), "bf16 forward launch");
}

cowa_status cowa_bwd_workspace_size(const cowa_params* p, size_t* bytes) {
  COWA_TRY(check_params(p));
  if (!bytes) return fail(COWA_ERR_INVALID_ARG, "bytes is NULL");
  const size_t rows = (size_t)p->batch * p->h_q * p->n_q;
  *bytes = align256(rows * sizeof(float));
  return COWA_OK;
}

// Checks shared by the backward stages; the workspace holds D = rowsum(O * dO).
static cowa_status check_bwd(const cowa_params* p, size_t ws_bytes, void* workspace, float** dsum) {
  COWA_TRY(check_params(p));
  if (p->dtype != COWA_BF16) return fail(COWA_ERR_UNSUPPORTED, "backward is built for bf16 only");
  if (!cowa::bwd_bf16_supported(p->head_dim, p->tile_q, p->tile_k))
    return fail(COWA_ERR_UNSUPPORTED, "bf16 backward is built for tile_q, tile_k in {64, 128} (got %d x %d)",
                p->tile_q, p->tile_k);
  // the dK/dV pass keeps a column's block list, the dQ pass a row's, in LDS
  const int64_t n_qt = ((int64_t)p->n_q + p->tile_q - 1) / p->tile_q;
  const int64_t n_kt = ((int64_t)p->n_k + p->tile_k - 1) / p->tile_k;
  if (n_qt > cowa::bwd_main_max_qblocks(p->head_dim, p->tile_k))
    return fail(COWA_ERR_UNSUPPORTED, "backward supports at most %d query blocks (got %lld)",
                cowa::bwd_main_max_qblocks(p->head_dim, p->tile_k), (long long)n_qt);
  if (n_kt > cowa::bwd_dq_max_kblocks(p->head_dim, p->tile_k))
    return fail(COWA_ERR_UNSUPPORTED, "backward supports at most %d key blocks (got %lld)",
                cowa::bwd_dq_max_kblocks(p->head_dim, p->tile_k), (long long)n_kt);
  // one workgroup per (KV block, KV head, sequence) in the dK/dV pass and per
  // (QO block, QO head, sequence) at most in the dQ pass: grid limit 2^31
  if (n_kt * p->h_k * p->batch >= (int64_t(1) << 31))
    return fail(COWA_ERR_UNSUPPORTED, "too many key blocks for one launch");
  if (n_qt * p->h_q * p->batch >= (int64_t(1) << 31))
    return fail(COWA_ERR_UNSUPPORTED, "too many query blocks for one launch");
  size_t need = 0;
  COWA_TRY(cowa_bwd_workspace_size(p, &need));
  if (p->batch > 0 && (!workspace || ws_bytes < need || !aligned(workspace, 256)))
    return fail(COWA_ERR_WORKSPACE, "backward needs a 256-byte aligned workspace of %zu bytes (got %zu)", need, ws_bytes);
  *dsum = static_cast<float*>(workspace);
  return COWA_OK;
}

// Pointer checks of each stage (after check_bwd; batch > 0).
static cowa_status check_prepare_ptrs(const void* o, const void* d_o) {
  COWA_TRY(check_tensor(o, "o", 16));
  return check_tensor(d_o, "d_o", 16);
}

static cowa_status check_qkv_lse_do(const void* q, const void* k, const void* v, const float* lse, const void* d_o) {
  COWA_TRY(check_tensor(q, "q", 16));
  COWA_TRY(check_tensor(k, "k", 16));
  COWA_TRY(check_tensor(v, "v", 16));
  COWA_TRY(check_tensor(lse, "lse", 4));
  return check_tensor(d_o, "d_o", 16);
}

static cowa_status check_main_ptrs(const void* q, const void* k, const void* v, const float* lse, const void* d_o,
                                   const void* dk, const void* dv) {
  COWA_TRY(check_qkv_lse_do(q, k, v, lse, d_o));
  COWA_TRY(check_tensor(dk, "dk", 16));
  return check_tensor(dv, "dv", 16);
}

static cowa_status check_dq_ptrs(const void* q, const void* k, const void* v, const float* lse, const void* d_o,
                                 const void* dq) {
  COWA_TRY(check_qkv_lse_do(q, k, v, lse, d_o));
  return check_tensor(dq, "dq", 16);
}

cowa_status cowa_bwd_prepare(const cowa_params* p, const void* o, const void* d_o, void* workspace, size_t ws_bytes,
                             void* stream) {
  float* dsum;
  COWA_TRY(check_bwd(p, ws_bytes, workspace, &dsum));
  if (p->batch == 0) return COWA_OK;
  COWA_TRY(check_prepare_ptrs(o, d_o));
  COWA_TRY(check_device());
  return hip_status(cowa::launch_bwd_prepare(*p, o, d_o, dsum, static_cast<hipStream_t>(stream)),
                    "backward prepare launch");
}

cowa_status cowa_bwd_main(const cowa_params* p, const cowa_schedule_t* s, const void* q, const void* k,
                          const void* v, const float* lse, const void* d_o, void* dk, void* dv, void* workspace,
                          size_t ws_bytes, void* stream) {
  float* dsum;
  COWA_TRY(check_bwd(p, ws_bytes, workspace, &dsum));
  COWA_TRY(check_schedule(p, s));
  if (p->batch == 0) return COWA_OK;
  COWA_TRY(check_main_ptrs(q, k, v, lse, d_o, dk, dv));
  COWA_TRY(check_device());
  return hip_status(cowa::launch_bwd_main(*p, cowa::sched_view(s), q, k, v, lse, d_o, dk, dv, dsum,
                                          static_cast<hipStream_t>(stream)),
                    "backward dK/dV launch");
}

cowa_status cowa_bwd_dq(const cowa_params* p, const cowa_schedule_t* s, const void* q, const void* k, const void* v,
                        const float* lse, const void* d_o, void* dq, void* workspace, size_t ws_bytes,
                        void* stream) {
  float* dsum;
  COWA_TRY(check_bwd(p, ws_bytes, workspace, &dsum));
  COWA_TRY(check_schedule(p, s));
  if (p->batch == 0) return COWA_OK;
  COWA_TRY(check_dq_ptrs(q, k, v, lse, d_o, dq));
  COWA_TRY(check_device());
  return hip_status(cowa::launch_bwd_dq(*p, cowa::sched_view(s), q, k, v, lse, d_o, dq, dsum,
                                        static_cast<hipStream_t>(stream)),
                    "backward dQ launch");
}

// All three stages; every check of every stage runs before the first launch.
cowa_status cowa_bwd(const cowa_params* p, const cowa_schedule_t* s, const void* q, const void* k, const void* v,
                     const void* o, const float* lse, const void* d_o, void* dq, void* dk, void* dv, void* workspace,
                     size_t ws_bytes, void* stream) {
  float* dsum;
  COWA_TRY(check_bwd(p, ws_bytes, workspace, &dsum));
  COWA_TRY(check_schedule(p, s));
  if (p->batch == 0) return COWA_OK;
  COWA_TRY(check_prepare_ptrs(o, d_o));
  COWA_TRY(check_main_ptrs(q, k, v, lse, d_o, dk, dv));
  COWA_TRY(check_dq_ptrs(q, k, v, lse, d_o, dq));
  COWA_TRY(check_device());
  hipStream_t st = static_cast<hipStream_t>(stream);
  const cowa::SchedView sv = cowa::sched_view(s);
  COWA_TRY(hip_status(cowa::launch_bwd_prepare(*p, o, d_o, dsum, st), "backward prepare launch"));
  COWA_TRY(hip_status(cowa::launch_bwd_main(*p, sv, q, k, v, lse, d_o, dk, dv, dsum, st), "backward dK/dV launch"));
  return hip_status(cowa::launch_bwd_dq(*p, sv, q, k, v, lse, d_o, dq, dsum, st), "backward dQ launch");
}

static cowa_status check_decode_params(const cowa_decode_params* p) {
  if (!p) return fail(COWA_ERR_INVALID_ARG, "params is NULL");
  if (p->batch < 0) return fail(COWA_ERR_INVALID_ARG, "batch must be >= 0");
  if (p->h_q < 1 || p->h_k < 1 || p->h_q % p->h_k != 0)
    return fail(COWA_ERR_INVALID_ARG, "need h_q >= 1, h_k >= 1 and h_q %% h_k == 0");
  if (p->head_dim != 64 && p->head_dim != 128) return fail(COWA_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (p->n_max < 1 || p->n_max >= (1 << 30)) return fail(COWA_ERR_INVALID_ARG, "n_max must be in [1, 2^30)");
  if (p->w_sink < 0 || p->w_near < 0) return fail(COWA_ERR_INVALID_ARG, "window widths must be >= 0");
  if (p->h_k_total < 1 || p->h_k_offset < 0 || (int64_t)p->h_k_offset + p->h_k > p->h_k_total)
    return fail(COWA_ERR_INVALID_ARG, "need 0 <= h_k_offset and h_k_offset + h_k <= h_k_total");
  if (p->split_keys < 0 || (p->split_keys > 0 && p->split_keys % 64 != 0))
    return fail(COWA_ERR_INVALID_ARG, "split_keys must be 0 or a positive multiple of 64");
  if (p->dtype != COWA_BF16) return fail(COWA_ERR_UNSUPPORTED, "decode is built for bf16 only");
  if (!cowa::decode_supported(p->head_dim, p->h_q / p->h_k))
    return fail(COWA_ERR_UNSUPPORTED, "decode is built for QO-head groups of 1, 2, 4 or 8");
  if (!std::isfinite(p->softmax_scale) || !(p->softmax_scale > 0.f))
    return fail(COWA_ERR_INVALID_ARG, "softmax_scale must be finite and > 0");
  return COWA_OK;
}

cowa_status cowa_decode_workspace_size(const cowa_decode_params* p, size_t* bytes) {
  COWA_TRY(check_decode_params(p));
  if (!bytes) return fail(COWA_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = cowa::decode_workspace_bytes(*p);
  return COWA_OK;
}

cowa_status cowa_decode(const cowa_decode_params* p, const void* q, const void* k_cache, const void* v_cache,
                        const int32_t* seqlens_k, void* o, float* lse, void* workspace, size_t ws_bytes,
                        void* stream) {
  COWA_TRY(check_decode_params(p));
  if (p->batch == 0) return COWA_OK;
  COWA_TRY(check_tensor(q, "q", 16));
  COWA_TRY(check_tensor(k_cache, "k_cache", 16));
  COWA_TRY(check_tensor(v_cache, "v_cache", 16));
  COWA_TRY(check_tensor(seqlens_k, "seqlens_k", 4));
  COWA_TRY(check_tensor(o, "o", 16));
  COWA_TRY(check_tensor(lse, "lse", 4));
  const size_t need = cowa::decode_workspace_bytes(*p);
  if (!workspace || ws_bytes < need || !aligned(workspace, 256))
    return fail(COWA_ERR_WORKSPACE, "decode needs a 256-byte aligned workspace of %zu bytes (got %zu)", need, ws_bytes);
  COWA_TRY(check_device());
  return hip_status(cowa::launch_decode(*p, q, k_cache, v_cache, seqlens_k, o, lse, workspace,
                                        static_cast<hipStream_t>(stream)),
                    "decode launch");
}

}  // extern "C"
