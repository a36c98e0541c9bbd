// C ABI of the CoWA library: argument validation, sizing, and launches on the
// caller's stream.  Every check runs before the first launch, so a failing call
// writes nothing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <set>
#include <utility>
#include <vector>

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

#define COWA_TRY(expr)                     \
  do {                                     \
    cowa_status st_ = (expr);              \
    if (st_ != COWA_OK) return st_;        \
  } while (0)

constexpr int64_t kDistCap = int64_t(1) << 30;  // causal distances are below N_k < 2^30

bool ragged(const cowa_params* p) { return p->cu_seqlens_q != nullptr; }

cowa_status check_params(const cowa_params* p) {
  if (!p) return fail(COWA_ERR_INVALID_ARG, "params is NULL");
  if (p->batch < 0) return fail(COWA_ERR_INVALID_ARG, "batch must be >= 0 (got %d)", p->batch);
  if ((p->cu_seqlens_q == nullptr) != (p->cu_seqlens_k == nullptr))
    return fail(COWA_ERR_INVALID_ARG, "cu_seqlens_q and cu_seqlens_k must both be given or both be NULL");
  if (!ragged(p)) {
    if (p->n_q < 1 || p->n_k < 1) return fail(COWA_ERR_INVALID_ARG, "n_q and n_k must be >= 1");
    if (p->n_q > p->n_k) return fail(COWA_ERR_INVALID_ARG, "n_q (%d) must not exceed n_k (%d)", p->n_q, p->n_k);
  } else if (p->n_q < 0 || p->n_k < 0) {
    return fail(COWA_ERR_INVALID_ARG, "packed totals n_q and n_k must be >= 0");
  }
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

// An explicit window tuple resolved to distance bounds (Sec. 2.1 four-tuple).
cowa_status resolve_tuple(const cowa_window& w, int h, cowa::WinDesc* out) {
  if (w.sink < 0 || w.near < 0 || w.gap < 0 || w.width < 0)
    return fail(COWA_ERR_INVALID_ARG, "window of KV head %d has a negative field (%d, %d, %d, %d)", h, w.sink,
                w.near, w.gap, w.width);
  const int64_t lo = (int64_t)w.near + w.gap, hi = lo + w.width;
  out->sink = (int32_t)cowa::imin64(w.sink, kDistCap);
  out->near = (int32_t)cowa::imin64(w.near, kDistCap);
  out->lo = (int32_t)cowa::imin64(lo, kDistCap);
  out->hi = (int32_t)cowa::imin64(hi, kDistCap);
  return COWA_OK;
}

// The default rule for key length n_k and global KV head hg (Eq. fwa_long_range_span).
cowa::WinDesc default_window(int64_t n_k, int32_t w_sink, int32_t w_near, int64_t hg, int64_t ht) {
  int64_t lo, hi;
  cowa::long_bounds(n_k, w_sink, w_near, hg, ht, &lo, &hi);
  cowa::WinDesc w;
  w.sink = (int32_t)cowa::imin64(w_sink, kDistCap);
  w.near = (int32_t)cowa::imin64(w_near, kDistCap);
  w.lo = (int32_t)cowa::imin64(lo, kDistCap);
  w.hi = (int32_t)cowa::imin64(hi, kDistCap);
  return w;
}

uint64_t fnv(uint64_t h, const void* data, size_t n) {
  const unsigned char* c = static_cast<const unsigned char*>(data);
  for (size_t i = 0; i < n; ++i) h = (h ^ c[i]) * 1099511628211ull;
  return h;
}

// Sequences, windows and block counts of one call, resolved on the host.
struct Layout {
  bool ragged = false, per_seq_win = false;
  std::vector<cowa::SeqDesc> seq;  // one entry per sequence (one for fixed lengths)
  std::vector<cowa::WinDesc> win;  // [n_win][h_k]
  int32_t n_qt = 0, n_kt = 0, max_qt = 0, max_kt = 0;
  uint64_t digest = 0;
  const cowa::WinDesc& window(int b, int h, int h_k) const { return win[(per_seq_win ? (size_t)b * h_k : 0) + h]; }
};

cowa_status resolve_layout(const cowa_params* p, Layout* L) {
  L->ragged = ragged(p);
  L->per_seq_win = L->ragged && p->windows == nullptr;
  uint64_t dg = 1469598103934665603ull;
  const int32_t flags[2] = {L->ragged ? 1 : 0, p->windows ? 1 : 0};
  dg = fnv(dg, flags, sizeof(flags));
  int64_t n_qt = 0, n_kt = 0;
  if (!L->ragged) {
    cowa::SeqDesc sd{};
    sd.n_q = p->n_q;
    sd.n_k = p->n_k;
    L->seq.assign(1, sd);
    n_qt = (p->n_q + p->tile_q - 1) / p->tile_q;
    n_kt = (p->n_k + p->tile_k - 1) / p->tile_k;
    L->max_qt = (int32_t)n_qt;
    L->max_kt = (int32_t)n_kt;
  } else {
    const int32_t* cq = p->cu_seqlens_q;
    const int32_t* ck = p->cu_seqlens_k;
    if (cq[0] != 0 || ck[0] != 0) return fail(COWA_ERR_INVALID_ARG, "cu_seqlens_q[0] and cu_seqlens_k[0] must be 0");
    if (cq[p->batch] != p->n_q || ck[p->batch] != p->n_k)
      return fail(COWA_ERR_INVALID_ARG, "n_q (%d) and n_k (%d) must equal cu_seqlens_q[B] (%d) and cu_seqlens_k[B] (%d)",
                  p->n_q, p->n_k, cq[p->batch], ck[p->batch]);
    L->seq.resize(p->batch);
    for (int b = 0; b < p->batch; ++b) {
      const int64_t nq = (int64_t)cq[b + 1] - cq[b], nk = (int64_t)ck[b + 1] - ck[b];
      if (nq < 0 || nk < 0) return fail(COWA_ERR_INVALID_ARG, "cu_seqlens decrease at sequence %d", b);
      if (nq > nk) return fail(COWA_ERR_INVALID_ARG, "sequence %d has more queries (%lld) than keys (%lld)", b,
                               (long long)nq, (long long)nk);
      cowa::SeqDesc& sd = L->seq[b];
      sd.q_start = cq[b];
      sd.k_start = ck[b];
      sd.n_q = (int32_t)nq;
      sd.n_k = (int32_t)nk;
      sd.qt_off = (int32_t)n_qt;
      sd.kt_off = (int32_t)n_kt;
      sd.pad0 = sd.pad1 = 0;
      const int64_t bq = (nq + p->tile_q - 1) / p->tile_q, bk = (nk + p->tile_k - 1) / p->tile_k;
      n_qt += bq;
      n_kt += bk;
      if (bq > L->max_qt) L->max_qt = (int32_t)bq;
      if (bk > L->max_kt) L->max_kt = (int32_t)bk;
    }
    dg = fnv(dg, &p->batch, sizeof(p->batch));
    dg = fnv(dg, cq, sizeof(int32_t) * ((size_t)p->batch + 1));
    dg = fnv(dg, ck, sizeof(int32_t) * ((size_t)p->batch + 1));
  }
  L->n_qt = (int32_t)n_qt;
  L->n_kt = (int32_t)n_kt;
  if (p->windows) {
    L->win.resize(p->h_k);
    for (int h = 0; h < p->h_k; ++h) COWA_TRY(resolve_tuple(p->windows[h], h, &L->win[h]));
    dg = fnv(dg, p->windows, sizeof(cowa_window) * (size_t)p->h_k);
  } else {
    const size_t n_win = L->per_seq_win ? L->seq.size() : 1;
    L->win.resize(n_win * p->h_k);
    for (size_t b = 0; b < n_win; ++b)
      for (int h = 0; h < p->h_k; ++h)
        L->win[b * p->h_k + h] =
            default_window(L->seq.empty() ? p->n_k : L->seq[b].n_k, p->w_sink, p->w_near,
                           (int64_t)p->h_k_offset + h, p->h_k_total);
  }
  L->digest = dg;
  return COWA_OK;
}

cowa::HeadGeo geo_of(const cowa_params* p, const Layout& L, int b, int h) {
  const cowa::WinDesc& w = L.window(b, h, p->h_k);
  return cowa::make_geo_bounds(L.seq[b].n_q, L.seq[b].n_k, w.sink, w.near, w.lo, w.hi, p->tile_q, p->tile_k);
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Split plan of the dK/dV pass (cowa::BwdSplit): the leading KV blocks that hold
// sink keys of some head are split into P parts, P = ceil(2 x longest such
// column / longest other column) (at most 16, and at most 256 MB of partials):
// parts of about half an ordinary column, which fill the ends of the other
// workgroups' queues when the grid is a few rounds of the device.  A
// column past the sink holds at most the query blocks of its near run
// (B_k + w_near - 1 distance-0 keys) and of its long-range run
// (B_k + hi - lo - 1), each spanning up to one block more than its length.
cowa::BwdSplit bwd_split_plan(const cowa_params* p, const Layout& L) {
  cowa::BwdSplit sp;
  if (p->tile_q < 1 || p->tile_k < 1 || L.max_kt == 0) return sp;
  int64_t S = 0;
  for (const cowa::WinDesc& w : L.win) S = std::max<int64_t>(S, ((int64_t)w.sink + p->tile_k - 1) / p->tile_k);
  S = std::min<int64_t>(S, L.max_kt);
  if (S == 0) return sp;
  int64_t l_sink = 0, l_other = 1;
  for (size_t b = 0; b < L.seq.size(); ++b) {
    const int64_t bq = ((int64_t)L.seq[b].n_q + p->tile_q - 1) / p->tile_q;
    const int64_t bk = ((int64_t)L.seq[b].n_k + p->tile_k - 1) / p->tile_k;
    for (int h = 0; h < p->h_k; ++h) {
      const cowa::HeadGeo g = geo_of(p, L, (int)b, h);
      for (int64_t j = 0; j < std::min(S, bk); ++j)
        l_sink = std::max<int64_t>(l_sink, cowa::ranges_count(cowa::bwd_block_ranges(g, (int32_t)j)));
      const int64_t near = std::min<int64_t>(g.w_near, g.n_k), width = std::min<int64_t>(g.hi, g.n_k) -
                                                                         std::min<int64_t>(g.lo, g.n_k);
      int64_t other = 0;
      if (near > 0) other += (p->tile_k + near - 2) / p->tile_q + 2;
      if (width > 0) other += (p->tile_k + width - 2) / p->tile_q + 2;
      l_other = std::max(l_other, std::min(bq, other));
    }
  }
  const int64_t seqs = L.ragged ? (int64_t)L.seq.size() : p->batch;
  int64_t P = std::min<int64_t>((2 * l_sink + l_other - 1) / l_other, 16);
  const size_t col_bytes = cowa::bwd_part_floats(*p) * sizeof(float);
  while (P > 1 && (size_t)(seqs * p->h_k * S * P) * col_bytes > (size_t(256) << 20)) --P;
  if (P <= 1) return sp;
  sp.S = (int32_t)S;
  sp.P = (int32_t)P;
  sp.n_cols = seqs * p->h_k * S;
  return sp;
}


// Every schedule-relevant field must match (the digest covers windows and lengths).
bool same_schedule(const cowa_params* a, const cowa_params* b) {
  return a->n_q == b->n_q && a->n_k == b->n_k && a->h_k == b->h_k && a->w_sink == b->w_sink &&
         a->w_near == b->w_near && a->h_k_total == b->h_k_total && a->h_k_offset == b->h_k_offset &&
         a->tile_q == b->tile_q && a->tile_k == b->tile_k && ragged(a) == ragged(b) &&
         (!ragged(a) || a->batch == b->batch) && (a->windows == nullptr) == (b->windows == nullptr);
}

cowa_status check_schedule(const cowa_params* p, const Layout& L, const cowa_schedule_t* s) {
  if (!s) return fail(COWA_ERR_INVALID_ARG, "schedule is NULL");
  if (!same_schedule(p, &s->p) || s->digest != L.digest)
    return fail(COWA_ERR_SCHEDULE_MISMATCH, "schedule was sized for other shapes, windows or sequence lengths");
  // the sized fields must be the ones cowa_schedule_size produces
  if (s->n_qt != L.n_qt || s->n_kt != L.n_kt || s->max_qt != L.max_qt || s->max_kt != L.max_kt)
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

// No work: no sequence, or a ragged batch without a single query.
bool no_work(const cowa_params* p) { return p->batch == 0 || (ragged(p) && p->n_q == 0 && p->n_k == 0); }

// Grid units of the launches: B H for fixed lengths, H for a ragged batch.
int64_t seq_factor(const cowa_params* p) { return ragged(p) ? 1 : p->batch; }

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

const char* cowa_version(void) { return "cowa-mi355x 0.2 (gfx950)"; }

const char* cowa_last_error(void) { return g_err; }

cowa_status cowa_windows(const cowa_params* p, cowa_window* out_host) {
  COWA_TRY(check_params(p));
  if (!out_host) return fail(COWA_ERR_INVALID_ARG, "out_host is NULL");
  for (int h = 0; h < p->h_k; ++h) {
    if (p->windows) {
      cowa::WinDesc w;
      COWA_TRY(resolve_tuple(p->windows[h], h, &w));
      out_host[h] = p->windows[h];
      continue;
    }
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
  Layout L;
  COWA_TRY(resolve_layout(p, &L));
  int64_t nnz = 0, nnz_b = 0;
  int32_t max_row = 0, max_col = 0;
  for (size_t b = 0; b < L.seq.size(); ++b) {
    const int32_t bq = (L.seq[b].n_q + p->tile_q - 1) / p->tile_q;
    const int32_t bk = (L.seq[b].n_k + p->tile_k - 1) / p->tile_k;
    for (int h = 0; h < p->h_k; ++h) {
      const cowa::HeadGeo g = geo_of(p, L, (int)b, h);
      for (int32_t i = 0; i < bq; ++i) {
        const int32_t c = cowa::ranges_count(cowa::fwd_block_ranges(g, i));
        nnz += c;
        if (c > max_row) max_row = c;
      }
      for (int32_t j = 0; j < bk; ++j) {
        const int32_t c = cowa::ranges_count(cowa::bwd_block_ranges(g, j));
        nnz_b += c;
        if (c > max_col) max_col = c;
      }
    }
  }
  if (nnz != nnz_b) return fail(COWA_ERR_INVALID_ARG, "internal: block-set sizes disagree (%lld vs %lld)",
                                (long long)nnz, (long long)nnz_b);
  if (nnz >= (int64_t(1) << 31)) return fail(COWA_ERR_UNSUPPORTED, "schedule has more than 2^31 entries");
  if ((int64_t)p->h_k * L.n_qt >= (int64_t(1) << 31) || (int64_t)p->h_k * L.n_kt >= (int64_t(1) << 31))
    return fail(COWA_ERR_UNSUPPORTED, "schedule has more than 2^31 rows");
  std::memset(out, 0, sizeof(*out));
  out->p = *p;
  out->n_qt = L.n_qt;
  out->n_kt = L.n_kt;
  out->max_qt = L.max_qt;
  out->max_kt = L.max_kt;
  out->max_row = max_row;
  out->max_col = max_col;
  out->nnz = nnz;
  out->digest = L.digest;
  size_t off = 0;
  out->off_fwd_row_ptr = off;
  off = align256(off + 4 * ((size_t)p->h_k * L.n_qt + 1));
  out->off_bwd_col_ptr = off;
  off = align256(off + 4 * ((size_t)p->h_k * L.n_kt + 1));
  out->off_fwd_ent = off;
  off = align256(off + 4 * (size_t)nnz);
  out->off_bwd_ent = off;
  off = align256(off + 4 * (size_t)nnz);
  out->off_windows = off;
  off = align256(off + sizeof(cowa::WinDesc) * L.win.size());
  out->off_seqs = off;
  if (L.ragged) {
    off = align256(off + sizeof(cowa::SeqDesc) * L.seq.size());
    out->off_qt_seq = off;
    off = align256(off + 4 * (size_t)L.n_qt);
    out->off_kt_seq = off;
    off = align256(off + 4 * (size_t)L.n_kt);
  } else {
    out->off_qt_seq = out->off_kt_seq = off;
  }
  out->bytes = off;
  out->buf = nullptr;
  return COWA_OK;
}

cowa_status cowa_legal_pairs(const cowa_params* p, int64_t* pairs) {
  COWA_TRY(check_params(p));
  if (!pairs) return fail(COWA_ERR_INVALID_ARG, "pairs is NULL");
  Layout L;
  COWA_TRY(resolve_layout(p, &L));
  int64_t total = 0;
  for (size_t b = 0; b < L.seq.size(); ++b) {
    const int64_t n_q = L.seq[b].n_q, off = (int64_t)L.seq[b].n_k - n_q;
    for (int h = 0; h < p->h_k; ++h) {
      const cowa::WinDesc& w = L.window((int)b, h, p->h_k);
      for (int64_t iq = 0; iq < n_q; ++iq)  // runs of the query whose distance-0 key is iq + off
        total += cowa::ranges_count(cowa::decode_key_runs(iq + off + 1, w.sink, w.near, w.lo, w.hi));
    }
  }
  *pairs = total * (p->h_q / p->h_k) * seq_factor(p);
  return COWA_OK;
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
  if (p->windows) {
    if (p->h_k > cowa::kDecodeMaxExplicitHeads)
      return fail(COWA_ERR_UNSUPPORTED, "decode with explicit windows takes at most %d local KV heads",
                  cowa::kDecodeMaxExplicitHeads);
    cowa::WinDesc w;
    for (int h = 0; h < p->h_k; ++h) COWA_TRY(resolve_tuple(p->windows[h], h, &w));
  }
  return COWA_OK;
}

cowa_status cowa_decode_visible_keys(const cowa_decode_params* p, const int32_t* seqlens_host, int64_t* keys) {
  if (!seqlens_host || !keys) return fail(COWA_ERR_INVALID_ARG, "NULL argument");
  COWA_TRY(check_decode_params(p));
  int64_t total = 0;
  for (int b = 0; b < p->batch; ++b) {
    const int64_t n_k = seqlens_host[b];
    if (n_k < 1 || n_k > p->n_max) continue;
    for (int h = 0; h < p->h_k; ++h) {
      cowa::WinDesc w;
      if (p->windows)
        resolve_tuple(p->windows[h], h, &w);
      else
        w = default_window(n_k, p->w_sink, p->w_near, (int64_t)p->h_k_offset + h, p->h_k_total);
      total += cowa::ranges_count(cowa::decode_key_runs(n_k, w.sink, w.near, w.lo, w.hi));
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
      ref.off_bwd_col_ptr != s->off_bwd_col_ptr || ref.off_windows != s->off_windows ||
      ref.off_seqs != s->off_seqs || ref.off_qt_seq != s->off_qt_seq || ref.off_kt_seq != s->off_kt_seq ||
      ref.digest != s->digest || ref.max_qt != s->max_qt || ref.max_kt != s->max_kt)
    return fail(COWA_ERR_SCHEDULE_MISMATCH, "schedule fields were not produced by cowa_schedule_size for its params");
  if (!s->buf || !aligned(s->buf, 256)) return fail(COWA_ERR_INVALID_ARG, "schedule buffer is NULL or not 256-byte aligned");
  Layout L;
  COWA_TRY(resolve_layout(&s->p, &L));
  // host image of the tables: windows at off_windows, the sequence table at off_seqs
  const size_t table_bytes = L.ragged ? s->off_seqs - s->off_windows + sizeof(cowa::SeqDesc) * L.seq.size()
                                      : sizeof(cowa::WinDesc) * L.win.size();
  std::vector<uint32_t> image((table_bytes + 3) / 4, 0u);
  std::memcpy(image.data(), L.win.data(), sizeof(cowa::WinDesc) * L.win.size());
  if (L.ragged)
    std::memcpy(reinterpret_cast<char*>(image.data()) + (s->off_seqs - s->off_windows), L.seq.data(),
                sizeof(cowa::SeqDesc) * L.seq.size());
  COWA_TRY(check_device());
  return hip_status(cowa::launch_schedule(s, image.data(), 4 * image.size(), static_cast<hipStream_t>(stream)),
                    "schedule launch");
}

cowa_status cowa_fwd(const cowa_params* p, const cowa_schedule_t* s, const void* q, const void* k, const void* v,
                     void* o, float* lse, void* stream) {
  COWA_TRY(check_params(p));
  Layout L;
  COWA_TRY(resolve_layout(p, &L));
  COWA_TRY(check_schedule(p, L, s));
  if (no_work(p)) return COWA_OK;
  COWA_TRY(check_tensor(q, "q", 16));
  COWA_TRY(check_tensor(k, "k", 16));
  COWA_TRY(check_tensor(v, "v", 16));
  COWA_TRY(check_tensor(o, "o", 16));
  COWA_TRY(check_tensor(lse, "lse", 4));
  if ((int64_t)s->n_qt * p->h_q * seq_factor(p) >= (int64_t(1) << 31))
    return fail(COWA_ERR_UNSUPPORTED, "too many query blocks for one launch");
  if (p->dtype == COWA_BF16 && !cowa::fwd_bf16_supported(p->head_dim, p->tile_q, p->tile_k))
    return fail(COWA_ERR_UNSUPPORTED, "bf16 forward is built for tile_q and tile_k in {64, 128} (got %d x %d)",
                p->tile_q, p->tile_k);
  if (p->dtype == COWA_BF16 && s->max_kt > cowa::fwd_bf16_max_kblocks(p->head_dim, p->tile_k))
    return fail(COWA_ERR_UNSUPPORTED, "bf16 forward supports at most %d key blocks per sequence (got %d)",
                cowa::fwd_bf16_max_kblocks(p->head_dim, p->tile_k), s->max_kt);
  COWA_TRY(check_device());
  if (s->n_qt == 0) return COWA_OK;
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
  Layout L;
  COWA_TRY(resolve_layout(p, &L));
  *bytes = cowa::bwd_workspace_bytes(*p, bwd_split_plan(p, L));
  return COWA_OK;
}

// Checks shared by the backward stages; the workspace holds -D and -LSE log2(e) per query row.
static cowa_status check_bwd(const cowa_params* p, const Layout& L, size_t ws_bytes, void* workspace,
                             cowa::BwdWork* w) {
  if (p->dtype != COWA_BF16) return fail(COWA_ERR_UNSUPPORTED, "backward is built for bf16 only");
  if (!cowa::bwd_bf16_supported(p->head_dim, p->tile_q, p->tile_k))
    return fail(COWA_ERR_UNSUPPORTED, "bf16 backward is built for tile_q, tile_k in {64, 128} (got %d x %d)",
                p->tile_q, p->tile_k);
  // the dK/dV pass keeps a column's block list, the dQ pass a row's, in LDS
  if (L.max_qt > cowa::bwd_main_max_qblocks(p->head_dim, p->tile_k))
    return fail(COWA_ERR_UNSUPPORTED, "backward supports at most %d query blocks per sequence (got %d)",
                cowa::bwd_main_max_qblocks(p->head_dim, p->tile_k), L.max_qt);
  if (L.max_kt > cowa::bwd_dq_max_kblocks(p->head_dim, p->tile_k))
    return fail(COWA_ERR_UNSUPPORTED, "backward supports at most %d key blocks per sequence (got %d)",
                cowa::bwd_dq_max_kblocks(p->head_dim, p->tile_k), L.max_kt);
  // one workgroup per (KV block, KV head, sequence) in the dK/dV pass and per
  // (QO block, QO head, sequence) at most in the dQ pass: grid limit 2^31
  if ((int64_t)L.n_kt * p->h_k * seq_factor(p) >= (int64_t(1) << 31))
    return fail(COWA_ERR_UNSUPPORTED, "too many key blocks for one launch");
  if ((int64_t)L.n_qt * p->h_q * seq_factor(p) >= (int64_t(1) << 31))
    return fail(COWA_ERR_UNSUPPORTED, "too many query blocks for one launch");
  const cowa::BwdSplit sp = bwd_split_plan(p, L);
  if ((int64_t)L.n_kt * p->h_k * seq_factor(p) + sp.n_cols * sp.P + 8 >= (int64_t(1) << 31))
    return fail(COWA_ERR_UNSUPPORTED, "too many key blocks for one launch");
  const size_t need = cowa::bwd_workspace_bytes(*p, sp);
  if (!no_work(p) && (!workspace || ws_bytes < need || !aligned(workspace, 256)))
    return fail(COWA_ERR_WORKSPACE, "backward needs a 256-byte aligned workspace of %zu bytes (got %zu)", need, ws_bytes);
  *w = cowa::bwd_work(*p, sp, workspace);
  return COWA_OK;
}

// Pointer checks of each stage (after check_bwd, when there is work).
static cowa_status check_prepare_ptrs(const void* o, const void* d_o, const float* lse) {
  COWA_TRY(check_tensor(o, "o", 16));
  COWA_TRY(check_tensor(lse, "lse", 4));
  return check_tensor(d_o, "d_o", 16);
}

static cowa_status check_qkv_do(const void* q, const void* k, const void* v, const void* d_o) {
  COWA_TRY(check_tensor(q, "q", 16));
  COWA_TRY(check_tensor(k, "k", 16));
  COWA_TRY(check_tensor(v, "v", 16));
  return check_tensor(d_o, "d_o", 16);
}

static cowa_status check_main_ptrs(const void* q, const void* k, const void* v, const void* d_o, const void* dk,
                                   const void* dv) {
  COWA_TRY(check_qkv_do(q, k, v, d_o));
  COWA_TRY(check_tensor(dk, "dk", 16));
  return check_tensor(dv, "dv", 16);
}

static cowa_status check_dq_ptrs(const void* q, const void* k, const void* v, const void* d_o, const void* dq) {
  COWA_TRY(check_qkv_do(q, k, v, d_o));
  return check_tensor(dq, "dq", 16);
}

cowa_status cowa_bwd_prepare(const cowa_params* p, const void* o, const void* d_o, const float* lse, void* workspace,
                             size_t ws_bytes, void* stream) {
  COWA_TRY(check_params(p));
  Layout L;
  COWA_TRY(resolve_layout(p, &L));
  cowa::BwdWork w;
  COWA_TRY(check_bwd(p, L, ws_bytes, workspace, &w));
  if (no_work(p)) return COWA_OK;
  COWA_TRY(check_prepare_ptrs(o, d_o, lse));
  COWA_TRY(check_device());
  if (cowa::q_rows(*p) == 0) return COWA_OK;
  return hip_status(cowa::launch_bwd_prepare(*p, o, d_o, lse, w, static_cast<hipStream_t>(stream)),
                    "backward prepare launch");
}

cowa_status cowa_bwd_main(const cowa_params* p, const cowa_schedule_t* s, const void* q, const void* k,
                          const void* v, const void* d_o, void* dk, void* dv, void* workspace, size_t ws_bytes,
                          void* stream) {
  COWA_TRY(check_params(p));
  Layout L;
  COWA_TRY(resolve_layout(p, &L));
  cowa::BwdWork w;
  COWA_TRY(check_bwd(p, L, ws_bytes, workspace, &w));
  COWA_TRY(check_schedule(p, L, s));
  if (no_work(p)) return COWA_OK;
  COWA_TRY(check_main_ptrs(q, k, v, d_o, dk, dv));
  COWA_TRY(check_device());
  if (s->n_kt == 0) return COWA_OK;
  return hip_status(cowa::launch_bwd_main(*p, cowa::sched_view(s), q, k, v, d_o, dk, dv, w,
                                          static_cast<hipStream_t>(stream)),
                    "backward dK/dV launch");
}

cowa_status cowa_bwd_dq(const cowa_params* p, const cowa_schedule_t* s, const void* q, const void* k, const void* v,
                        const void* d_o, void* dq, void* workspace, size_t ws_bytes, void* stream) {
  COWA_TRY(check_params(p));
  Layout L;
  COWA_TRY(resolve_layout(p, &L));
  cowa::BwdWork w;
  COWA_TRY(check_bwd(p, L, ws_bytes, workspace, &w));
  COWA_TRY(check_schedule(p, L, s));
  if (no_work(p)) return COWA_OK;
  COWA_TRY(check_dq_ptrs(q, k, v, d_o, dq));
  COWA_TRY(check_device());
  if (s->n_qt == 0) return COWA_OK;
  return hip_status(cowa::launch_bwd_dq(*p, cowa::sched_view(s), q, k, v, d_o, dq, w,
                                        static_cast<hipStream_t>(stream)),
                    "backward dQ launch");
}

// All three stages; every check of every stage runs before the first launch.
cowa_status cowa_bwd(const cowa_params* p, const cowa_schedule_t* s, const void* q, const void* k, const void* v,
                     const void* o, const float* lse, const void* d_o, void* dq, void* dk, void* dv, void* workspace,
                     size_t ws_bytes, void* stream) {
  COWA_TRY(check_params(p));
  Layout L;
  COWA_TRY(resolve_layout(p, &L));
  cowa::BwdWork w;
  COWA_TRY(check_bwd(p, L, ws_bytes, workspace, &w));
  COWA_TRY(check_schedule(p, L, s));
  if (no_work(p)) return COWA_OK;
  COWA_TRY(check_prepare_ptrs(o, d_o, lse));
  COWA_TRY(check_main_ptrs(q, k, v, d_o, dk, dv));
  COWA_TRY(check_dq_ptrs(q, k, v, d_o, dq));
  COWA_TRY(check_device());
  hipStream_t st = static_cast<hipStream_t>(stream);
  const cowa::SchedView sv = cowa::sched_view(s);
  if (cowa::q_rows(*p) > 0)
    COWA_TRY(hip_status(cowa::launch_bwd_prepare(*p, o, d_o, lse, w, st), "backward prepare launch"));
  if (s->n_kt > 0)
    COWA_TRY(hip_status(cowa::launch_bwd_main(*p, sv, q, k, v, d_o, dk, dv, w, st), "backward dK/dV launch"));
  if (s->n_qt == 0) return COWA_OK;
  return hip_status(cowa::launch_bwd_dq(*p, sv, q, k, v, d_o, dq, w, st), "backward dQ launch");
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

cowa_status cowa_decode_noalloc(const cowa_decode_params* p, const void* q, const void* k_cache, const void* v_cache,
                                const int32_t* seqlens_k, void* o, float* lse, void* stream) {
  COWA_TRY(check_decode_params(p));
  if (p->batch == 0) return COWA_OK;
  COWA_TRY(check_tensor(q, "q", 16));
  COWA_TRY(check_tensor(k_cache, "k_cache", 16));
  COWA_TRY(check_tensor(v_cache, "v_cache", 16));
  COWA_TRY(check_tensor(seqlens_k, "seqlens_k", 4));
  COWA_TRY(check_tensor(o, "o", 16));
  COWA_TRY(check_tensor(lse, "lse", 4));
  const size_t need = cowa::decode_workspace_bytes(*p);
  if (need > cowa::kDecodeScratchBytes)
    return fail(COWA_ERR_UNSUPPORTED,
                "cowa_decode_noalloc: this step needs %zu bytes of split partials, more than its %zu-byte device "
                "scratch; use cowa_decode with a workspace, or a larger split_keys",
                need, cowa::kDecodeScratchBytes);
  COWA_TRY(check_device());
  void* ws = nullptr;
  COWA_TRY(hip_status(cowa::decode_scratch(&ws), "decode scratch address"));
  return hip_status(cowa::launch_decode(*p, q, k_cache, v_cache, seqlens_k, o, lse, ws,
                                        static_cast<hipStream_t>(stream)),
                    "decode launch");
}

}  // extern "C"
