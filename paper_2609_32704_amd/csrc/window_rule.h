// Window rule and block-set construction shared by the host sizing code and
// the device kernels of the library.
//
// Sec. 2.1: with the bottom-right causal distance delta = i_q + (N_k - N_q) - i_k
// (Eq. fwa_distance), KV head h sees
//   near : 0 <= delta < w_near
//   sink : i_k < w_sink and delta >= 0
//   long : lo_h <= delta < hi_h,  lo_h = w_near + b_h,  hi_h = w_near + b_{h+1}
// with L = max(N_k - w_sink - w_near, 0) and b_h = floor(h L / H_k) over the
// global KV-head index (Eq. fwa_long_range_span, Eq. fwa_global_head).
//
// Sec. 2.3: J_h(i) is the set of KV blocks holding at least one legal pair with
// QO block i, I_h(j) its inverse.  Each window is one contiguous key run per
// query and the runs slide by one key per query, so over a QO block every
// window covers one contiguous key range; J_h(i) is the union of at most three
// block ranges and is found in O(1) per block (likewise I_h(j)).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cowa {

struct HeadGeo {
  int32_t n_q, n_k, w_sink, w_near, tile_q, tile_k;
  int64_t lo, hi;  // long-window distance bounds [lo, hi)
};

__host__ __device__ inline int64_t imin64(int64_t a, int64_t b) { return a < b ? a : b; }
__host__ __device__ inline int64_t imax64(int64_t a, int64_t b) { return a > b ? a : b; }

// Long-window bounds of global KV head hg out of ht heads (64-bit products).
__host__ __device__ inline void long_bounds(int64_t n_k, int64_t w_sink, int64_t w_near, int64_t hg,
                                            int64_t ht, int64_t* lo, int64_t* hi) {
  int64_t span = imax64(n_k - w_sink - w_near, 0);
  *lo = w_near + (hg * span) / ht;
  *hi = w_near + ((hg + 1) * span) / ht;
}

// The same from resolved window bounds (sink, near, long-range [lo, hi)).
__host__ __device__ inline HeadGeo make_geo_bounds(int32_t n_q, int32_t n_k, int32_t sink, int32_t near, int64_t lo,
                                                   int64_t hi, int32_t tile_q, int32_t tile_k) {
  HeadGeo g;
  g.n_q = n_q; g.n_k = n_k; g.w_sink = sink; g.w_near = near; g.tile_q = tile_q; g.tile_k = tile_k;
  g.lo = lo; g.hi = hi;
  return g;
}

__host__ __device__ inline HeadGeo make_geo(int32_t n_q, int32_t n_k, int32_t w_sink, int32_t w_near,
                                            int32_t tile_q, int32_t tile_k, int32_t hg, int32_t ht) {
  HeadGeo g;
  g.n_q = n_q; g.n_k = n_k; g.w_sink = w_sink; g.w_near = w_near; g.tile_q = tile_q; g.tile_k = tile_k;
  long_bounds(n_k, w_sink, w_near, hg, ht, &g.lo, &g.hi);
  return g;
}

// Element predicate of Eq. fwa_support (set union of the three windows).
__host__ __device__ inline bool legal_pair(const HeadGeo& g, int64_t q, int64_t k) {
  if (q >= g.n_q || k >= g.n_k) return false;
  int64_t d = q + (int64_t)(g.n_k - g.n_q) - k;
  if (d < 0) return false;
  return d < g.w_near || k < g.w_sink || (d >= g.lo && d < g.hi);
}

// 32-bit form of the element predicate for kernels: window bounds clamped to
// n_k (a distance never reaches n_k, so a larger bound behaves the same).
struct Geo32 {
  int32_t off, w_near, w_sink, lo, hi, n_q, n_k;
};

__host__ __device__ inline Geo32 geo32(const HeadGeo& g) {
  Geo32 r;
  r.off = g.n_k - g.n_q;
  r.w_near = g.w_near < g.n_k ? g.w_near : g.n_k;
  r.w_sink = g.w_sink < g.n_k ? g.w_sink : g.n_k;
  r.lo = (int32_t)imin64(g.lo, g.n_k);
  r.hi = (int32_t)imin64(g.hi, g.n_k);
  r.n_q = g.n_q;
  r.n_k = g.n_k;
  return r;
}

// Same predicate as legal_pair for in-range positions (q < n_q, k < n_k).
__host__ __device__ inline bool legal32(const Geo32& g, int32_t q, int32_t k) {
  const int32_t d = q + g.off - k;
  // bitwise, not short-circuit: a mask evaluated without branches
  return (q < g.n_q) & (k < g.n_k) & (d >= 0) & ((d < g.w_near) | (k < g.w_sink) | ((d >= g.lo) & (d < g.hi)));
}

// Bits a..b (inclusive) of a 32-bit word, for any a, b (none when a > b or the
// range misses 0..31).
__host__ __device__ inline uint32_t bit_range32(int32_t a, int32_t b) {
  const int32_t lo = a < 0 ? 0 : (a > 32 ? 32 : a);
  const int32_t hi = b < 0 ? 0 : (b > 31 ? 32 : b + 1);
  const int32_t w = hi - lo;  // (32-bit arithmetic only: few registers)
  return w <= 0 ? 0u : (w >= 32 ? ~0u : ((1u << (w & 31)) - 1u) << (lo & 31));
}
__host__ __device__ inline int32_t imin32(int32_t a, int32_t b) { return a < b ? a : b; }
__host__ __device__ inline int32_t imax32(int32_t a, int32_t b) { return a > b ? a : b; }

// legal32 over 32 consecutive keys at once: bit j is legal32(g, q, key0 + j).
// For one query the legal keys are the union of three runs (near, long, sink)
// cut to d >= 0 and k < n_k; each run becomes a range of bits, so a partial
// block's element mask costs a few operations per query and chunk instead of
// the window rule per element.
__host__ __device__ inline uint32_t legal_keys32(const Geo32& g, int32_t q, int32_t key0) {
  const int32_t d0 = q + g.off - key0;                // distance of key0
  const int32_t up = imin32(d0, g.n_k - 1 - key0);    // d >= 0, k < n_k
  const uint32_t m = bit_range32(d0 - g.w_near + 1, up) | bit_range32(d0 - g.hi + 1, imin32(up, d0 - g.lo)) |
                     bit_range32(0, imin32(up, g.w_sink - 1 - key0));
  return q < g.n_q ? m : 0u;  // (a select, not a branch)
}
// The same over 32 consecutive queries for one key: bit i is legal32(g, q0 + i, k).
__host__ __device__ inline uint32_t legal_queries32(const Geo32& g, int32_t q0, int32_t k) {
  const int32_t e0 = q0 + g.off - k;                  // distance of query q0
  const int32_t up = g.n_q - 1 - q0;                  // q < n_q
  const uint32_t m = bit_range32(-e0, imin32(up, g.w_near - 1 - e0)) |
                     bit_range32(imax32(-e0, g.lo - e0), imin32(up, g.hi - 1 - e0)) |
                     (k < g.w_sink ? bit_range32(-e0, up) : 0u);
  return k < g.n_k ? m : 0u;
}

// Up to three inclusive ranges, merged (overlapping or adjacent ranges join).
struct Ranges {
  int32_t n;
  int32_t a[3], b[3];
};

__host__ __device__ inline void ranges_add(Ranges& r, int64_t a, int64_t b) {
  if (a <= b) { r.a[r.n] = (int32_t)a; r.b[r.n] = (int32_t)b; ++r.n; }
}

// Sort by start (ascending) and merge.
__host__ __device__ inline void ranges_merge(Ranges& r) {
  for (int x = 0; x < r.n; ++x)
    for (int y = x + 1; y < r.n; ++y)
      if (r.a[y] < r.a[x]) {
        int32_t ta = r.a[x], tb = r.b[x];
        r.a[x] = r.a[y]; r.b[x] = r.b[y]; r.a[y] = ta; r.b[y] = tb;
      }
  int m = 0;
  for (int x = 0; x < r.n; ++x) {
    if (m > 0 && r.a[x] <= r.b[m - 1] + 1) {
      if (r.b[x] > r.b[m - 1]) r.b[m - 1] = r.b[x];
    } else {
      r.a[m] = r.a[x]; r.b[m] = r.b[x]; ++m;
    }
  }
  r.n = m;
}

__host__ __device__ inline int32_t ranges_count(const Ranges& r) {
  int32_t c = 0;
  for (int x = 0; x < r.n; ++x) c += r.b[x] - r.a[x] + 1;
  return c;
}

// KV-block ranges of J_h(i) (ascending, merged).
__host__ __device__ inline Ranges fwd_block_ranges(const HeadGeo& g, int32_t i) {
  int64_t q0 = (int64_t)i * g.tile_q;
  int64_t q1 = imin64(q0 + g.tile_q, g.n_q) - 1;
  int64_t off = (int64_t)g.n_k - g.n_q;
  int64_t c0 = q0 + off, c1 = q1 + off;  // keys at distance 0 of the first / last query
  Ranges r; r.n = 0;
  if (g.w_near >= 1) ranges_add(r, imax64(0, c0 - g.w_near + 1) / g.tile_k, c1 / g.tile_k);
  if (g.w_sink >= 1) ranges_add(r, 0, imin64(g.w_sink - 1, c1) / g.tile_k);
  if (g.hi > g.lo && c1 - g.lo >= 0) ranges_add(r, imax64(0, c0 - g.hi + 1) / g.tile_k, (c1 - g.lo) / g.tile_k);
  ranges_merge(r);
  return r;
}

// QO-block ranges of I_h(j) (ascending, merged).
__host__ __device__ inline Ranges bwd_block_ranges(const HeadGeo& g, int32_t j) {
  int64_t k0 = (int64_t)j * g.tile_k;
  int64_t k1 = imin64(k0 + g.tile_k, g.n_k) - 1;
  int64_t off = (int64_t)g.n_k - g.n_q;
  int64_t cmin = off, cmax = (int64_t)g.n_k - 1;  // range of distance-0 keys over all queries
  Ranges r; r.n = 0;
  auto add_c = [&](int64_t ca, int64_t cb) {
    ca = imax64(ca, cmin); cb = imin64(cb, cmax);
    if (ca <= cb) ranges_add(r, (ca - off) / g.tile_q, (cb - off) / g.tile_q);
  };
  if (g.w_near >= 1) add_c(k0, k1 + g.w_near - 1);
  if (g.w_sink >= 1 && k0 < g.w_sink) add_c(k0, cmax);
  if (g.hi > g.lo) add_c(k0 + g.lo, k1 + g.hi - 1);
  ranges_merge(r);
  return r;
}

// FULL iff the tile lies inside both sequences and every element pair is legal.
__host__ __device__ inline bool tile_full(const HeadGeo& g, int32_t i, int32_t j) {
  int64_t q0 = (int64_t)i * g.tile_q, k0 = (int64_t)j * g.tile_k;
  if (q0 + g.tile_q > g.n_q || k0 + g.tile_k > g.n_k) return false;
  int64_t q1 = q0 + g.tile_q - 1, k1 = k0 + g.tile_k - 1;
  int64_t off = (int64_t)g.n_k - g.n_q;
  int64_t c0 = q0 + off, c1 = q1 + off;
  if (k0 < g.w_sink) {  // sink keys: legal iff causal
    int64_t ks1 = imin64(k1, (int64_t)g.w_sink - 1);
    if (c0 - ks1 < 0) return false;
  }
  int64_t kn0 = imax64(k0, g.w_sink);
  if (kn0 <= k1) {  // other keys: every distance in [a, b] must be in [0, w_near) u [lo, hi)
    int64_t a = c0 - k1, b = c1 - kn0;
    bool ok = (a >= 0 && b < g.w_near) || (a >= g.lo && b < g.hi) ||
              (g.lo == g.w_near && a >= 0 && b < g.hi);
    if (!ok) return false;
  }
  return true;
}

}  // namespace cowa

namespace cowa {

// Key runs of the single decoding query (N_q = 1, distance-0 key c = N_k - 1),
// ascending and merged: the visible set A_h of Sec. 2.3 (decoding execution).
__host__ __device__ inline Ranges decode_key_runs(int64_t n_k, int64_t w_sink, int64_t w_near, int64_t lo,
                                                  int64_t hi) {
  const int64_t c = n_k - 1;
  Ranges r; r.n = 0;
  if (w_near >= 1) ranges_add(r, imax64(0, c - w_near + 1), c);
  if (w_sink >= 1) ranges_add(r, 0, imin64(w_sink - 1, c));
  if (hi > lo && c - lo >= 0) ranges_add(r, imax64(0, c - hi + 1), c - lo);
  ranges_merge(r);
  return r;
}

// The key at position v (0-based) of the ascending visible list.
__host__ __device__ inline int32_t run_key(const Ranges& r, int32_t v) {
  for (int x = 0; x < r.n; ++x) {
    const int32_t sz = r.b[x] - r.a[x] + 1;
    if (v < sz) return r.a[x] + v;
    v -= sz;
  }
  return r.n > 0 ? r.b[r.n - 1] : 0;
}

}  // namespace cowa
