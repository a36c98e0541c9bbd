// CoWA decoding step (Sec. 2.3, decoding execution): the forward with N_q = 1,
// N_k = seqlens_k[b], breakpoints recomputed from that N_k.
//
// Split kernel: one workgroup per (split s, local KV head h, sequence b).  The
// visible keys of (b, h) are the merged key runs of sink, long-range window and
// near window; split s takes positions [s * SK, (s + 1) * SK) of that ascending
// list.  Loads are 16-byte and coalesced: a 64-lane wave reads whole K and V
// rows (d/8 lanes per row), so every wave step streams a contiguous run of
// cache rows.  Each lane group keeps, for each of the G QO heads of the group,
// an online-softmax state (m, l, O slice) in registers; the workgroup merges
// its 4 x (64 / (d/8)) states and writes one partial (m, l, O) per QO head.
//
// Combine kernel: one 64-lane wave per (sequence, QO head) merges the split
// partials (max of m, rescaled sums) and writes O and the natural-log LSE.
// Everything is fp32 apart from the bf16 loads; scores are kept in base 2.
#include <map>
#include <mutex>

#include "internal.h"
#include "window_rule.h"

namespace cowa {
namespace {

constexpr int kDefaultSplitKeys = 256;   // smallest default split
constexpr int64_t kTargetPrograms = 1024;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

constexpr int kHeadsPerLaunch = 32;  // explicit windows travel in the kernel arguments, 32 heads at a time

struct DecArgs {
  const __bf16* q;
  const __bf16* kc;
  const __bf16* vc;
  const int32_t* seqlens;
  __bf16* o;
  float* lse;
  float* part_o;   // [B][H_q][S][D]
  float* part_ml;  // [B][H_q][S][2]
  int32_t batch, h_q, h_k, n_max, w_sink, w_near, h_total, h_offset, splits, split_keys;
  float c;  // softmax_scale * log2(e)
  int32_t explicit_win;            // windows below (else the default rule from each sequence's N_k)
  int32_t head_base;               // first local KV head of this launch
  WinDesc win[kHeadsPerLaunch];    // explicit windows of heads head_base .. head_base + 31
};

// The visible keys of the decoding query (distance-0 key c = N_k - 1) as up to
// three ascending, merged key runs [a, b] -- the union of the sink, long-range
// and near windows of Sec. 2.1 -- computed with scalar selects only (no
// indexed arrays, which the compiler would place in scratch memory).  Empty
// runs have a = kNone.
constexpr int32_t kNone = 0x3fffffff;
struct Runs3 {
  int32_t a0, b0, a1, b1, a2, b2;
};
__device__ inline void order2(int32_t& a, int32_t& b, int32_t& c, int32_t& d) {  // (a, b) before (c, d)
  const bool sw = c < a;
  const int32_t ta = sw ? c : a, tb = sw ? d : b, tc = sw ? a : c, td = sw ? b : d;
  a = ta; b = tb; c = tc; d = td;
}
__device__ inline Runs3 key_runs3(int32_t n_k, int32_t sink, int32_t near, int32_t lo, int32_t hi) {
  const int32_t c = n_k - 1;
  Runs3 r;
  // near: delta in [0, near); sink: keys below sink; long: delta in [lo, hi)
  r.a0 = near >= 1 ? max(0, c - near + 1) : kNone;
  r.b0 = near >= 1 ? c : kNone - 1;
  r.a1 = sink >= 1 ? 0 : kNone;
  r.b1 = sink >= 1 ? min(sink - 1, c) : kNone - 1;
  const bool has_long = hi > lo && c - lo >= 0;
  r.a2 = has_long ? max(0, c - hi + 1) : kNone;
  r.b2 = has_long ? c - lo : kNone - 1;
  order2(r.a0, r.b0, r.a1, r.b1);
  order2(r.a1, r.b1, r.a2, r.b2);
  order2(r.a0, r.b0, r.a1, r.b1);
  // merge overlapping or touching runs (an empty run starts at kNone and never merges)
  if (r.a1 != kNone && r.a1 <= r.b0 + 1) {
    r.b0 = max(r.b0, r.b1);
    r.a1 = r.a2; r.b1 = r.b2;
    r.a2 = kNone; r.b2 = kNone - 1;
  }
  if (r.a1 != kNone && r.a1 <= r.b0 + 1) {
    r.b0 = max(r.b0, r.b1);
    r.a1 = kNone; r.b1 = kNone - 1;
  }
  if (r.a2 != kNone && r.a2 <= r.b1 + 1) {
    r.b1 = max(r.b1, r.b2);
    r.a2 = kNone; r.b2 = kNone - 1;
  }
  return r;
}

// Sum over the DC lanes of each lane group (DC = 8 or 16 consecutive lanes,
// inside one 16-lane DPP row), the result in every lane of the group:
// quad butterflies, then mirrors within 8 and within 16 lanes.
template <int DC>
__device__ inline float group_sum(float x) {
  auto dpp = [](float v, int ctrl) -> float {
    switch (ctrl) {  // the DPP control must be a constant
      case 0xB1: return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
      case 0x4E: return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, false));
      case 0x141: return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x141, 0xF, 0xF, false));
      default: return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x140, 0xF, 0xF, false));
    }
  };
  x += dpp(x, 0xB1);   // quad_perm [1,0,3,2]: lane ^ 1
  x += dpp(x, 0x4E);   // quad_perm [2,3,0,1]: lane ^ 2
  x += dpp(x, 0x141);  // row_half_mirror: lane i <-> 7 - i within 8 lanes (the other quad)
  if constexpr (DC == 16) x += dpp(x, 0x140);  // row_mirror: lane i <-> 15 - i (the other half row)
  return x;
}

// The visible K/V rows are read once per step: non-temporal loads stream
// them measurably faster than ordinary loads (7.1 against 6.3 TB/s for a plain
// 5 GiB read on MI355X), since the data need not be kept in the caches.
__device__ inline uint4 ld_stream16(const __bf16* ptr) {
  typedef unsigned v4u __attribute__((ext_vector_type(4)));
  const v4u t = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(ptr));
  return make_uint4(t.x, t.y, t.z, t.w);
}

template <int D, int G>
__global__ void __launch_bounds__(256) decode_split(DecArgs a) {
  constexpr int DC = D / 8;               // lanes per cache row (16-byte chunks)
  constexpr int KG = 64 / DC;             // rows per wave load instruction
  constexpr int STEP = 4 * KG;            // keys per workgroup step (4 waves)
  constexpr int U = G >= 8 ? 4 : 8;       // steps in flight per iteration
  __shared__ float sm_m[4][G], sm_l[4][G];
  __shared__ float sm_o[4][G][D];

  const int s = blockIdx.x, hk = a.head_base + blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int kg = lane / DC, dc = lane % DC;

  const int32_t n_k = a.seqlens[b];
  const bool valid = n_k >= 1 && n_k <= a.n_max;
  Runs3 runs{kNone, kNone - 1, kNone, kNone - 1, kNone, kNone - 1};
  if (valid) {
    WinDesc w;
    if (a.explicit_win) {
      w = a.win[blockIdx.y];
    } else {
      int64_t lo, hi;
      long_bounds(n_k, a.w_sink, a.w_near, (int64_t)a.h_offset + hk, a.h_total, &lo, &hi);
      w = WinDesc{a.w_sink, a.w_near, (int32_t)lo, (int32_t)hi};
    }
    runs = key_runs3(n_k, min(w.sink, n_k), min(w.near, n_k), min(w.lo, n_k), min(w.hi, n_k));
  }
  const int32_t total = (runs.b0 - runs.a0 + 1) + (runs.b1 - runs.a1 + 1) + (runs.b2 - runs.a2 + 1);
  const int32_t v0 = s * a.split_keys;
  const int32_t v1 = min(v0 + a.split_keys, total);

  // query chunk of each QO head as packed bf16 pairs (dot products in fp32)
  uint32_t qp[G][4];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint4 w = *reinterpret_cast<const uint4*>(a.q + ((int64_t)b * a.h_q + hk * G + g) * D + dc * 8);
    qp[g][0] = w.x; qp[g][1] = w.y; qp[g][2] = w.z; qp[g][3] = w.w;
  }
  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[g][t] = 0.f;
  }

  const int64_t head_off = ((int64_t)b * a.h_k + hk) * a.n_max * D;
  const __bf16* kbase = a.kc + head_off + dc * 8;
  const __bf16* vbase = a.vc + head_off + dc * 8;
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

  // the split's visible positions [v0, v1) cover at most three contiguous key
  // runs; each run is streamed as a contiguous key range
  int32_t off = 0;
#pragma unroll
  for (int r = 0; r < 3; ++r) {
    const int32_t ra = r == 0 ? runs.a0 : r == 1 ? runs.a1 : runs.a2;
    const int32_t rb = r == 0 ? runs.b0 : r == 1 ? runs.b1 : runs.b2;
    if (ra == kNone) break;
    const int32_t len = rb - ra + 1;
    const int32_t lo = max(v0, off), hi = min(v1, off + len);
    off += len;
    if (lo >= hi) continue;
    const int32_t k_lo = ra + (lo - off + len), k_hi = ra + (hi - off + len);  // keys [k_lo, k_hi)
    for (int32_t kb = k_lo; kb < k_hi; kb += STEP * U) {
      uint4 kr[U], vr[U];
      bool ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int32_t key = kb + u * STEP + wave * KG + kg;
        ok[u] = key < k_hi;
        const int64_t kc = ok[u] ? key : k_hi - 1;
        kr[u] = ld_stream16(kbase + kc * D);
        vr[u] = ld_stream16(vbase + kc * D);
      }
      float sc[U][G];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t kw[4] = {kr[u].x, kr[u].y, kr[u].z, kr[u].w};
#pragma unroll
        for (int g = 0; g < G; ++g) {
          float part = 0.f;
#pragma unroll
          for (int t = 0; t < 4; ++t)
            part = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, qp[g][t]),
                                                   __builtin_bit_cast(bf16x2, kw[t]), part, false);
          part = group_sum<DC>(part);
          sc[u][g] = ok[u] ? part * a.c : -INFINITY;
        }
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float mx = sc[0][g];
#pragma unroll
        for (int u = 1; u < U; ++u) mx = fmaxf(mx, sc[u][g]);
        const float m_new = fmaxf(m[g], mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m[g] - m_use);
        l[g] *= alpha;
#pragma unroll
        for (int t = 0; t < 8; ++t) acc[g][t] *= alpha;
        m[g] = m_new;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const float p = __builtin_amdgcn_exp2f(sc[u][g] - m_use);
          l[g] += p;
          const uint32_t vw[4] = {vr[u].x, vr[u].y, vr[u].z, vr[u].w};
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            acc[g][2 * t] = fmaf(p, __uint_as_float(vw[t] << 16), acc[g][2 * t]);
            acc[g][2 * t + 1] = fmaf(p, __uint_as_float(vw[t] & 0xffff0000u), acc[g][2 * t + 1]);
          }
        }
      }
    }
  }

  // merge the KG lane groups of each wave (lanes dc, dc + DC, ... hold the same d slice)
#pragma unroll
  for (int off = DC; off < 64; off <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float mo = __shfl_xor(m[g], off);
      const float lo2 = __shfl_xor(l[g], off);
      const float mm = fmaxf(m[g], mo);
      const float mu = mm == -INFINITY ? 0.f : mm;
      const float f1 = __builtin_amdgcn_exp2f(m[g] - mu), f2 = __builtin_amdgcn_exp2f(mo - mu);
      l[g] = l[g] * f1 + lo2 * f2;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float ao = __shfl_xor(acc[g][t], off);
        acc[g][t] = acc[g][t] * f1 + ao * f2;
      }
      m[g] = mm;
    }
  }
  // then the four waves through LDS
  if (kg == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (dc == 0) { sm_m[wave][g] = m[g]; sm_l[wave][g] = l[g]; }
#pragma unroll
      for (int t = 0; t < 8; ++t) sm_o[wave][g][dc * 8 + t] = acc[g][t];
    }
  }
  __syncthreads();

  const int64_t part_base = (((int64_t)b * a.h_q + hk * G) * a.splits + s);
  for (int x = tid; x < G * D; x += 256) {
    const int g = x / D, d = x % D;
    float mm = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) mm = fmaxf(mm, sm_m[r][g]);
    const float mu = mm == -INFINITY ? 0.f : mm;
    float ov = 0.f, lv = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float f = __builtin_amdgcn_exp2f(sm_m[r][g] - mu);
      ov = fmaf(sm_o[r][g][d], f, ov);
      lv = fmaf(sm_l[r][g], f, lv);
    }
    const int64_t pidx = part_base + (int64_t)g * a.splits;  // [b][hk*G + g][s]
    a.part_o[pidx * D + d] = ov;
    if (d == 0) {
      a.part_ml[pidx * 2] = mm;
      a.part_ml[pidx * 2 + 1] = lv;
    }
  }
}

// One wave per (sequence, QO head); lanes own D/64 output elements each.
template <int D>
__global__ void __launch_bounds__(256) decode_combine(DecArgs a) {
  constexpr int PER = D / 64;
  const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  if (wave >= a.batch * a.h_q) return;
  const int64_t base = (int64_t)wave * a.splits;
  float mm = -INFINITY;
  for (int s = lane; s < a.splits; s += 64) mm = fmaxf(mm, a.part_ml[(base + s) * 2]);
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mm = fmaxf(mm, __shfl_xor(mm, off));
  const float mu = mm == -INFINITY ? 0.f : mm;
  float ov[PER], lv = 0.f;
#pragma unroll
  for (int t = 0; t < PER; ++t) ov[t] = 0.f;
  for (int s = 0; s < a.splits; ++s) {
    const float ms = a.part_ml[(base + s) * 2];
    const float f = __builtin_amdgcn_exp2f(ms - mu);
    lv = fmaf(a.part_ml[(base + s) * 2 + 1], f, lv);
#pragma unroll
    for (int t = 0; t < PER; ++t) ov[t] = fmaf(a.part_o[(base + s) * D + lane * PER + t], f, ov[t]);
  }
  const float inv = lv > 0.f ? 1.f / lv : 0.f;
#pragma unroll
  for (int t = 0; t < PER; ++t) a.o[(int64_t)wave * D + lane * PER + t] = (__bf16)(ov[t] * inv);
  if (lane == 0) a.lse[wave] = lv > 0.f ? (mm + __log2f(lv)) * kLn2 : -INFINITY;
}

// An upper bound of the visible keys of any (sequence, KV head): sink + near +
// the long-range width, at most n_max.
int32_t max_visible(const cowa_decode_params& p) {
  int64_t v = 0;
  if (p.windows) {
    for (int h = 0; h < p.h_k; ++h) {
      const cowa_window& w = p.windows[h];
      const int64_t x = (int64_t)w.sink + w.near + w.width;
      v = x > v ? x : v;
    }
  } else {
    const int64_t span = p.n_max - (int64_t)p.w_sink - p.w_near;
    const int64_t width = span > 0 ? (span + p.h_k_total - 1) / p.h_k_total : 0;
    v = (int64_t)p.w_sink + p.w_near + width;
  }
  return (int32_t)(v < p.n_max ? v : p.n_max);
}

template <int D, int G>
hipError_t launch_dg(DecArgs a, const cowa_window* windows, hipStream_t stream) {
  if (!windows) {
    a.explicit_win = 0;
    a.head_base = 0;
    hipLaunchKernelGGL((decode_split<D, G>), dim3(a.splits, a.h_k, a.batch), dim3(256), 0, stream, a);
  } else {
    a.explicit_win = 1;
    for (int h0 = 0; h0 < a.h_k; h0 += kHeadsPerLaunch) {
      const int nh = a.h_k - h0 < kHeadsPerLaunch ? a.h_k - h0 : kHeadsPerLaunch;
      a.head_base = h0;
      for (int x = 0; x < nh; ++x) {
        const cowa_window& w = windows[h0 + x];
        const int64_t lo = (int64_t)w.near + w.gap, hi = lo + w.width, cap = int64_t(1) << 30;
        a.win[x] = WinDesc{w.sink, w.near, (int32_t)(lo < cap ? lo : cap), (int32_t)(hi < cap ? hi : cap)};
      }
      hipLaunchKernelGGL((decode_split<D, G>), dim3(a.splits, nh, a.batch), dim3(256), 0, stream, a);
    }
  }
  const int waves = a.batch * a.h_q;
  hipLaunchKernelGGL(decode_combine<D>, dim3((waves + 3) / 4), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

// Default split size: about kTargetPrograms split programs in total (four
// per compute unit of an MI355X), each streaming one contiguous share of a
// (sequence, KV head)'s visible keys; at least kDefaultSplitKeys keys, a
// multiple of 256.  Fewer, longer splits amortise each program's start-up
// (the first loads' latency, the key-run set-up) and its merge.
int32_t decode_split_keys(const cowa_decode_params& p) {
  if (p.split_keys > 0) return p.split_keys;
  const int64_t per = (int64_t)p.batch * p.h_k;
  const int64_t splits = per >= kTargetPrograms ? 1 : (kTargetPrograms + per - 1) / per;
  const int64_t v = max_visible(p);
  int64_t sk = (v + splits - 1) / splits;
  sk = (sk + 255) / 256 * 256;
  return (int32_t)(sk < kDefaultSplitKeys ? kDefaultSplitKeys : sk);
}

int32_t decode_num_splits(const cowa_decode_params& p) {
  const int32_t sk = decode_split_keys(p);
  const int32_t v = max_visible(p);
  return v > 0 ? (v + sk - 1) / sk : 1;
}

size_t decode_workspace_bytes(const cowa_decode_params& p) {
  const size_t parts = (size_t)p.batch * p.h_q * decode_num_splits(p);
  const size_t o_bytes = (parts * p.head_dim * sizeof(float) + 255) & ~size_t(255);
  return o_bytes + ((parts * 2 * sizeof(float) + 255) & ~size_t(255));
}

// Scratch of the allocation-free decoding entry point: the split partials live
// in this file-scope device array (one copy per GPU, held until the process
// ends) instead of a caller workspace.  Host code never uses the array's name
// as an address: decode_scratch() looks the device address up once per device
// and every launch takes that pointer.
__device__ __align__(256) unsigned char scratch[kDecodeScratchBytes];

hipError_t decode_scratch(void** ptr) {
  int dev = -1;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  static std::mutex mu;
  static std::map<int, void*> addr;  // device -> address of its copy of `scratch`
  std::lock_guard<std::mutex> lock(mu);
  auto it = addr.find(dev);
  if (it == addr.end()) {
    void* a = nullptr;
    err = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    if (a == nullptr) return hipErrorInvalidSymbol;
    it = addr.emplace(dev, a).first;
  }
  *ptr = it->second;
  return hipSuccess;
}

bool decode_supported(int head_dim, int group) {
  return (head_dim == 64 || head_dim == 128) && (group == 1 || group == 2 || group == 4 || group == 8);
}

hipError_t launch_decode(const cowa_decode_params& p, const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* seqlens, void* o, float* lse, void* ws, hipStream_t stream) {
  DecArgs a;
  a.q = static_cast<const __bf16*>(q);
  a.kc = static_cast<const __bf16*>(k_cache);
  a.vc = static_cast<const __bf16*>(v_cache);
  a.seqlens = seqlens;
  a.o = static_cast<__bf16*>(o);
  a.lse = lse;
  a.batch = p.batch; a.h_q = p.h_q; a.h_k = p.h_k; a.n_max = p.n_max; a.w_sink = p.w_sink; a.w_near = p.w_near;
  a.h_total = p.h_k_total; a.h_offset = p.h_k_offset;
  a.splits = decode_num_splits(p);
  a.split_keys = decode_split_keys(p);
  a.c = p.softmax_scale * kLog2e;
  const size_t parts = (size_t)p.batch * p.h_q * a.splits;
  a.part_o = static_cast<float*>(ws);
  a.part_ml = reinterpret_cast<float*>(static_cast<char*>(ws) + ((parts * p.head_dim * sizeof(float) + 255) & ~size_t(255)));
  const int G = p.h_q / p.h_k;
#define COWA_DEC_CASE(D_, G_) if (p.head_dim == D_ && G == G_) return launch_dg<D_, G_>(a, p.windows, stream);
  COWA_DEC_CASE(128, 4) COWA_DEC_CASE(128, 1) COWA_DEC_CASE(128, 2) COWA_DEC_CASE(128, 8)
  COWA_DEC_CASE(64, 4) COWA_DEC_CASE(64, 1) COWA_DEC_CASE(64, 2) COWA_DEC_CASE(64, 8)
#undef COWA_DEC_CASE
  return hipErrorInvalidValue;
}

}  // namespace cowa
