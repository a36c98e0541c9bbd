// CoWA forward in bfloat16 on the CDNA4 matrix cores (Alg. 1).
//
// Work decomposition.  One workgroup per (QO block i, group of HPW QO heads
// that share one KV head, sequence b): every QO head of a GQA group has the
// same block set J_{h_k}(i), so the heads of a workgroup share each K/V block
// staged in LDS.  Each 64-lane wave owns NQW query rows of one head (up to
// 256 rows and 8 waves per workgroup).
//
// Per KV block j of J_{h_k}(i), visited in the schedule's descending order:
//   * K_j and V_j are copied global -> LDS with direct 16-byte loads
//     (global_load_lds), double buffered: block e+1 is in flight while block e
//     is computed.  Rows are stored unpadded with their 16-byte chunks XOR
//     swizzled by row, so both the row reads of K and the transposed reads of
//     V hit distinct banks.
//   * S^T = K_j Q^T on v_mfma_f32_16x16x32_bf16 (fp32 accumulate); Q^T stays
//     in registers for the whole block.  Computing the transpose puts one
//     query per lane column, which is the B-operand layout of the second
//     product, so P never leaves registers.
//   * only blocks flagged partial evaluate the element mask of Eq. fwa_support;
//   * online softmax in registers, base 2, with scale * log2(e) folded into one
//     fused multiply-add per score; the O accumulator is rescaled only when a
//     running maximum moved;
//   * O^T += V_j^T P^T; the V^T fragments come straight from the row-major
//     V_j in LDS through the transposing LDS read (ds_read_b64_tr_b16).
// Finally O = O / l and LSE = (m + log2 l) ln 2 (natural log).
#include "internal.h"
#include "window_rule.h"
#include "mfma_tiles.h"

namespace cowa {
namespace {

template <int D, int BQ, int BK>
struct FwdCfg {
  static constexpr int NQW = 64;          // query rows per wave
  static constexpr int NTQ = NQW / 16;    // query tiles per wave (columns of S^T)
  static constexpr int KSD = D / 32;      // k-steps over d
  static constexpr int MTD = D / 16;      // d tiles of O^T
  static constexpr int NCH = BK / 32;     // 32-key chunks per block (one k-step of O^T += V^T P^T)
  static constexpr int WPH = BQ / NQW;    // waves per QO head
  using T = SwzTile<D, BK>;
  static constexpr int MAIN_BYTES = 4 * T::BYTES;  // K, V of two blocks; then the row's entry lists
  static constexpr int LDS_MAX = 160 * 1024;
  static int lds_bytes(int n_kt) { return MAIN_BYTES + 4 * n_kt + 16; }  // + a vote word
  static int max_kblocks() { return (LDS_MAX - MAIN_BYTES - 16) / 4; }
};

template <int D, int BQ, int BK>
__global__ void __launch_bounds__(256) fwd_bf16_kernel(cowa_params p, SchedView sv, int hpw, int n_hgroups,
                                                       const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                                                       const __bf16* __restrict__ v, __bf16* __restrict__ o,
                                                       float* __restrict__ lse) {
  using C = FwdCfg<D, BQ, BK>;
  using T = typename C::T;
  constexpr int NTQ = C::NTQ, KSD = C::KSD, MTD = C::MTD, NCH = C::NCH;
  extern __shared__ __align__(1024) unsigned char smem[];

  const int nw = blockDim.x >> 6;
  const int G = p.h_q / p.h_k;
  const int total = sv.n_qt * n_hgroups * p.batch;
  const int work = xcd_remap(blockIdx.x, total);
  const int per_i = n_hgroups * p.batch;
  const int i = sv.n_qt - 1 - work / per_i;  // latest (longest) QO blocks first
  const int rest = work % per_i;
  const int hgi = rest % n_hgroups, b = rest / n_hgroups;
  const int hk = hgi / (G / hpw);
  const int h0 = hgi * hpw;  // first QO head of this workgroup (all in KV group hk)

  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int h = h0 + wave / C::WPH;
  const int q_first = i * BQ + (wave % C::WPH) * C::NQW;
  const Geo32 g = geo32(make_geo(p.n_q, p.n_k, p.w_sink, p.w_near, BQ, BK, p.h_k_offset + hk, p.h_k_total));

  const __bf16* kbase = k + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  const __bf16* vbase = v + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  const uint32_t smem_base = lds_addr(smem);

  // the row's entries, split into full (from the front) and partial (from the back) lists
  const int r = hk * sv.n_qt + i;
  const int e0 = sv.fwd_row_ptr[r], e1 = sv.fwd_row_ptr[r + 1];
  const int n_ent = e1 - e0;
  const int cap = sv.n_kt;
  uint32_t* list = reinterpret_cast<uint32_t*>(smem + C::MAIN_BYTES);
  int n_full = 0;
  for (int c0 = 0; c0 < n_ent; c0 += 64) {
    const bool in = c0 + lane < n_ent;
    const uint32_t ent = in ? sv.fwd_ent[e0 + c0 + lane] : 0u;
    const uint64_t full = __ballot(in && !(ent & 1u));
    const uint64_t part = __ballot(in && (ent & 1u));
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    if (wave == 0 && in) {
      if (ent & 1u)
        list[cap - 1 - (c0 - n_full + __popcll(part & below))] = ent;
      else
        list[n_full + __popcll(full & below)] = ent;
    }
    n_full += __popcll(full);
  }
  auto entry_at = [&](int t) -> uint32_t {
    const int tt = t < n_ent ? t : n_ent - 1;
    const int idx = tt < n_full ? tt : cap - 1 - (tt - n_full);
    return __builtin_amdgcn_readfirstlane(list[idx]);
  };
  auto stage = [&](uint32_t ent, int buf) {
    const int kf = (int)(ent >> 1) * BK;
    load_tile_asm_nw<D, BK>(kbase, kf, p.n_k, smem_base + buf * 2 * T::BYTES, wave, nw, lane);
    load_tile_asm_nw<D, BK>(vbase, kf, p.n_k, smem_base + buf * 2 * T::BYTES + T::BYTES, wave, nw, lane);
  };
  __syncthreads();  // the lists are in LDS

  // Q^T fragments (B operands): query column nt*16 + lr, d = ks*32 + 8*lg + 0..7
  const int64_t row_base = ((int64_t)b * p.h_q + h) * p.n_q;
  bf16x8 qf[NTQ][KSD];
#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) {
    const int qp = q_first + nt * 16 + lr;
    const bool ok = qp < p.n_q;
    const __bf16* qrow = q + (row_base + (ok ? qp : 0)) * D;
#pragma unroll
    for (int ks = 0; ks < KSD; ++ks) {
      const bf16x8 val = *reinterpret_cast<const bf16x8*>(qrow + ks * 32 + 8 * lg);
      qf[nt][ks] = ok ? val : bf16x8{};
    }
  }
  f32x4 oacc[MTD][NTQ];  // O^T: rows d, columns queries
#pragma unroll
  for (int md = 0; md < MTD; ++md)
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt) oacc[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  // The exponent offset m (base 2, per query column) is fixed once per row:
  // the maximum over the first 32 keys of the row's first block.  P = exp2(s c - m)
  // can then exceed 1, but O and l share the offset, so O / l and
  // LSE = (m + log2 l) ln 2 are unaffected; no O rescaling is ever needed.  If a
  // later score exceeds m by more than kLimit (P > 2^kLimit, where bf16 P and
  // fp32 sums would approach their range), the workgroup runs the row again
  // with m set to the row maximum found by the first pass.
  constexpr float kLimit = 64.f;
  float m_fix[NTQ], m_hi[NTQ], l_run[NTQ];  // m_hi: this lane's maximum raw score per column
#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) {
    m_fix[nt] = -INFINITY;
    m_hi[nt] = -INFINITY;
    l_run[nt] = 0.f;
  }
  const float c = p.softmax_scale * kLog2e;
  int offr[KSD], offt[MTD];
#pragma unroll
  for (int ks = 0; ks < KSD; ++ks) offr[ks] = row8_off<D>(lr, lg, ks);
#pragma unroll
  for (int md = 0; md < MTD; ++md) offt[md] = tr8_off<D>(lr, lg, md);

  f32x4 sacc[2][NTQ];    // S^T of the chunk's two 16-key tiles: rows keys 4 lg + rr, column query 16 nt + lr
  bf16x8 pb[2][NTQ];     // P^T of the current and the previous chunk as B operands

  // softmax of a chunk (key0: its first key) into pb[sl]
  auto softmax = [&](int sl, bool masked, int key0) __attribute__((always_inline)) {
    if (masked) {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int nt = 0; nt < NTQ; ++nt)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr)
            // an add that reads the accumulator: a plain masked store of -inf
            // into an MFMA destination could be overtaken by the MFMA write
            sacc[t][nt][rr] += legal32(g, q_first + nt * 16 + lr, key0 + t * 16 + 4 * lg + rr) ? 0.f : -INFINITY;
    }
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt) {
      const float lm = fmaxf(fmaxf(fmaxf(sacc[0][nt][0], sacc[0][nt][1]), fmaxf(sacc[0][nt][2], sacc[0][nt][3])),
                             fmaxf(fmaxf(sacc[1][nt][0], sacc[1][nt][1]), fmaxf(sacc[1][nt][2], sacc[1][nt][3])));
      m_hi[nt] = fmaxf(m_hi[nt], lm);
    }
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt) {
      const float mu = m_fix[nt] == -INFINITY ? 0.f : m_fix[nt];
      float ls = 0.f;
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const float pv = __builtin_amdgcn_exp2f(fmaf(sacc[t][nt][rr], c, -mu));
          ls += pv;
          pb[sl][nt][4 * t + rr] = (__bf16)pv;
        }
      l_run[nt] += ls;
    }
  };

  // A block: for each chunk, 2 KSD groups of S^T (one K row fragment, NTQ
  // MFMAs each), then MTD groups of O^T += V^T P^T for the previous chunk (one
  // V^T fragment, NTQ MFMAs each) beside this chunk's softmax; a last MTD
  // groups for the block's final chunk.  Fragments are read one group ahead.
  constexpr int GPC = 2 * KSD + MTD, NGB = NCH * GPC + MTD;
  auto load_g = [&](const unsigned char* Kt, const unsigned char* Vt, int gg, bf16x8& fa) __attribute__((always_inline)) {
    if (gg < NCH * GPC) {
      const int ch = gg / GPC, rr = gg % GPC;
      if (rr < 2 * KSD) {
        const int t = rr / KSD, ks = rr % KSD;
        fa = ld_row8(Kt + offr[ks] + (ch * 32 + t * 16) * D * 2);
      } else if (ch > 0) {
        fa = ld_tr8(Vt + offt[rr - 2 * KSD] + (ch - 1) * 32 * D * 2, D * 2);
      }
    } else {
      fa = ld_tr8(Vt + offt[gg - NCH * GPC] + (NCH - 1) * 32 * D * 2, D * 2);
    }
  };

  auto block = [&](int t, bool masked) {
    const int buf = t & 1;
    const uint32_t ent = entry_at(t);
    const int k_first = (int)(ent >> 1) * BK;
    if (t + 1 < n_ent) stage(entry_at(t + 1), buf ^ 1);  // prefetch the next block
    const unsigned char* Kt = smem + buf * 2 * T::BYTES;
    const unsigned char* Vt = Kt + T::BYTES;
    bf16x8 fa[2];
    load_g(Kt, Vt, 0, fa[0]);
    __builtin_amdgcn_sched_barrier(0);
    static_for<NGB>([&](auto ic) {
      constexpr int gg = decltype(ic)::value;
      if constexpr (gg + 1 < NGB) load_g(Kt, Vt, gg + 1, fa[(gg + 1) & 1]);
      const bf16x8& a = fa[gg & 1];
      if constexpr (gg < NCH * GPC) {
        constexpr int ch = gg / GPC, rr = gg % GPC;
        if constexpr (rr < 2 * KSD) {
          constexpr int tt = rr / KSD, ks = rr % KSD;
#pragma unroll
          for (int nt = 0; nt < NTQ; ++nt)
            sacc[tt][nt] = mfma16(a, qf[nt][ks], ks == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : sacc[tt][nt]);
        } else {
          constexpr int md = rr - 2 * KSD;
          if constexpr (ch > 0) {
#pragma unroll
            for (int nt = 0; nt < NTQ; ++nt) oacc[md][nt] = mfma16(a, pb[(ch - 1) & 1][nt], oacc[md][nt]);
          }
          if constexpr (md == 0) softmax(ch & 1, masked, k_first + ch * 32);
        }
      } else {
        constexpr int md = gg - NCH * GPC;
#pragma unroll
        for (int nt = 0; nt < NTQ; ++nt) oacc[md][nt] = mfma16(a, pb[(NCH - 1) & 1][nt], oacc[md][nt]);
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    // register placement: O^T accumulators in VGPRs, Q^T fragments in AGPRs
    // (read directly as B operands); these statements emit nothing
#pragma unroll
    for (int md = 0; md < MTD; ++md)
#pragma unroll
      for (int nt = 0; nt < NTQ; ++nt) asm volatile("" : "+v"(oacc[md][nt]));
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt)
#pragma unroll
      for (int ks = 0; ks < KSD; ++ks) asm volatile("" : "+a"(qf[nt][ks]));
    __builtin_amdgcn_s_waitcnt(0);  // the next block has landed
    __syncthreads();                 // ... for every wave, and this block is no longer read
  };
  for (int pass = 0; pass < 2; ++pass) {
    if (n_ent > 0) stage(entry_at(0), 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (pass == 0 && n_ent > 0) {
      // offsets from the first 32 keys of the row's first block (in processing
      // order: a full block when the row has one; its first key is legal for
      // every query of a causal row either way)
      const int key0 = (int)(entry_at(0) >> 1) * BK;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int ks = 0; ks < KSD; ++ks) {
          const bf16x8 a = ld_row8(smem + offr[ks] + tt * 16 * D * 2);
#pragma unroll
          for (int nt = 0; nt < NTQ; ++nt)
            sacc[tt][nt] = mfma16(a, qf[nt][ks], ks == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : sacc[tt][nt]);
        }
#pragma unroll
      for (int nt = 0; nt < NTQ; ++nt) {
        float cm = -INFINITY;
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const float sv2 = sacc[tt][nt][rr] + (legal32(g, q_first + nt * 16 + lr, key0 + tt * 16 + 4 * lg + rr) ? 0.f : -INFINITY);
            cm = fmaxf(cm, sv2);
          }
        cm = fmaxf(cm, __shfl_xor(cm, 16));
        cm = fmaxf(cm, __shfl_xor(cm, 32));
        m_fix[nt] = cm * c;  // -inf for a column without a legal key there
      }
    }
    int t = 0;
    for (; t < n_full; ++t) block(t, false);
    for (; t < n_ent; ++t) block(t, true);
    // did a score exceed its column's offset by more than kLimit?
    bool far = false;
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt) {
      float cm = m_hi[nt];
      cm = fmaxf(cm, __shfl_xor(cm, 16));
      cm = fmaxf(cm, __shfl_xor(cm, 32));
      m_hi[nt] = cm * c;  // the column's maximum, in exponent units
      // (a column whose offset is unset but which met legal keys later is run again too)
      far |= m_hi[nt] != -INFINITY && (m_fix[nt] == -INFINITY || m_hi[nt] > m_fix[nt] + kLimit);
    }
    // workgroup vote through a word past the block lists
    int* vote = reinterpret_cast<int*>(smem + C::MAIN_BYTES + 4 * cap);
    if (tid == 0) *vote = 0;
    __syncthreads();
    if (far) *vote = 1;
    __syncthreads();
    const bool again = *vote != 0;
    __syncthreads();
    if (!again) break;
    // run the row again with the row maxima as offsets (then P <= 1 everywhere)
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt) {
      m_fix[nt] = m_hi[nt];
      m_hi[nt] = -INFINITY;
      l_run[nt] = 0.f;
#pragma unroll
      for (int md = 0; md < MTD; ++md) oacc[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  }

  // O = O / l; LSE = (m + log2 l) ln 2 (m already in base-2 units)
#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) {
    float lt = l_run[nt];
    lt += __shfl_xor(lt, 16);
    lt += __shfl_xor(lt, 32);
    const int qp = q_first + nt * 16 + lr;
    if (qp >= p.n_q) continue;
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    __bf16* orow = o + (row_base + qp) * D;
#pragma unroll
    for (int md = 0; md < MTD; ++md) {
      bf16x4 ov;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) ov[rr] = (__bf16)(oacc[md][nt][rr] * inv);
      *reinterpret_cast<bf16x4*>(orow + md * 16 + 4 * lg) = ov;
    }
    if (lg == 0) lse[row_base + qp] = lt > 0.f ? (m_fix[nt] + __log2f(lt)) * kLn2 : -INFINITY;
  }
}

template <int D, int BQ, int BK>
hipError_t launch_cfg(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                      void* o, float* lse, hipStream_t stream) {
  using C = FwdCfg<D, BQ, BK>;
  if (sv.n_kt > C::max_kblocks()) return hipErrorInvalidValue;
  auto kern = fwd_bf16_kernel<D, BQ, BK>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_MAX);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const int G = p.h_q / p.h_k;
  int hpw = 256 / BQ;  // QO heads per workgroup: up to 256 query rows (four waves)
  while (hpw > 1 && G % hpw != 0) hpw >>= 1;
  const int n_hgroups = p.h_q / hpw;
  const int waves = hpw * C::WPH;
  const unsigned blocks = (unsigned)sv.n_qt * n_hgroups * p.batch;
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(64 * waves), C::lds_bytes(sv.n_kt), stream, p, sv, hpw, n_hgroups,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), static_cast<const __bf16*>(v),
                     static_cast<__bf16*>(o), lse);
  return hipGetLastError();
}

}  // namespace

int fwd_bf16_max_kblocks(int d, int tk) {
  if (d == 128) return tk == 128 ? FwdCfg<128, 128, 128>::max_kblocks() : tk == 64 ? FwdCfg<128, 128, 64>::max_kblocks()
                                                                                 : FwdCfg<128, 128, 32>::max_kblocks();
  return tk == 128 ? FwdCfg<64, 128, 128>::max_kblocks() : tk == 64 ? FwdCfg<64, 128, 64>::max_kblocks()
                                                                     : FwdCfg<64, 128, 32>::max_kblocks();
}

bool fwd_bf16_supported(int d, int tq, int tk) {
  return (d == 64 || d == 128) && (tq == 64 || tq == 128) && (tk == 32 || tk == 64 || tk == 128);
}

hipError_t launch_fwd_bf16(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                           void* o, float* lse, hipStream_t stream) {
#define COWA_FWD_CASE(D_, BQ_, BK_) \
  if (p.head_dim == D_ && p.tile_q == BQ_ && p.tile_k == BK_) return launch_cfg<D_, BQ_, BK_>(p, sv, q, k, v, o, lse, stream);
  COWA_FWD_CASE(128, 128, 128)
  COWA_FWD_CASE(128, 128, 64)
  COWA_FWD_CASE(128, 128, 32)
  COWA_FWD_CASE(128, 64, 128)
  COWA_FWD_CASE(128, 64, 64)
  COWA_FWD_CASE(128, 64, 32)
  COWA_FWD_CASE(64, 128, 128)
  COWA_FWD_CASE(64, 128, 64)
  COWA_FWD_CASE(64, 128, 32)
  COWA_FWD_CASE(64, 64, 128)
  COWA_FWD_CASE(64, 64, 64)
  COWA_FWD_CASE(64, 64, 32)
#undef COWA_FWD_CASE
  return hipErrorInvalidValue;
}

}  // namespace cowa
