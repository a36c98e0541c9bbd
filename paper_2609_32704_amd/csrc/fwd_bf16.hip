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
  static constexpr int NCH = BK / 32;     // 32-key chunks per block
  static constexpr int NG = 2 * KSD + MTD;  // MFMA groups per chunk (NTQ MFMAs each)
  static constexpr int WPH = BQ / NQW;    // waves per QO head
  using T = SwzTile<D, BK>;
  static constexpr int MAIN_BYTES = 4 * T::BYTES;  // K and V of two blocks; then the row's entry lists
  static constexpr int LDS_MAX = 160 * 1024;
  static int lds_bytes(int n_kt) { return MAIN_BYTES + 4 * n_kt + 16; }  // + a vote word
  static int max_kblocks() { return (LDS_MAX - MAIN_BYTES - 16) / 4; }
  static_assert(2 * KSD == MTD, "S and O groups alternate one to one");
};

// S^T = K Q^T products with the accumulator in VGPRs (read by the softmax on the
// vector ALUs) while O^T accumulates in AGPRs: written as assembly because the
// compiler gives all products of a kernel one accumulator register file.  The
// compiler does not see these as matrix instructions and inserts no wait states
// for them, so the schedule keeps their results at least four products away
// from any reader (the softmax of a chunk runs one chunk after its S^T; the
// k-steps of one tile are four products apart), and a block ends with explicit
// wait states before its last S^T can be read.
__device__ inline f32x4 mfma_v0(const bf16x8& a, const bf16x8& b) {
  f32x4 d;
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=&v"(d) : "v"(a), "a"(b));
  return d;
}
__device__ inline f32x4 mfma_v(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  // accumulator input not tied to the output: the register allocator never
  // needs a copy of a result that may still be in flight
  f32x4 d;
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %3" : "=&v"(d) : "v"(a), "a"(b), "v"(c));
  return d;
}

// max(a, b, c) in one instruction (fmaxf would first quiet each operand that
// the compiler cannot prove canonical: the products above are opaque to it)
__device__ inline float max3(float a, float b, float c) {
  float d;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
  return d;
}

#ifndef FWD_OPIN
#define FWD_OPIN "a"
#endif
#ifndef FWD_QPIN
#define FWD_QPIN "a"
#endif
template <int D, int BQ, int BK>
__global__ void __launch_bounds__(256) fwd_bf16_kernel(cowa_params p, SchedView sv, int hpw, int n_hgroups,
                                                       const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                                                       const __bf16* __restrict__ v, __bf16* __restrict__ o,
                                                       float* __restrict__ lse) {
  using C = FwdCfg<D, BQ, BK>;
  using T = typename C::T;
  constexpr int NTQ = C::NTQ, KSD = C::KSD, MTD = C::MTD, NCH = C::NCH, NG = C::NG;
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
  // LDS: K of block t in K buffer t % 2, V of block t in V buffer t % 2
  auto kbuf_off = [](int t) { return (t & 1) * 2 * T::BYTES; };
  auto vbuf_off = [](int t) { return (t & 1) * 2 * T::BYTES + T::BYTES; };
  auto stage_k = [&](int t) {
    load_tile_asm_nw<D, BK>(kbase, (int)(entry_at(t) >> 1) * BK, p.n_k, smem_base + kbuf_off(t), wave, nw, lane);
  };
  auto stage_v = [&](int t) {
    load_tile_asm_nw<D, BK>(vbase, (int)(entry_at(t) >> 1) * BK, p.n_k, smem_base + vbuf_off(t), wave, nw, lane);
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
  // The exponent offset m (base 2, per query column) is fixed once per row:
  // the maximum over the first 32 keys of the row's first block.  P = exp2(s c - m)
  // can then exceed 1, but O and l share the offset, so O / l and
  // LSE = (m + log2 l) ln 2 are unaffected; no O rescaling is ever needed.  If a
  // later score exceeds m by more than kLimit (P > 2^kLimit, where bf16 P and
  // fp32 sums would approach their range), the workgroup runs the row again
  // with m set to the row maximum found by the first pass.
  constexpr float kLimit = 64.f;
  float m_fix[NTQ], m_hi[NTQ], l_run[NTQ], mu[NTQ];  // m_hi: this lane's maximum raw score per column
#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) m_fix[nt] = -INFINITY;
  const float c = p.softmax_scale * kLog2e;
  int offr[KSD], offt[MTD];
#pragma unroll
  for (int ks = 0; ks < KSD; ++ks) offr[ks] = row8_off<D>(lr, lg, ks);
#pragma unroll
  for (int md = 0; md < MTD; ++md) offt[md] = tr8_off<D>(lr, lg, md);

  // Software pipeline over the row's 32-key chunks.  While the matrix cores
  // compute S^T of chunk n (K fragments of the current block) and O^T += V^T P^T
  // of a chunk one block back (V fragments of the previous block), the vector
  // ALUs turn S^T of chunk n - 1 into P^T: the two streams are independent, so
  // the exponentials of the softmax hide under the products.
  f32x4 sacc[2][2][NTQ];  // S^T of two chunks ([chunk % 2][16-key tile][query tile])
  bf16x8 pb[NCH][NTQ];    // P^T of the chunks of one block, as B operands

  // The softmax of one chunk is split into 32 element steps (element e: query
  // tile e / 8, key tile (e / 4) % 2, row e % 4), spread evenly over NS slots
  // of one MFMA each: first exponent, then sum, running maximum and packing.
  float pv[32];  // exponentials in flight between the two halves of an element step
  auto soft_a = [&](auto ec, auto rpc, bool masked, int key0) __attribute__((always_inline)) {
    constexpr int e = decltype(ec)::value, rp = decltype(rpc)::value;
    constexpr int nt = e / 8, tt = (e / 4) % 2, rr = e % 4;
    if (masked)
      sacc[rp][tt][nt][rr] += legal32(g, q_first + nt * 16 + lr, key0 + tt * 16 + 4 * lg + rr) ? 0.f : -INFINITY;
    pv[e] = __builtin_amdgcn_exp2f(fmaf(sacc[rp][tt][nt][rr], c, -mu[nt]));
  };
  auto soft_b = [&](auto ec, auto rpc, auto psc) __attribute__((always_inline)) {
    constexpr int e = decltype(ec)::value, rp = decltype(rpc)::value, ps = decltype(psc)::value;
    constexpr int nt = e / 8, tt = (e / 4) % 2, rr = e % 4;
    l_run[nt] += pv[e];
    if constexpr (rr & 1) {
      m_hi[nt] = max3(m_hi[nt], sacc[rp][tt][nt][rr - 1], sacc[rp][tt][nt][rr]);
      pb[ps][nt][4 * tt + rr - 1] = (__bf16)pv[e - 1];
      pb[ps][nt][4 * tt + rr] = (__bf16)pv[e];
    }
  };
  // the element steps of slot `slot` out of NS
  auto soft_slot = [&](auto slotc, auto nsc, auto rpc, auto psc, bool masked, int key0) __attribute__((always_inline)) {
    constexpr int slot = decltype(slotc)::value, NS = decltype(nsc)::value;
    constexpr int LAG = NS >= 64 ? NS / 64 : 0;  // slots between the two halves of an element step
    static_for<32>([&](auto ec) {
      constexpr int e = decltype(ec)::value;
      constexpr int sa = e * NS / 32;
      if constexpr (sa == slot) soft_a(ec, rpc, masked, key0);
      if constexpr (sa + LAG == slot) soft_b(ec, rpc, psc);
    });
  };

  // O^T += V^T P^T for chunk j of a block (V tile Vt) and S^T of chunk j (K tile
  // Kt), group by group, fragments read PF groups ahead.  gi -> S group or O group.
  constexpr int PF = 2;
  int k_prev = 0;  // first key of the previous block
  // One block of the pipeline.  FIRST: the row's first block (no previous block:
  // no O^T products, no softmax before the first chunk).  MPREV / MCUR: the
  // chunks softmaxed here from the previous / this block need the element mask.
  auto step = [&](int t, auto firstc, auto mprevc, auto mcurc) __attribute__((always_inline)) {
    constexpr bool FIRST = decltype(firstc)::value, MPREV = decltype(mprevc)::value, MCUR = decltype(mcurc)::value;
    const int k_first = (int)(entry_at(t) >> 1) * BK;
    if (t + 1 < n_ent) stage_k(t + 1);  // K buffer of block t - 1: free
    stage_v(t);                         // V buffer of block t - 2: free
    const unsigned char* Kt = smem + kbuf_off(t);
    const unsigned char* Vp = smem + vbuf_off(t + 1);  // V of block t - 1
    constexpr int NGS = NCH * NG;
    bf16x8 fa[PF + 1];
    auto load = [&](auto gc, bf16x8& dst) __attribute__((always_inline)) {
      constexpr int GG = decltype(gc)::value, j = GG / NG, gi = GG % NG;
      constexpr bool S = NCH >= 2 ? (gi % 2 == 0) : (gi < 2 * KSD);
      constexpr int x = NCH >= 2 ? gi / 2 : (S ? gi : gi - 2 * KSD);
      if constexpr (S) {
        dst = ld_row8(Kt + offr[x % KSD] + (j * 32 + (x / KSD) * 16) * D * 2);
      } else if constexpr (!FIRST) {
        dst = ld_tr8(Vp + offt[x] + j * 32 * D * 2, D * 2);
      }
    };
    static_for<PF>([&](auto ic) { load(ic, fa[decltype(ic)::value]); });
    __builtin_amdgcn_sched_barrier(0);
    static_for<NGS>([&](auto gc) {
      constexpr int GG = decltype(gc)::value, j = GG / NG, gi = GG % NG;
      constexpr bool S = NCH >= 2 ? (gi % 2 == 0) : (gi < 2 * KSD);
      constexpr int x = NCH >= 2 ? gi / 2 : (S ? gi : gi - 2 * KSD);
      if constexpr (GG + PF < NGS) load(std::integral_constant<int, GG + PF>{}, fa[(GG + PF) % (PF + 1)]);
      const bf16x8& a = fa[GG % (PF + 1)];
      // the softmax of the chunk before chunk j: chunk j - 1 of this block, or
      // the last chunk of the previous block; spread over all groups, or for a
      // one-chunk block over the S groups (its P^T is consumed within the block)
      constexpr int NS = NCH >= 2 ? 4 * NG : 4 * 2 * KSD;
      constexpr int ps = (j + NCH - 1) % NCH;
      static_for<NTQ>([&](auto mc) {
        constexpr int m = decltype(mc)::value;
        if constexpr (S) {
          constexpr int tt = x / KSD, ks = x % KSD;
          if constexpr (ks == 0)
            sacc[j & 1][tt][m] = mfma_v0(a, qf[m][ks]);
          else
            sacc[j & 1][tt][m] = mfma_v(a, qf[m][ks], sacc[j & 1][tt][m]);
        } else if constexpr (!FIRST) {
          oacc[x][m] = mfma16(a, pb[j][m], oacc[x][m]);
        }
        constexpr int slot = gi * NTQ + m;
        if constexpr (!(FIRST && j == 0) && slot < NS) {
          using SL = std::integral_constant<int, slot>;
          using NSC = std::integral_constant<int, NS>;
          using PS = std::integral_constant<int, ps>;
          if constexpr (j == 0)
            soft_slot(SL{}, NSC{}, std::integral_constant<int, 1>{}, PS{}, MPREV, k_prev + (NCH - 1) * 32);
          else
            soft_slot(SL{}, NSC{}, std::integral_constant<int, (j + 1) & 1>{}, PS{}, MCUR, k_first + (j - 1) * 32);
        }
        __builtin_amdgcn_sched_barrier(0);
      });
    });
    // the last S^T products of the block may still be in flight (a first block
    // has no O^T products after them): 16 wait states before anything reads them
    asm volatile("s_nop 7\n\ts_nop 7");
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (NCH == 1) {
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int nt = 0; nt < NTQ; ++nt) sacc[1][tt][nt] = sacc[0][tt][nt];
    }
    // register placement: O^T accumulators and Q^T fragments in AGPRs (read
    // directly by the matrix cores), S^T and P^T in VGPRs; these emit nothing
#pragma unroll
    for (int md = 0; md < MTD; ++md)
#pragma unroll
      for (int nt = 0; nt < NTQ; ++nt) asm volatile("" : "+" FWD_OPIN(oacc[md][nt]));
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt)
#pragma unroll
      for (int ks = 0; ks < KSD; ++ks) asm volatile("" : "+" FWD_QPIN(qf[nt][ks]));
    k_prev = k_first;
    __builtin_amdgcn_s_waitcnt(0);  // block t + 1's K and block t's V have landed
    __syncthreads();                 // ... for every wave, and the freed buffers are no longer read
  };
  // after the last block: the softmax of its last chunk, then its O^T products
  auto drain = [&](int t) __attribute__((always_inline)) {
    using R1 = std::integral_constant<int, 1>;
    static_for<32>([&](auto ec) { soft_a(ec, R1{}, true, k_prev + (NCH - 1) * 32); });
    static_for<32>([&](auto ec) { soft_b(ec, R1{}, std::integral_constant<int, NCH - 1>{}); });
    const unsigned char* Vt = smem + vbuf_off(t);
    static_for<NCH * MTD>([&](auto gc) {
      constexpr int GG = decltype(gc)::value, j = GG / MTD, md = GG % MTD;
      const bf16x8 a = ld_tr8(Vt + offt[md] + j * 32 * D * 2, D * 2);
#pragma unroll
      for (int nt = 0; nt < NTQ; ++nt) oacc[md][nt] = mfma16(a, pb[j][nt], oacc[md][nt]);
    });
  };

  for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt) {
      m_hi[nt] = -INFINITY;
      l_run[nt] = 0.f;
#pragma unroll
      for (int md = 0; md < MTD; ++md) oacc[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    if (n_ent > 0) stage_k(0);
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
            sacc[0][tt][nt] = mfma16(a, qf[nt][ks], ks == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : sacc[0][tt][nt]);
        }
#pragma unroll
      for (int nt = 0; nt < NTQ; ++nt) {
        float cm = -INFINITY;
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const float sv2 = sacc[0][tt][nt][rr] + (legal32(g, q_first + nt * 16 + lr, key0 + tt * 16 + 4 * lg + rr) ? 0.f : -INFINITY);
            cm = fmaxf(cm, sv2);
          }
        cm = fmaxf(cm, __shfl_xor(cm, 16));
        cm = fmaxf(cm, __shfl_xor(cm, 32));
        m_fix[nt] = cm * c;  // -inf for a column without a legal key there
      }
    }
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt) mu[nt] = m_fix[nt] == -INFINITY ? 0.f : m_fix[nt];
    using TT = std::true_type;
    using FF = std::false_type;
    int t = 0;
    if (n_full > 0) {
      step(0, TT{}, FF{}, FF{});
      for (t = 1; t < n_full; ++t) step(t, FF{}, FF{}, FF{});
    }
    if (t < n_ent) {
      if (t == 0) {
        step(0, TT{}, TT{}, TT{});
        t = 1;
      }
      for (; t < n_ent; ++t) step(t, FF{}, TT{}, TT{});
    }
    if (n_ent > 0) drain(n_ent - 1);
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
    for (int nt = 0; nt < NTQ; ++nt) m_fix[nt] = m_hi[nt];
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
