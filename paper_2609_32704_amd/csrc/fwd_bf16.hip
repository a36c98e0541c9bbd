// CoWA forward in bfloat16 on the CDNA4 matrix cores (Alg. 1).
//
// Work decomposition.  One workgroup per (QO block i, group of HPW QO heads
// that share one KV head, sequence b): every QO head of a GQA group has the
// same block set J_{h_k}(i), so the heads of a workgroup share each K/V block
// staged in LDS.  Each 64-lane wave owns 64 query rows of one head (up to 256
// rows, four waves, per workgroup).  Workgroups are grouped per XCD so that
// rows sharing K/V blocks run together on one L2 (cluster_item).
//
// Per KV block j of J_{h_k}(i), full blocks first, then partial ones:
//   * K_j and V_j are copied global -> LDS with direct 16-byte buffer loads,
//     double buffered and issued a block (K) or half a block (V) ahead.  Rows
//     are stored unpadded with their 16-byte chunks XOR swizzled by row, so the
//     row reads of K and the transposing reads of V hit distinct banks.
//   * S^T = K_j Q^T on v_mfma_f32_32x32x16_bf16 (fp32 accumulate); Q^T stays in
//     registers for the whole row.  The accumulator layout of S^T is the
//     B-operand layout of P^T for O^T += V^T P^T, so P never leaves registers;
//     the V^T fragments come from the row-major V_j through the transposing
//     LDS read (ds_read_b64_tr_b16).
//   * only blocks flagged partial apply the element mask of Eq. fwa_support,
//     as a 32-bit mask of legal keys per query and chunk;
//   * softmax in base 2 with a per-row exponent offset that moves only at
//     block ends and rarely (see below), the scale * log2(e) folded into one
//     fused multiply-add per score, and the row sum l accumulated from the
//     rounded bf16 P^T that enters O, on the matrix cores (one 16x16x32
//     product per 16 keys with a 0/1 selector as A), which keeps the vector
//     ALUs, the busier unit, for the exponentials;
//   * the 32-key chunks of a row form a software pipeline: S^T of chunk n and
//     O^T of chunk n - 2 on the matrix cores while the vector ALUs exponentiate
//     chunk n - 1.
// Finally O = O / l and LSE = (m + log2 l) ln 2 (natural log); O leaves through
// LDS as whole rows.
//
// Two launches per call (TRACK false, then true).  The first tracks no running
// maximum: its offset moves on the row sums, and rows it cannot finish (an
// overflow, or a column without a starting offset whose sum stays tiny) leave
// LSE = NaN.  The second runs the tracked algorithm described below, but only
// in workgroups holding such a row; the others end at once.
#include "internal.h"
#include "window_rule.h"
#include "mfma_tiles.h"
#include "work_item.h"

namespace cowa {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// S^T = K Q^T products with the accumulator in VGPRs (read by the softmax on the
// vector ALUs) while O^T accumulates in AGPRs: written as assembly because the
// compiler gives all products of a kernel one accumulator register file.  The
// compiler does not see these as matrix instructions and inserts no wait states
// for them, so the schedule keeps every reader of a result at least three
// products behind it (the softmax of a chunk runs one chunk after its S^T; the
// k-steps of one tile are three products apart, or separated by explicit wait
// states), and a block ends with explicit wait states before its last S^T can
// be read.  (A k-step chain accumulates in place; the schedule gives the
// register allocator no reason to copy a result that may still be in flight,
// which the kernel's assembly is checked for.)
__device__ inline f32x16 mfma32_v0(const bf16x8& a, const bf16x8& b) {
  f32x16 d;
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(d) : "v"(a), "a"(b));
  return d;
}
__device__ inline f32x16 mfma32_v(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  f32x16 d = c;
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(d) : "v"(a), "a"(b));
  return d;
}
__device__ inline f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// wait states after the products above before their results are read; the
// accumulators pass through the statement, so no reader is moved above it
__device__ inline void mfma_settle(f32x16& a, f32x16& b) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(a), "+v"(b));
}
__device__ inline void mfma_settle(f32x16 (&r)[2]) { mfma_settle(r[0], r[1]); }

// max(a, b, c) in one instruction (fmaxf would first quiet each operand that
// the compiler cannot prove canonical: the products above are opaque to it)
__device__ inline float max3(float a, float b, float c) {
  float d;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
  return d;
}

template <int D, int BQ, int BK>
struct FwdCfg {
  static constexpr int NQW = 64;          // query rows per wave
  static constexpr int NWF = 256 / NQW;   // waves of a full workgroup (256 query rows)
  static constexpr int NQT = NQW / 32;    // 32-query tiles per wave (columns of S^T)
  static constexpr int KS = D / 16;       // k-steps over d of S^T = K Q^T
  static constexpr int MD = D / 32;       // 32-row d tiles of O^T
  static constexpr int NCH = BK / 32;     // 32-key chunks per block (2 or 4)
  static constexpr int NG = KS + 2 * MD;  // product groups per chunk (NQT products each)
  static constexpr int WPH = BQ / NQW;    // waves per QO head
  using T = SwzTile<D, BK>;
  static constexpr int MAIN_BYTES = 4 * T::BYTES;  // K and V of two blocks; then the row's entry lists
  static constexpr int LDS_MAX = 160 * 1024;
  static constexpr int OUT_PITCH = 2 * D + 16;               // staged output rows (bytes)
  static constexpr int OUT_BYTES = NWF * NQW * OUT_PITCH;    // reuses the K/V buffers and lists at the end
  static int lds_bytes(int n_kt) {                           // + a vote word
    return MAIN_BYTES + 4 * n_kt + 16 > OUT_BYTES ? MAIN_BYTES + 4 * n_kt + 16 : OUT_BYTES;
  }
  static int max_kblocks() { return (LDS_MAX - MAIN_BYTES - 16) / 4; }
  static_assert(KS == 2 * MD, "S and O groups alternate one to one");
  static_assert(NCH == 2 || NCH == 4, "64- or 128-key blocks");
};

// FULL: launched with NWF waves (the fast copy path; a compile-time choice
// keeps the block step free of branches)
template <int D, int BQ, int BK, bool FULL, bool TRACK>
__global__ void __launch_bounds__(256) fwd_bf16_kernel(cowa_params p, SchedView sv, int hpw,
                                                       const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                                                       const __bf16* __restrict__ v, __bf16* __restrict__ o,
                                                       float* __restrict__ lse) {
  using C = FwdCfg<D, BQ, BK>;
  using T = typename C::T;
  constexpr int NQT = C::NQT, KS = C::KS, MD = C::MD, NCH = C::NCH, NG = C::NG;
  extern __shared__ __align__(1024) unsigned char smem[];

  const int nw = blockDim.x >> 6;
  const int G = p.h_q / p.h_k;
  // rows of 16 QO blocks x the head groups of one KV head share an XCD's L2;
  // latest (longest) QO blocks first
  const WorkItem wi = cluster_item(blockIdx.x, sv.n_qt, G / hpw, grid_units(p, sv),
                                   cluster_rows(sv.n_qt, grid_units(p, sv), 16), true);
  int hk;
  const SeqCtx sc = seq_ctx(p, sv, wi.row, wi.unit, true, hk);
  const int i = sc.tile;
  const int hgi = hk * (G / hpw) + wi.group;
  const int h0 = hgi * hpw;  // first QO head of this workgroup (all in KV group hk)

  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int l32 = lane & 31, hh = lane >> 5;  // MFMA column and half
  const int hq = h0 + wave / C::WPH;
  const int q_first = i * BQ + (wave % C::WPH) * C::NQW;
  const Geo32 g = sc.g;
  const int n_q = sc.n_q, n_k = sc.n_k;
  const __bf16* kbase = k + (sc.k0 + (int64_t)hk * sc.kh) * D;
  const __bf16* vbase = v + (sc.k0 + (int64_t)hk * sc.kh) * D;
  const uint32_t smem_base = lds_addr(smem);

  // Q^T fragments (B operands): query column 32 nq + l32, d = 16 ks + 8 hh + 0..7;
  // loaded first, so that their latency overlaps that of the entry lists
  const int64_t row_base = sc.q0 + (int64_t)hq * sc.qh;
  if constexpr (TRACK) {
    // only the workgroups with a row that the untracked launch left to this
    // one (LSE = NaN) run; the rest end here, uniformly
    int* flag = reinterpret_cast<int*>(smem + C::MAIN_BYTES + 4 * sv.max_kt);
    if (tid == 0) *flag = 0;
    __syncthreads();
    const int qr = q_first + lane;
    if (__ballot(qr < n_q && __builtin_isnan(lse[row_base + qr])) != 0 && lane == 0) *flag = 1;
    __syncthreads();
    const bool mine = *flag != 0;
    __syncthreads();
    if (!mine) return;
  }
  bf16x8 qf[NQT][KS];
#pragma unroll
  for (int nq = 0; nq < NQT; ++nq) {
    const int qp = q_first + nq * 32 + l32;
    const bool ok = qp < n_q;
    const __bf16* qrow = q + (row_base + (ok ? qp : 0)) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 val = *reinterpret_cast<const bf16x8*>(qrow + ks * 16 + 8 * hh);
      qf[nq][ks] = ok ? val : bf16x8{};
    }
  }
  // Move the Q^T fragments into AGPRs here, long before the first product: the
  // assembly products read them from AGPRs, and the compiler could otherwise
  // copy them there just before that read, without the wait states a product
  // needs after a vector write of its operands.  (These statements emit
  // nothing themselves.)
#pragma unroll
  for (int nq = 0; nq < NQT; ++nq)
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+a"(qf[nq][ks]));
  // zero the K/V buffers once when the last KV block is partial: key rows past
  // the end of the sequence are not copied and must hold finite values
  if (n_k % BK != 0)
    for (int x = tid; x < C::MAIN_BYTES / 16; x += blockDim.x) reinterpret_cast<u32x4*>(smem)[x] = u32x4{0u, 0u, 0u, 0u};

  // the row's entries, split into full (from the front) and partial (from the back) lists
  const int r = sc.sched;
  const int e0 = sv.fwd_row_ptr[r], e1 = sv.fwd_row_ptr[r + 1];
  const int n_ent = e1 - e0;
  const int cap = sv.max_kt;
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

  // Global -> LDS copies of K and V blocks.  With four waves each lane copies
  // the same 16-byte column of its row in every 1 KB piece it takes: its byte
  // offsets within a block are fixed, and the block position goes into the
  // (scalar) buffer resource, whose size bounds the reads to the sequence.
  constexpr int RPL = 1024 / (D * 2);  // rows per 1 KB piece
  constexpr int NWF = C::NWF;
  constexpr int PPW = T::LOADS / NWF;  // pieces per wave
  uint32_t dma_off[PPW];
  {
    const int row0 = wave * RPL + lane / T::CH;
    const int col = (lane % T::CH) ^ swz<T::CH>(row0);
#pragma unroll
    for (int n = 0; n < PPW; ++n) dma_off[n] = (uint32_t)(((n * NWF * RPL + row0) * D + col * 8) * 2);
  }
  auto kbuf_off = [](int t) { return (t & 1) * 2 * T::BYTES; };
  auto vbuf_off = [](int t) { return (t & 1) * 2 * T::BYTES + T::BYTES; };
  auto stage = [&](const __bf16* base, int t, int buf_off) {
    const int kf = (int)(entry_at(t) >> 1) * BK;
    if constexpr (FULL) {
      const i32x4 rs = buffer_rsrc(base + (int64_t)kf * D, (uint32_t)(n_k - kf) * D * 2);
      const uint32_t lds0 = smem_base + buf_off + wave * 1024;
#pragma unroll
      for (int n = 0; n < PPW; ++n) dma16_buf(dma_off[n], rs, lds0 + n * NWF * 1024);
    } else {
      load_tile_asm_nw<D, BK>(base, kf, n_k, smem_base + buf_off, wave, nw, lane);
    }
  };
  // piece n of a block copy (full waves only), issued on its own
  auto stage_piece = [&](const __bf16* base, int kf, int buf_off, int n) {
    const i32x4 rs = buffer_rsrc(base + (int64_t)kf * D, (uint32_t)(n_k - kf) * D * 2);
    dma16_buf(dma_off[n], rs, smem_base + buf_off + wave * 1024 + n * NWF * 1024);
  };
  __syncthreads();  // the lists and the zeroed buffers are in LDS

  // LDS fragment offsets for chunk 0 of a tile (the swizzle depends on row % 16,
  // so chunks 32 rows further and k-steps 16 rows further add plain row bytes)
  //  K (A operand of S^T): row l32, columns 16 ks + 8 hh + 0..7;
  //  V^T (A operand of O^T): transposing reads of rows 4 hh + (lane % 16) / 4
  //  (+ 8 for slots 4..7), columns 32 md + 16 ((lane / 16) % 2) + 4 (lane % 4).
  int offk[KS], offv[MD][2];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) offk[ks] = T::off(l32, 2 * ks + hh);
#pragma unroll
  for (int md = 0; md < MD; ++md)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
      offv[md][hf] = T::off_col(4 * hh + ((lane & 15) >> 2) + 8 * hf, 32 * md + 16 * ((lane >> 4) & 1) + 4 * (lane & 3));
  auto ld_v = [&](const unsigned char* tile, int md, int row_bytes) -> bf16x8 {
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + offv[md][0] + row_bytes));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + offv[md][1] + row_bytes));
    const bf16x4 a = __builtin_bit_cast(bf16x4, lo), c2 = __builtin_bit_cast(bf16x4, hi);
    return bf16x8{a[0], a[1], a[2], a[3], c2[0], c2[1], c2[2], c2[3]};
  };

  // O^T accumulators: element (lane, e) is d = 32 md + 8 (e / 4) + 4 hh + e % 4, query 32 nq + l32
  f32x16 oacc[MD][NQT];
  // S^T of two chunks: element (lane, e) is key 8 (e / 4) + 4 hh + e % 4 of the
  // chunk, query 32 nq + l32.  Slots e = 8 kk .. 8 kk + 7 are exactly the keys
  // that lane holds in k-step kk of O^T += V^T P^T (16 keys each), so P^T needs
  // no data movement.
  f32x16 sacc[2][NQT];
  u32x4 pbw[2][2][NQT];  // P^T of two chunks: bf16 pairs, [chunk % 2][k-step][query tile]

  // The exponent offset m (base 2, per query column) starts kHead above the
  // maximum over the first 32 keys of the row's first block, so P = exp2(s c - m)
  // is at most 2^-kHead there and a later score may pass that maximum by
  // kHead + ~110 before P, l or O could overflow (keys more than ~60 below the
  // maximum underflow, 2^-60 of the largest term).  O and l share the offset,
  // so O / l and LSE = (m + log2 l) ln 2 are unaffected, and O is rescaled
  // only when, at the end of a block, a column's maximum has passed the one
  // that m was set from by more than kLimit: then m moves to kHead above it
  // and O, l and the P^T not yet in O are multiplied by 2^(m_old - m) once
  // (rare after the first blocks of a row, never for scores within kLimit).
  // If P, l or O overflowed anyway, the workgroup runs the row again with m
  // set from the row maximum found by the first pass, as it does when m was
  // unset (no legal key among the first 32) but the row has legal keys.
  constexpr float kHead = 64.f, kLimit = 32.f;
  float m_fix[NQT], m_hi[NQT], mu[NQT];  // m_hi: this lane's maximum raw score per column
#pragma unroll
  for (int nq = 0; nq < NQT; ++nq) m_fix[nq] = -INFINITY;
  const float c = p.softmax_scale * kLog2e;
  // Row sums l = sum of the rounded P^T over the keys, per query column, on the
  // matrix cores: the P^T fragment of a 16-key k-step, read as the B operand of
  // a 16x16x32 product, holds in lane L column L % 16 of k-group L / 16, which
  // is query 32 nq + (L % 32) with the keys of half L / 32 (k-groups 0 and 2:
  // queries 0-15, 1 and 3: queries 16-31).  The selector A has ones where
  // (row & 4) == 0 equals (k-group even), so rows 0-3 and 8-11 sum queries 0-15
  // and rows 4-7 and 12-15 queries 16-31; the result rows 4 (L / 16) .. + 3 of
  // lane L then all hold the sum of lane L's own query column L % 32.
  f32x4 lacc[NQT];
  const bf16x8 lsel = ((lane & 4) == 0) == (((lane >> 4) & 1) == 0)
                          ? bf16x8{(__bf16)1.f, (__bf16)1.f, (__bf16)1.f, (__bf16)1.f,
                                   (__bf16)1.f, (__bf16)1.f, (__bf16)1.f, (__bf16)1.f}
                          : bf16x8{};

  float pv[32];  // exponentials in flight between the two halves of an element step
  uint32_t lmask[NQT];  // legal keys of the chunk being masked, per query tile
  // element step e of a chunk's softmax (query tile e / 16, slot e % 16), first half
  auto soft_a = [&](auto ec, auto rpc, bool masked, int key0) __attribute__((always_inline)) {
    constexpr int e = decltype(ec)::value, rp = decltype(rpc)::value;
    constexpr int nq = e / 16, s = e % 16;
    if (masked) {  // key0: this lane's first key of the chunk
      // the window rule as a bit mask over the lane's keys key0 .. key0 + 31,
      // once per chunk and query tile; slot s holds key key0 + cs, which an
      // illegal pair turns into -inf (bit select, no compare)
      constexpr int cs = 8 * (s >> 2) + (s & 3);
      if constexpr (s == 0) lmask[nq] = legal_keys32(g, q_first + nq * 32 + l32, key0);
      const uint32_t m = (uint32_t)((int32_t)(lmask[nq] << (31 - cs)) >> 31);
      sacc[rp][nq][s] = __uint_as_float((__float_as_uint(sacc[rp][nq][s]) & m) | (0xff800000u & ~m));
    }
    pv[e] = __builtin_amdgcn_exp2f(fmaf(sacc[rp][nq][s], c, -mu[nq]));
  };
  // second half (odd e): running maximum (TRACK only), bf16 pair
  auto soft_b = [&](auto ec, auto rpc, auto psc) __attribute__((always_inline)) {
    constexpr int e = decltype(ec)::value, rp = decltype(rpc)::value, ps = decltype(psc)::value;
    constexpr int nq = e / 16, s = e % 16;
    if constexpr (s & 1) {
      if constexpr (TRACK) m_hi[nq] = max3(m_hi[nq], sacc[rp][nq][s - 1], sacc[rp][nq][s]);
      const bf16x2 pk = {(__bf16)pv[e - 1], (__bf16)pv[e]};
      pbw[ps][s / 8][nq][(s & 7) >> 1] = __builtin_bit_cast(uint32_t, pk);
    }
  };
  // the element steps that belong to slot `slot` of NS
  auto soft_slot = [&](auto slotc, auto nsc, auto rpc, auto psc, bool masked, int key0) __attribute__((always_inline)) {
    constexpr int slot = decltype(slotc)::value, NS = decltype(nsc)::value;
    static_for<16 * NQT>([&](auto ec) {
      constexpr int e = decltype(ec)::value;
      constexpr int sa = e * NS / (16 * NQT);
      constexpr int sb = sa + 1 < NS ? sa + 1 : sa;
      if constexpr (sa == slot) soft_a(ec, rpc, masked, key0);
      if constexpr (sb == slot) soft_b(ec, rpc, psc);
    });
  };

  // End of a block: move the offset of columns whose maximum has passed it by
  // more than kLimit.  P^T of the block's second-to-last chunk is computed but
  // not yet in O (it enters in the next block's first chunk step), so it is
  // rescaled with O and l; the last chunk is exponentiated after this point.
  // The test is per lane (a column's two lanes hold disjoint keys, and the one
  // holding the maximum sees it); the new offset is kHead above the column
  // maximum.  `hot` records a P above 2^kHot, the only way P, l or O can
  // approach the float range, so the overflow check at the end of a pass runs
  // only then.
  constexpr float kHot = 64.f;
  bool hot = false;
  auto rebase = [&]() __attribute__((always_inline)) {
    bool need = false;
#pragma unroll
    for (int nq = 0; nq < NQT; ++nq) {
      const float e = m_hi[nq] * c - mu[nq];
      need |= e > kLimit - kHead;
      hot |= e > kHot;
    }
    if (__builtin_expect(__ballot(need) == 0, 1)) return;  // (rare: keep it a branch)
    constexpr int PS = (NCH - 2) & 1;  // pair buffer of the pending chunk
#pragma unroll
    for (int nq = 0; nq < NQT; ++nq) {
      const float mh = fmaxf(m_hi[nq], __shfl_xor(m_hi[nq], 32)) * c + kHead;
      const bool mv = mh > mu[nq] + kLimit;
      // the factor 2^(m_old - m) is applied as its square root twice: a jump of
      // the maximum by more than 126 within one block would make it underflow,
      // although the products (the new maximum's own terms among them) are
      // ordinary numbers; the square root stays normal up to a jump of 252,
      // beyond which P has overflowed and the row runs again anyway
      const float f = mv ? __builtin_amdgcn_exp2f(0.5f * (mu[nq] - mh)) : 1.f;
      mu[nq] = mv ? mh : mu[nq];
      lacc[nq] = lacc[nq] * f * f;
#pragma unroll
      for (int md = 0; md < MD; ++md) {  // one tile at a time, back into its AGPRs
#pragma unroll
        for (int x = 0; x < 16; ++x) oacc[md][nq][x] = oacc[md][nq][x] * f * f;
        asm volatile("" : "+a"(oacc[md][nq]));
      }
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          // (a vector element is copied out first: bit-casting the element
          // expression itself reads element 0)
          const uint32_t u = pbw[PS][kk][nq][w];
          const bf16x2 pk = __builtin_bit_cast(bf16x2, u);
          const bf16x2 sc2 = {(__bf16)((float)pk[0] * f * f), (__bf16)((float)pk[1] * f * f)};
          pbw[PS][kk][nq][w] = __builtin_bit_cast(uint32_t, sc2);
        }
    }
  };

  // The same move without a tracked maximum (TRACK false): the row sum l of a
  // column bounds each of its P from above, so when it passes 2^(kLimit -
  // kHead) at a block end (never before some score has passed the first keys'
  // maximum by 15 or more: at most 2^31 keys of at most 2^-kHead each) the
  // offset moves by log2 l + kHead, which leaves every P so far at most
  // 2^-kHead (l itself becomes 2^-kHead) and overshoots the move the maximum
  // would give by at most log2 of the row length.  Both lanes of a column hold
  // the same sum, so they move alike.  The sum lags by the chunks not yet in
  // it (the pending P^T and the last chunk); a P that overflows in the
  // meantime makes l infinite, and the row is left to the tracked launch.
  auto rebase_sum = [&]() __attribute__((always_inline)) {
    bool need = false;
#pragma unroll
    for (int nq = 0; nq < NQT; ++nq) {
      const float l = lacc[nq][0];
      need |= l > 0x1p-32f;
      hot |= !(l <= 0x1p64f);
    }
    if (__builtin_expect(__ballot(need) == 0, 1)) return;  // (rare: keep it a branch)
    constexpr int PS = (NCH - 2) & 1;  // pair buffer of the pending chunk
#pragma unroll
    for (int nq = 0; nq < NQT; ++nq) {
      const float l = lacc[nq][0];
      const bool mv = l > 0x1p-32f && l < INFINITY;  // (an overflowed sum: the row goes to the tracked launch)
      const float dm = mv ? __log2f(l) + kHead : 0.f;
      const float f = mv ? __builtin_amdgcn_exp2f(-0.5f * dm) : 1.f;  // applied twice, as above
      mu[nq] += dm;
      lacc[nq] = lacc[nq] * f * f;
#pragma unroll
      for (int md = 0; md < MD; ++md) {
#pragma unroll
        for (int x = 0; x < 16; ++x) oacc[md][nq][x] = oacc[md][nq][x] * f * f;
        asm volatile("" : "+a"(oacc[md][nq]));
      }
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t u = pbw[PS][kk][nq][w];
          const bf16x2 pk = __builtin_bit_cast(bf16x2, u);
          const bf16x2 sc2 = {(__bf16)((float)pk[0] * f * f), (__bf16)((float)pk[1] * f * f)};
          pbw[PS][kk][nq][w] = __builtin_bit_cast(uint32_t, sc2);
        }
    }
  };

  // Software pipeline over the row's 32-key chunks: chunk n has its S^T
  // computed in chunk step n, is exponentiated in step n + 1 and enters
  // O^T += V^T P^T in step n + 2.  Within a chunk step the matrix cores work on
  // S^T (chunk n) and O^T (chunk n - 2) while the vector ALUs turn S^T of chunk
  // n - 1 into P^T: the streams are independent, so the exponentials hide under
  // the products.  Fragments are read PF groups ahead.
  //
  // LDS: K of block t in K buffer t % 2, V of block t in V buffer t % 2.  The
  // O^T products of block t's steps read V of block t - 1 for the chunks two
  // back; with 128-key blocks, V of block t is needed from its third step on,
  // so it is copied in the middle of block t - 1, once V of block t - 2 is no
  // longer read.
  constexpr int PF = 2, RING = PF + 2;
  int k_prev = 0;  // first key of the previous block
  // One block.  FIRST: the row's first block (nothing before its first chunk).
  // MPREV / MCUR: the chunks exponentiated here from the previous / this block
  // need the element mask.
  auto step = [&](int t, auto firstc, auto mprevc, auto mcurc) __attribute__((always_inline)) {
    constexpr bool FIRST = decltype(firstc)::value, MPREV = decltype(mprevc)::value;
    constexpr bool MCUR = decltype(mcurc)::value;
    const int k_first = (int)(entry_at(t) >> 1) * BK;
    // K of block t + 1 goes into the K buffer of block t - 1, which is free
    // (the last block repeats itself).  With 128-key blocks and full waves the
    // copies of K (from the block start) and of V (from the mid-block barrier)
    // go out one 1 KB piece per product group: a burst of them would hold the
    // wave at the vector memory queue.
    constexpr bool SPREAD = FULL && NCH == 4;
    [[maybe_unused]] const int kf_next = (int)(entry_at(t + 1) >> 1) * BK;
    if constexpr (!SPREAD) stage(kbase, t + 1, kbuf_off(t + 1));
    if constexpr (NCH == 2) stage(vbase, t, vbuf_off(t));  // V buffer of block t - 2: free
    const unsigned char* Kt = smem + kbuf_off(t);
    const unsigned char* Vt = smem + vbuf_off(t);
    const unsigned char* Vp = smem + vbuf_off(t + 1);  // V of block t - 1
    constexpr int NGS = NCH * NG;
    bf16x8 fa[RING];
    // group GG of the block: chunk step j, S^T k-step or O^T (k-step kk, d tile md)
    auto load = [&](auto gc, bf16x8& dst) __attribute__((always_inline)) {
      constexpr int GG = decltype(gc)::value, j = GG / NG, gi = GG % NG;
      constexpr bool S = gi % 2 == 0;
      constexpr int x = gi / 2;
      constexpr int jo = (j + NCH - 2) % NCH;  // chunk of the O^T products within its block
      constexpr bool OLD = j < 2;              // ... of the previous block
      if constexpr (S) {
        dst = ld_row8(Kt + offk[x] + j * 32 * D * 2);
      } else if constexpr (!(FIRST && OLD)) {
        constexpr int kk = x / MD, md = x % MD;
        dst = ld_v(OLD ? Vp : Vt, md, (jo * 32 + kk * 16) * D * 2);
      }
    };
    static_for<PF>([&](auto ic) { load(ic, fa[decltype(ic)::value]); });
    __builtin_amdgcn_sched_barrier(0);
    static_for<NGS>([&](auto gc) {
      constexpr int GG = decltype(gc)::value, j = GG / NG, gi = GG % NG;
      constexpr bool S = gi % 2 == 0;
      constexpr int x = gi / 2;
      constexpr bool OLD = j < 2;
      if constexpr (NCH == 4 && GG == 2 * NG - PF) {
        // middle of a 128-key block, before the first read of V of block t
        // (fragments run PF groups ahead) and after the last read of V of
        // block t - 1 was issued: V of block t is in (its copies were issued
        // before this block's K copies), and once every wave's reads of V of
        // block t - 1 are done, the copy of block t + 1 may overwrite it
        if constexpr (FULL)
          __builtin_amdgcn_s_waitcnt(vmcnt_only(PPW));
        else
          __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if constexpr (!SPREAD) stage(vbase, t + 1, vbuf_off(t + 1));
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (SPREAD && GG < PPW) stage_piece(kbase, kf_next, kbuf_off(t + 1), GG);
      if constexpr (SPREAD && GG >= 2 * NG - PF && GG < 2 * NG - PF + PPW)
        stage_piece(vbase, kf_next, vbuf_off(t + 1), GG - (2 * NG - PF));
      if constexpr (GG + PF < NGS) load(std::integral_constant<int, GG + PF>{}, fa[(GG + PF) % RING]);
      const bf16x8& a = fa[GG % RING];
      static_for<NQT>([&](auto mc) {
        constexpr int m = decltype(mc)::value;
        if constexpr (S) {
          if constexpr (x == 0)
            sacc[j & 1][m] = mfma32_v0(a, qf[m][0]);
          else
            sacc[j & 1][m] = mfma32_v(a, qf[m][x], sacc[j & 1][m]);
        } else if constexpr (!(FIRST && OLD)) {
          constexpr int kk = x / MD, md = x % MD;
          oacc[md][m] = mfma32(a, __builtin_bit_cast(bf16x8, pbw[j & 1][kk][m]), oacc[md][m]);
          if constexpr (md == 0) lacc[m] = mfma16(lsel, __builtin_bit_cast(bf16x8, pbw[j & 1][kk][m]), lacc[m]);
        }
        // the softmax of the chunk before chunk j (chunk j - 1 of this block,
        // or the last chunk of the previous block), spread over the products
        constexpr int slot = gi * NQT + m;
        if constexpr (!(FIRST && j == 0)) {
          using SL = std::integral_constant<int, slot>;
          using NSC = std::integral_constant<int, NQT * NG>;
          using RP = std::integral_constant<int, (j + 1) & 1>;
          if constexpr (j == 0)
            soft_slot(SL{}, NSC{}, RP{}, RP{}, MPREV, k_prev + (NCH - 1) * 32 + 4 * hh);
          else
            soft_slot(SL{}, NSC{}, RP{}, RP{}, MCUR, k_first + (j - 1) * 32 + 4 * hh);
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      // a chunk step without O^T products (start of the row): its S^T results
      // are read early in the next step, so settle them here
      if constexpr (FIRST && OLD && gi == NG - 1) {
        mfma_settle(sacc[j & 1]);
        __builtin_amdgcn_sched_barrier(0);
      }
    });
    // the last S^T products may still be in flight: wait states before
    // anything reads them
    mfma_settle(sacc[1]);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (TRACK)
      rebase();
    else
      rebase_sum();
    // register placement: O^T accumulators and Q^T fragments in AGPRs (read
    // directly by the matrix cores), S^T and P^T in VGPRs; these emit nothing
#pragma unroll
    for (int md = 0; md < MD; ++md)
#pragma unroll
      for (int nq = 0; nq < NQT; ++nq) asm volatile("" : "+a"(oacc[md][nq]));
#pragma unroll
    for (int nq = 0; nq < NQT; ++nq)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+a"(qf[nq][ks]));
    k_prev = k_first;
    // the next block's K has landed (with 128-key blocks the next V may still
    // be in flight)
    if constexpr (NCH == 4 && FULL)
      __builtin_amdgcn_s_waitcnt(vmcnt_only(PPW));
    else
      __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();  // ... for every wave, and the freed buffers are no longer read
  };
  // after the last block: the softmax of its last chunk, then the O^T products
  // of its last two chunks
  auto drain = [&](int t) __attribute__((always_inline)) {
    using R1 = std::integral_constant<int, 1>;
    static_for<16 * NQT>([&](auto ec) { soft_a(ec, R1{}, true, k_prev + (NCH - 1) * 32 + 4 * hh); });
    static_for<16 * NQT>([&](auto ec) { soft_b(ec, R1{}, R1{}); });
    if constexpr (NCH == 4 && FULL) __builtin_amdgcn_s_waitcnt(0);  // (the repeated V copy of the mid-block)
    const unsigned char* Vt = smem + vbuf_off(t);
    static_for<2 * 2 * MD>([&](auto gc) {
      constexpr int GG = decltype(gc)::value, jj = GG / (2 * MD), kk = (GG / MD) % 2, md = GG % MD;
      constexpr int jo = NCH - 2 + jj;  // chunk within the block
      const bf16x8 a = ld_v(Vt, md, (jo * 32 + kk * 16) * D * 2);
#pragma unroll
      for (int nq = 0; nq < NQT; ++nq)
        oacc[md][nq] = mfma32(a, __builtin_bit_cast(bf16x8, pbw[jo & 1][kk][nq]), oacc[md][nq]);
      if constexpr (md == 0)
#pragma unroll
        for (int nq = 0; nq < NQT; ++nq)
          lacc[nq] = mfma16(lsel, __builtin_bit_cast(bf16x8, pbw[jo & 1][kk][nq]), lacc[nq]);
    });
  };
  using TT = std::true_type;
  using FF = std::false_type;
  auto sweep = [&]() __attribute__((always_inline)) {
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
  };

  int* vote = reinterpret_cast<int*>(smem + C::MAIN_BYTES + 4 * cap);
  // TRACK false: one pass without a tracked maximum (its offset moves on the
  // row sums); rows it cannot finish get LSE = NaN and are run again by the
  // TRACK launch, with up to two passes as described above
  bool flagged = false;
  for (int pass = 0; pass < (TRACK ? 2 : 1); ++pass) {
#pragma unroll
    for (int nq = 0; nq < NQT; ++nq) {
      m_hi[nq] = -INFINITY;
      lacc[nq] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int md = 0; md < MD; ++md) oacc[md][nq] = f32x16{};
    }
    if (n_ent > 0) {
      stage(kbase, 0, kbuf_off(0));
      if (NCH == 4) stage(vbase, 0, vbuf_off(0));  // (needed from the block's third chunk)
    }
    // K of the first block has landed; with 128-key blocks and full waves its V
    // may still be in flight (the first block's mid-block wait covers it)
    if constexpr (NCH == 4 && FULL)
      __builtin_amdgcn_s_waitcnt(vmcnt_only(PPW));
    else
      __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (pass == 0 && n_ent > 0) {
      // offsets from the first 32 keys of the row's first block (in processing
      // order: a full block when the row has one)
      const int kb = (int)(entry_at(0) >> 1) * BK + 4 * hh;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 a = ld_row8(smem + offk[ks]);
#pragma unroll
        for (int nq = 0; nq < NQT; ++nq)
          sacc[0][nq] = ks == 0 ? mfma32_v0(a, qf[nq][0]) : mfma32_v(a, qf[nq][ks], sacc[0][nq]);
        mfma_settle(sacc[0]);  // the next k-step reads these accumulators
      }
#pragma unroll
      for (int nq = 0; nq < NQT; ++nq) {
        float cm = -INFINITY;
        const uint32_t lm = legal_keys32(g, q_first + nq * 32 + l32, kb);
#pragma unroll
        for (int x = 0; x < 16; ++x) {
          const bool ok = (lm >> (8 * (x >> 2) + (x & 3))) & 1u;
          cm = fmaxf(cm, ok ? sacc[0][nq][x] : -INFINITY);
        }
        cm = fmaxf(cm, __shfl_xor(cm, 32));
        m_fix[nq] = cm * c;  // -inf for a column without a legal key there
      }
    }
#pragma unroll
    for (int nq = 0; nq < NQT; ++nq) mu[nq] = m_fix[nq] == -INFINITY ? 0.f : m_fix[nq] + kHead;
    sweep();
    bool far = false;
    if constexpr (TRACK) {
      // was a column's offset unset although it met legal keys later, or did
      // P, l or O overflow (possible only after a P above 2^kHot)?
#pragma unroll
      for (int nq = 0; nq < NQT; ++nq) {
        hot |= m_hi[nq] * c - mu[nq] > kHot;  // (the last chunk came after the last block end)
        const float mh = fmaxf(m_hi[nq], __shfl_xor(m_hi[nq], 32)) * c;  // the column maximum, exponent units
        far |= mh != -INFINITY && m_fix[nq] == -INFINITY;
        m_fix[nq] = mh;  // the offset of a second pass: then P <= 2^-kHead everywhere
      }
    } else {
      // a column without an offset at the start (m = 0) keeps its sum only if
      // that sum is comfortably normal (otherwise it met no legal key, or its
      // P underflowed); an overflow shows in the sum
#pragma unroll
      for (int nq = 0; nq < NQT; ++nq) {
        const float l = lacc[nq][0];
        hot |= !(l <= 0x1p64f);
        far |= m_fix[nq] == -INFINITY && q_first + nq * 32 + l32 < n_q && !(l >= 0x1p-60f);
      }
    }
    if (__ballot(hot) != 0) {
#pragma unroll
      for (int nq = 0; nq < NQT; ++nq) {
        far |= !__builtin_isfinite(lacc[nq][0]);
#pragma unroll
        for (int md = 0; md < MD; ++md) {
#pragma unroll
          for (int x = 0; x < 16; ++x) far |= !__builtin_isfinite(oacc[md][nq][x]);
          asm volatile("" : "+a"(oacc[md][nq]));
        }
      }
    }
    hot = false;
    // workgroup vote through a word past the block lists
    if (tid == 0) *vote = 0;
    __syncthreads();
    if (far) *vote = 1;
    __syncthreads();
    const bool again = *vote != 0;
    __syncthreads();
    if (!TRACK) flagged = again;
    if (!again) break;
  }

  // O = O / l; LSE = (m + log2 l) ln 2 with the offset m of the last pass (base 2).
  // O goes out through LDS (free here: every wave is past the vote's barriers,
  // its reads are done and its copies have landed): each wave stages its 64
  // rows and stores whole rows, 16 bytes per lane, instead of 16-byte pieces of
  // 32 rows per store in the accumulator layout.
  constexpr int OP = C::OUT_PITCH;
  unsigned char* ot = smem + wave * C::NQW * OP;
#pragma unroll
  for (int nq = 0; nq < NQT; ++nq) {
    const float lt = lacc[nq][0];
    const int qp = q_first + nq * 32 + l32;
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
#pragma unroll
    for (int md = 0; md < MD; ++md)
#pragma unroll
      for (int j4 = 0; j4 < 4; ++j4) {
        bf16x4 ov;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) ov[rr] = (__bf16)(oacc[md][nq][4 * j4 + rr] * inv);
        *reinterpret_cast<bf16x4*>(ot + (nq * 32 + l32) * OP + (md * 32 + 8 * j4 + 4 * hh) * 2) = ov;
      }
    if (hh == 0 && qp < n_q) lse[row_base + qp] = flagged ? __builtin_nanf("") : lt > 0.f ? (mu[nq] + __log2f(lt)) * kLn2 : -INFINITY;
  }
  constexpr int CPR = D / 8;  // 16-byte chunks per row
#pragma unroll
  for (int x = 0; x < C::NQW * CPR / 64; ++x) {
    const int idx = x * 64 + lane, row = idx / CPR, ch = idx % CPR;
    if (q_first + row < n_q)
      *reinterpret_cast<u32x4*>(o + (row_base + q_first + row) * D + ch * 8) =
          *reinterpret_cast<const u32x4*>(ot + row * OP + ch * 16);
  }
}

template <int D, int BQ, int BK, bool FULL>
hipError_t launch_waves(const cowa_params& p, const SchedView& sv, int hpw, int n_hgroups, int waves, const void* q,
                        const void* k, const void* v, void* o, float* lse, hipStream_t stream) {
  using C = FwdCfg<D, BQ, BK>;
  // the untracked launch, then the tracked one for the rows it flagged
  auto kern0 = fwd_bf16_kernel<D, BQ, BK, FULL, false>;
  auto kern1 = fwd_bf16_kernel<D, BQ, BK, FULL, true>;
  for (const void* kp : {reinterpret_cast<const void*>(kern0), reinterpret_cast<const void*>(kern1)}) {
    const hipError_t err = allow_lds(kp, C::LDS_MAX);
    if (err != hipSuccess) return err;
  }
  const unsigned blocks = (unsigned)sv.n_qt * n_hgroups * (sv.ragged ? 1 : p.batch);
  hipLaunchKernelGGL(kern0, dim3(blocks), dim3(64 * waves), C::lds_bytes(sv.max_kt), stream, p, sv, hpw,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), static_cast<const __bf16*>(v),
                     static_cast<__bf16*>(o), lse);
  hipLaunchKernelGGL(kern1, dim3(blocks), dim3(64 * waves), C::lds_bytes(sv.max_kt), stream, p, sv, hpw,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), static_cast<const __bf16*>(v),
                     static_cast<__bf16*>(o), lse);
  return hipGetLastError();
}

template <int D, int BQ, int BK>
hipError_t launch_cfg(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                      void* o, float* lse, hipStream_t stream) {
  using C = FwdCfg<D, BQ, BK>;
  if (sv.max_kt > C::max_kblocks()) return hipErrorInvalidValue;
  const int G = p.h_q / p.h_k;
  int hpw = 256 / BQ;  // QO heads per workgroup: up to 256 query rows
  while (hpw > 1 && G % hpw != 0) hpw >>= 1;
  const int n_hgroups = p.h_q / hpw;
  const int waves = hpw * C::WPH;
  if (waves == C::NWF) return launch_waves<D, BQ, BK, true>(p, sv, hpw, n_hgroups, waves, q, k, v, o, lse, stream);
  return launch_waves<D, BQ, BK, false>(p, sv, hpw, n_hgroups, waves, q, k, v, o, lse, stream);
}

}  // namespace

int fwd_bf16_max_kblocks(int d, int tk) {
  if (d == 128) return tk == 128 ? FwdCfg<128, 128, 128>::max_kblocks() : FwdCfg<128, 128, 64>::max_kblocks();
  return tk == 128 ? FwdCfg<64, 128, 128>::max_kblocks() : FwdCfg<64, 128, 64>::max_kblocks();
}

bool fwd_bf16_supported(int d, int tq, int tk) {
  return (d == 64 || d == 128) && (tq == 64 || tq == 128) && (tk == 64 || tk == 128);
}

hipError_t launch_fwd_bf16(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                           void* o, float* lse, hipStream_t stream) {
#define COWA_FWD_CASE(D_, BQ_, BK_) \
  if (p.head_dim == D_ && p.tile_q == BQ_ && p.tile_k == BK_) return launch_cfg<D_, BQ_, BK_>(p, sv, q, k, v, o, lse, stream);
  COWA_FWD_CASE(128, 128, 128)
  COWA_FWD_CASE(128, 128, 64)
  COWA_FWD_CASE(128, 64, 128)
  COWA_FWD_CASE(128, 64, 64)
  COWA_FWD_CASE(64, 128, 128)
  COWA_FWD_CASE(64, 128, 64)
  COWA_FWD_CASE(64, 64, 128)
  COWA_FWD_CASE(64, 64, 64)
#undef COWA_FWD_CASE
  return hipErrorInvalidValue;
}

}  // namespace cowa
