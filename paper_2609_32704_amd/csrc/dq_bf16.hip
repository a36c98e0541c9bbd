// CoWA backward, dQ pass, in bfloat16 on the CDNA4 matrix cores (Alg. 2, the
// dQ = scale dS K term), for 128-key blocks and four-wave workgroups.
//
// One workgroup per (QO block i, QO heads of one KV group, sequence b): four
// waves of 64 query rows (two heads of a 128-row block, or four of a 64-row
// block).  Every QO head of a group has the same block set J_{h_k}(i), so the
// heads share each K/V block staged in LDS.  Per KV block, full blocks first:
//   S^T = K Q^T and dP^T = V dO^T on v_mfma_f32_32x32x16_bf16, with Q^T and dO^T
//     in registers for the whole row;
//   P^T = exp2(S^T c - LSE log2 e) (LSE from the forward: P is exact, no
//     running maximum) and dS^T = P^T (dP^T - D) on the vector ALUs;
//   dQ^T += K^T dS^T, K^T from the transposing LDS read of the row-major K
//     block.  The S^T accumulator layout is the B-operand layout of dS^T, so dS
//     never leaves registers.
// The 32-key chunks of a row form a software pipeline: in chunk step n the
// matrix cores compute S^T and dP^T of chunk n and dQ^T of chunk n - 2 while
// the vector ALUs turn chunk n - 1 into dS^T.  Alg. 2 adds the dQ terms of
// different KV blocks with atomics; here each row's dQ is complete in
// registers and written once.  The pass recomputes S and dP (the dK/dV pass
// computed them too).
#include "internal.h"
#include "window_rule.h"
#include "mfma_tiles.h"
#include "work_item.h"

namespace cowa {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// S^T and dP^T products with the accumulator in VGPRs (read by the vector ALUs)
// while dQ^T accumulates in AGPRs through the builtin: written as assembly
// because the compiler gives all products of a kernel one accumulator register
// file.  The compiler inserts no wait states for these, so the schedule keeps
// every reader of a result at least three products behind it, and a block
// ends with explicit wait states (settle) before its last results are read.
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
__device__ inline void settle(f32x16 (&s)[2], f32x16 (&d)[2]) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" : "+v"(s[0]), "+v"(s[1]), "+v"(d[0]), "+v"(d[1]));
}

template <int D, int BQ>
struct Dq32Cfg {
  static constexpr int BK = 128;          // keys per block
  static constexpr int NQW = 64;          // query rows per wave
  static constexpr int NQT = NQW / 32;    // 32-query tiles per wave (columns of S^T)
  static constexpr int KS = D / 16;       // k-steps over d of S^T and dP^T
  static constexpr int MD = D / 32;       // 32-row d tiles of dQ^T
  static constexpr int NCH = BK / 32;     // 32-key chunks per block
  static constexpr int NG = 3 * KS;       // groups per chunk step: S^T, dP^T and dQ^T per slot x < KS
  static constexpr int WPH = BQ / NQW;    // waves per QO head
  static constexpr int HPW = 4 / WPH;     // QO heads per workgroup
  using T = SwzTile<D, BK>;
  static constexpr int MAIN_BYTES = 4 * T::BYTES;  // K and V of two blocks; then the row's entry lists
  static constexpr int LDS_MAX = 160 * 1024;
  static int lds_bytes(int n_kt) { return MAIN_BYTES + 4 * n_kt; }
  static constexpr int OUT_PITCH = 2 * D + 16;  // staged dQ rows (bytes), in the K/V buffers at the end
  static_assert(KS == 2 * MD, "one dQ^T product group per k-step slot");
  static_assert(4 * NQW * OUT_PITCH <= MAIN_BYTES, "staged rows fit the K/V buffers");
};

template <int D, int BQ>
__global__ void __launch_bounds__(256) bwd_dq32(cowa_params p, SchedView sv, const __bf16* __restrict__ q,
                                                const __bf16* __restrict__ k, const __bf16* __restrict__ v,
                                                const __bf16* __restrict__ d_o, const float* __restrict__ nl,
                                                const float* __restrict__ nd, __bf16* __restrict__ dq) {
  using C = Dq32Cfg<D, BQ>;
  using T = typename C::T;
  constexpr int NQT = C::NQT, KS = C::KS, MD = C::MD, NCH = C::NCH, NG = C::NG, BK = C::BK;
  extern __shared__ __align__(1024) unsigned char smem[];

  const int G = p.h_q / p.h_k;
  // rows of 16 QO blocks x the head groups of one KV head share an XCD's L2;
  // latest (longest) QO blocks first
  const WorkItem wi = cluster_item(blockIdx.x, sv.n_qt, G / C::HPW, grid_units(p, sv),
                                   cluster_rows(sv.n_qt, grid_units(p, sv), 16), true);
  int hk;
  const SeqCtx sc = seq_ctx(p, sv, wi.row, wi.unit, true, hk);
  const int i = sc.tile;
  const int h0 = (hk * (G / C::HPW) + wi.group) * C::HPW;  // first QO head (all in KV group hk)

  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int l32 = lane & 31, hh = lane >> 5;  // MFMA column and half
  const int hq = h0 + wave / C::WPH;
  const int q_first = i * BQ + (wave % C::WPH) * C::NQW;
  const Geo32 g = sc.g;
  const int n_q = sc.n_q, n_k = sc.n_k;
  const __bf16* kbase = k + (sc.k0 + (int64_t)hk * sc.kh) * D;
  const __bf16* vbase = v + (sc.k0 + (int64_t)hk * sc.kh) * D;
  const uint32_t smem_base = lds_addr(smem);

  // Q^T and dO^T fragments (B operands): query column 32 nq + l32, d = 16 ks + 8 hh + 0..7;
  // the row values of that query: the exponent offset -LSE log2 e (-inf for a
  // row past n_q or without keys, so P = 0 there) and -D.  Loaded first, so
  // that their latency overlaps that of the entry lists.
  const int64_t row_base = sc.q0 + (int64_t)hq * sc.qh;
  bf16x8 qf[NQT][KS], gf[NQT][KS];
  float mlse[NQT], dn[NQT];
#pragma unroll
  for (int nq = 0; nq < NQT; ++nq) {
    const int qp = q_first + nq * 32 + l32;
    const bool ok = qp < n_q;
    const int64_t row = row_base + (ok ? qp : 0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(q + row * D + ks * 16 + 8 * hh);
      const bf16x8 b = *reinterpret_cast<const bf16x8*>(d_o + row * D + ks * 16 + 8 * hh);
      qf[nq][ks] = ok ? a : bf16x8{};
      gf[nq][ks] = ok ? b : bf16x8{};
    }
    const float nlv = ok ? nl[row] : -INFINITY;
    mlse[nq] = nlv == INFINITY ? -INFINITY : nlv;
    dn[nq] = ok ? nd[row] : 0.f;
  }
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

  // Global -> LDS copies of K and V blocks: each lane copies the same 16-byte
  // column of its row in every 1 KB piece it takes (fixed byte offsets within a
  // block); the block position goes into the buffer resource, whose size
  // bounds the reads to the sequence.
  constexpr int RPL = 1024 / (D * 2);  // rows per 1 KB piece
  constexpr int PPW = T::LOADS / 4;    // pieces per wave
  static_assert(T::LOADS % 4 == 0 && (4 * RPL) % 16 == 0, "piece layout");
  uint32_t dma_off[PPW];
  {
    const int row0 = wave * RPL + lane / T::CH;
    const int col = (lane % T::CH) ^ swz<T::CH>(row0);
#pragma unroll
    for (int n = 0; n < PPW; ++n) dma_off[n] = (uint32_t)(((n * 4 * RPL + row0) * D + col * 8) * 2);
  }
  auto kbuf_off = [](int t) { return (t & 1) * 2 * T::BYTES; };
  auto vbuf_off = [](int t) { return (t & 1) * 2 * T::BYTES + T::BYTES; };
  auto stage_piece = [&](const __bf16* base, int kf, int buf_off, int n) {
    const i32x4 rs = buffer_rsrc(base + (int64_t)kf * D, (uint32_t)(n_k - kf) * D * 2);
    dma16_buf(dma_off[n], rs, smem_base + buf_off + wave * 1024 + n * 4 * 1024);
  };
  auto stage = [&](const __bf16* base, int t, int buf_off) {
    const int kf = (int)(entry_at(t) >> 1) * BK;
#pragma unroll
    for (int n = 0; n < PPW; ++n) stage_piece(base, kf, buf_off, n);
  };
  __syncthreads();  // the lists and the zeroed buffers are in LDS

  // dQ^T accumulators: element (lane, e) is d = 32 md + 8 (e / 4) + 4 hh + e % 4, query 32 nq + l32
  f32x16 qacc[MD][NQT];
#pragma unroll
  for (int md = 0; md < MD; ++md)
#pragma unroll
    for (int nq = 0; nq < NQT; ++nq) qacc[md][nq] = f32x16{};
  // Move the fragments and accumulators into AGPRs here, long before the first
  // product: the assembly products read Q^T / dO^T from AGPRs, and the compiler
  // would otherwise copy them there just before that read without the wait
  // states a product needs after a vector write of its operands.  These
  // statements emit nothing themselves.
#pragma unroll
  for (int nq = 0; nq < NQT; ++nq) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+a"(qf[nq][ks]), "+a"(gf[nq][ks]));
#pragma unroll
    for (int md = 0; md < MD; ++md) asm volatile("" : "+a"(qacc[md][nq]));
  }
  // LDS fragment offsets for chunk 0 of a block (the swizzle depends on row % 16,
  // so chunks 32 rows further and k-steps 16 rows further add plain row bytes)
  //  K and V rows (A operands of S^T, dP^T): row l32, columns 16 ks + 8 hh + 0..7;
  //  K^T (A operand of dQ^T): transposing reads of rows 4 hh + (lane % 16) / 4
  //  (+ 8 for slots 4..7), columns 32 md + 16 ((lane / 16) % 2) + 4 (lane % 4).
  int offk[KS], offt[MD][2];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) offk[ks] = T::off(l32, 2 * ks + hh);
#pragma unroll
  for (int md = 0; md < MD; ++md)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
      offt[md][hf] = T::off_col(4 * hh + ((lane & 15) >> 2) + 8 * hf, 32 * md + 16 * ((lane >> 4) & 1) + 4 * (lane & 3));
  auto ld_kt = [&](const unsigned char* tile, int md, int row_bytes) -> bf16x8 {
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + offt[md][0] + row_bytes));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + offt[md][1] + row_bytes));
    const bf16x4 a = __builtin_bit_cast(bf16x4, lo), c2 = __builtin_bit_cast(bf16x4, hi);
    return bf16x8{a[0], a[1], a[2], a[3], c2[0], c2[1], c2[2], c2[3]};
  };

  // S^T and dP^T of two chunks: element (lane, e) is key 8 (e / 4) + 4 hh + e % 4 of
  // the chunk, query 32 nq + l32.  Slots e = 8 kk .. 8 kk + 7 are exactly the keys
  // that lane holds in k-step kk of dQ^T += K^T dS^T (16 keys each).
  f32x16 sacc[2][NQT], pacc[2][NQT];
  u32x4 dsw[2][2][NQT];  // dS^T of two chunks: bf16 pairs, [chunk % 2][k-step][query tile]
  const float c = p.softmax_scale * kLog2e;

  float pv[16 * NQT];  // exponentials in flight between the two halves of an element step
  uint32_t lmask[NQT];  // legal keys of the chunk being masked, per query tile
  // element step e of a chunk (query tile e / 16, slot e % 16), first half: P
  auto soft_a = [&](auto ec, auto rpc, bool masked, int key0) __attribute__((always_inline)) {
    constexpr int e = decltype(ec)::value, rp = decltype(rpc)::value;
    constexpr int nq = e / 16, s = e % 16;
    if (masked) {  // key0: this lane's first key of the chunk
      // the window rule as a bit mask over the lane's keys key0 .. key0 + 31,
      // once per chunk and query tile (slot s holds key key0 + cs)
      constexpr int cs = 8 * (s >> 2) + (s & 3);
      if constexpr (s == 0) lmask[nq] = legal_keys32(g, q_first + nq * 32 + l32, key0);
      const uint32_t m = (uint32_t)((int32_t)(lmask[nq] << (31 - cs)) >> 31);
      sacc[rp][nq][s] = __uint_as_float((__float_as_uint(sacc[rp][nq][s]) & m) | (0xff800000u & ~m));
    }
    pv[e] = __builtin_amdgcn_exp2f(fmaf(sacc[rp][nq][s], c, mlse[nq]));
  };
  // second half (odd e): dS = P (dP - D) of the pair, rounded to bf16
  auto soft_b = [&](auto ec, auto rpc, auto psc) __attribute__((always_inline)) {
    constexpr int e = decltype(ec)::value, rp = decltype(rpc)::value, ps = decltype(psc)::value;
    constexpr int nq = e / 16, s = e % 16;
    if constexpr (s & 1) {
      const float d0 = pv[e - 1] * (pacc[rp][nq][s - 1] + dn[nq]);
      const float d1 = pv[e] * (pacc[rp][nq][s] + dn[nq]);
      const bf16x2 pk = {(__bf16)d0, (__bf16)d1};
      dsw[ps][s / 8][nq][(s & 7) >> 1] = __builtin_bit_cast(uint32_t, pk);
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

  // LDS: K of block t in K buffer t % 2, V of block t in V buffer t % 2.  The
  // dQ^T products of block t's first two chunk steps read K of block t - 1
  // (chunks two back), so K of block t + 1 is copied from the middle of block
  // t, once every wave has read K of block t - 1 for the last time; V of block
  // t + 1 is copied from the start of block t.  Both copies go out one 1 KB
  // piece per product group (a burst would hold the wave at the vector memory
  // queue) and land by the end of block t.
  constexpr int PF = 2, RING = PF + 2;
  int k_prev = 0;  // first key of the previous block
  // One block.  FIRST: the row's first block (nothing before its first chunk).
  // MPREV / MCUR: the chunks turned into dS here from the previous / this block
  // need the element mask.
  auto step = [&](int t, auto firstc, auto mprevc, auto mcurc) __attribute__((always_inline)) {
    constexpr bool FIRST = decltype(firstc)::value, MPREV = decltype(mprevc)::value;
    constexpr bool MCUR = decltype(mcurc)::value;
    const int k_first = (int)(entry_at(t) >> 1) * BK;
    const int kf_next = (int)(entry_at(t + 1) >> 1) * BK;  // (the last block repeats itself)
    const unsigned char* Kt = smem + kbuf_off(t);
    const unsigned char* Vt = smem + vbuf_off(t);
    const unsigned char* Kp = smem + kbuf_off(t + 1);  // K of block t - 1
    constexpr int NGS = NCH * NG;
    constexpr int MID = 2 * NG - PF;  // group of the mid-block barrier
    bf16x8 fa[RING];
    // group GG of the block: chunk step j, slot x, product 0 S^T / 1 dP^T / 2 dQ^T
    auto load = [&](auto gc, bf16x8& dst) __attribute__((always_inline)) {
      constexpr int GG = decltype(gc)::value, j = GG / NG, gi = GG % NG, x = gi / 3, kind = gi % 3;
      constexpr int jo = (j + NCH - 2) % NCH;  // chunk of the dQ^T products within its block
      constexpr bool OLD = j < 2;              // ... of the previous block
      if constexpr (kind == 0) {
        dst = ld_row8(Kt + offk[x] + j * 32 * D * 2);
      } else if constexpr (kind == 1) {
        dst = ld_row8(Vt + offk[x] + j * 32 * D * 2);
      } else if constexpr (!(FIRST && OLD)) {
        constexpr int kk = x / MD, md = x % MD;
        dst = ld_kt(OLD ? Kp : Kt, md, (jo * 32 + kk * 16) * D * 2);
      }
    };
    static_for<PF>([&](auto ic) { load(ic, fa[decltype(ic)::value]); });
    __builtin_amdgcn_sched_barrier(0);
    static_for<NGS>([&](auto gc) {
      constexpr int GG = decltype(gc)::value, j = GG / NG, gi = GG % NG, x = gi / 3, kind = gi % 3;
      constexpr bool OLD = j < 2;
      if constexpr (GG == MID) {
        // every read of K of block t - 1 has been issued (fragments run PF
        // groups ahead): once all waves are past them, K of block t + 1 may
        // overwrite that buffer
        __syncthreads();
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (GG < PPW) stage_piece(vbase, kf_next, vbuf_off(t + 1), GG);
      if constexpr (GG >= MID && GG < MID + PPW) stage_piece(kbase, kf_next, kbuf_off(t + 1), GG - MID);
      if constexpr (GG + PF < NGS) load(std::integral_constant<int, GG + PF>{}, fa[(GG + PF) % RING]);
      const bf16x8& a = fa[GG % RING];
      static_for<NQT>([&](auto mc) {
        constexpr int m = decltype(mc)::value;
        if constexpr (kind == 0) {
          if constexpr (x == 0)
            sacc[j & 1][m] = mfma32_v0(a, qf[m][0]);
          else
            sacc[j & 1][m] = mfma32_v(a, qf[m][x], sacc[j & 1][m]);
        } else if constexpr (kind == 1) {
          if constexpr (x == 0)
            pacc[j & 1][m] = mfma32_v0(a, gf[m][0]);
          else
            pacc[j & 1][m] = mfma32_v(a, gf[m][x], pacc[j & 1][m]);
        } else if constexpr (!(FIRST && OLD)) {
          constexpr int kk = x / MD, md = x % MD;
          qacc[md][m] = mfma32(a, __builtin_bit_cast(bf16x8, dsw[j & 1][kk][m]), qacc[md][m]);
        }
        // dS^T of the chunk before chunk j (chunk j - 1 of this block, or the
        // last chunk of the previous block), spread over the products
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
      // a chunk step without dQ^T products (start of the row): its S^T and dP^T
      // results are read early in the next step, so settle them here
      if constexpr (FIRST && OLD && gi == NG - 1) {
        settle(sacc[j & 1], pacc[j & 1]);
        __builtin_amdgcn_sched_barrier(0);
      }
    });
    // the last S^T / dP^T products may still be in flight: wait states before
    // anything reads them
    settle(sacc[1], pacc[1]);
    __builtin_amdgcn_sched_barrier(0);
    // register placement: dQ^T accumulators and Q^T / dO^T fragments in AGPRs
    // (read directly by the matrix cores), S^T, dP^T and dS^T in VGPRs; these
    // statements emit nothing
#pragma unroll
    for (int md = 0; md < MD; ++md)
#pragma unroll
      for (int nq = 0; nq < NQT; ++nq) asm volatile("" : "+a"(qacc[md][nq]));
#pragma unroll
    for (int nq = 0; nq < NQT; ++nq)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+a"(qf[nq][ks]), "+a"(gf[nq][ks]));
    k_prev = k_first;
    __builtin_amdgcn_s_waitcnt(0);  // K and V of block t + 1 have landed
    __syncthreads();                // ... for every wave
  };
  // after the last block: dS^T of its last chunk, then the dQ^T products of its
  // last two chunks
  auto drain = [&](int t) __attribute__((always_inline)) {
    using R1 = std::integral_constant<int, 1>;
    static_for<16 * NQT>([&](auto ec) { soft_a(ec, R1{}, true, k_prev + (NCH - 1) * 32 + 4 * hh); });
    static_for<16 * NQT>([&](auto ec) { soft_b(ec, R1{}, R1{}); });
    const unsigned char* Kt = smem + kbuf_off(t);
    static_for<2 * 2 * MD>([&](auto gc) {
      constexpr int GG = decltype(gc)::value, jj = GG / (2 * MD), kk = (GG / MD) % 2, md = GG % MD;
      constexpr int jo = NCH - 2 + jj;  // chunk within the block
      const bf16x8 a = ld_kt(Kt, md, (jo * 32 + kk * 16) * D * 2);
#pragma unroll
      for (int nq = 0; nq < NQT; ++nq)
        qacc[md][nq] = mfma32(a, __builtin_bit_cast(bf16x8, dsw[jo & 1][kk][nq]), qacc[md][nq]);
    });
  };
  using TT = std::true_type;
  using FF = std::false_type;

  if (n_ent > 0) {
    stage(kbase, 0, kbuf_off(0));
    stage(vbase, 0, vbuf_off(0));
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  {
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
  }

  // dQ = scale dQ^T, written once per row through LDS: once every wave's last
  // reads are done, each wave stages its 64 rows and stores whole rows, 16
  // bytes per lane, instead of 16-byte pieces of 32 rows per store in the
  // accumulator layout
  const float scale = p.softmax_scale;
  constexpr int OP = C::OUT_PITCH;
  unsigned char* ot = smem + wave * C::NQW * OP;
  __syncthreads();
#pragma unroll
  for (int nq = 0; nq < NQT; ++nq)
#pragma unroll
    for (int md = 0; md < MD; ++md)
#pragma unroll
      for (int j4 = 0; j4 < 4; ++j4) {
        bf16x4 ov;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) ov[rr] = (__bf16)(scale * qacc[md][nq][4 * j4 + rr]);
        *reinterpret_cast<bf16x4*>(ot + (nq * 32 + l32) * OP + (md * 32 + 8 * j4 + 4 * hh) * 2) = ov;
      }
  constexpr int CPR = D / 8;  // 16-byte chunks per row
#pragma unroll
  for (int x = 0; x < C::NQW * CPR / 64; ++x) {
    const int idx = x * 64 + lane, row = idx / CPR, ch = idx % CPR;
    if (q_first + row < n_q)
      *reinterpret_cast<u32x4*>(dq + (row_base + q_first + row) * D + ch * 8) =
          *reinterpret_cast<const u32x4*>(ot + row * OP + ch * 16);
  }
}

template <int D, int BQ>
hipError_t launch(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                  const void* d_o, const float* nl, const float* nd, void* dq, hipStream_t stream) {
  using C = Dq32Cfg<D, BQ>;
  auto kern = bwd_dq32<D, BQ>;
  {
    const hipError_t err = allow_lds(reinterpret_cast<const void*>(kern), C::LDS_MAX);
    if (err != hipSuccess) return err;
  }
  const unsigned blocks = (unsigned)sv.n_qt * (p.h_q / C::HPW) * (sv.ragged ? 1 : p.batch);
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), C::lds_bytes(sv.max_kt), stream, p, sv,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), static_cast<const __bf16*>(v),
                     static_cast<const __bf16*>(d_o), nl, nd, static_cast<__bf16*>(dq));
  return hipGetLastError();
}

}  // namespace

bool bwd_dq32_supported(const cowa_params& p) {
  const int G = p.h_q / p.h_k;
  if (p.tile_k != 128 || (p.head_dim != 128 && p.head_dim != 64)) return false;
  if (p.tile_q == 128) return G % 2 == 0;
  if (p.tile_q == 64) return G % 4 == 0;
  return false;
}

hipError_t launch_bwd_dq32(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                           const void* d_o, void* dq, const BwdWork& w, hipStream_t stream) {
  if (p.head_dim == 128 && p.tile_q == 128) return launch<128, 128>(p, sv, q, k, v, d_o, w.nl, w.nd, dq, stream);
  if (p.head_dim == 128 && p.tile_q == 64) return launch<128, 64>(p, sv, q, k, v, d_o, w.nl, w.nd, dq, stream);
  if (p.head_dim == 64 && p.tile_q == 128) return launch<64, 128>(p, sv, q, k, v, d_o, w.nl, w.nd, dq, stream);
  if (p.head_dim == 64 && p.tile_q == 64) return launch<64, 64>(p, sv, q, k, v, d_o, w.nl, w.nd, dq, stream);
  return hipErrorInvalidValue;
}

}  // namespace cowa
