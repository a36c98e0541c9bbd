// CoWA backward in bfloat16 on the CDNA4 matrix cores (Alg. 2).
//
// Three launches on the caller's stream:
//
//  1. bwd_pre: D = rowsum(O * dO) per query row (fp32).
//  2. bwd_main (dK, dV): one workgroup of four waves per (KV block j, local KV
//     head h_k, sequence b).  K_j and V_j stay in registers for the whole
//     workgroup (wave w owns keys [w BK/4, (w+1) BK/4)).  The workgroup walks
//     every QO head of the group and, for each, the QO blocks of I_{h_k}(j)
//     in ascending order, 64 query rows per step; Q and dO of the next step are
//     copied global -> LDS while the current step computes
//       S = Q K^T, dP = dO V^T, P = exp(S - LSE), dS = P (dP - D),
//       dV^T += dO^T P, dK^T += scale Q^T dS.
//     dK and dV of the block are summed over every QO head of the group
//     inside the workgroup and written once, without atomics; keys that no
//     query sees get zeros.
//  3. bwd_dq (dQ): one workgroup per (QO block i, QO heads of one KV group,
//     sequence b), like the forward: K_j and V_j of J_{h_k}(i) are staged in
//     double-buffered LDS and shared by the heads, Q^T and dO^T stay in
//     registers, and per KV block
//       S^T = K Q^T, dP^T = V dO^T, dS^T = P^T (dP^T - D), dQ^T += scale K^T dS^T.
//     Alg. 2 adds dQ contributions of different KV blocks with atomics; at the
//     paper's 128K scale that is ~5e10 fp32 atomic adds, more than the L2
//     atomic units sustain, so dQ is instead computed in its own pass that
//     recomputes S and dP (4d extra FLOPs per legal pair) and writes each dQ
//     row once.
#include "internal.h"
#include "window_rule.h"
#include "mfma_tiles.h"
#include "work_item.h"

namespace cowa {
namespace {



// Per query row: nd = -D with D = sum_d O[row, d] dO[row, d] (D/8 lanes per
// row), and nl = -LSE log2(e), the row's exponent offset in base 2; the dK/dV
// pass folds nd into the accumulator input of dP = dO V^T (dP - D comes out of
// the products) and adds nl to the scaled scores.
template <int D>
__global__ void __launch_bounds__(256) bwd_pre(const __bf16* __restrict__ o, const __bf16* __restrict__ d_o,
                                               const float* __restrict__ lse, float* __restrict__ nd,
                                               float* __restrict__ nl, int64_t rows) {
  constexpr int CH = D / 8;
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = c / CH;
  const int ch = (int)(c % CH);
  float part = 0.f;
  if (row < rows) {
    const uint4 a = *reinterpret_cast<const uint4*>(o + row * D + ch * 8);
    const uint4 g = *reinterpret_cast<const uint4*>(d_o + row * D + ch * 8);
    const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, gw[4] = {g.x, g.y, g.z, g.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      part = fmaf(__uint_as_float(aw[t] << 16), __uint_as_float(gw[t] << 16), part);
      part = fmaf(__uint_as_float(aw[t] & 0xffff0000u), __uint_as_float(gw[t] & 0xffff0000u), part);
    }
  }
#pragma unroll
  for (int off = 1; off < CH; off <<= 1) part += __shfl_xor(part, off);
  if (row < rows && ch == 0) {
    nd[row] = -part;
    nl[row] = -lse[row] * kLog2e;
  }
}

template <int D, int BK, int NW_ = 4>
struct BwdCfg {
  static constexpr int NW = NW_;          // waves per workgroup
  static constexpr int BQ = 64;           // query rows per step
  static constexpr int NKW = BK / NW;     // keys per wave
  static constexpr int NTK = NKW / 16;    // key tiles per wave
  static constexpr int MTQ = BQ / 16;     // query tiles per step
  static constexpr int KSD = D / 32;      // k-steps over d
  static constexpr int MD = D / 16;       // d tiles
  static constexpr int KSQ = BQ / 32;     // k-steps over queries
  using QT = SwzTile<D, BQ>;              // Q or dO rows of one step
  static constexpr int ROWV = 2 * BQ * 4; // per-step row values: LSE [BQ], then D [BQ]
  // LDS: a ring of three stages (Q, dO, row values), then the column's entry lists
  static constexpr int NST = 3;
  __device__ static int q_off(int s) { return s * QT::BYTES; }
  __device__ static int do_off(int s) { return (NST + s) * QT::BYTES; }
  __device__ static int rv_off(int s) { return 2 * NST * QT::BYTES + s * ROWV; }
  static constexpr int MAIN_BYTES = 2 * NST * QT::BYTES + NST * ROWV;
  static constexpr int LOADS_PER_STEP = 2 * QT::LOADS / NW + 1;  // direct loads each wave issues per step
  static constexpr int OUT_BYTES = 2 * BK * (D + 8) * 2;        // dK, dV staging at the end
  static constexpr int LDS_MAX = 160 * 1024;
  // LDS for a schedule with n_qt query blocks
  static int lds_bytes(int n_qt) {
    const int main = MAIN_BYTES + 4 * n_qt;
    return main > OUT_BYTES ? main : OUT_BYTES;
  }
  static int max_qblocks() { return (LDS_MAX - MAIN_BYTES) / 4; }
};

// Parts of the split columns (BwdSplit): the first n_extra workgroups (a
// multiple of 8, so the XCD order of the others is unchanged) take parts
// 1 .. P-1 of the first S KV blocks of every (sequence, KV head); the other
// workgroups take one column each (part 0 of a split column).
struct SplitArgs {
  float* part;       // [split column][P][2][BK * D] float32 partials
  int32_t S, P;      // split blocks per (sequence, KV head); parts (1: no split)
  int32_t n_extra;   // workgroups of parts 1 .. P-1, rounded up to a multiple of 8
};

template <int D, int BK, int NW>
__global__ void __launch_bounds__(64 * NW) bwd_main(cowa_params p, SchedView sv, SplitArgs sa,
                                                const __bf16* __restrict__ q,
                                                const __bf16* __restrict__ k, const __bf16* __restrict__ v,
                                                const __bf16* __restrict__ d_o, const float* __restrict__ nl,
                                                const float* __restrict__ nd, __bf16* __restrict__ dk,
                                                __bf16* __restrict__ dv) {
  using C = BwdCfg<D, BK, NW>;
  extern __shared__ __align__(1024) unsigned char smem[];

  // clusters of 32 consecutive KV blocks of one KV head share an XCD's L2;
  // first blocks (the sink, with the longest query lists) first
  int part = 0;
  WorkItem wi;
  if ((int)blockIdx.x < sa.n_extra) {
    const int e = blockIdx.x;
    part = 1 + e % (sa.P - 1);
    const int rest = e / (sa.P - 1);
    const int tile = rest % sa.S, us = rest / sa.S;  // us = sequence * h_k + KV head
    if (us >= p.batch * p.h_k) return;               // padding
    wi.group = 0;
    if (!sv.ragged) {
      wi.row = tile;
      wi.unit = us;
    } else {
      const SeqDesc sd = sv.seq[us / p.h_k];
      if (tile * BK >= sd.n_k) return;  // a sequence with fewer blocks
      wi.row = sd.kt_off + tile;
      wi.unit = us % p.h_k;
    }
  } else {
    wi = cluster_item(blockIdx.x - sa.n_extra, sv.n_kt, 1, grid_units(p, sv),
                      cluster_rows(sv.n_kt, grid_units(p, sv), 32), false);
  }
  int hk;
  const SeqCtx sc = seq_ctx(p, sv, wi.row, wi.unit, false, hk);
  const int j = sc.tile;
  const bool split = sa.P > 1 && j < sa.S;
  const int n_parts = split ? sa.P : 1;
  const int G = p.h_q / p.h_k;
  const Geo32 g = sc.g;
  const int n_q = sc.n_q, n_k = sc.n_k;

  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t k_first = (int64_t)j * BK;
  const int64_t kv_row0 = sc.k0 + (int64_t)hk * sc.kh;
  const __bf16* kbase = k + kv_row0 * D;
  const __bf16* vbase = v + kv_row0 * D;

  // The steps: every QO head of the group x every QO block of I(j) x 64-row
  // sub-blocks.  Full blocks are taken first, then partial ones, so that each
  // of the two step loops below is straight-line code (the partial loop adds
  // the element mask).  The column's entries are split once into two lists in
  // LDS: full entries from the front, partial entries from the back.
  const int col = sc.sched;
  const int e0 = sv.bwd_col_ptr[col], e1 = sv.bwd_col_ptr[col + 1];
  const int n_ent = e1 - e0;
  const int cap = sv.max_qt;  // list capacity (entries of one column)
  uint32_t* list = reinterpret_cast<uint32_t*>(smem + C::MAIN_BYTES);
  int n_full = 0;
  for (int c0 = 0; c0 < n_ent; c0 += 64) {  // every wave builds the same counts; wave 0 writes
    const bool in = c0 + lane < n_ent;
    const uint32_t ent = in ? sv.bwd_ent[e0 + c0 + lane] : 0u;
    const uint64_t full = __ballot(in && !(ent & 1u));
    const uint64_t part = __ballot(in && (ent & 1u));
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int n_part_before = c0 - n_full;
    if (wave == 0 && in) {
      if (ent & 1u)
        list[cap - 1 - (n_part_before + __popcll(part & below))] = ent;
      else
        list[n_full + __popcll(full & below)] = ent;
    }
    n_full += __popcll(full);
  }
  const int n_part = n_ent - n_full;
  const int subs = p.tile_q / C::BQ;
  const int steps_full = G * n_full * subs, n_steps = G * n_ent * subs;
  // this workgroup's steps: all of them, or part `part` of n_parts contiguous shares
  const int s_begin = (int)((int64_t)n_steps * part / n_parts);
  const int s_end = (int)((int64_t)n_steps * (part + 1) / n_parts);
  // cursor (phase: 0 full / 1 partial, QO head, list index, sub-block) of step s_begin
  int c_ph, c_k, c_sub, c_hh;
  {
    c_ph = s_begin < steps_full ? 0 : 1;
    const int r = c_ph ? s_begin - steps_full : s_begin;
    const int nl_ = c_ph ? n_part : n_full;
    c_hh = nl_ > 0 ? r / (nl_ * subs) : 0;
    c_k = nl_ > 0 ? (r / subs) % nl_ : 0;
    c_sub = r % subs;
  }
  int n1_ph = c_ph, n1_hh = c_hh, n1_k = c_k, n1_sub = c_sub;  // the next step (staged)
  int n2_ph = c_ph, n2_hh = c_hh, n2_k = c_k, n2_sub = c_sub;  // the step after (being staged)
  auto advance = [&](int& ph, int& hh, int& kk, int& sub) {
    if (++sub == subs) {
      sub = 0;
      if (++kk == (ph == 0 ? n_full : n_part)) {
        kk = 0;
        if (++hh == G) {
          hh = 0;
          ++ph;
          if (ph == 1 && n_part == 0) ph = 2;  // past the end
        }
      }
    }
  };
  // list entry of a cursor; a cursor past the end names the first entry
  auto entry_of = [&](int ph, int kk) -> uint32_t {
    const int idx = ph == 0 ? kk : (ph == 1 ? cap - 1 - kk : (n_full > 0 ? 0 : cap - 1));
    return __builtin_amdgcn_readfirstlane(list[idx]);
  };

  // Every operand of a step goes global -> LDS directly, through copies the
  // compiler does not track (dma16/dma4): the Q and dO tiles, and the LSE and
  // D values of its 64 rows (waves 0 and 2 copy the LSE, 1 and 3 the D values,
  // the same data twice).  Each wave issues LOADS_PER_STEP copies per step and
  // waits for them two steps later.  Rows past n_q (partial blocks only, where
  // the mask gives them P = 0) hold zeros or an earlier step's rows.  A cursor
  // past the last step stages a copy of the last head's rows, never read.
  const uint32_t smem_base = lds_addr(smem);
  // Each lane copies the same 16-byte column of its row in every 1 KB piece it
  // takes: its byte offsets within a tile are fixed, and the tile position
  // goes into the (scalar) buffer resource, whose size bounds the reads to the
  // sequence (rows past n_q read as zero).
  constexpr int RPL = 1024 / (D * 2);     // rows per 1 KB piece
  constexpr int PPW = C::QT::LOADS / NW;  // pieces per wave and tile
  uint32_t tile_off[PPW];
  {
    const int row0 = wave * RPL + lane / C::QT::CH;
    const int col = (lane % C::QT::CH) ^ swz<C::QT::CH>(row0);
#pragma unroll
    for (int n = 0; n < PPW; ++n) tile_off[n] = (uint32_t)(((n * NW * RPL + row0) * D + col * 8) * 2);
  }
  // A step's copies are issued in pieces (piece n: 1 KB of Q and of dO per
  // wave; and the row values), one piece every other product group early in
  // the step two before it: issued back to back they hold the wave at the
  // vector memory queue for hundreds of cycles.  (Spread over the whole step
  // they would keep more scalar registers live than the kernel has.)
  struct StageSrc {
    int64_t off;       // byte offset of the step's first row in Q and in dO
    uint32_t bytes;    // bytes from there to the end of the sequence
    const float* rv;   // this lane's LSE or D value
  };
  auto stage_src = [&](uint32_t ent, int hh, int sub) -> StageSrc {
    hh = hh < G ? hh : G - 1;
    const int q0 = (int)(ent >> 1) * p.tile_q + sub * C::BQ;
    const int64_t row_base = sc.q0 + (int64_t)(hk * G + hh) * sc.qh;
    // a sub-block wholly past n_q (the last QO block's second half) reads nothing
    const uint32_t bytes = q0 < n_q ? (uint32_t)(n_q - q0) * D * 2 : 0u;
    const int r = q0 + lane;
    const int rc = r < n_q ? r : n_q - 1;
    return StageSrc{(row_base + q0) * D * 2, bytes, ((wave & 1) ? nd : nl) + row_base + rc};
  };
  auto stage_piece = [&](const StageSrc& src, int n, int slot) {
    const unsigned char* qb = reinterpret_cast<const unsigned char*>(q) + src.off;
    const unsigned char* ob = reinterpret_cast<const unsigned char*>(d_o) + src.off;
    dma16_buf(tile_off[n], buffer_rsrc(qb, src.bytes), smem_base + C::q_off(slot) + (n * NW + wave) * 1024);
    dma16_buf(tile_off[n], buffer_rsrc(ob, src.bytes), smem_base + C::do_off(slot) + (n * NW + wave) * 1024);
  };
  auto stage_rows = [&](const StageSrc& src, int slot) {
    dma4(src.rv, __builtin_amdgcn_readfirstlane(smem_base + C::rv_off(slot) + (wave & 1) * C::BQ * 4));
  };
  auto stage = [&](uint32_t ent, int hh, int sub, int slot) {
    const StageSrc src = stage_src(ent, hh, sub);
#pragma unroll
    for (int n = 0; n < PPW; ++n) stage_piece(src, n, slot);
    stage_rows(src, slot);
  };

  // rows past the end of the sequence are not copied: give them finite values
  for (int x = tid; x < 2 * C::NST * C::QT::BYTES / 16; x += blockDim.x)
    reinterpret_cast<uint4*>(smem)[x] = uint4{0u, 0u, 0u, 0u};
  __syncthreads();  // the entry lists and the zeroed stages are in LDS
  // prologue: the first two steps in flight
  if (s_end > s_begin) {
    stage(entry_of(n2_ph, n2_k), n2_hh, n2_sub, 0);  // step s_begin
    advance(n2_ph, n2_hh, n2_k, n2_sub);
    n1_ph = n2_ph, n1_hh = n2_hh, n1_k = n2_k, n1_sub = n2_sub;
    stage(entry_of(n2_ph, n2_k), n2_hh, n2_sub, 1);  // step 1
    advance(n2_ph, n2_hh, n2_k, n2_sub);
  }

  // K and V rows of this wave's keys as B fragments: key nt*16 + lr, d = ks*32 + 8*lg + 0..7
  bf16x8 kf[C::NTK][C::KSD], vf[C::NTK][C::KSD];
#pragma unroll
  for (int nt = 0; nt < C::NTK; ++nt) {
    int64_t kp = k_first + wave * C::NKW + nt * 16 + lr;
    if (kp >= n_k) kp = n_k - 1;  // masked: such keys are in partial blocks only
#pragma unroll
    for (int ks = 0; ks < C::KSD; ++ks) {
      kf[nt][ks] = *reinterpret_cast<const bf16x8*>(kbase + kp * D + ks * 32 + 8 * lg);
      vf[nt][ks] = *reinterpret_cast<const bf16x8*>(vbase + kp * D + ks * 32 + 8 * lg);
    }
  }
  f32x4 dka[C::MD][C::NTK], dva[C::MD][C::NTK];  // dK^T / scale, dV^T: rows d, columns keys
#pragma unroll
  for (int md = 0; md < C::MD; ++md)
#pragma unroll
    for (int nt = 0; nt < C::NTK; ++nt) {
      dka[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      dva[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  // per-lane LDS offsets of the row-fragment and transposing reads
  int offr[C::KSD], offt[C::MD];
#pragma unroll
  for (int ks = 0; ks < C::KSD; ++ks) offr[ks] = row8_off<D>(lr, lg, ks);
#pragma unroll
  for (int md = 0; md < C::MD; ++md) offt[md] = tr8_off<D>(lr, lg, md);
  const float c = p.softmax_scale * kLog2e;
  const int k0 = (int)k_first + wave * C::NKW + lr;  // key of column nt*16 + lr
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // One step on ring slot `slot`:
  //   S = Q K^T, dP = dO V^T, P = exp(S - LSE), dS = P (dP - D),
  //   dV^T += dO^T P, dK^T += Q^T dS (the softmax scale is applied to dK at the end).
  // The 64 rows are taken in two halves of 32 (one k-step of the dV/dK
  // products).  The step is a fixed schedule of groups of four MFMAs, each
  // with the LDS reads of the next group and, where there is one, a chunk of a
  // softmax, so that the matrix cores always have independent work while the
  // vector units run the exponentials:
  //   S/dP(half 0) | S/dP(half 1) + softmax(half 0) | dV/dK(half 0) + softmax(half 1) | dV/dK(half 1)
  // Scheduling fences between groups keep that order.
  f32x4 sacc[C::MTQ][C::NTK], pacc[C::MTQ][C::NTK];  // rows q = mt*16 + 4*lg + r, column key = nt*16 + lr
  bf16x8 pb[C::KSQ][C::NTK], sb[C::KSQ][C::NTK];     // P and dS as B operands, k-slots = queries of a half
  constexpr int NG = 2 * C::KSD;  // S/dP groups per half: (k-step, query tile)
  static_assert(C::MTQ == 4 && C::MD == NG && (8 * C::NTK) % NG == 0, "group schedule layout");
  // S/dP group gi of half hf: k-step gi / 2, query tile 2 hf + gi % 2
  auto sdp_load = [&](const unsigned char* qs, const unsigned char* dos, int hf, int gi, bf16x8& fa, bf16x8& fb) {
    const int ks = gi >> 1, mt = 2 * hf + (gi & 1);
    fa = ld_row8(qs + offr[ks] + mt * 16 * D * 2);
    fb = ld_row8(dos + offr[ks] + mt * 16 * D * 2);
  };
  // (dP accumulates on top of -D of its rows, so it holds dP - D)
  auto sdp_mfma = [&](int hf, int gi, const bf16x8& fa, const bf16x8& fb, const f32x4 (&nd4)[C::MTQ]) {
    const int ks = gi >> 1, mt = 2 * hf + (gi & 1);
#pragma unroll
    for (int nt = 0; nt < C::NTK; ++nt) {
      sacc[mt][nt] = mfma16(fa, kf[nt][ks], ks == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : sacc[mt][nt]);
      pacc[mt][nt] = mfma16(fb, vf[nt][ks], ks == 0 ? nd4[mt] : pacc[mt][nt]);
    }
  };
  // dV/dK group md of half hf: d tile md, queries of the half as k-slots
  auto dvdk_load = [&](const unsigned char* qs, const unsigned char* dos, int hf, int md, bf16x8& fa, bf16x8& fb) {
    fa = ld_tr8(dos + offt[md] + hf * 32 * D * 2, D * 2);
    fb = ld_tr8(qs + offt[md] + hf * 32 * D * 2, D * 2);
  };
  auto dvdk_mfma = [&](int hf, int md, const bf16x8& fa, const bf16x8& fb) {
#pragma unroll
    for (int nt = 0; nt < C::NTK; ++nt) {
      dva[md][nt] = mfma16(fa, pb[hf][nt], dva[md][nt]);
      dka[md][nt] = mfma16(fb, sb[hf][nt], dka[md][nt]);
    }
  };
  // Softmax chunk ci of half hf: elements e = ci * EPC .. ci * EPC + EPC - 1 of
  // the lane's 8 NTK, where element e is row r = e % 4 of the lane's four in
  // query tile 2 hf + e / (4 NTK), key tile (e / 4) % NTK.  P and dS are rounded
  // to bf16 into the B-operand layout: k-slot 4 i + r is query row
  // (2 hf + i) * 16 + 4 lg + r.  In a partial block the masked pairs get P = 0
  // through a -inf exponent, selected after the exponent has read the MFMA result.
  constexpr int EPC = 8 * C::NTK / NG;
  // (the row values are nl = -LSE log2(e), so x = S c + nl = (S - LSE) log2(e);
  // pacc already holds dP - D)
  // In a partial block the window rule comes as a bit mask over the half's 32
  // query rows per key (once per half and key tile, shifted to the lane's rows
  // 4 lg + 16 i + r); an illegal pair's exponent becomes -inf by a bit select.
  uint32_t qmask[C::NTK];
  auto soft_chunk = [&](int hf, int ci, const float4 (&l4)[2], bool masked, int q0) {
    if (masked && ci == 0)
#pragma unroll
      for (int nt = 0; nt < C::NTK; ++nt) qmask[nt] = legal_queries32(g, q0 + 32 * hf, k0 + nt * 16) >> (4 * lg);
#pragma unroll
    for (int jj = 0; jj < EPC; ++jj) {
      const int e = ci * EPC + jj, r = e & 3, nt = (e >> 2) % C::NTK, i = e / (4 * C::NTK), mt = 2 * hf + i;
      const float lv = r == 0 ? l4[i].x : r == 1 ? l4[i].y : r == 2 ? l4[i].z : l4[i].w;
      float x = fmaf(sacc[mt][nt][r], c, lv);
      // (a row of a full block has a finite LSE; a masked pair may have LSE = -inf)
      if (masked) {
        const uint32_t m = (uint32_t)((int32_t)(qmask[nt] << (31 - (16 * i + r))) >> 31);
        x = __uint_as_float((__float_as_uint(x) & m) | (0xff800000u & ~m));
      }
      const float pv = __builtin_amdgcn_exp2f(x);
      pb[hf][nt][4 * i + r] = (__bf16)pv;
      sb[hf][nt][4 * i + r] = (__bf16)(pv * pacc[mt][nt][r]);
    }
  };
  // nl of query tile 2 hf + i (the lane's rows 4 lg .. 4 lg + 3)
  auto load_rowv = [&](const float* rowv, int hf, int i, float4 (&l4)[2]) {
    l4[i] = *reinterpret_cast<const float4*>(rowv + (2 * hf + i) * 16 + 4 * lg);
  };

  int slot = 0;  // ring slot of the step being computed (t mod 3)
  auto step = [&](bool masked) {
    const int slot2 = slot == 0 ? 2 : slot - 1;  // (t + 2) mod 3
    const unsigned char* qs = smem + C::q_off(slot);
    const unsigned char* dos = smem + C::do_off(slot);
    const float* rowv = reinterpret_cast<const float*>(smem + C::rv_off(slot));
    const int q0 = (int)(entry_of(c_ph, c_k) >> 1) * p.tile_q + c_sub * C::BQ;
    const StageSrc src2 = stage_src(entry_of(n2_ph, n2_k), n2_hh, n2_sub);

    // groups 0 .. 4 NG - 1: S/dP(half 0), S/dP(half 1), dV/dK(half 0), dV/dK(half 1);
    // operand fragments are read PD groups ahead of their MFMAs
    constexpr int NGT = 4 * NG, PD = 1;
    static_assert(2 * PPW <= NGT, "copy pieces per step");
    auto load_group = [&](int gg, bf16x8& fa, bf16x8& fb) {
      if (gg < NG)
        sdp_load(qs, dos, 0, gg, fa, fb);
      else if (gg < 2 * NG)
        sdp_load(qs, dos, 1, gg - NG, fa, fb);
      else if (gg < 3 * NG)
        dvdk_load(qs, dos, 0, gg - 2 * NG, fa, fb);
      else
        dvdk_load(qs, dos, 1, gg - 3 * NG, fa, fb);
    };
    bf16x8 fa[PD + 1], fb[PD + 1];
    float4 l4[2];  // nl of the half in the softmax
    f32x4 nd4[C::MTQ];  // -D of the step's rows, the accumulator input of dP
#pragma unroll
    for (int mt = 0; mt < C::MTQ; ++mt) nd4[mt] = *reinterpret_cast<const f32x4*>(rowv + C::BQ + mt * 16 + 4 * lg);
#pragma unroll
    for (int gg = 0; gg < PD; ++gg) load_group(gg, fa[gg], fb[gg]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int gg = 0; gg < NGT; ++gg) {
      if (gg + PD < NGT) load_group(gg + PD, fa[(gg + PD) % (PD + 1)], fb[(gg + PD) % (PD + 1)]);
      if (gg % 2 == 0 && gg < 2 * PPW) stage_piece(src2, gg / 2, slot2);
      if (gg == 1) stage_rows(src2, slot2);
      // the row values of a half's first and second query tile are needed by
      // its softmax chunks [0, NG/2) and [NG/2, NG); each is loaded once the
      // previous half no longer reads that register
      if (gg == NG - 2) {
        load_rowv(rowv, 0, 0, l4);
        load_rowv(rowv, 0, 1, l4);
      }
      if (gg == NG + NG / 2) load_rowv(rowv, 1, 0, l4);
      if (gg == 2 * NG) load_rowv(rowv, 1, 1, l4);
      bf16x8& a0 = fa[gg % (PD + 1)];
      bf16x8& b0 = fb[gg % (PD + 1)];
      if (gg < NG)
        sdp_mfma(0, gg, a0, b0, nd4);
      else if (gg < 2 * NG)
        sdp_mfma(1, gg - NG, a0, b0, nd4);
      else if (gg < 3 * NG)
        dvdk_mfma(0, gg - 2 * NG, a0, b0);
      else
        dvdk_mfma(1, gg - 3 * NG, a0, b0);
      if (gg >= NG && gg < 2 * NG) soft_chunk(0, gg - NG, l4, masked, q0);
      if (gg >= 2 * NG && gg < 3 * NG) soft_chunk(1, gg - 2 * NG, l4, masked, q0);
      __builtin_amdgcn_sched_barrier(0);
    }

    // Register placement (the library builds this file with MFMA results in
    // VGPRs): the dK/dV accumulators stay in VGPRs and the K/V fragments in
    // AGPRs, which the MFMAs read directly as B operands.  These empty
    // statements emit nothing; they only pin the register class across steps
    // (otherwise the allocator shuffles values between the two files).
#pragma unroll
    for (int md = 0; md < C::MD; ++md)
#pragma unroll
      for (int nt = 0; nt < C::NTK; ++nt) asm volatile("" : "+v"(dka[md][nt]), "+v"(dva[md][nt]));
#pragma unroll
    for (int nt = 0; nt < C::NTK; ++nt)
#pragma unroll
      for (int ks = 0; ks < C::KSD; ++ks) asm volatile("" : "+a"(kf[nt][ks]), "+a"(vf[nt][ks]));
    // the next step's operands have landed (only the step after may still be in
    // flight), for every wave; and this step's slot is no longer read
    __builtin_amdgcn_s_waitcnt(vmcnt_only(C::LOADS_PER_STEP));
    __syncthreads();
    c_ph = n1_ph, c_k = n1_k, c_sub = n1_sub;
    n1_ph = n2_ph, n1_hh = n2_hh, n1_k = n2_k, n1_sub = n2_sub;
    advance(n2_ph, n2_hh, n2_k, n2_sub);
    slot = slot == 2 ? 0 : slot + 1;
  };
  int t = s_begin;
  for (; t < (s_end < steps_full ? s_end : steps_full); ++t) step(false);
  for (; t < s_end; ++t) step(true);

  // the copies staged past the last step must land before their LDS is reused
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  const float scale = p.softmax_scale;
  if (split) {
    // float32 partials in register order: element ((md NTK + nt) NW + wave) 64 + lane
    // holds rows d = 16 md + 4 (lane / 16) + 0..3, key wave NKW + 16 nt + lane % 16
    const int64_t col = ((int64_t)(sc.b * p.h_k + hk) * sa.S + j) * sa.P + part;
    f32x4* pk = reinterpret_cast<f32x4*>(sa.part + col * 2 * BK * D);
    f32x4* pv = pk + BK * D / 4;
#pragma unroll
    for (int md = 0; md < C::MD; ++md)
#pragma unroll
      for (int nt = 0; nt < C::NTK; ++nt) {
        const int x = ((md * C::NTK + nt) * NW + wave) * 64 + lane;
        pk[x] = scale * dka[md][nt];
        pv[x] = dva[md][nt];
      }
    return;
  }
  // write dK and dV of the block: through LDS as [key][d], then 16-byte rows
  __bf16* tk = reinterpret_cast<__bf16*>(smem);                        // [BK][D + 8]
  __bf16* tv = reinterpret_cast<__bf16*>(smem) + BK * (D + 8);         // [BK][D + 8]
#pragma unroll
  for (int md = 0; md < C::MD; ++md)
#pragma unroll
    for (int nt = 0; nt < C::NTK; ++nt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int key = wave * C::NKW + nt * 16 + lr, d = md * 16 + 4 * lg + rr;
        tk[key * (D + 8) + d] = (__bf16)(scale * dka[md][nt][rr]);
        tv[key * (D + 8) + d] = (__bf16)dva[md][nt][rr];
      }
  __syncthreads();
  __bf16* dkb = dk + kv_row0 * D;
  __bf16* dvb = dv + kv_row0 * D;
  for (int x = tid; x < BK * (D / 8); x += blockDim.x) {
    const int key = x / (D / 8), ch = x % (D / 8);
    const int64_t kp = k_first + key;
    if (kp < n_k) {
      *reinterpret_cast<uint4*>(dkb + kp * D + ch * 8) = *reinterpret_cast<const uint4*>(tk + key * (D + 8) + ch * 8);
      *reinterpret_cast<uint4*>(dvb + kp * D + ch * 8) = *reinterpret_cast<const uint4*>(tv + key * (D + 8) + ch * 8);
    }
  }
}

// Sum of the P partials of each split column (in part order) -> bf16 dK, dV;
// one workgroup per (split column, 16-row d tile), each thread the
// register-order elements a lane of bwd_main held for that d tile.
template <int D, int BK, int NW>
__global__ void __launch_bounds__(64 * NW) bwd_split_sum(cowa_params p, SchedView sv, SplitArgs sa,
                                                     __bf16* __restrict__ dk, __bf16* __restrict__ dv) {
  using C = BwdCfg<D, BK, NW>;
  const int c = blockIdx.x;  // (sequence * h_k + KV head) * S + block
  const int j = c % sa.S, us = c / sa.S, b = us / p.h_k, hk = us % p.h_k;
  int n_k;
  int64_t row0;  // row of key 0 of this (sequence, KV head) in K, V, dK, dV
  if (!sv.ragged) {
    n_k = p.n_k;
    row0 = ((int64_t)b * p.h_k + hk) * p.n_k;
  } else {
    const SeqDesc sd = sv.seq[b];
    n_k = sd.n_k;
    row0 = (int64_t)hk * p.n_k + sd.k_start;
  }
  if (j * BK >= n_k) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 15, lg = lane >> 4;
  const f32x4* src = reinterpret_cast<const f32x4*>(sa.part + (int64_t)c * sa.P * 2 * BK * D);
  const int md = blockIdx.y;
#pragma unroll
  for (int nt = 0; nt < C::NTK; ++nt) {
    const int x = ((md * C::NTK + nt) * NW + wave) * 64 + lane;
    f32x4 a = src[x], g = src[BK * D / 4 + x];
    for (int pt = 1; pt < sa.P; ++pt) {
      a += src[pt * (2 * BK * D / 4) + x];
      g += src[pt * (2 * BK * D / 4) + BK * D / 4 + x];
    }
    const int64_t kp = (int64_t)j * BK + wave * C::NKW + nt * 16 + lr;
    if (kp >= n_k) continue;
    bf16x4 ka, va;
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      ka[rr] = (__bf16)a[rr];
      va[rr] = (__bf16)g[rr];
    }
    const int64_t off = (row0 + kp) * D + md * 16 + 4 * lg;
    *reinterpret_cast<bf16x4*>(dk + off) = ka;
    *reinterpret_cast<bf16x4*>(dv + off) = va;
  }
}

template <int D, int BK, int NW = 4>
hipError_t launch_main(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                       const void* d_o, const BwdWork& w, void* dk, void* dv, hipStream_t stream) {
  using C = BwdCfg<D, BK, NW>;
  static_assert(C::OUT_BYTES <= C::LDS_MAX && C::MAIN_BYTES < C::LDS_MAX, "LDS budget");
  if (sv.max_qt > C::max_qblocks()) return hipErrorInvalidValue;
  auto kern = bwd_main<D, BK, NW>;
  {
    const hipError_t err = allow_lds(reinterpret_cast<const void*>(kern), C::LDS_MAX);
    if (err != hipSuccess) return err;
  }
  SplitArgs sa;
  sa.part = w.part;
  sa.S = w.split.S;
  sa.P = w.split.P;
  sa.n_extra = sa.P > 1 ? (int32_t)(((int64_t)p.batch * p.h_k * sa.S * (sa.P - 1) + 7) / 8 * 8) : 0;
  const unsigned blocks = (unsigned)sv.n_kt * p.h_k * (sv.ragged ? 1 : p.batch) + (unsigned)sa.n_extra;
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(64 * NW), C::lds_bytes(sv.max_qt), stream, p, sv, sa,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), static_cast<const __bf16*>(v),
                     static_cast<const __bf16*>(d_o), w.nl, w.nd, static_cast<__bf16*>(dk),
                     static_cast<__bf16*>(dv));
  if (sa.P > 1)
    hipLaunchKernelGGL((bwd_split_sum<D, BK, NW>), dim3((unsigned)w.split.n_cols, C::MD), dim3(64 * NW), 0, stream, p, sv,
                       sa, static_cast<__bf16*>(dk), static_cast<__bf16*>(dv));
  return hipGetLastError();
}

// dQ pass: one workgroup per (QO block i, HPW QO heads of one KV group,
// sequence b); each 64-lane wave owns 64 query rows of one head, and one wave
// runs per SIMD.  Q^T and dO^T of the wave's rows stay in registers (as MFMA B
// operands, pinned to AGPRs) for the whole row of KV blocks; K_j and V_j are
// double buffered in LDS and shared by the heads.  Full blocks are taken first,
// then partial ones (each kind a straight-line loop body).  Per chunk of 32 keys:
//   phase A: S^T = K Q^T and dP^T = V dO^T for 16 keys (32 MFMAs),
//   phase B: dS^T = P^T (dP^T - D) for those keys on the vector units while the
//            matrix cores run half of dQ^T += K^T dS^T of the previous chunk,
// twice per chunk;
// the softmax scale is applied to dQ when it is written.
template <int D, int BQ, int BK, int NQW_ = 64>
struct DqCfg {
  static constexpr int NQW = NQW_;          // query rows per wave
  static constexpr int NTQ = NQW / 16;      // query tiles per wave
  static constexpr int BKC = 32;            // keys per chunk (one k-step of dQ^T += K^T dS^T)
  static constexpr int NCH = BK / BKC;      // chunks per block
  static constexpr int KSD = D / 32;        // k-steps over d
  static constexpr int MTD = D / 16;        // d tiles of dQ^T
  static constexpr int WPH = BQ / NQW;      // waves per QO head
  using T = SwzTile<D, BK>;
  static constexpr int MAIN_BYTES = 4 * T::BYTES;  // K, V of two blocks; then the row's entry lists
  static constexpr int LDS_MAX = 160 * 1024;
  static int lds_bytes(int n_kt) { return MAIN_BYTES + 4 * n_kt; }
  static int max_kblocks() { return (LDS_MAX - MAIN_BYTES) / 4; }
};

// W4: the workgroup has exactly four waves (then the next block's copies are
// spread over the block's product groups).
template <int D, int BQ, int BK, int NQW, bool W4>
__global__ void __launch_bounds__(256 * 64 / NQW) bwd_dq_kernel(cowa_params p, SchedView sv, int hpw,
                                                     const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                                                     const __bf16* __restrict__ v, const __bf16* __restrict__ d_o,
                                                     const float* __restrict__ nl, const float* __restrict__ nd,
                                                     __bf16* __restrict__ dq) {
  using C = DqCfg<D, BQ, BK, NQW>;
  using T = typename C::T;
  constexpr int NTQ = C::NTQ, KSD = C::KSD, MTD = C::MTD;
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
  const int h0 = hgi * hpw;

  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int h = h0 + wave / C::WPH;
  const int q_first = i * BQ + (wave % C::WPH) * C::NQW;
  const Geo32 g = sc.g;
  const int n_q = sc.n_q, n_k = sc.n_k;

  const __bf16* kbase = k + (sc.k0 + (int64_t)hk * sc.kh) * D;
  const __bf16* vbase = v + (sc.k0 + (int64_t)hk * sc.kh) * D;
  const uint32_t smem_base = lds_addr(smem);

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
  // list position of the t-th block in processing order (full ones, then partial ones)
  auto entry_at = [&](int t) -> uint32_t {
    const int tt = t < n_ent ? t : n_ent - 1;
    const int idx = tt < n_full ? tt : cap - 1 - (tt - n_full);
    return __builtin_amdgcn_readfirstlane(list[idx]);
  };
  auto stage = [&](uint32_t ent, int buf) {
    const int kf = (int)(ent >> 1) * BK;
    load_tile_asm_nw<D, BK>(kbase, kf, n_k, smem_base + buf * 2 * T::BYTES, wave, nw, lane);
    load_tile_asm_nw<D, BK>(vbase, kf, n_k, smem_base + buf * 2 * T::BYTES + T::BYTES, wave, nw, lane);
  };
  __syncthreads();  // the lists are in LDS
  if (n_ent > 0) stage(entry_at(0), 0);
  // With four waves, the next block's K and V copies go out one 1 KB piece per
  // product group (K piece n, then V piece n) instead of a burst that would
  // hold the wave at the vector memory queue; past the last block the last
  // block is copied again (into the free buffer, never read).
  constexpr int RPL = 1024 / (D * 2), PPW4 = T::LOADS / 4;
  static_assert(!W4 || (T::LOADS % 4 == 0 && (4 * RPL) % 16 == 0), "piece layout");
  const int row0 = wave * RPL + lane / T::CH;
  const int col0 = ((lane % T::CH) ^ swz<T::CH>(row0)) << 3;
  auto stage_piece = [&](const __bf16* base, int kf, int buf, int n, int isv) {
    int r = kf + n * 4 * RPL + row0;
    r = r < n_k ? r : n_k - 1;
    dma16(base + (int64_t)r * D + col0,
          __builtin_amdgcn_readfirstlane(smem_base + buf * 2 * T::BYTES + isv * T::BYTES + (n * 4 + wave) * 1024));
  };

  // Q^T and dO^T fragments (B operands): query column nt*16 + lr, d = ks*32 + 8*lg + 0..7;
  // per-query LSE (base 2; a row without keys or past n_q gets +inf, so P = 0) and D
  const int64_t row_base = sc.q0 + (int64_t)h * sc.qh;
  bf16x8 qf[NTQ][KSD], gf[NTQ][KSD];
  float l2[NTQ], dd[NTQ];
#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) {
    const int qp = q_first + nt * 16 + lr;
    const bool ok = qp < n_q;
    const int64_t row = row_base + (ok ? qp : 0);
#pragma unroll
    for (int ks = 0; ks < KSD; ++ks) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(q + row * D + ks * 32 + 8 * lg);
      const bf16x8 c2 = *reinterpret_cast<const bf16x8*>(d_o + row * D + ks * 32 + 8 * lg);
      qf[nt][ks] = ok ? a : bf16x8{};
      gf[nt][ks] = ok ? c2 : bf16x8{};
    }
    // nl = -LSE log2(e); a row without keys (LSE = -inf) or past n_q gets +inf, so P = 0
    const float nlv = ok ? nl[row] : INFINITY;
    l2[nt] = nlv == INFINITY ? INFINITY : -nlv;
    dd[nt] = ok ? -nd[row] : 0.f;
  }

  f32x4 qacc[MTD][NTQ];  // dQ^T / scale: rows d, columns queries
#pragma unroll
  for (int md = 0; md < MTD; ++md)
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt) qacc[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float c = p.softmax_scale * kLog2e;
  // per-lane offsets: K/V row fragments (row lr of a 16-row tile, chunk 4 ks + lg)
  // and the transposing K^T reads (rows 4 lg + lr / 4, column 16 md + 4 (lr % 4))
  int offr[KSD], offt[MTD];
#pragma unroll
  for (int ks = 0; ks < KSD; ++ks) offr[ks] = row8_off<D>(lr, lg, ks);
#pragma unroll
  for (int md = 0; md < MTD; ++md) offt[md] = tr8_off<D>(lr, lg, md);

  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  f32x4 sacc[NTQ], pacc[NTQ];  // S^T, dP^T of 16 keys: rows keys 4 lg + rr, column query 16 nt + lr
  bf16x8 sb[2][NTQ];           // dS^T of the current and the previous chunk as B operands

  // dS^T of key tile kt, query tile nt into sb[sl], k-slots 4 (kt % 2) + rr
  // (key 16 kt + 4 lg + rr of the block); the chunk's k-slot order is the one
  // the transposing K^T read produces
  auto ds_tile = [&](int sl, int kt, int nt, bool masked, int k_first) {
    const int qp = q_first + nt * 16 + lr;
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
      float x = fmaf(sacc[nt][rr], c, -l2[nt]);
      if (masked) x = legal32(g, qp, k_first + kt * 16 + 4 * lg + rr) ? x : -INFINITY;
      const float pv = __builtin_amdgcn_exp2f(x);
      sb[sl][nt][4 * (kt & 1) + rr] = (__bf16)(pv * (pacc[nt][rr] - dd[nt]));
    }
  };
  // A block is a fixed sequence of groups, each an LDS read (issued PD groups
  // ahead) and the MFMAs that consume it:
  //   per key tile kt (16 keys): KSD groups of S^T/dP^T, then MTD/2 groups of
  //   dQ^T for the previous 32-key chunk interleaved with dS^T of tile kt;
  //   finally MTD groups of dQ^T for the last chunk.
  constexpr int GPS = KSD + MTD / 2, NKT = 2 * C::NCH, NGB = NKT * GPS + MTD, PD = 1;
  static_assert(!W4 || 2 * PPW4 <= NGB, "copy pieces per block");
  auto load_g = [&](const unsigned char* Kt, const unsigned char* Vt, int gg, bf16x8& fa, bf16x8& fb) {
    if (gg < NKT * GPS) {
      const int kt = gg / GPS, r = gg % GPS;
      if (r < KSD) {
        fa = ld_row8(Kt + offr[r] + kt * 16 * D * 2);
        fb = ld_row8(Vt + offr[r] + kt * 16 * D * 2);
      } else if (kt >= 2) {
        const int md = (kt & 1) * (MTD / 2) + (r - KSD);
        fa = ld_tr8(Kt + offt[md] + (kt / 2 - 1) * C::BKC * D * 2, D * 2);
      }
    } else {
      const int md = gg - NKT * GPS;
      fa = ld_tr8(Kt + offt[md] + (C::NCH - 1) * C::BKC * D * 2, D * 2);
    }
  };
  auto exec_g = [&](int gg, const bf16x8& fa, const bf16x8& fb, bool masked, int k_first) {
    if (gg < NKT * GPS) {
      const int kt = gg / GPS, r = gg % GPS;
      if (r < KSD) {
#pragma unroll
        for (int nt = 0; nt < NTQ; ++nt) {
          sacc[nt] = mfma16(fa, qf[nt][r], r == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : sacc[nt]);
          pacc[nt] = mfma16(fb, gf[nt][r], r == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : pacc[nt]);
        }
      } else {
        const int x = r - KSD;
        if (kt >= 2) {
          const int md = (kt & 1) * (MTD / 2) + x, sl = (kt / 2 - 1) & 1;
#pragma unroll
          for (int nt = 0; nt < NTQ; ++nt) qacc[md][nt] = mfma16(fa, sb[sl][nt], qacc[md][nt]);
        }
#pragma unroll
        for (int nt = x * NTQ / (MTD / 2); nt < (x + 1) * NTQ / (MTD / 2); ++nt)
          ds_tile((kt / 2) & 1, kt, nt, masked, k_first);
      }
    } else {
      const int md = gg - NKT * GPS, sl = (C::NCH - 1) & 1;
#pragma unroll
      for (int nt = 0; nt < NTQ; ++nt) qacc[md][nt] = mfma16(fa, sb[sl][nt], qacc[md][nt]);
    }
  };

  auto block = [&](int t, bool masked) {
    const int buf = t & 1;
    const uint32_t ent = entry_at(t);
    const int k_first = (int)(ent >> 1) * BK;
    [[maybe_unused]] const int kf_next = (int)(entry_at(t + 1) >> 1) * BK;
    if constexpr (!W4) {
      if (t + 1 < n_ent) stage(entry_at(t + 1), buf ^ 1);  // prefetch the next block
    }
    const unsigned char* Kt = smem + buf * 2 * T::BYTES;
    const unsigned char* Vt = Kt + T::BYTES;
    bf16x8 fa[PD + 1], fb[PD + 1];
    static_for<PD>([&](auto ic) { load_g(Kt, Vt, ic.value, fa[ic.value], fb[ic.value]); });
    __builtin_amdgcn_sched_barrier(0);
    static_for<NGB>([&](auto ic) {
      constexpr int gg = decltype(ic)::value;
      if constexpr (W4 && gg < 2 * PPW4) stage_piece((gg & 1) ? vbase : kbase, kf_next, buf ^ 1, gg >> 1, gg & 1);
      if constexpr (gg + PD < NGB) load_g(Kt, Vt, gg + PD, fa[(gg + PD) % (PD + 1)], fb[(gg + PD) % (PD + 1)]);
      exec_g(gg, fa[gg % (PD + 1)], fb[gg % (PD + 1)], masked, k_first);
      __builtin_amdgcn_sched_barrier(0);
    });
    // register placement: dQ^T accumulators in VGPRs, Q^T / dO^T fragments in
    // AGPRs (read directly as B operands); these statements emit nothing
#pragma unroll
    for (int md = 0; md < MTD; ++md)
#pragma unroll
      for (int nt = 0; nt < NTQ; ++nt) asm volatile("" : "+v"(qacc[md][nt]));
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt)
#pragma unroll
      for (int ks = 0; ks < KSD; ++ks) asm volatile("" : "+a"(qf[nt][ks]), "+a"(gf[nt][ks]));
    __builtin_amdgcn_s_waitcnt(0);  // the next block has landed
    __syncthreads();                 // ... for every wave, and this block is no longer read
  };
  int t = 0;
  for (; t < n_full; ++t) block(t, false);
  for (; t < n_ent; ++t) block(t, true);

  const float scale = p.softmax_scale;
#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) {
    const int qp = q_first + nt * 16 + lr;
    if (qp >= n_q) continue;
    __bf16* drow = dq + (row_base + qp) * D;
#pragma unroll
    for (int md = 0; md < MTD; ++md) {
      bf16x4 w4;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) w4[rr] = (__bf16)(scale * qacc[md][nt][rr]);
      *reinterpret_cast<bf16x4*>(drow + md * 16 + 4 * lg) = w4;
    }
  }
}

template <int D, int BQ, int BK, int NQW, bool W4>
hipError_t launch_dq_w(const cowa_params& p, const SchedView& sv, int hpw, int waves, const void* q, const void* k,
                       const void* v, const void* d_o, const float* nl, const float* nd, void* dq,
                       hipStream_t stream) {
  using C = DqCfg<D, BQ, BK, NQW>;
  auto kern = bwd_dq_kernel<D, BQ, BK, NQW, W4>;
  {
    const hipError_t err = allow_lds(reinterpret_cast<const void*>(kern), C::LDS_MAX);
    if (err != hipSuccess) return err;
  }
  const int n_hgroups = p.h_q / hpw;
  const unsigned blocks = (unsigned)sv.n_qt * n_hgroups * (sv.ragged ? 1 : p.batch);
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(64 * waves), C::lds_bytes(sv.max_kt), stream, p, sv, hpw,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), static_cast<const __bf16*>(v),
                     static_cast<const __bf16*>(d_o), nl, nd, static_cast<__bf16*>(dq));
  return hipGetLastError();
}

template <int D, int BQ, int BK, int NQW = 64>
hipError_t launch_dq(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                     const void* d_o, const float* nl, const float* nd, void* dq, hipStream_t stream) {
  using C = DqCfg<D, BQ, BK, NQW>;
  if (sv.max_kt > C::max_kblocks()) return hipErrorInvalidValue;
  const int G = p.h_q / p.h_k;
  int hpw = 256 / BQ;  // up to 256 query rows per workgroup
  while (hpw > 1 && G % hpw != 0) hpw >>= 1;
  const int waves = hpw * C::WPH;
  if (waves == 4) return launch_dq_w<D, BQ, BK, NQW, true>(p, sv, hpw, waves, q, k, v, d_o, nl, nd, dq, stream);
  return launch_dq_w<D, BQ, BK, NQW, false>(p, sv, hpw, waves, q, k, v, d_o, nl, nd, dq, stream);
}

}  // namespace

int bwd_main_max_qblocks(int d, int tk) {
  if (d == 128) return tk == 128 ? BwdCfg<128, 128>::max_qblocks() : BwdCfg<128, 64>::max_qblocks();
  return tk == 128 ? BwdCfg<64, 128>::max_qblocks() : BwdCfg<64, 64>::max_qblocks();
}

int bwd_dq_max_kblocks(int d, int tk) {
  // the LDS of the dQ pass: two K/V blocks, then one row's block list
  if (d == 128) return tk == 128 ? DqCfg<128, 128, 128>::max_kblocks() : DqCfg<128, 128, 64>::max_kblocks();
  return tk == 128 ? DqCfg<64, 128, 128>::max_kblocks() : DqCfg<64, 128, 64>::max_kblocks();
}

bool bwd_bf16_supported(int d, int tq, int tk) {
  return (d == 64 || d == 128) && (tq == 64 || tq == 128) && (tk == 64 || tk == 128);
}

hipError_t launch_bwd_prepare(const cowa_params& p, const void* o, const void* d_o, const float* lse,
                              const BwdWork& w, hipStream_t stream) {
  const int64_t rows = q_rows(p);
  const int64_t chunks = rows * (p.head_dim / 8);
  const unsigned blocks = (unsigned)((chunks + 255) / 256);
  if (p.head_dim == 128)
    hipLaunchKernelGGL(bwd_pre<128>, dim3(blocks), dim3(256), 0, stream, static_cast<const __bf16*>(o),
                       static_cast<const __bf16*>(d_o), lse, w.nd, w.nl, rows);
  else
    hipLaunchKernelGGL(bwd_pre<64>, dim3(blocks), dim3(256), 0, stream, static_cast<const __bf16*>(o),
                       static_cast<const __bf16*>(d_o), lse, w.nd, w.nl, rows);
  return hipGetLastError();
}

hipError_t launch_bwd_main(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                           const void* d_o, void* dk, void* dv, const BwdWork& w, hipStream_t stream) {
  if (p.head_dim == 128 && p.tile_k == 128) return launch_main<128, 128>(p, sv, q, k, v, d_o, w, dk, dv, stream);
  if (p.head_dim == 128 && p.tile_k == 64) return launch_main<128, 64>(p, sv, q, k, v, d_o, w, dk, dv, stream);
  if (p.head_dim == 64 && p.tile_k == 128) return launch_main<64, 128>(p, sv, q, k, v, d_o, w, dk, dv, stream);
  if (p.head_dim == 64 && p.tile_k == 64) return launch_main<64, 64>(p, sv, q, k, v, d_o, w, dk, dv, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_bwd_dq(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                         const void* d_o, void* dq, const BwdWork& w, hipStream_t stream) {
  if (bwd_dq32_supported(p)) return launch_bwd_dq32(p, sv, q, k, v, d_o, dq, w, stream);
#define COWA_DQ_CASE(D_, BQ_, BK_) \
  if (p.head_dim == D_ && p.tile_q == BQ_ && p.tile_k == BK_) return launch_dq<D_, BQ_, BK_>(p, sv, q, k, v, d_o, w.nl, w.nd, dq, stream);
  COWA_DQ_CASE(128, 128, 128)
  COWA_DQ_CASE(128, 128, 64)
  COWA_DQ_CASE(128, 64, 128)
  COWA_DQ_CASE(128, 64, 64)
  COWA_DQ_CASE(64, 128, 128)
  COWA_DQ_CASE(64, 128, 64)
  COWA_DQ_CASE(64, 64, 128)
  COWA_DQ_CASE(64, 64, 64)
#undef COWA_DQ_CASE
  return hipErrorInvalidValue;
}

}  // namespace cowa
