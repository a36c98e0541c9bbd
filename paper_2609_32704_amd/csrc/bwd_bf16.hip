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

namespace cowa {
namespace {

// D[row] = sum_d O[row, d] dO[row, d], D/8 lanes per row.
template <int D>
__global__ void __launch_bounds__(256) bwd_pre(const __bf16* __restrict__ o, const __bf16* __restrict__ d_o,
                                               float* __restrict__ dsum, int64_t rows) {
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
  if (row < rows && ch == 0) dsum[row] = part;
}

template <int D, int BK>
struct BwdCfg {
  static constexpr int BQ = 64;           // query rows per step
  static constexpr int NKW = BK / 4;      // keys per wave
  static constexpr int NTK = NKW / 16;    // key tiles per wave
  static constexpr int MTQ = BQ / 16;     // query tiles per step
  static constexpr int KSD = D / 32;      // k-steps over d
  static constexpr int MD = D / 16;       // d tiles
  static constexpr int KSQ = BQ / 32;     // k-steps over queries
  static constexpr int KSK = BK / 32;     // k-steps over keys
  using QT = SwzTile<D, BQ>;              // Q or dO rows of one step
  static constexpr int ROWV = 2 * BQ * 4; // per-step row values: LSE [BQ], then D [BQ]
  static constexpr int STAGE = 2 * QT::BYTES + ROWV;     // Q, dO and row values of one step
  static constexpr int OUT_BYTES = 2 * BK * (D + 8) * 2;  // dK, dV staging at the end
  static constexpr int LDS_BYTES = 2 * STAGE > OUT_BYTES ? 2 * STAGE : OUT_BYTES;
};

template <int D, int BK>
__global__ void __launch_bounds__(256) bwd_main(cowa_params p, SchedView sv, const __bf16* __restrict__ q,
                                                const __bf16* __restrict__ k, const __bf16* __restrict__ v,
                                                const __bf16* __restrict__ d_o, const float* __restrict__ lse,
                                                const float* __restrict__ dsum, __bf16* __restrict__ dk,
                                                __bf16* __restrict__ dv) {
  using C = BwdCfg<D, BK>;
  extern __shared__ __align__(1024) unsigned char smem[];

  const int total = sv.n_kt * p.h_k * p.batch;
  const int work = xcd_remap(blockIdx.x, total);
  const int j = work % sv.n_kt;  // KV block (sink blocks, with the longest query lists, first)
  const int hk = (work / sv.n_kt) % p.h_k;
  const int b = work / (sv.n_kt * p.h_k);
  const int G = p.h_q / p.h_k;
  const Geo32 g = geo32(make_geo(p.n_q, p.n_k, p.w_sink, p.w_near, p.tile_q, BK, p.h_k_offset + hk, p.h_k_total));

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int nw = blockDim.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t k_first = (int64_t)j * BK;
  const __bf16* kbase = k + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  const __bf16* vbase = v + ((int64_t)b * p.h_k + hk) * p.n_k * D;

  // the step list: every QO head of the group x every QO block of I(j) x 64-row sub-steps
  const int col = hk * sv.n_kt + j;
  const int e0 = sv.bwd_col_ptr[col], e1 = sv.bwd_col_ptr[col + 1];
  const int subs = p.tile_q / C::BQ;
  const int per_head = (e1 - e0) * subs;
  const int n_steps = G * per_head;
  auto step_rows = [&](int t, int& h, int64_t& q0, bool& partial) {
    const int hh = t / per_head, rem = t % per_head;
    const uint32_t ent = sv.bwd_ent[e0 + rem / subs];
    h = hk * G + hh;
    q0 = (int64_t)(ent >> 1) * p.tile_q + (rem % subs) * C::BQ;
    partial = ent & 1u;
  };
  // Q and dO rows of step t go global -> LDS directly; the step's LSE and D
  // values go through registers of the last wave (rows past n_q: LSE = -inf, D = 0)
  auto stage_step = [&](int t, unsigned char* st, float& lv, float& dv2) {
    int h;
    int64_t q0;
    bool partial;
    step_rows(t, h, q0, partial);
    const int64_t row_base = ((int64_t)b * p.h_q + h) * p.n_q;
    load_tile<D, C::BQ>(q + row_base * D, q0, p.n_q, st, wave, nw, lane);
    load_tile<D, C::BQ>(d_o + row_base * D, q0, p.n_q, st + C::QT::BYTES, wave, nw, lane);
    if (wave == nw - 1) {
      const int64_t r = q0 + lane;
      lv = r < p.n_q ? lse[row_base + r] : -INFINITY;
      dv2 = r < p.n_q ? dsum[row_base + r] : 0.f;
    }
  };
  auto store_rowv = [&](unsigned char* st, float lv, float dv2) {
    if (wave == nw - 1) {
      float* rv = reinterpret_cast<float*>(st + 2 * C::QT::BYTES);
      rv[lane] = lv;
      rv[C::BQ + lane] = dv2;
    }
  };

  float nlv = 0.f, ndv = 0.f;  // row values of the step being staged
  if (n_steps > 0) {
    stage_step(0, smem, nlv, ndv);
    store_rowv(smem, nlv, ndv);
  }

  // K and V rows of this wave's keys as B fragments: key nt*16 + lr, d = ks*32 + 8*lg + 0..7
  bf16x8 kf[C::NTK][C::KSD], vf[C::NTK][C::KSD];
#pragma unroll
  for (int nt = 0; nt < C::NTK; ++nt) {
    int64_t kp = k_first + wave * C::NKW + nt * 16 + lr;
    if (kp >= p.n_k) kp = p.n_k - 1;  // masked below: such keys are in partial blocks only
#pragma unroll
    for (int ks = 0; ks < C::KSD; ++ks) {
      kf[nt][ks] = *reinterpret_cast<const bf16x8*>(kbase + kp * D + ks * 32 + 8 * lg);
      vf[nt][ks] = *reinterpret_cast<const bf16x8*>(vbase + kp * D + ks * 32 + 8 * lg);
    }
  }
  f32x4 dka[C::MD][C::NTK], dva[C::MD][C::NTK];  // dK^T, dV^T: rows d, columns keys
#pragma unroll
  for (int md = 0; md < C::MD; ++md)
#pragma unroll
    for (int nt = 0; nt < C::NTK; ++nt) {
      dka[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      dva[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  const float c = p.softmax_scale * kLog2e;
  const float scale = p.softmax_scale;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int t = 0; t < n_steps; ++t) {
    unsigned char* st = smem + (t & 1) * C::STAGE;
    unsigned char* nst = smem + ((t + 1) & 1) * C::STAGE;
    if (t + 1 < n_steps) stage_step(t + 1, nst, nlv, ndv);
    int h;
    int64_t q0;
    bool partial;
    step_rows(t, h, q0, partial);
    const unsigned char* qs = st;
    const unsigned char* dos = st + C::QT::BYTES;
    const float* rowv = reinterpret_cast<const float*>(st + 2 * C::QT::BYTES);

    // S = Q K^T and dP = dO V^T: rows q = mt*16 + 4*lg + r, column key = nt*16 + lr
    f32x4 sacc[C::MTQ][C::NTK], pacc[C::MTQ][C::NTK];
#pragma unroll
    for (int mt = 0; mt < C::MTQ; ++mt)
#pragma unroll
      for (int nt = 0; nt < C::NTK; ++nt) {
        sacc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        pacc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
    for (int ks = 0; ks < C::KSD; ++ks)
#pragma unroll
      for (int mt = 0; mt < C::MTQ; ++mt) {
        const bf16x8 aq = read_row8<D, C::BQ>(qs, mt * 16 + lr, ks * 4 + lg);
        const bf16x8 ag = read_row8<D, C::BQ>(dos, mt * 16 + lr, ks * 4 + lg);
#pragma unroll
        for (int nt = 0; nt < C::NTK; ++nt) {
          sacc[mt][nt] = mfma16(aq, kf[nt][ks], sacc[mt][nt]);
          pacc[mt][nt] = mfma16(ag, vf[nt][ks], pacc[mt][nt]);
        }
      }

    // P = exp(S - LSE) and scale * dS = scale * P (dP - D); masked pairs get P = 0
    // through an additive -inf in the exponent (the value read keeps the MFMA
    // result ordering).  A row whose LSE is -inf has no legal key: P = 0.
    const int64_t qrow = q0 + 4 * lg;  // + mt*16 + r
    const int k0 = (int)k_first + wave * C::NKW + lr;
#pragma unroll
    for (int mt = 0; mt < C::MTQ; ++mt) {
      const float4 lv = *reinterpret_cast<const float4*>(rowv + mt * 16 + 4 * lg);
      const float4 dv4 = *reinterpret_cast<const float4*>(rowv + C::BQ + mt * 16 + 4 * lg);
      const float lsev[4] = {lv.x, lv.y, lv.z, lv.w}, dd[4] = {dv4.x, dv4.y, dv4.z, dv4.w};
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const float l2 = lsev[rr] == -INFINITY ? INFINITY : lsev[rr] * kLog2e;
        const int qi = (int)qrow + mt * 16 + rr;
#pragma unroll
        for (int nt = 0; nt < C::NTK; ++nt) {
          const float bias = (!partial || legal32(g, qi, k0 + nt * 16)) ? 0.f : -INFINITY;
          const float pv = __builtin_amdgcn_exp2f(fmaf(sacc[mt][nt][rr], c, -l2) + bias);
          sacc[mt][nt][rr] = pv;
          pacc[mt][nt][rr] = scale * pv * (pacc[mt][nt][rr] - dd[rr]);
        }
      }
    }

    // dV^T += dO^T P and dK^T += Q^T (scale dS): k-slots are queries 32ks + 4lg + t, 32ks + 16 + 4lg + t
#pragma unroll
    for (int ks = 0; ks < C::KSQ; ++ks) {
      bf16x8 pb[C::NTK], sb[C::NTK];
#pragma unroll
      for (int nt = 0; nt < C::NTK; ++nt)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          pb[nt][rr] = (__bf16)sacc[2 * ks][nt][rr];
          pb[nt][4 + rr] = (__bf16)sacc[2 * ks + 1][nt][rr];
          sb[nt][rr] = (__bf16)pacc[2 * ks][nt][rr];
          sb[nt][4 + rr] = (__bf16)pacc[2 * ks + 1][nt][rr];
        }
#pragma unroll
      for (int md = 0; md < C::MD; ++md) {
        const bf16x8 ag = read_tr8<D, C::BQ>(dos, ks * 32, md * 16, lr, lg);
        const bf16x8 aq = read_tr8<D, C::BQ>(qs, ks * 32, md * 16, lr, lg);
#pragma unroll
        for (int nt = 0; nt < C::NTK; ++nt) {
          dva[md][nt] = mfma16(ag, pb[nt], dva[md][nt]);
          dka[md][nt] = mfma16(aq, sb[nt], dka[md][nt]);
        }
      }
    }

    if (t + 1 < n_steps) store_rowv(nst, nlv, ndv);
    __builtin_amdgcn_s_waitcnt(0);  // the next step's tiles have landed
    __syncthreads();                 // ... for every wave; this step's LDS is no longer read
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
        tk[key * (D + 8) + d] = (__bf16)dka[md][nt][rr];
        tv[key * (D + 8) + d] = (__bf16)dva[md][nt][rr];
      }
  __syncthreads();
  __bf16* dkb = dk + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  __bf16* dvb = dv + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  for (int x = tid; x < BK * (D / 8); x += blockDim.x) {
    const int key = x / (D / 8), ch = x % (D / 8);
    const int64_t kp = k_first + key;
    if (kp < p.n_k) {
      *reinterpret_cast<uint4*>(dkb + kp * D + ch * 8) = *reinterpret_cast<const uint4*>(tk + key * (D + 8) + ch * 8);
      *reinterpret_cast<uint4*>(dvb + kp * D + ch * 8) = *reinterpret_cast<const uint4*>(tv + key * (D + 8) + ch * 8);
    }
  }
}

template <int D, int BK>
hipError_t launch_main(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                       const void* d_o, const float* lse, const float* dsum, void* dk, void* dv,
                       hipStream_t stream) {
  using C = BwdCfg<D, BK>;
  static_assert(C::LDS_BYTES <= 160 * 1024, "LDS budget");
  auto kern = bwd_main<D, BK>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const unsigned blocks = (unsigned)sv.n_kt * p.h_k * p.batch;
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), C::LDS_BYTES, stream, p, sv, static_cast<const __bf16*>(q),
                     static_cast<const __bf16*>(k), static_cast<const __bf16*>(v), static_cast<const __bf16*>(d_o),
                     lse, dsum, static_cast<__bf16*>(dk), static_cast<__bf16*>(dv));
  return hipGetLastError();
}

// dQ pass: one workgroup per (QO block i, HPW QO heads of one KV group,
// sequence b); each 64-lane wave owns 32 query rows of one head.
template <int D, int BQ, int BK>
__global__ void __launch_bounds__(512) bwd_dq_kernel(cowa_params p, SchedView sv, int hpw, int n_hgroups,
                                                     const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                                                     const __bf16* __restrict__ v, const __bf16* __restrict__ d_o,
                                                     const float* __restrict__ lse, const float* __restrict__ dsum,
                                                     __bf16* __restrict__ dq) {
  using T = SwzTile<D, BK>;
  constexpr int NQW = 32;                 // query rows per wave
  constexpr int NTQ = NQW / 16;           // query tiles per wave
  constexpr int BKC = D > 64 ? 32 : 64;   // keys per step (register budget of two waves per SIMD)
  constexpr int MTK = BKC / 16;           // key tiles of S^T
  constexpr int KSD = D / 32;             // k-steps over d
  constexpr int MTD = D / 16;             // d tiles of dQ^T
  constexpr int KSK = BKC / 32;           // k-steps over keys
  constexpr int WAVES_PER_HEAD = BQ / NQW;
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
  const int h0 = hgi * hpw;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int h = h0 + wave / WAVES_PER_HEAD;
  const int64_t q_first = (int64_t)i * BQ + (wave % WAVES_PER_HEAD) * NQW;
  const Geo32 g = geo32(make_geo(p.n_q, p.n_k, p.w_sink, p.w_near, BQ, BK, p.h_k_offset + hk, p.h_k_total));

  const __bf16* kbase = k + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  const __bf16* vbase = v + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  const int r = hk * sv.n_qt + i;
  const int e0 = sv.fwd_row_ptr[r], e1 = sv.fwd_row_ptr[r + 1];
  if (e0 < e1) {
    const int64_t kf = (int64_t)(sv.fwd_ent[e0] >> 1) * BK;
    load_tile<D, BK>(kbase, kf, p.n_k, smem, wave, nw, lane);
    load_tile<D, BK>(vbase, kf, p.n_k, smem + T::BYTES, wave, nw, lane);
  }

  // Q^T and dO^T fragments (B operands): query column nt*16 + lr, d = ks*32 + 8*lg + 0..7;
  // per-query LSE (base 2; an empty row gets +inf so that P = 0) and D
  const int64_t row_base = ((int64_t)b * p.h_q + h) * p.n_q;
  bf16x8 qf[NTQ][KSD], gf[NTQ][KSD];
  float l2[NTQ], dd[NTQ];
#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) {
    const int64_t qp = q_first + nt * 16 + lr;
    const bool ok = qp < p.n_q;
    const int64_t row = row_base + (ok ? qp : 0);
#pragma unroll
    for (int ks = 0; ks < KSD; ++ks) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(q + row * D + ks * 32 + 8 * lg);
      const bf16x8 c2 = *reinterpret_cast<const bf16x8*>(d_o + row * D + ks * 32 + 8 * lg);
      qf[nt][ks] = ok ? a : bf16x8{};
      gf[nt][ks] = ok ? c2 : bf16x8{};
    }
    const float lv = ok ? lse[row] : -INFINITY;
    l2[nt] = lv == -INFINITY ? INFINITY : lv * kLog2e;
    dd[nt] = ok ? dsum[row] : 0.f;
  }

  f32x4 qacc[MTD][NTQ];  // dQ^T: rows d, columns queries
#pragma unroll
  for (int md = 0; md < MTD; ++md)
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt) qacc[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const float c = p.softmax_scale * kLog2e;
  const float scale = p.softmax_scale;

  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int e = e0; e < e1; ++e) {
    const int buf = (e - e0) & 1;
    const uint32_t ent = sv.fwd_ent[e];
    const bool partial = ent & 1u;
    const int64_t k_first = (int64_t)(ent >> 1) * BK;
    if (e + 1 < e1) {
      const int64_t kf = (int64_t)(sv.fwd_ent[e + 1] >> 1) * BK;
      unsigned char* nb = smem + (buf ^ 1) * 2 * T::BYTES;
      load_tile<D, BK>(kbase, kf, p.n_k, nb, wave, nw, lane);
      load_tile<D, BK>(vbase, kf, p.n_k, nb + T::BYTES, wave, nw, lane);
    }
    const unsigned char* Kt = smem + buf * 2 * T::BYTES;
    const unsigned char* Vt = Kt + T::BYTES;

#pragma unroll 1
    for (int kc = 0; kc < BK; kc += BKC) {
      // S^T = K Q^T and dP^T = V dO^T: rows keys kc + mt*16 + 4*lg + rr, column query nt*16 + lr
      f32x4 sacc[MTK][NTQ], pacc[MTK][NTQ];
#pragma unroll
      for (int mt = 0; mt < MTK; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTQ; ++nt) {
          sacc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
          pacc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
      for (int ks = 0; ks < KSD; ++ks)
#pragma unroll
        for (int mt = 0; mt < MTK; ++mt) {
          const bf16x8 ak = read_row8<D, BK>(Kt, kc + mt * 16 + lr, ks * 4 + lg);
          const bf16x8 av = read_row8<D, BK>(Vt, kc + mt * 16 + lr, ks * 4 + lg);
#pragma unroll
          for (int nt = 0; nt < NTQ; ++nt) {
            sacc[mt][nt] = mfma16(ak, qf[nt][ks], sacc[mt][nt]);
            pacc[mt][nt] = mfma16(av, gf[nt][ks], pacc[mt][nt]);
          }
        }

      // P^T = exp(S^T - LSE), scale dS^T = scale P^T (dP^T - D); masked pairs: an
      // additive -inf in the exponent (an update that reads the MFMA result)
      const int k0 = (int)k_first + kc + 4 * lg;
#pragma unroll
      for (int nt = 0; nt < NTQ; ++nt) {
        const int qp = (int)q_first + nt * 16 + lr;
#pragma unroll
        for (int mt = 0; mt < MTK; ++mt)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const float bias = (!partial || legal32(g, qp, k0 + mt * 16 + rr)) ? 0.f : -INFINITY;
            const float pv = __builtin_amdgcn_exp2f(fmaf(sacc[mt][nt][rr], c, -l2[nt]) + bias);
            sacc[mt][nt][rr] = scale * pv * (pacc[mt][nt][rr] - dd[nt]);
          }
      }

      // dQ^T += K^T (scale dS^T): k-slots are keys kc + 32ks + 4lg + t and kc + 32ks + 16 + 4lg + t
#pragma unroll
      for (int ks = 0; ks < KSK; ++ks) {
        bf16x8 sb[NTQ];
#pragma unroll
        for (int nt = 0; nt < NTQ; ++nt)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            sb[nt][rr] = (__bf16)sacc[2 * ks][nt][rr];
            sb[nt][4 + rr] = (__bf16)sacc[2 * ks + 1][nt][rr];
          }
#pragma unroll
        for (int md = 0; md < MTD; ++md) {
          const bf16x8 a = read_tr8<D, BK>(Kt, kc + ks * 32, md * 16, lr, lg);
#pragma unroll
          for (int nt = 0; nt < NTQ; ++nt) qacc[md][nt] = mfma16(a, sb[nt], qacc[md][nt]);
        }
      }
    }

    __builtin_amdgcn_s_waitcnt(0);  // the prefetch of block e+1 has landed
    __syncthreads();                 // ... for every wave, and block e is no longer read
  }

#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) {
    const int64_t qp = q_first + nt * 16 + lr;
    if (qp >= p.n_q) continue;
    __bf16* drow = dq + (row_base + qp) * D;
#pragma unroll
    for (int md = 0; md < MTD; ++md) {
      bf16x4 w4;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) w4[rr] = (__bf16)qacc[md][nt][rr];
      *reinterpret_cast<bf16x4*>(drow + md * 16 + 4 * lg) = w4;
    }
  }
}

template <int D, int BQ, int BK>
hipError_t launch_dq(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                     const void* d_o, const float* lse, const float* dsum, void* dq, hipStream_t stream) {
  constexpr int LDS = 4 * SwzTile<D, BK>::BYTES;
  static_assert(LDS <= 160 * 1024, "LDS budget");
  auto kern = bwd_dq_kernel<D, BQ, BK>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const int G = p.h_q / p.h_k;
  int hpw = 256 / BQ;  // up to 256 query rows per workgroup
  while (hpw > 1 && G % hpw != 0) hpw >>= 1;
  const int n_hgroups = p.h_q / hpw;
  const int waves = hpw * (BQ / 32);
  const unsigned blocks = (unsigned)sv.n_qt * n_hgroups * p.batch;
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(64 * waves), LDS, stream, p, sv, hpw, n_hgroups,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), static_cast<const __bf16*>(v),
                     static_cast<const __bf16*>(d_o), lse, dsum, static_cast<__bf16*>(dq));
  return hipGetLastError();
}

}  // namespace

bool bwd_bf16_supported(int d, int tq, int tk) {
  return (d == 64 || d == 128) && (tq == 64 || tq == 128) && (tk == 64 || tk == 128);
}

hipError_t launch_bwd_prepare(const cowa_params& p, const void* o, const void* d_o, float* dsum,
                              hipStream_t stream) {
  const int64_t rows = (int64_t)p.batch * p.h_q * p.n_q;
  const int64_t chunks = rows * (p.head_dim / 8);
  const unsigned blocks = (unsigned)((chunks + 255) / 256);
  if (p.head_dim == 128)
    hipLaunchKernelGGL(bwd_pre<128>, dim3(blocks), dim3(256), 0, stream, static_cast<const __bf16*>(o),
                       static_cast<const __bf16*>(d_o), dsum, rows);
  else
    hipLaunchKernelGGL(bwd_pre<64>, dim3(blocks), dim3(256), 0, stream, static_cast<const __bf16*>(o),
                       static_cast<const __bf16*>(d_o), dsum, rows);
  return hipGetLastError();
}

hipError_t launch_bwd_main(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                           const float* lse, const void* d_o, void* dk, void* dv, const float* dsum,
                           hipStream_t stream) {
  if (p.head_dim == 128 && p.tile_k == 128) return launch_main<128, 128>(p, sv, q, k, v, d_o, lse, dsum, dk, dv, stream);
  if (p.head_dim == 128 && p.tile_k == 64) return launch_main<128, 64>(p, sv, q, k, v, d_o, lse, dsum, dk, dv, stream);
  if (p.head_dim == 64 && p.tile_k == 128) return launch_main<64, 128>(p, sv, q, k, v, d_o, lse, dsum, dk, dv, stream);
  if (p.head_dim == 64 && p.tile_k == 64) return launch_main<64, 64>(p, sv, q, k, v, d_o, lse, dsum, dk, dv, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_bwd_dq(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                         const float* lse, const void* d_o, void* dq, const float* dsum, hipStream_t stream) {
#define COWA_DQ_CASE(D_, BQ_, BK_) \
  if (p.head_dim == D_ && p.tile_q == BQ_ && p.tile_k == BK_) return launch_dq<D_, BQ_, BK_>(p, sv, q, k, v, d_o, lse, dsum, dq, stream);
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
