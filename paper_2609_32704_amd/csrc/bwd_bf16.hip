// CoWA backward in bfloat16 on the CDNA4 matrix cores (Alg. 2).
//
// Three launches on the caller's stream:
//
//  1. bwd_pre: D = rowsum(O * dO) per query row (fp32), and the fp32 dQ
//     accumulator set to zero.
//  2. bwd_main: one workgroup of four waves per (KV block j, local KV head h_k,
//     sequence b).  K_j and V_j stay in registers for the whole workgroup (wave
//     w owns keys [w BK/4, (w+1) BK/4) of the block), K_j^T is staged once in
//     LDS.  The workgroup walks all QO heads of the group and, for each, the
//     QO blocks of I_{h_k}(j) in ascending order (in 64-row steps).  Per step:
//       S = Q K^T, dP = dO V^T                (A from LDS, B from registers)
//       P = exp(S - LSE), dS = P * (dP - D)   (partial blocks masked)
//       dV^T += dO^T P, dK^T += scale Q^T dS  (accumulated in registers)
//       dQ += scale dS K                      (dS through LDS; fp32 atomics)
//     dK and dV of the block are therefore summed over every QO head of the
//     group inside the workgroup and written once, without atomics; keys that
//     no query sees get zeros.  Only dQ, which many KV blocks touch, is
//     reduced with atomic adds.
//  3. bwd_dq: dQ = bf16(dQ accumulator).
#include "internal.h"
#include "window_rule.h"

namespace cowa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;

__device__ inline int xcd_remap(int id, int total) {
  const int full = (total / 64) * 64;
  if (id >= full) return id;
  const int xcd = id & 7, slot = id >> 3;
  const int chunk = (slot >> 3) * 8 + xcd;
  return chunk * 8 + (slot & 7);
}

// D[row] = sum_d O[row, d] dO[row, d]; dq_acc[row, :] = 0.  D/8 lanes per row.
template <int D>
__global__ void __launch_bounds__(256) bwd_pre(const __bf16* __restrict__ o, const __bf16* __restrict__ d_o,
                                               float* __restrict__ dsum, float* __restrict__ dq_acc, int64_t rows) {
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
    float4* z = reinterpret_cast<float4*>(dq_acc + row * D + ch * 8);
    z[0] = make_float4(0.f, 0.f, 0.f, 0.f);
    z[1] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
#pragma unroll
  for (int off = 1; off < CH; off <<= 1) part += __shfl_xor(part, off);
  if (row < rows && ch == 0) dsum[row] = part;
}

__global__ void __launch_bounds__(256) bwd_dq(const float* __restrict__ dq_acc, __bf16* __restrict__ dq, int64_t n8) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= n8) return;
  const float4 a = reinterpret_cast<const float4*>(dq_acc)[2 * c];
  const float4 b = reinterpret_cast<const float4*>(dq_acc)[2 * c + 1];
  bf16x8 out = {(__bf16)a.x, (__bf16)a.y, (__bf16)a.z, (__bf16)a.w,
                (__bf16)b.x, (__bf16)b.y, (__bf16)b.z, (__bf16)b.w};
  reinterpret_cast<bf16x8*>(dq)[c] = out;
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
  static constexpr int RPAD = D + 8;      // row-major [q][d] stride
  static constexpr int TPAD = BQ + 4;     // transposed [d][q] stride
  static constexpr int SPAD = BK + 8;     // dS [q][key] and K^T [d][key] stride
  static constexpr int OFF_Q = 0;
  static constexpr int OFF_DO = OFF_Q + BQ * RPAD;
  static constexpr int OFF_QT = OFF_DO + BQ * RPAD;
  static constexpr int OFF_DOT = OFF_QT + D * TPAD;
  static constexpr int OFF_DS = OFF_DOT + D * TPAD;
  static constexpr int OFF_KT = OFF_DS + BQ * SPAD;
  static constexpr int ELEMS = OFF_KT + D * SPAD;  // bf16 elements
  static constexpr int LDS_BYTES = ELEMS * 2 + 2 * BQ * 4;
};

// rows [q0, q0 + 4) x d chunk [8 ch, 8 ch + 8) -> row-major and transposed copies
template <int D, int RPAD, int TPAD>
__device__ inline void stage_rows4(const __bf16* src, int64_t row0, int64_t n_rows, int qloc, int ch, __bf16* rm,
                                   __bf16* tr) {
  uint4 rv[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    rv[u] = make_uint4(0, 0, 0, 0);
    if (row0 + qloc + u < n_rows) rv[u] = *reinterpret_cast<const uint4*>(src + (row0 + qloc + u) * D + ch * 8);
    *reinterpret_cast<uint4*>(rm + (qloc + u) * RPAD + ch * 8) = rv[u];
  }
  const uint32_t* w0 = reinterpret_cast<const uint32_t*>(&rv[0]);
  const uint32_t* w1 = reinterpret_cast<const uint32_t*>(&rv[1]);
  const uint32_t* w2 = reinterpret_cast<const uint32_t*>(&rv[2]);
  const uint32_t* w3 = reinterpret_cast<const uint32_t*>(&rv[3]);
#pragma unroll
  for (int dd = 0; dd < 8; ++dd) {
    const int wd = dd >> 1;
    uint2 pk;
    if (dd & 1) {
      pk.x = (w0[wd] >> 16) | (w1[wd] & 0xffff0000u);
      pk.y = (w2[wd] >> 16) | (w3[wd] & 0xffff0000u);
    } else {
      pk.x = (w0[wd] & 0xffffu) | (w1[wd] << 16);
      pk.y = (w2[wd] & 0xffffu) | (w3[wd] << 16);
    }
    *reinterpret_cast<uint2*>(tr + (ch * 8 + dd) * TPAD + qloc) = pk;
  }
}

template <int D, int BK>
__global__ void __launch_bounds__(256) bwd_main(cowa_params p, SchedView sv, const __bf16* __restrict__ q,
                                                const __bf16* __restrict__ k, const __bf16* __restrict__ v,
                                                const __bf16* __restrict__ d_o, const float* __restrict__ lse,
                                                const float* __restrict__ dsum, float* __restrict__ dq_acc,
                                                __bf16* __restrict__ dk, __bf16* __restrict__ dv) {
  using C = BwdCfg<D, BK>;
  extern __shared__ __align__(16) unsigned char smem[];
  __bf16* lds = reinterpret_cast<__bf16*>(smem);
  __bf16* Qs = lds + C::OFF_Q;
  __bf16* dOs = lds + C::OFF_DO;
  __bf16* Qt = lds + C::OFF_QT;
  __bf16* dOt = lds + C::OFF_DOT;
  __bf16* dSs = lds + C::OFF_DS;
  __bf16* Kt = lds + C::OFF_KT;
  float* lse2 = reinterpret_cast<float*>(lds + C::ELEMS);
  float* dsm = lse2 + C::BQ;

  const int total = sv.n_kt * p.h_k * p.batch;
  const int work = xcd_remap(blockIdx.x, total);
  const int j = work % sv.n_kt;  // KV block (sink blocks, with the longest query lists, first)
  const int hk = (work / sv.n_kt) % p.h_k;
  const int b = work / (sv.n_kt * p.h_k);
  const int G = p.h_q / p.h_k;
  const HeadGeo g = make_geo(p.n_q, p.n_k, p.w_sink, p.w_near, p.tile_q, BK, p.h_k_offset + hk, p.h_k_total);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t k_first = (int64_t)j * BK;
  const __bf16* kbase = k + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  const __bf16* vbase = v + ((int64_t)b * p.h_k + hk) * p.n_k * D;

  // K and V rows of this wave's keys as B fragments: key nt*16 + lr, d = ks*32 + 8*lg + 0..7
  bf16x8 kf[C::NTK][C::KSD], vf[C::NTK][C::KSD];
#pragma unroll
  for (int nt = 0; nt < C::NTK; ++nt) {
    const int64_t kp = k_first + wave * C::NKW + nt * 16 + lr;
#pragma unroll
    for (int ks = 0; ks < C::KSD; ++ks) {
      bf16x8 a = bf16x8{}, c2 = bf16x8{};
      if (kp < p.n_k) {
        a = *reinterpret_cast<const bf16x8*>(kbase + kp * D + ks * 32 + 8 * lg);
        c2 = *reinterpret_cast<const bf16x8*>(vbase + kp * D + ks * 32 + 8 * lg);
      }
      kf[nt][ks] = a;
      vf[nt][ks] = c2;
    }
  }
  // K^T of the whole block in LDS: Kt[d][key]
  for (int x = tid; x < (BK / 4) * (D / 8); x += 256) {
    const int kg = x / (D / 8), ch = x % (D / 8);
    uint4 rv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t kp = k_first + kg * 4 + u;
      rv[u] = make_uint4(0, 0, 0, 0);
      if (kp < p.n_k) rv[u] = *reinterpret_cast<const uint4*>(kbase + kp * D + ch * 8);
    }
    const uint32_t* w0 = reinterpret_cast<const uint32_t*>(&rv[0]);
    const uint32_t* w1 = reinterpret_cast<const uint32_t*>(&rv[1]);
    const uint32_t* w2 = reinterpret_cast<const uint32_t*>(&rv[2]);
    const uint32_t* w3 = reinterpret_cast<const uint32_t*>(&rv[3]);
#pragma unroll
    for (int dd = 0; dd < 8; ++dd) {
      const int wd = dd >> 1;
      uint2 pk;
      if (dd & 1) {
        pk.x = (w0[wd] >> 16) | (w1[wd] & 0xffff0000u);
        pk.y = (w2[wd] >> 16) | (w3[wd] & 0xffff0000u);
      } else {
        pk.x = (w0[wd] & 0xffffu) | (w1[wd] << 16);
        pk.y = (w2[wd] & 0xffffu) | (w3[wd] << 16);
      }
      *reinterpret_cast<uint2*>(Kt + (ch * 8 + dd) * C::SPAD + kg * 4) = pk;
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
  const int col = hk * sv.n_kt + j;
  const int e0 = sv.bwd_col_ptr[col], e1 = sv.bwd_col_ptr[col + 1];
  const int sub_per_tile = p.tile_q / C::BQ;

  for (int hh = 0; hh < G; ++hh) {
    const int h = hk * G + hh;
    const int64_t row_base = ((int64_t)b * p.h_q + h) * p.n_q;
    const __bf16* qh = q + row_base * D;
    const __bf16* doh = d_o + row_base * D;
    for (int e = e0; e < e1; ++e) {
      const uint32_t ent = sv.bwd_ent[e];
      const int i = (int)(ent >> 1);
      const bool partial = ent & 1u;
      for (int sub = 0; sub < sub_per_tile; ++sub) {
        const int64_t q0 = (int64_t)i * p.tile_q + sub * C::BQ;
        if (q0 >= p.n_q) break;
        __syncthreads();  // previous step's LDS reads are done
        {
          const int x = tid;  // 16 row quads x 16 d chunks (D = 128) or 16 x 8 (D = 64)
          for (int y = x; y < (C::BQ / 4) * (D / 8); y += 256) {
            const int quad = y / (D / 8), ch = y % (D / 8);
            stage_rows4<D, C::RPAD, C::TPAD>(qh, q0, p.n_q, quad * 4, ch, Qs, Qt);
            stage_rows4<D, C::RPAD, C::TPAD>(doh, q0, p.n_q, quad * 4, ch, dOs, dOt);
          }
          if (tid < C::BQ) {
            const int64_t qp = q0 + tid;
            const bool ok = qp < p.n_q;
            lse2[tid] = ok ? lse[row_base + qp] * kLog2e : INFINITY;
            dsm[tid] = ok ? dsum[row_base + qp] : 0.f;
          }
        }
        __syncthreads();

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
            const bf16x8 aq = *reinterpret_cast<const bf16x8*>(Qs + (mt * 16 + lr) * C::RPAD + ks * 32 + 8 * lg);
            const bf16x8 ag = *reinterpret_cast<const bf16x8*>(dOs + (mt * 16 + lr) * C::RPAD + ks * 32 + 8 * lg);
#pragma unroll
            for (int nt = 0; nt < C::NTK; ++nt) {
              sacc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq, kf[nt][ks], sacc[mt][nt], 0, 0, 0);
              pacc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ag, vf[nt][ks], pacc[mt][nt], 0, 0, 0);
            }
          }

        // P = exp(S - LSE), dS = P (dP - D); sacc <- P, pacc <- scale * dS
#pragma unroll
        for (int mt = 0; mt < C::MTQ; ++mt)
#pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const int ql = mt * 16 + 4 * lg + rr;
            const float l2 = lse2[ql], dd = dsm[ql];
#pragma unroll
            for (int nt = 0; nt < C::NTK; ++nt) {
              const int64_t kp = k_first + wave * C::NKW + nt * 16 + lr;
              float pv = __builtin_amdgcn_exp2f(sacc[mt][nt][rr] * c - l2);
              if (partial && !legal_pair(g, q0 + ql, kp)) pv = 0.f;
              sacc[mt][nt][rr] = pv;
              pacc[mt][nt][rr] = scale * pv * (pacc[mt][nt][rr] - dd);
            }
          }

        // dV^T += dO^T P and dK^T += Q^T dS over this step's queries
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
            const __bf16* gr = dOt + (md * 16 + lr) * C::TPAD + ks * 32 + 4 * lg;
            const __bf16* qr = Qt + (md * 16 + lr) * C::TPAD + ks * 32 + 4 * lg;
            const bf16x4 g0 = *reinterpret_cast<const bf16x4*>(gr), g1 = *reinterpret_cast<const bf16x4*>(gr + 16);
            const bf16x4 q0v = *reinterpret_cast<const bf16x4*>(qr), q1v = *reinterpret_cast<const bf16x4*>(qr + 16);
            const bf16x8 ag = {g0[0], g0[1], g0[2], g0[3], g1[0], g1[1], g1[2], g1[3]};
            const bf16x8 aq = {q0v[0], q0v[1], q0v[2], q0v[3], q1v[0], q1v[1], q1v[2], q1v[3]};
#pragma unroll
            for (int nt = 0; nt < C::NTK; ++nt) {
              dva[md][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ag, pb[nt], dva[md][nt], 0, 0, 0);
              dka[md][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aq, sb[nt], dka[md][nt], 0, 0, 0);
            }
          }
        }

        // dS -> LDS [q][key] (bf16) for the dQ product
#pragma unroll
        for (int mt = 0; mt < C::MTQ; ++mt)
#pragma unroll
          for (int nt = 0; nt < C::NTK; ++nt)
#pragma unroll
            for (int rr = 0; rr < 4; ++rr)
              dSs[(mt * 16 + 4 * lg + rr) * C::SPAD + wave * C::NKW + nt * 16 + lr] = (__bf16)pacc[mt][nt][rr];
        __syncthreads();

        // dQ rows [16 wave, 16 wave + 16) += dS K over all BK keys: column d = md*16 + lr, row 4*lg + r
        f32x4 qacc[C::MD];
#pragma unroll
        for (int md = 0; md < C::MD; ++md) qacc[md] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < C::KSK; ++ks) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(dSs + (wave * 16 + lr) * C::SPAD + ks * 32 + 8 * lg);
#pragma unroll
          for (int md = 0; md < C::MD; ++md) {
            const bf16x8 bk = *reinterpret_cast<const bf16x8*>(Kt + (md * 16 + lr) * C::SPAD + ks * 32 + 8 * lg);
            qacc[md] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bk, qacc[md], 0, 0, 0);
          }
        }
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const int64_t qp = q0 + wave * 16 + 4 * lg + rr;
          if (qp < p.n_q) {
            float* dst = dq_acc + (row_base + qp) * D + lr;
#pragma unroll
            for (int md = 0; md < C::MD; ++md) unsafeAtomicAdd(dst + md * 16, qacc[md][rr]);
          }
        }
      }
    }
  }

  // write dK and dV of the block: through LDS as [key][d], then 16-byte rows
  __syncthreads();
  __bf16* tk = lds;                   // [BK][RPAD]
  __bf16* tv = lds + BK * C::RPAD;    // [BK][RPAD]
#pragma unroll
  for (int md = 0; md < C::MD; ++md)
#pragma unroll
    for (int nt = 0; nt < C::NTK; ++nt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int key = wave * C::NKW + nt * 16 + lr, d = md * 16 + 4 * lg + rr;
        tk[key * C::RPAD + d] = (__bf16)dka[md][nt][rr];
        tv[key * C::RPAD + d] = (__bf16)dva[md][nt][rr];
      }
  __syncthreads();
  __bf16* dkb = dk + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  __bf16* dvb = dv + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  for (int x = tid; x < BK * (D / 8); x += 256) {
    const int key = x / (D / 8), ch = x % (D / 8);
    const int64_t kp = k_first + key;
    if (kp < p.n_k) {
      *reinterpret_cast<uint4*>(dkb + kp * D + ch * 8) = *reinterpret_cast<const uint4*>(tk + key * C::RPAD + ch * 8);
      *reinterpret_cast<uint4*>(dvb + kp * D + ch * 8) = *reinterpret_cast<const uint4*>(tv + key * C::RPAD + ch * 8);
    }
  }
}

template <int D, int BK>
hipError_t launch_main(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                       const void* d_o, const float* lse, const float* dsum, float* dq_acc, void* dk, void* dv,
                       hipStream_t stream) {
  using C = BwdCfg<D, BK>;
  static_assert(C::LDS_BYTES <= 160 * 1024, "LDS budget");
  static_assert(2 * BK * C::RPAD <= C::ELEMS, "dK/dV staging must fit in the step buffers");
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
                     lse, dsum, dq_acc, static_cast<__bf16*>(dk), static_cast<__bf16*>(dv));
  return hipGetLastError();
}

}  // namespace

bool bwd_bf16_supported(int d, int tq, int tk) {
  return (d == 64 || d == 128) && (tq == 64 || tq == 128) && (tk == 64 || tk == 128);
}

hipError_t launch_bwd_prepare(const cowa_params& p, const void* o, const void* d_o, float* dq_acc, float* dsum,
                              hipStream_t stream) {
  const int64_t rows = (int64_t)p.batch * p.h_q * p.n_q;
  const int64_t chunks = rows * (p.head_dim / 8);
  const unsigned blocks = (unsigned)((chunks + 255) / 256);
  if (p.head_dim == 128)
    hipLaunchKernelGGL(bwd_pre<128>, dim3(blocks), dim3(256), 0, stream, static_cast<const __bf16*>(o),
                       static_cast<const __bf16*>(d_o), dsum, dq_acc, rows);
  else
    hipLaunchKernelGGL(bwd_pre<64>, dim3(blocks), dim3(256), 0, stream, static_cast<const __bf16*>(o),
                       static_cast<const __bf16*>(d_o), dsum, dq_acc, rows);
  return hipGetLastError();
}

hipError_t launch_bwd_main(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                           const float* lse, const void* d_o, void* dk, void* dv, float* dq_acc, const float* dsum,
                           hipStream_t stream) {
  if (p.head_dim == 128 && p.tile_k == 128) return launch_main<128, 128>(p, sv, q, k, v, d_o, lse, dsum, dq_acc, dk, dv, stream);
  if (p.head_dim == 128 && p.tile_k == 64) return launch_main<128, 64>(p, sv, q, k, v, d_o, lse, dsum, dq_acc, dk, dv, stream);
  if (p.head_dim == 64 && p.tile_k == 128) return launch_main<64, 128>(p, sv, q, k, v, d_o, lse, dsum, dq_acc, dk, dv, stream);
  if (p.head_dim == 64 && p.tile_k == 64) return launch_main<64, 64>(p, sv, q, k, v, d_o, lse, dsum, dq_acc, dk, dv, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_bwd_finish(const cowa_params& p, const float* dq_acc, void* dq, hipStream_t stream) {
  const int64_t n8 = (int64_t)p.batch * p.h_q * p.n_q * p.head_dim / 8;
  hipLaunchKernelGGL(bwd_dq, dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, stream, dq_acc,
                     static_cast<__bf16*>(dq), n8);
  return hipGetLastError();
}

}  // namespace cowa
