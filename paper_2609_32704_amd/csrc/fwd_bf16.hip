// CoWA forward in bfloat16 on the CDNA4 matrix cores (Alg. 1).
//
// One workgroup of four 64-lane waves per (QO block i, QO head h, sequence b);
// wave w owns queries [w * BQ/4, (w+1) * BQ/4) of the block.  For every KV
// block j of J_{h_k}(i), visited in the schedule's descending order:
//
//   * K_j is staged in LDS row-major ([key][d], 16-byte padded rows) and V_j
//     transposed ([d][key]), both with coalesced 16-byte global loads;
//   * S^T = K_j Q^T on v_mfma_f32_16x16x32_bf16 (fp32 accumulate), with Q^T
//     held in registers for the whole block;
//   * only blocks flagged partial evaluate the element mask of Eq. fwa_support;
//   * online softmax per query column in registers (running max m, running
//     sum l, rescale of the O accumulator), base-2 with scale * log2(e) folded
//     into the scores;
//   * O^T += V_j^T P^T on the matrix cores, P rounded to bf16.  S^T is
//     computed transposed so that its accumulator layout (query = lane % 16)
//     is already the B-operand layout of the second product.
//
// Finally O = O / l and LSE = (m + log2 l) ln 2 (natural log).
#include "internal.h"
#include "window_rule.h"

namespace cowa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Workgroups id, id + 8, id + 16, ... land on the same XCD (round-robin
// dispatch over the 8 XCDs).  Hand each XCD whole chunks of 8 consecutive work
// items so that items sharing K/V blocks share that XCD's L2.
__device__ inline int xcd_remap(int id, int total) {
  const int full = (total / 64) * 64;
  if (id >= full) return id;
  const int xcd = id & 7, slot = id >> 3;
  const int chunk = (slot >> 3) * 8 + xcd;
  return chunk * 8 + (slot & 7);
}

template <int D, int BQ, int BK>
struct FwdCfg {
  static constexpr int NW = 4;
  static constexpr int NQW = BQ / NW;   // queries per wave
  static constexpr int NTQ = NQW / 16;  // 16-wide query tiles per wave
  static constexpr int MTK = BK / 16;   // key tiles of S^T
  static constexpr int KSD = D / 32;    // k-steps over d
  static constexpr int MTD = D / 16;    // d tiles of O^T
  static constexpr int KSK = BK / 32;   // k-steps over keys
  static constexpr int KPAD = D + 8;    // Ks row stride (elements)
  static constexpr int VPAD = BK + 4;   // Vt row stride (elements)
  static constexpr int LDS_BYTES = (BK * KPAD + D * VPAD) * 2;
};

template <int D, int BQ, int BK>
__global__ void __launch_bounds__(256) fwd_bf16_kernel(cowa_params p, SchedView sv, const __bf16* __restrict__ q,
                                                       const __bf16* __restrict__ k, const __bf16* __restrict__ v,
                                                       __bf16* __restrict__ o, float* __restrict__ lse) {
  using C = FwdCfg<D, BQ, BK>;
  extern __shared__ __align__(16) unsigned char smem[];
  __bf16* Ks = reinterpret_cast<__bf16*>(smem);
  __bf16* Vt = Ks + BK * C::KPAD;

  const int total = sv.n_qt * p.h_q * p.batch;
  const int work = xcd_remap(blockIdx.x, total);
  const int hb = p.h_q * p.batch;
  const int i = sv.n_qt - 1 - work / hb;  // latest (longest) QO blocks first
  const int h = (work % hb) % p.h_q, b = (work % hb) / p.h_q;
  const int hk = (int)(((int64_t)h * p.h_k) / p.h_q);
  const HeadGeo g = make_geo(p.n_q, p.n_k, p.w_sink, p.w_near, BQ, BK, p.h_k_offset + hk, p.h_k_total);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int64_t q_first = (int64_t)i * BQ + wave * C::NQW;

  const __bf16* kbase = k + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  const __bf16* vbase = v + ((int64_t)b * p.h_k + hk) * p.n_k * D;

  // Q^T fragments (B operand): query column nt*16 + lr, d = ks*32 + 8*lg + 0..7.
  bf16x8 qf[C::NTQ][C::KSD];
#pragma unroll
  for (int nt = 0; nt < C::NTQ; ++nt) {
    const int64_t qp = q_first + nt * 16 + lr;
    const __bf16* qrow = q + (((int64_t)b * p.h_q + h) * p.n_q + (qp < p.n_q ? qp : 0)) * D;
#pragma unroll
    for (int ks = 0; ks < C::KSD; ++ks) {
      bf16x8 val = *reinterpret_cast<const bf16x8*>(qrow + ks * 32 + 8 * lg);
      if (qp >= p.n_q) val = bf16x8{};
      qf[nt][ks] = val;
    }
  }

  f32x4 oacc[C::MTD][C::NTQ];
#pragma unroll
  for (int md = 0; md < C::MTD; ++md)
#pragma unroll
    for (int nt = 0; nt < C::NTQ; ++nt) oacc[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[C::NTQ], l_run[C::NTQ];
#pragma unroll
  for (int nt = 0; nt < C::NTQ; ++nt) { m_run[nt] = -INFINITY; l_run[nt] = 0.f; }

  const float c = p.softmax_scale * kLog2e;
  const int r = hk * sv.n_qt + i;
  const int e0 = sv.fwd_row_ptr[r], e1 = sv.fwd_row_ptr[r + 1];

  for (int e = e0; e < e1; ++e) {
    const uint32_t ent = sv.fwd_ent[e];
    const int j = (int)(ent >> 1);
    const bool partial = ent & 1u;
    const int64_t k_first = (int64_t)j * BK;

    __syncthreads();  // previous block's LDS reads are done
    // K_j -> Ks[key][d]
    for (int x = tid; x < BK * (D / 8); x += 256) {
      const int key = x / (D / 8), ch = x % (D / 8);
      const int64_t kp = k_first + key;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (kp < p.n_k) val = *reinterpret_cast<const uint4*>(kbase + kp * D + ch * 8);
      *reinterpret_cast<uint4*>(Ks + key * C::KPAD + ch * 8) = val;
    }
    // V_j -> Vt[d][key], four keys x eight d per unit
    for (int x = tid; x < (BK / 4) * (D / 8); x += 256) {
      const int kg = x / (D / 8), ch = x % (D / 8);
      uint4 rv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t kp = k_first + kg * 4 + u;
        rv[u] = make_uint4(0, 0, 0, 0);
        if (kp < p.n_k) rv[u] = *reinterpret_cast<const uint4*>(vbase + kp * D + ch * 8);
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
        *reinterpret_cast<uint2*>(Vt + (ch * 8 + dd) * C::VPAD + kg * 4) = pk;
      }
    }
    __syncthreads();

    // S^T = K_j Q^T : rows = keys (mt*16 + 4*lg + rr), column = query nt*16 + lr
    f32x4 sacc[C::MTK][C::NTQ];
#pragma unroll
    for (int mt = 0; mt < C::MTK; ++mt)
#pragma unroll
      for (int nt = 0; nt < C::NTQ; ++nt) sacc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < C::KSD; ++ks)
#pragma unroll
      for (int mt = 0; mt < C::MTK; ++mt) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(Ks + (mt * 16 + lr) * C::KPAD + ks * 32 + 8 * lg);
#pragma unroll
        for (int nt = 0; nt < C::NTQ; ++nt)
          sacc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[nt][ks], sacc[mt][nt], 0, 0, 0);
      }

    // online softmax per query column
#pragma unroll
    for (int nt = 0; nt < C::NTQ; ++nt) {
      const int64_t qp = q_first + nt * 16 + lr;
      float mx = -INFINITY;
#pragma unroll
      for (int mt = 0; mt < C::MTK; ++mt)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          float s = sacc[mt][nt][rr] * c;
          if (partial && !legal_pair(g, qp, k_first + mt * 16 + 4 * lg + rr)) s = -INFINITY;
          sacc[mt][nt][rr] = s;
          mx = fmaxf(mx, s);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[nt], mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run[nt] - m_use);
      m_run[nt] = m_new;
      float lsum = 0.f;
#pragma unroll
      for (int mt = 0; mt < C::MTK; ++mt)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          const float pv = __builtin_amdgcn_exp2f(sacc[mt][nt][rr] - m_use);
          sacc[mt][nt][rr] = pv;
          lsum += pv;
        }
      l_run[nt] = l_run[nt] * alpha + lsum;
#pragma unroll
      for (int md = 0; md < C::MTD; ++md) oacc[md][nt] *= alpha;
    }

    // O^T += V_j^T P^T : k-slot s of step ks is key 32ks + 4lg + s (s < 4) or 32ks + 16 + 4lg + (s - 4)
#pragma unroll
    for (int ks = 0; ks < C::KSK; ++ks) {
      bf16x8 pb[C::NTQ];
#pragma unroll
      for (int nt = 0; nt < C::NTQ; ++nt) {
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
          pb[nt][rr] = (__bf16)sacc[2 * ks][nt][rr];
          pb[nt][4 + rr] = (__bf16)sacc[2 * ks + 1][nt][rr];
        }
      }
#pragma unroll
      for (int md = 0; md < C::MTD; ++md) {
        const __bf16* vr = Vt + (md * 16 + lr) * C::VPAD + ks * 32 + 4 * lg;
        const bf16x4 lo = *reinterpret_cast<const bf16x4*>(vr);
        const bf16x4 hi = *reinterpret_cast<const bf16x4*>(vr + 16);
        const bf16x8 a = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
        for (int nt = 0; nt < C::NTQ; ++nt)
          oacc[md][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[nt], oacc[md][nt], 0, 0, 0);
      }
    }
  }

  // O = O / l; LSE = (m + log2 l) ln 2
#pragma unroll
  for (int nt = 0; nt < C::NTQ; ++nt) {
    float lt = l_run[nt];
    lt += __shfl_xor(lt, 16);
    lt += __shfl_xor(lt, 32);
    const int64_t qp = q_first + nt * 16 + lr;
    if (qp >= p.n_q) continue;
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    __bf16* orow = o + (((int64_t)b * p.h_q + h) * p.n_q + qp) * D;
#pragma unroll
    for (int md = 0; md < C::MTD; ++md) {
      bf16x4 ov;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) ov[rr] = (__bf16)(oacc[md][nt][rr] * inv);
      *reinterpret_cast<bf16x4*>(orow + md * 16 + 4 * lg) = ov;
    }
    if (lg == 0)
      lse[((int64_t)b * p.h_q + h) * p.n_q + qp] = lt > 0.f ? (m_run[nt] + __log2f(lt)) * kLn2 : -INFINITY;
  }
}

template <int D, int BQ, int BK>
hipError_t launch_cfg(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                      void* o, float* lse, hipStream_t stream) {
  using C = FwdCfg<D, BQ, BK>;
  auto kern = fwd_bf16_kernel<D, BQ, BK>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const unsigned blocks = (unsigned)sv.n_qt * p.h_q * p.batch;
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), C::LDS_BYTES, stream, p, sv,
                     static_cast<const __bf16*>(q), static_cast<const __bf16*>(k), static_cast<const __bf16*>(v),
                     static_cast<__bf16*>(o), lse);
  return hipGetLastError();
}

}  // namespace

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
