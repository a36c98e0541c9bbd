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

template <int D, int BQ, int BK, int NQW>
__global__ void __launch_bounds__(512) fwd_bf16_kernel(cowa_params p, SchedView sv, int hpw, int n_hgroups,
                                                       const __bf16* __restrict__ q, const __bf16* __restrict__ k,
                                                       const __bf16* __restrict__ v, __bf16* __restrict__ o,
                                                       float* __restrict__ lse) {
  using T = SwzTile<D, BK>;
  constexpr int NTQ = NQW / 16;           // query tiles per wave
  constexpr int BKC = BK > 64 ? 64 : BK;   // keys per softmax step (a KV block is 1 or 2 steps)
  constexpr int MTK = BKC / 16;           // key tiles of S^T
  constexpr int KSD = D / 32;             // k-steps over d
  constexpr int MTD = D / 16;             // d tiles of O^T
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
  const int h0 = hgi * hpw;  // first QO head of this workgroup (all in KV group hk)

  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int h = h0 + wave / WAVES_PER_HEAD;
  const int64_t q_first = (int64_t)i * BQ + (wave % WAVES_PER_HEAD) * NQW;
  const Geo32 g = geo32(make_geo(p.n_q, p.n_k, p.w_sink, p.w_near, BQ, BK, p.h_k_offset + hk, p.h_k_total));

  const __bf16* kbase = k + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  const __bf16* vbase = v + ((int64_t)b * p.h_k + hk) * p.n_k * D;
  const int r = hk * sv.n_qt + i;
  const int e0 = sv.fwd_row_ptr[r], e1 = sv.fwd_row_ptr[r + 1];

  // buffer s: K at smem + 2 s BYTES, V right after it
  if (e0 < e1) {
    const int64_t kf = (int64_t)(sv.fwd_ent[e0] >> 1) * BK;
    load_tile_asm_nw<D, BK>(kbase, (int)kf, p.n_k, lds_addr(smem), wave, nw, lane);
    load_tile_asm_nw<D, BK>(vbase, (int)kf, p.n_k, lds_addr(smem) + T::BYTES, wave, nw, lane);
  }

  // Q^T fragments (B operand): query column nt*16 + lr, d = ks*32 + 8*lg + 0..7
  bf16x8 qf[NTQ][KSD];
#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) {
    const int64_t qp = q_first + nt * 16 + lr;
    const bool ok = qp < p.n_q;
    const __bf16* qrow = q + (((int64_t)b * p.h_q + h) * p.n_q + (ok ? qp : 0)) * D;
#pragma unroll
    for (int ks = 0; ks < KSD; ++ks) {
      bf16x8 val = *reinterpret_cast<const bf16x8*>(qrow + ks * 32 + 8 * lg);
      qf[nt][ks] = ok ? val : bf16x8{};
    }
  }

  f32x4 oacc[MTD][NTQ];
#pragma unroll
  for (int md = 0; md < MTD; ++md)
#pragma unroll
    for (int nt = 0; nt < NTQ; ++nt) oacc[md][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[NTQ], l_run[NTQ];
#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) { m_run[nt] = -INFINITY; l_run[nt] = 0.f; }
  const float c = p.softmax_scale * kLog2e;

  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // schedule entries one and two blocks ahead are read early, so that no
  // iteration waits on the load of the entry it prefetches
  uint32_t ent_cur = e0 < e1 ? sv.fwd_ent[e0] : 0u;
  uint32_t ent_nxt = e0 + 1 < e1 ? sv.fwd_ent[e0 + 1] : 0u;
  for (int e = e0; e < e1; ++e) {
    const int buf = (e - e0) & 1;
    const uint32_t ent = ent_cur;
    const int j = (int)(ent >> 1);
    const bool partial = ent & 1u;
    const int64_t k_first = (int64_t)j * BK;
    if (e + 1 < e1) {  // prefetch the next block into the other buffer
      const int64_t kf = (int64_t)(ent_nxt >> 1) * BK;
      unsigned char* nb = smem + (buf ^ 1) * 2 * T::BYTES;
      load_tile_asm_nw<D, BK>(kbase, (int)kf, p.n_k, lds_addr(nb), wave, nw, lane);
      load_tile_asm_nw<D, BK>(vbase, (int)kf, p.n_k, lds_addr(nb) + T::BYTES, wave, nw, lane);
    }
    ent_cur = ent_nxt;
    ent_nxt = sv.fwd_ent[e + 2 < e1 ? e + 2 : e1 - 1];  // unconditional: no merge of wait states
    const unsigned char* Kt = smem + buf * 2 * T::BYTES;
    const unsigned char* Vt = Kt + T::BYTES;

#pragma unroll 1
    for (int kc = 0; kc < BK; kc += BKC) {
      // S^T = K_j Q^T : rows = keys (mt*16 + 4*lg + rr), column = query nt*16 + lr
      f32x4 sacc[MTK][NTQ];
  #pragma unroll
      for (int mt = 0; mt < MTK; ++mt)
  #pragma unroll
        for (int nt = 0; nt < NTQ; ++nt) sacc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  #pragma unroll
      for (int ks = 0; ks < KSD; ++ks)
  #pragma unroll
        for (int mt = 0; mt < MTK; ++mt) {
          const int row = kc + mt * 16 + lr;
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(Kt + T::off(row, ks * 4 + lg));
  #pragma unroll
          for (int nt = 0; nt < NTQ; ++nt)
            sacc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[nt][ks], sacc[mt][nt], 0, 0, 0);
        }

      // online softmax per query column (raw-score units; c folded into the exponent)
      if (partial) {
  #pragma unroll
        for (int nt = 0; nt < NTQ; ++nt) {
          const int qp = (int)q_first + nt * 16 + lr;
          const int k0 = (int)k_first + kc + 4 * lg;
  #pragma unroll
          for (int mt = 0; mt < MTK; ++mt)
  #pragma unroll
            for (int rr = 0; rr < 4; ++rr)
              // an add that reads the accumulator: a plain masked store of -inf
              // into an MFMA destination could be overtaken by the MFMA write
              sacc[mt][nt][rr] += legal32(g, qp, k0 + mt * 16 + rr) ? 0.f : -INFINITY;
        }
      }
      float alpha[NTQ];
      bool moved = false;
  #pragma unroll
      for (int nt = 0; nt < NTQ; ++nt) {
        float mx = -INFINITY;
  #pragma unroll
        for (int mt = 0; mt < MTK; ++mt)
  #pragma unroll
          for (int rr = 0; rr < 4; ++rr) mx = fmaxf(mx, sacc[mt][nt][rr]);
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run[nt], mx);
        moved |= m_new > m_run[nt];
        const float mc = m_new == -INFINITY ? 0.f : m_new * c;
        alpha[nt] = __builtin_amdgcn_exp2f(m_run[nt] * c - mc);
        m_run[nt] = m_new;
        float lsum = 0.f;
  #pragma unroll
        for (int mt = 0; mt < MTK; ++mt)
  #pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            const float pv = __builtin_amdgcn_exp2f(fmaf(sacc[mt][nt][rr], c, -mc));
            sacc[mt][nt][rr] = pv;
            lsum += pv;
          }
        l_run[nt] = l_run[nt] * alpha[nt] + lsum;
      }
      if (__any(moved)) {
  #pragma unroll
        for (int md = 0; md < MTD; ++md)
  #pragma unroll
          for (int nt = 0; nt < NTQ; ++nt) oacc[md][nt] *= alpha[nt];
      }

      // O^T += V_j^T P^T.  k-slot t of step ks is key 32ks + 4lg + t (t < 4) or
      // 32ks + 16 + 4lg + (t - 4); the transposing read gives lane lr the column
      // d = md*16 + lr of four keys, supplied by lanes 4*t + (lr / 4) of its group.
  #pragma unroll
      for (int ks = 0; ks < KSK; ++ks) {
        bf16x8 pb[NTQ];
  #pragma unroll
        for (int nt = 0; nt < NTQ; ++nt)
  #pragma unroll
          for (int rr = 0; rr < 4; ++rr) {
            pb[nt][rr] = (__bf16)sacc[2 * ks][nt][rr];
            pb[nt][4 + rr] = (__bf16)sacc[2 * ks + 1][nt][rr];
          }
  #pragma unroll
        for (int md = 0; md < MTD; ++md) {
          const bf16x8 a = read_tr8<D, BK>(Vt, kc + ks * 32, md * 16, lr, lg);
  #pragma unroll
          for (int nt = 0; nt < NTQ; ++nt) oacc[md][nt] = mfma16(a, pb[nt], oacc[md][nt]);
        }
      }
    }

    __builtin_amdgcn_s_waitcnt(0);  // the prefetch of block e+1 has landed
    __syncthreads();                 // ... for every wave, and block e is no longer read
  }

  // O = O / l; LSE = (m c + log2 l) ln 2
#pragma unroll
  for (int nt = 0; nt < NTQ; ++nt) {
    float lt = l_run[nt];
    lt += __shfl_xor(lt, 16);
    lt += __shfl_xor(lt, 32);
    const int64_t qp = q_first + nt * 16 + lr;
    if (qp >= p.n_q) continue;
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    __bf16* orow = o + (((int64_t)b * p.h_q + h) * p.n_q + qp) * D;
#pragma unroll
    for (int md = 0; md < MTD; ++md) {
      bf16x4 ov;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) ov[rr] = (__bf16)(oacc[md][nt][rr] * inv);
      *reinterpret_cast<bf16x4*>(orow + md * 16 + 4 * lg) = ov;
    }
    if (lg == 0)
      lse[((int64_t)b * p.h_q + h) * p.n_q + qp] = lt > 0.f ? (m_run[nt] * c + __log2f(lt)) * kLn2 : -INFINITY;
  }
}

template <int D, int BQ, int BK, int NQW = 32>
hipError_t launch_cfg(const cowa_params& p, const SchedView& sv, const void* q, const void* k, const void* v,
                      void* o, float* lse, hipStream_t stream) {
  constexpr int LDS = 4 * SwzTile<D, BK>::BYTES;
  static_assert(LDS <= 160 * 1024, "LDS budget");
  auto kern = fwd_bf16_kernel<D, BQ, BK, NQW>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, LDS);
    if (err != hipSuccess) return err;
    attr_set = true;
  }
  const int G = p.h_q / p.h_k;
  int hpw = 256 / BQ;  // QO heads per workgroup: up to 256 query rows
  while (hpw > 1 && G % hpw != 0) hpw >>= 1;
  const int n_hgroups = p.h_q / hpw;
  const int waves = hpw * (BQ / NQW);
  const unsigned blocks = (unsigned)sv.n_qt * n_hgroups * p.batch;
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(64 * waves), LDS, stream, p, sv, hpw, n_hgroups,
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
