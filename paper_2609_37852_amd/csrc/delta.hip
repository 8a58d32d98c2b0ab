// Matched correction pass (Sec. 3.4; App. B.6.3 "Matched correction").
//
// delta_i = (sum_j P_ij dP_ij) / (sum_j P_ij) with the FP32 probabilities
// P = 2^(S tau log2e - LSE log2e) recomputed from the FP8 scores, and
// dP = dO_row V_row^T (MX MFMA, FP32).  Keys are visited in ascending order;
// sum P dP and sum P are reduced in FP32 over each aligned 32-key group, the
// group sums are accumulated in FP64, and delta is stored as an FP32 pair
// (hi, lo) with hi + lo the FP64 quotient to about 2^-48.  Dividing by sum P
// makes the pair the exact centring constant of the P the backward
// recomputes, even where the stored LSE leaves sum P a few ulp away from 1.
//
// Geometry as in the forward: NW waves x 32 queries per workgroup, 64-key
// tiles of K and V (row copies) staged in LDS; S^T and dP^T are computed so
// that each lane owns one query.  P and dP use exactly the operations of the
// backward kernel (same MX MFMA operands and k order, bwd_prob()), so the
// backward's dS = P (dP - delta) sums to zero over every row up to FP32
// rounding of its own terms.
#include "common.hpp"
#include "kernels.hpp"
#include "tiles.hpp"

namespace afp8 {

template <int DQK, int DV, int NW>
__global__ __launch_bounds__(64 * NW) void delta_matching_kernel(AttnArgs a) {
  constexpr int BQ = 32 * NW, BK = 64;
  constexpr int KS = DQK / 64, VS = DV / 64;
  constexpr int KST = DQK + 16, VST = DV + 16;
  __shared__ __attribute__((aligned(16))) uint8_t sK[BK * KST];
  __shared__ __attribute__((aligned(16))) uint8_t sKs[BK * DQK / 32];
  __shared__ __attribute__((aligned(16))) uint8_t sV[BK * VST];
  __shared__ __attribute__((aligned(16))) uint8_t sVs[BK * DV / 32];
  __shared__ __attribute__((aligned(16))) float sKh[BK];
  __shared__ int hot_slot;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hf = lane >> 5, li = lane & 31;
  const int64_t nqb = (a.N + BQ - 1) / BQ;
  const int64_t qb = nqb - 1 - (int64_t)blockIdx.x;
  const int64_t h = blockIdx.y, b = blockIdx.z, kh = h / a.G;
  const int64_t q0 = qb * BQ + 32 * w;
  const bool live = q0 < a.N;
  const int64_t qi = q0 + li;
  const int hot = select_hot_channel<DQK>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, &hot_slot);

  v8i qf[KS], df[VS];
  int qsc[KS], dsc[VS];
  float L = 0.f;
#pragma unroll
  for (int s = 0; s < KS; s++) { qf[s] = v8i{0, 0, 0, 0, 0, 0, 0, 0}; qsc[s] = 0; }
#pragma unroll
  for (int s = 0; s < VS; s++) { df[s] = v8i{0, 0, 0, 0, 0, 0, 0, 0}; dsc[s] = 0; }
  if (live) {
    const int64_t row = (b * a.Hq + h) * a.N + qi;
#pragma unroll
    for (int s = 0; s < KS; s++) {
      qf[s] = frag_rows_global(a.q_code + row * DQK, s, hf);
      clear_channel(qf[s], s, hf, hot);
      qsc[s] = a.q_scale[row * (DQK / 32) + 2 * s + hf];
    }
#pragma unroll
    for (int s = 0; s < VS; s++) {
      df[s] = frag_rows_global(a.do_code + row * DV, s, hf);
      dsc[s] = a.do_scale[row * (DV / 32) + 2 * s + hf];
    }
    L = a.lse[row] * kLog2e;
  }
  const float qhot = (live && hot >= 0) ? row_value<DQK>(a.q_code, a.q_scale, (b * a.Hq + h) * a.N + qi, hot) : 0.f;
  double num = 0.0, den = 0.0;

  const int64_t qend = ((qb + 1) * BQ < a.N) ? (qb + 1) * BQ : a.N;
  const int ntiles = (int)((qend + BK - 1) / BK);
  const uint8_t* kcode = a.k_code + (b * a.Hkv + kh) * a.N * DQK;
  const uint8_t* kscale = a.k_scale + (b * a.Hkv + kh) * a.N * (DQK / 32);
  const uint8_t* vcode = a.v_code + (b * a.Hkv + kh) * a.N * DV;
  const uint8_t* vscale = a.v_scale + (b * a.Hkv + kh) * a.N * (DV / 32);

  for (int t = 0; t < ntiles; t++) {
    const int64_t j0 = (int64_t)t * BK;
    __syncthreads();
    stage_rows<BK, DQK, KST, 64 * NW>(sK, sKs, kcode, kscale, j0, a.N, hot);
    stage_rows<BK, DV, VST, 64 * NW>(sV, sVs, vcode, vscale, j0, a.N);
    if (threadIdx.x < BK)
      sKh[threadIdx.x] = (hot >= 0 && j0 + threadIdx.x < a.N) ? row_value<DQK>(kcode, kscale, j0 + threadIdx.x, hot) : 0.f;
    __syncthreads();
    if (!live || j0 > q0) continue;

    const bool diag = j0 + BK - 1 > q0;
    float gnum[2], gden[2];
#pragma unroll
    for (int kb = 0; kb < 2; kb++) {
      v16f s, dp;
#pragma unroll
      for (int r = 0; r < 16; r++) { s[r] = 0.f; dp[r] = 0.f; }
#pragma unroll
      for (int st = 0; st < KS; st++) {
        const v8i kf = frag_rows<KST>(sK, 32 * kb + li, st, hf);
        s = mfma_mx(kf, qf[st], s, sKs[(32 * kb + li) * (DQK / 32) + 2 * st + hf], qsc[st]);
      }
#pragma unroll
      for (int st = 0; st < VS; st++) {
        const v8i vf = frag_rows<VST>(sV, 32 * kb + li, st, hf);
        dp = mfma_mx(vf, df[st], dp, sVs[(32 * kb + li) * (DV / 32) + 2 * st + hf], dsc[st]);
      }
      float pn = 0.f, pd = 0.f;
      float kh4[16];
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const float4 v4 = *reinterpret_cast<const float4*>(&sKh[32 * kb + 8 * g + 4 * hf]);
        kh4[4 * g] = v4.x; kh4[4 * g + 1] = v4.y; kh4[4 * g + 2] = v4.z; kh4[4 * g + 3] = v4.w;
      }
#pragma unroll
      for (int r = 0; r < 16; r++) {
        float p = bwd_prob(__builtin_fmaf(qhot, kh4[r], s[r]), a.c, L);
        if (diag) {
          const int64_t key = j0 + 32 * kb + 8 * (r >> 2) + 4 * hf + (r & 3);
          p = key > qi ? 0.f : p;
        }
        pn = __builtin_fmaf(p, dp[r], pn);
        pd += p;
      }
      gnum[kb] = pn;
      gden[kb] = pd;
    }
    // 32-key group sums: this lane's 16 keys plus the partner's 16 (FP32)
#pragma unroll
    for (int kb = 0; kb < 2; kb++) {
      const float n32 = gnum[kb] + partner(gnum[kb]);
      const float d32 = gden[kb] + partner(gden[kb]);
      num += (double)n32;
      den += (double)d32;
    }
  }
  if (!live || hf != 0) return;
  const double d = den > 0.0 ? num / den : 0.0;
  const float hi = (float)d;
  const float lo = (float)(d - (double)hi);
  float* dst = a.delta_out + ((b * a.Hq + h) * a.N + qi) * 2;
  *reinterpret_cast<float2*>(dst) = make_float2(hi, lo);
}

template <int DQK, int DV>
static hipError_t delta_dispatch(const AttnArgs& a, hipStream_t s) {
  constexpr int NW = 4;
  const int64_t nqb = (a.N + 32 * NW - 1) / (32 * NW);
  dim3 grid((unsigned)nqb, (unsigned)a.Hq, (unsigned)a.B);
  hipLaunchKernelGGL((delta_matching_kernel<DQK, DV, NW>), grid, dim3(64 * NW), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_delta_matching(const AttnArgs& a, int dqk, int dv, hipStream_t s) {
  if (dqk == 64 && dv == 64) return delta_dispatch<64, 64>(a, s);
  if (dqk == 128 && dv == 128) return delta_dispatch<128, 128>(a, s);
  if (dqk == 256 && dv == 256) return delta_dispatch<256, 256>(a, s);
  if (dqk == 192 && dv == 128) return delta_dispatch<192, 128>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace afp8
