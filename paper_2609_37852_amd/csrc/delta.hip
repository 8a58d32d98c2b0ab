// Matched correction pass (Sec. 3.4; App. B.6.3 "Matched correction").
//
// delta_i = (sum_j P_ij dP_ij) / (sum_j P_ij) with the FP32 probabilities
// P = 2^(tau log2e (S - LSE / tau)) recomputed from the FP8 scores, and
// dP = dO_row V_row^T (MX MFMA, FP32).  Sums of P dP and of P are formed in
// FP32 over each aligned 32-key group, the group sums are accumulated in
// FP64, and delta is stored as an FP32 pair (hi, lo) with hi + lo the FP64
// quotient to about 2^-48.  Dividing by sum P makes the pair the exact
// centring constant of the P the backward recomputes, even where the stored
// LSE leaves sum P a few ulp away from 1.  Compensated variant (COMP): every
// product P dP is formed exactly in FP64 and all sums run in FP64, so delta
// carries no FP32 rounding of the terms it cancels.
//
// Workgroup: NW waves x 32 queries of one (batch, query head); 128-key tiles
// (64 at wide heads) of K and V (row copies) reach LDS by direct loads,
// double-buffered, so the next tile streams in while the current one is
// computed.  S^T and dP^T put one query in each lane (row reductions in-lane
// plus one exchange with lane l ^ 32).  The isolated score channel (if any)
// is zeroed in the Q operand; its product and the shift -LSE / tau are added
// to the scores by one FP32 rank-2 MFMA.  P and dP use exactly the
// operations of the backward kernel (same MX MFMA products and k order, the
// same rank-2 update, bwd_prob()), so the backward's dS = P (dP - delta) sums
// to zero over every row up to FP32 rounding of its own terms.  Only the 32-key group holding the
// diagonal is masked; groups in a wave's future (causal) or past the last key
// are skipped.
#include <type_traits>

#include "common.hpp"
#include "dma.hpp"
#include "kernels.hpp"
#include "tiles.hpp"

namespace afp8 {

template <int DQK, int DV, int NH = 1, bool CAUSAL = true>
struct DeltaCfg {
  // Wide heads (dqk + dv > 256) take 64-key tiles, so that two
  // double-buffered workgroups fit a CU (with 128-key tiles one did, a single
  // wave per SIMD, 15 % slower on the d = 256 and 192 / 128 problems); dv =
  // 256 without the mask keeps 128-key tiles and one workgroup, since two do
  // not fit its registers (they spilled, 3x slower).
  static constexpr bool WIDE = DQK + DV > 256;
  static constexpr int NW = 4, NT = 64 * NW, BQ = 32 * NW, BK = WIDE && (CAUSAL || DV <= 128) ? 64 : 128;
  static constexpr int al16(int x) { return (x + 15) & ~15; }
  static constexpr int K_OFF = 0;                               // K row codes [BK][DQK], swizzled
  static constexpr int V_OFF = K_OFF + BK * DQK;                // V row codes [BK][DV], swizzled
  static constexpr int KS_OFF = V_OFF + BK * DV;                // K row scales [BK][DQK/32]
  static constexpr int VS_OFF = al16(KS_OFF + BK * DQK / 32);   // V row scales [BK][DV/32]
  static constexpr int KH_OFF = al16(VS_OFF + BK * DV / 32);    // isolated-channel key values [NH][BK] FP32
  static constexpr int STAGE = KH_OFF + BK * 4 * NH;
  // two workgroups per CU where both stage buffers fit 80 KB
  static constexpr int WGS = 2 * STAGE <= 80 * 1024 ? 2 : 1;
};

// CAUSAL: the mask (key length = query length) or every key of Nk; COMP:
// FP64 products and sums; NH: isolated score channels (with 3, channels 1
// and 2 take a second rank-2 FP32 MFMA, the first shares one with the shift)
template <int DQK, int DV, bool CAUSAL, bool COMP, int NH = 1>
__global__ __launch_bounds__(256, (DeltaCfg<DQK, DV, NH, CAUSAL>::WGS)) void delta_matching_kernel(AttnArgs a) {
  using C = DeltaCfg<DQK, DV, NH, CAUSAL>;
  constexpr int NW = C::NW, BQ = C::BQ, BK = C::BK;
  constexpr int KS = DQK / 64, VS = DV / 64;
  __shared__ __attribute__((aligned(16))) uint8_t stA[C::STAGE];
  __shared__ __attribute__((aligned(16))) uint8_t stB[C::STAGE];
  __shared__ int hot_slot[NH];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hf = lane >> 5, li = lane & 31;
  constexpr bool causal = CAUSAL;
  const int N = (int)a.N, Nk = CAUSAL ? N : (int)a.Nk;
  const int nqb = (N + BQ - 1) / BQ;
  const WgCoord wc = query_major_coord((int)blockIdx.x, (int)a.B, (int)a.Hq, (int)a.Hkv, a.lens_q != nullptr);
  const int qb = nqb - 1 - wc.r;              // longest causal rows first
  const int h = wc.h, b = wc.b, kh = h / (int)a.G;
  // the sequence's own lengths bound the work; N and Nk remain the strides
  const SeqLens L = seq_lens<CAUSAL>(a, b, N, Nk);
  if (qb * BQ >= L.q) return;                 // the whole block is past the sequence
  const int q0 = qb * BQ + 32 * w;
  const bool live = q0 < L.q;
  const int qi = q0 + li;
  // groups visible to the wave's queries start before klim (a multiple of 32)
  const int klim = causal ? q0 + 32 : L.k;
  int hots[NH];
  if constexpr (NH == 1) hots[0] = select_hot_channel<DQK>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, hot_slot);
  else select_hot_channels<DQK, NH>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, hot_slot, hots);
  const int hot = hots[0];

  const size_t bhq = (size_t)b * a.Hq + h, bhk = (size_t)b * a.Hkv + kh;
  v8i qf[KS], df[VS];
  int qsc[KS], dsc[VS];
  // B operand of the score's rank-2 update: isolated-channel value (lanes
  // < 32), -LSE / tau (lanes >= 32) of the lane's query
  float qv = 0.f;
  float qv12 = 0.f;   // NH = 3: channel 1 (lanes < 32) and 2 (lanes >= 32) of the lane's query
  {
    const size_t row = bhq * N + (live ? qi : 0);
#pragma unroll
    for (int s = 0; s < KS; s++) {
      qf[s] = frag_rows_global(a.q_code + row * DQK, s, hf);
#pragma unroll
      for (int i = 0; i < NH; i++) clear_channel(qf[s], s, hf, hots[i]);
      qsc[s] = a.q_scale[row * (DQK / 32) + 2 * s + hf];
    }
#pragma unroll
    for (int s = 0; s < VS; s++) {
      df[s] = frag_rows_global(a.do_code + row * DV, s, hf);
      dsc[s] = a.do_scale[row * (DV / 32) + 2 * s + hf];
    }
    const float qhot = hot >= 0 ? row_value<DQK>(a.q_code, a.q_scale, (int64_t)row, hot) : 0.f;
    qv = hf ? neg_lse_over_tau(a.lse[row], a.tau) : qhot;
    if constexpr (NH == 3) {
      if (hot >= 0) qv12 = row_value<DQK>(a.q_code, a.q_scale, (int64_t)row, hf ? hots[2] : hots[1]);
    }
  }
  double num = 0.0, den = 0.0;

  const uint8_t* kcode = a.k_code + bhk * Nk * DQK;
  const uint8_t* kscale = a.k_scale + bhk * Nk * (DQK / 32);
  const uint8_t* vcode = a.v_code + bhk * Nk * DV;
  const uint8_t* vscale = a.v_scale + bhk * Nk * (DV / 32);
  // key tiles up to the block's last query, or over all keys
  const int kend = causal ? ((qb + 1) * BQ < L.q ? (qb + 1) * BQ : L.q) : L.k;
  const int ntiles = (kend + BK - 1) / BK;

  // loads of tile j0 (raw isolated-channel bytes in registers, decoded when
  // they are stored to LDS)
  uint32_t khc[NH] = {}, khs[NH] = {};
  RowLoads<DQK, NW, BK> kload;
  RowLoads<DV, NW, BK> vload;
  kload.init(w, lane);
  vload.init(w, lane);
  auto issue = [&](lds8* st, int j0) __attribute__((always_inline)) {
    // keys past the sequence are clamped to its last ones (never the padding)
    kload.issue(st + C::K_OFF, kcode, j0, L.k, w, lane);
    vload.issue(st + C::V_OFF, vcode, j0, L.k, w, lane);
    dma_row_scales<DQK, NW, BK>(st + C::KS_OFF, kscale, j0, L.k, w, lane, 0);
    dma_row_scales<DV, NW, BK>(st + C::VS_OFF, vscale, j0, L.k, w, lane, 1);
    if (hot >= 0 && threadIdx.x < BK) {
      const int r = j0 + (int)threadIdx.x < L.k ? j0 + (int)threadIdx.x : L.k - 1;
#pragma unroll
      for (int i = 0; i < NH; i++) {
        khc[i] = kcode[(int64_t)r * DQK + hots[i]];
        khs[i] = kscale[(int64_t)r * (DQK / 32) + hots[i] / 32];
      }
    }
    __builtin_amdgcn_sched_barrier(0);   // keep every load ahead of the tile's compute
  };
  auto finish = [&](uint8_t* st) __attribute__((always_inline)) {
    if (threadIdx.x < BK) {
#pragma unroll
      for (int i = 0; i < NH; i++)
        reinterpret_cast<float*>(st + C::KH_OFF)[i * BK + threadIdx.x] = hot >= 0 ? scaled_value(khc[i], khs[i]) : 0.f;
    }
  };

  // Scores (with the rank-2 update) and dP of one 32-key group (keys
  // j0 + 32 g ..) of the tile in st.
  auto group_mfma = [&](const uint8_t* st, int g, v16f& s, v16f& dp) __attribute__((always_inline)) {
    const uint8_t* K = st + C::K_OFF;
    const uint8_t* Ks = st + C::KS_OFF;
    const uint8_t* V = st + C::V_OFF;
    const uint8_t* Vs = st + C::VS_OFF;
    const float* Kh = reinterpret_cast<const float*>(st + C::KH_OFF);
#pragma unroll
    for (int r = 0; r < 16; r++) { s[r] = 0.f; dp[r] = 0.f; }
#pragma unroll
    for (int t = 0; t < KS; t++)
      s = mfma_mx(frag_rows_swz<DQK>(K, 32 * g + li, t, hf), qf[t], s, Ks[(32 * g + li) * (DQK / 32) + 2 * t + hf],
                  qsc[t]);
#pragma unroll
    for (int t = 0; t < VS; t++)
      dp = mfma_mx(frag_rows_swz<DV>(V, 32 * g + li, t, hf), df[t], dp, Vs[(32 * g + li) * (DV / 32) + 2 * t + hf],
                   dsc[t]);
    // S + k_c* q_c* - LSE / tau: A = isolated-channel key value (lanes
    // < 32) or 1 (lanes >= 32), B = qv
    s = rank2_update(hf ? 1.0f : Kh[32 * g + li], qv, s);
    if constexpr (NH == 3) s = rank2_update(Kh[(hf ? 2 * BK : BK) + 32 * g + li], qv12, s);
  };
  // P, then the group's sums of P dP and P; DIAG: the group holding the
  // wave's diagonal (keys after the query masked).  The lane holds keys
  // 32 g + 8 (r/4) + 4 hf + r % 4 of the tile, query qi.
  auto group_sums = [&](const v16f& s, const v16f& dp, auto diag_tag) __attribute__((always_inline)) {
    constexpr bool DIAG = decltype(diag_tag)::value;
    if constexpr (COMP) {
      double qn = 0.0, qd = 0.0;
#pragma unroll
      for (int q4 = 0; q4 < 4; q4++) {
#pragma unroll
        for (int e = 0; e < 4; e++) {
          const int r = 4 * q4 + e;
          float p = bwd_prob(s[r], a.c);
          if (DIAG) p = (8 * q4 + 4 * hf + e) > li ? 0.f : p;
          qn = __builtin_fma((double)p, (double)dp[r], qn);   // the product is exact in FP64
          qd += (double)p;
        }
      }
      num += qn + __shfl_xor(qn, 32);
      den += qd + __shfl_xor(qd, 32);
      return;
    }
    float pn = 0.f, pd = 0.f;
#pragma unroll
    for (int q4 = 0; q4 < 4; q4++) {
#pragma unroll
      for (int e = 0; e < 4; e++) {
        const int r = 4 * q4 + e;
        float p = bwd_prob(s[r], a.c);
        if (DIAG) p = (8 * q4 + 4 * hf + e) > li ? 0.f : p;
        pn = __builtin_fmaf(p, dp[r], pn);
        pd += p;
      }
    }
    // 32-key group sums: this lane's 16 keys plus the partner's 16 (FP32)
    num += (double)(pn + partner(pn));
    den += (double)(pd + partner(pd));
  };

  auto tile = [&](const uint8_t* st, int j0) __attribute__((always_inline)) {
    if (!live || j0 >= klim) return;
    v16f s0, dp0, s1, dp1;
    if (causal ? j0 + BK <= q0 : j0 + BK <= L.k) {
      // every key visible to every query of the wave: every group, no mask;
      // the MFMAs of group g + 1 are issued before the vector work of group g
      group_mfma(st, 0, s0, dp0);
#pragma unroll
      for (int g = 0; g < BK / 32; g += 2) {
        group_mfma(st, g + 1, s1, dp1);
        group_sums(s0, dp0, std::false_type{});
        if (g + 2 < BK / 32) group_mfma(st, g + 2, s0, dp0);
        group_sums(s1, dp1, std::false_type{});
      }
      return;
    }
#pragma unroll
    for (int g = 0; g < BK / 32; g++) {
      const int g0 = j0 + 32 * g;              // first key of the group
      if (g0 >= klim) break;                   // this and later groups are invisible to the wave
      group_mfma(st, g, s0, dp0);
      if (causal && g0 == q0) group_sums(s0, dp0, std::true_type{});
      else group_sums(s0, dp0, std::false_type{});
    }
  };

  issue((lds8*)stA, 0);
  finish(stA);
  lds_barrier();
  for (int t = 0; t < ntiles; t += 2) {
    if (t + 1 < ntiles) issue((lds8*)stB, (t + 1) * BK);
    tile(stA, t * BK);
    if (t + 1 < ntiles) finish(stB);
    lds_barrier();
    if (t + 1 >= ntiles) break;
    if (t + 2 < ntiles) issue((lds8*)stA, (t + 2) * BK);
    tile(stB, (t + 1) * BK);
    if (t + 2 < ntiles) finish(stA);
    lds_barrier();
  }
  if (!live || hf != 0) return;
  const double d = den > 0.0 ? num / den : 0.0;
  const float hi = (float)d;
  const float lo = (float)(d - (double)hi);
  *reinterpret_cast<float2*>(a.delta_out + (bhq * N + qi) * 2) = make_float2(hi, lo);
}

template <int DQK, int DV>
static hipError_t delta_dispatch(const AttnArgs& a, hipStream_t s) {
  using C = DeltaCfg<DQK, DV>;
  const int64_t nqb = (a.N + C::BQ - 1) / C::BQ;
  const dim3 grid((unsigned)(nqb * a.Hq * a.B));
  if (a.iso3) {
    if (a.causal) hipLaunchKernelGGL((delta_matching_kernel<DQK, DV, true, false, 3>), grid, dim3(C::NT), 0, s, a);
    else hipLaunchKernelGGL((delta_matching_kernel<DQK, DV, false, false, 3>), grid, dim3(C::NT), 0, s, a);
  } else if (a.causal) {
    if (a.comp) hipLaunchKernelGGL((delta_matching_kernel<DQK, DV, true, true>), grid, dim3(C::NT), 0, s, a);
    else hipLaunchKernelGGL((delta_matching_kernel<DQK, DV, true, false>), grid, dim3(C::NT), 0, s, a);
  } else {
    if (a.comp) hipLaunchKernelGGL((delta_matching_kernel<DQK, DV, false, true>), grid, dim3(C::NT), 0, s, a);
    else hipLaunchKernelGGL((delta_matching_kernel<DQK, DV, false, false>), grid, dim3(C::NT), 0, s, a);
  }
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
