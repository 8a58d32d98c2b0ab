// Backward pass (Sec. 2.3; App. B.6.3 with power-of-two casts).
//
// Key-major: a workgroup owns BKB = 32*NWK keys of one (batch, KV head); wave
// w owns keys 32w..32w+31 of them.  The workgroup loops over the query heads
// of the KV group and over 64-query tiles from the causal diagonal to the end
// of the sequence.  dK and dV for its keys stay in registers (FP32) across
// the whole loop, which is the GQA group sum.  The next query tile's codes
// are loaded into registers while the current one is computed (LDS
// double-buffered where it fits).
//
// Per wave, tile and 32-query sub-block qs (near the diagonal a sub-block is
// skipped when it lies wholly before the wave's keys or past the sequence,
// and masked when it holds them; tiles wholly after the workgroup's keys take
// a path without either):
//   S  = Q K^T, dP = dO V^T   MX MFMA (A = Q / dO row tiles in LDS, B = the
//                             wave's K / V row codes in registers); lane l
//                             owns key l % 32 and holds 16 queries.
//   P  = bwd_prob(S + q_c* k_c*), dS = P ((dP - hi) - lo).
//   P' = C8(256 P) with scale 2^-8;  dS' = C8(dS / 2^e) with one exponent e
//        per aligned 32x32 block (the wave's 32 keys x 32 queries).
//   dV += P'^T dO_col,  dK += dS'^T Q_col   (A = codes straight from
//                             registers, B = col tiles in LDS permuted to the
//                             lane's queries).
// dQ: every wave writes its dS' codes to LDS ([key][query]); after the tile's
// barrier the 64 x Dqk dQ tile = dS'(64 x BKB) K_col(BKB x Dqk) is split over
// the waves, the dS' operand read with the 8-bit LDS transpose, and added to
// the FP32 workspace with atomics (dQ = tau * workspace is stored by a second
// kernel).
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "tiles.hpp"

namespace afp8 {

template <int DQK, int DV>
struct BwdCfg {
  // waves per workgroup (eight only where their dK/dV accumulators leave
  // room for two waves per SIMD) and LDS buffers, within 160 KB of LDS
  static constexpr int NWK = (DQK + DV <= 128) ? 8 : 4;
  static constexpr int NBUF = (DQK + DV <= 320) ? 2 : 1;   // staging buffers
  static constexpr int NT = 64 * NWK, BKB = 32 * NWK, BQ = 64;
  static constexpr int QST = DQK + 16, OST = DV + 16, CST = BQ + 16, KCST = BKB + 16, DST = BQ + 16;
  static constexpr int NDS = (DQK == 128 && DV == 128) || (DQK == 64) ? 2 : 1;  // dS buffers
  static constexpr int QU = BQ * DQK / 16, OU = BQ * DV / 16;   // uint4 per row tile
  static constexpr int QCU = DQK * BQ / 16, OCU = DV * BQ / 16; // uint4 per col tile
  static constexpr int PQ = (QU + NT - 1) / NT, PO = (OU + NT - 1) / NT;
  static constexpr int PQC = (QCU + NT - 1) / NT, POC = (OCU + NT - 1) / NT;
  static constexpr int QSD = BQ * DQK / 128, OSD = BQ * DV / 128;  // row-copy scale dwords per tile
  static_assert(QSD <= NT && OSD <= NT && DQK <= NT && DV <= NT && BQ <= NT, "one element per thread");
};

// One query tile in flight from global memory: raw loaded words only.  Every
// use of a loaded value waits for the load, so all decoding is left to
// bwd_store, after the current tile has been computed.
template <int DQK, int DV>
struct BwdStage {
  using C = BwdCfg<DQK, DV>;
  uint4 q[C::PQ], o[C::PO], qc[C::PQC], oc[C::POC];
  uint32_t qs, os;              // row-copy scale dwords
  uint32_t qcs0, qcs1;          // col-copy scale bytes of one Q channel (query groups 0, 1)
  uint32_t ocs0, ocs1;          // same for dO
  float L, dhi, dlo;            // LSE and delta (hi, lo) of one query
  uint32_t qhc, qhs;            // isolated-channel code and scale byte of one query
};

// Per-(batch, query head) base pointers of the query-side operands.
struct BwdHead {
  const uint8_t *qrow, *qsc, *orow, *osc, *qcol, *qcsc, *ocol, *ocsc;
  const float *lse, *delta;
};

template <int DQK, int DV>
__device__ __forceinline__ BwdHead bwd_head(const AttnArgs& a, size_t bh, int N) {
  BwdHead p;
  p.qrow = a.q_code + bh * N * DQK;
  p.qsc = a.q_scale + bh * N * (DQK / 32);
  p.orow = a.do_code + bh * N * DV;
  p.osc = a.do_scale + bh * N * (DV / 32);
  p.qcol = a.qc_code + bh * DQK * N;
  p.qcsc = a.qc_scale + bh * DQK * (N / 32);
  p.ocol = a.doc_code + bh * DV * N;
  p.ocsc = a.doc_scale + bh * DV * (N / 32);
  p.lse = a.lse + bh * N;
  p.delta = a.delta + bh * N * 2;
  return p;
}

template <int DQK, int DV>
__device__ __forceinline__ void bwd_load(BwdStage<DQK, DV>& st, const BwdHead& hp, int i0, int N, int hot) {
  using C = BwdCfg<DQK, DV>;
  const int tid = threadIdx.x;
  // row tiles: contiguous; bytes past the sequence are read from its last
  // valid 16 bytes (those queries are skipped)
  const uint8_t* qrow = hp.qrow + i0 * DQK;
  const uint8_t* orow = hp.orow + i0 * DV;
  const uint32_t qlim = (N - i0) * DQK - 16, olim = (N - i0) * DV - 16;
#pragma unroll
  for (int i = 0; i < C::PQ; i++) {
    const uint32_t u = tid + i * C::NT;
    const uint32_t off = (u < C::QU ? u : 0) * 16;
    st.q[i] = *reinterpret_cast<const uint4*>(qrow + (off < qlim ? off : qlim));
  }
#pragma unroll
  for (int i = 0; i < C::PO; i++) {
    const uint32_t u = tid + i * C::NT;
    const uint32_t off = (u < C::OU ? u : 0) * 16;
    st.o[i] = *reinterpret_cast<const uint4*>(orow + (off < olim ? off : olim));
  }
  const int cl = N - 16 - i0;   // last valid 16-byte column piece, relative to i0
#pragma unroll
  for (int i = 0; i < C::PQC; i++) {
    const uint32_t u = (tid + i * C::NT) < C::QCU ? tid + i * C::NT : 0, c = u >> 2, q = u & 3;
    const int col = (int)q * 16 < cl ? (int)q * 16 : cl;
    st.qc[i] = *reinterpret_cast<const uint4*>(hp.qcol + i0 + (c * N + col));
  }
#pragma unroll
  for (int i = 0; i < C::POC; i++) {
    const uint32_t u = (tid + i * C::NT) < C::OCU ? tid + i * C::NT : 0, c = u >> 2, q = u & 3;
    const int col = (int)q * 16 < cl ? (int)q * 16 : cl;
    st.oc[i] = *reinterpret_cast<const uint4*>(hp.ocol + i0 + (c * N + col));
  }
  if (tid < C::QSD) {
    const uint32_t off = i0 * (DQK / 32) + tid * 4, lim = N * (DQK / 32) - 4;
    st.qs = *reinterpret_cast<const uint32_t*>(hp.qsc + (off < lim ? off : lim));
  }
  if (tid < C::OSD) {
    const uint32_t off = i0 * (DV / 32) + tid * 4, lim = N * (DV / 32) - 4;
    st.os = *reinterpret_cast<const uint32_t*>(hp.osc + (off < lim ? off : lim));
  }
  const int g0 = i0 / 32, g1 = (i0 + 32 < N ? i0 + 32 : i0) / 32;
  if (tid < DQK) {
    st.qcs0 = hp.qcsc[tid * (N / 32) + g0];
    st.qcs1 = hp.qcsc[tid * (N / 32) + g1];
  }
  if (tid < DV) {
    st.ocs0 = hp.ocsc[tid * (N / 32) + g0];
    st.ocs1 = hp.ocsc[tid * (N / 32) + g1];
  }
  if (tid < C::BQ) {
    const int r = i0 + tid < N ? i0 + tid : N - 1;
    st.L = hp.lse[r];
    st.dhi = hp.delta[2 * r];
    st.dlo = hp.delta[2 * r + 1];
    if (hot >= 0) {
      st.qhc = hp.qrow[r * DQK + hot];
      st.qhs = hp.qsc[r * (DQK / 32) + hot / 32];
    }
  }
}

template <int DQK, int DV>
__device__ __forceinline__ void bwd_store(const BwdStage<DQK, DV>& st, uint8_t* sQ, uint8_t* sQs, uint8_t* sO,
                                          uint8_t* sOs, uint8_t* sQc, uint8_t* sQcs, uint8_t* sOc, uint8_t* sOcs,
                                          float* sRow, int hot) {
  using C = BwdCfg<DQK, DV>;
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < C::PQ; i++) {
    const int u = tid + i * C::NT;
    if (C::QU % C::NT == 0 || u < C::QU) {
      const int r = (u * 16) / DQK, c = (u * 16) % DQK;
      uint4 v = st.q[i];
      if (hot >= c && hot < c + 16) clear_byte(v, hot - c);
      *reinterpret_cast<uint4*>(sQ + r * C::QST + c) = v;
    }
  }
#pragma unroll
  for (int i = 0; i < C::PO; i++) {
    const int u = tid + i * C::NT;
    if (C::OU % C::NT == 0 || u < C::OU)
      *reinterpret_cast<uint4*>(sO + ((u * 16) / DV) * C::OST + (u * 16) % DV) = st.o[i];
  }
  // col tiles, permuted within each 32-query group (stage_cols_perm); 32-bit
  // stores keep the compiler from pairing the loaded registers early
#pragma unroll
  for (int i = 0; i < C::PQC; i++) {
    const int u = tid + i * C::NT;
    if (C::QCU % C::NT == 0 || u < C::QCU) {
      const int c = u >> 2, q = u & 3;
      uint32_t* base = reinterpret_cast<uint32_t*>(sQc + c * C::CST + (q >> 1) * 32 + (q & 1) * 8);
      base[0] = st.qc[i].x;
      base[1] = st.qc[i].z;
      base[4] = st.qc[i].y;
      base[5] = st.qc[i].w;
    }
  }
#pragma unroll
  for (int i = 0; i < C::POC; i++) {
    const int u = tid + i * C::NT;
    if (C::OCU % C::NT == 0 || u < C::OCU) {
      const int c = u >> 2, q = u & 3;
      uint32_t* base = reinterpret_cast<uint32_t*>(sOc + c * C::CST + (q >> 1) * 32 + (q & 1) * 8);
      base[0] = st.oc[i].x;
      base[1] = st.oc[i].z;
      base[4] = st.oc[i].y;
      base[5] = st.oc[i].w;
    }
  }
  if (tid < C::QSD) *reinterpret_cast<uint32_t*>(sQs + tid * 4) = st.qs;
  if (tid < C::OSD) *reinterpret_cast<uint32_t*>(sOs + tid * 4) = st.os;
  if (tid < DQK) *reinterpret_cast<uint16_t*>(sQcs + tid * 2) = (uint16_t)(st.qcs0 | (st.qcs1 << 8));
  if (tid < DV) *reinterpret_cast<uint16_t*>(sOcs + tid * 2) = (uint16_t)(st.ocs0 | (st.ocs1 << 8));
  if (tid < C::BQ) {
    sRow[tid] = st.L * kLog2e;
    sRow[C::BQ + tid] = st.dhi;
    sRow[2 * C::BQ + tid] = st.dlo;
    sRow[3 * C::BQ + tid] = hot >= 0 ? scaled_value(st.qhc, st.qhs) : 0.f;
  }
}

// Columns [k0, k0 + W) of a col-copy code matrix [D, N] into LDS [D][W]
// (natural order, row stride ST) and their scales into [D][W/32].
template <int D, int W, int ST, int NT>
__device__ __forceinline__ void stage_col_slice(uint8_t* lds, uint8_t* lds_scale, const uint8_t* code,
                                                const uint8_t* scale, int k0, int N) {
  constexpr int PER = W / 16;
  for (int u = threadIdx.x; u < D * PER; u += NT) {
    const int c = u / PER, q = u % PER;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (k0 + q * 16 < N) v = *reinterpret_cast<const uint4*>(code + (size_t)c * N + k0 + q * 16);
    *reinterpret_cast<uint4*>(lds + c * ST + q * 16) = v;
  }
  for (int u = threadIdx.x; u < D * (W / 32); u += NT) {
    const int c = u / (W / 32), g = u % (W / 32);
    lds_scale[u] = (k0 + g * 32 < N) ? scale[(size_t)c * (N / 32) + k0 / 32 + g] : (uint8_t)0;
  }
}

__device__ __forceinline__ double half_sum_d(double v) {
#pragma unroll
  for (int m = 1; m < 32; m <<= 1) v += __shfl_xor(v, m);
  return v;
}
__device__ __forceinline__ float half_max(float v) {
#pragma unroll
  for (int m = 1; m < 32; m <<= 1) v = fmaxf(v, __shfl_xor(v, m));
  return v;
}

template <int DQK, int DV, bool STATS>
__global__ __launch_bounds__((64 * BwdCfg<DQK, DV>::NWK)) void bwd_kernel(AttnArgs a) {
  using C = BwdCfg<DQK, DV>;
  constexpr int NWK = C::NWK, BKB = C::BKB, BQ = C::BQ;
  constexpr int KS = DQK / 64, VS = DV / 64, CK = DQK / 32, CV = DV / 32;
  __shared__ __attribute__((aligned(16))) uint8_t sQ[C::NBUF][BQ * C::QST];
  __shared__ __attribute__((aligned(16))) uint8_t sQs[C::NBUF][BQ * DQK / 32];
  __shared__ __attribute__((aligned(16))) uint8_t sO[C::NBUF][BQ * C::OST];
  __shared__ __attribute__((aligned(16))) uint8_t sOs[C::NBUF][BQ * DV / 32];
  __shared__ __attribute__((aligned(16))) uint8_t sQc[C::NBUF][DQK * C::CST];
  __shared__ __attribute__((aligned(16))) uint8_t sQcs[C::NBUF][DQK * 2];
  __shared__ __attribute__((aligned(16))) uint8_t sOc[C::NBUF][DV * C::CST];
  __shared__ __attribute__((aligned(16))) uint8_t sOcs[C::NBUF][DV * 2];
  __shared__ __attribute__((aligned(16))) float sRow[C::NBUF][4 * BQ];
  __shared__ __attribute__((aligned(16))) uint8_t sKc[DQK * C::KCST];
  __shared__ __attribute__((aligned(16))) uint8_t sKcs[DQK * BKB / 32];
  __shared__ __attribute__((aligned(16))) uint8_t sdS[C::NDS][BKB * C::DST];
  __shared__ __attribute__((aligned(16))) uint8_t sdSs[C::NDS][NWK * 2];
  __shared__ int hot_slot;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hf = lane >> 5, li = lane & 31;
  const int N = (int)a.N;
  const int kb0 = blockIdx.x * BKB;             // key block (block 0 has the most work)
  const int kh = blockIdx.y, b = blockIdx.z;
  const int kw0 = kb0 + 32 * w;                 // this wave's first key
  const bool live = kw0 < N;
  const int kj = kw0 + li;                      // this lane's key
  const int hot = select_hot_channel<DQK>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, &hot_slot);
  const size_t bhk = (size_t)b * a.Hkv + kh;
  const int Hq = (int)a.Hq, G = (int)a.G;
  const float c = a.c;

  // K and V row codes of this lane's key (B operands of S and dP)
  v8i kf[KS], vf[VS];
  int ksc[KS], vsc[VS];
  float khot = 0.f;
  {
    const int row = live ? kj : 0;
    const uint8_t* kr = a.k_code + (bhk * N + row) * DQK;
    const uint8_t* vr = a.v_code + (bhk * N + row) * DV;
#pragma unroll
    for (int s = 0; s < KS; s++) {
      kf[s] = frag_rows_global(kr, s, hf);
      clear_channel(kf[s], s, hf, hot);
      ksc[s] = a.k_scale[(bhk * N + row) * (DQK / 32) + 2 * s + hf];
    }
#pragma unroll
    for (int s = 0; s < VS; s++) {
      vf[s] = frag_rows_global(vr, s, hf);
      vsc[s] = a.v_scale[(bhk * N + row) * (DV / 32) + 2 * s + hf];
    }
    if (hot >= 0) khot = row_value<DQK>(a.k_code + bhk * N * DQK, a.k_scale + bhk * N * (DQK / 32), row, hot);
  }
  // K col codes of the workgroup's keys (B operand of dQ), once
  stage_col_slice<DQK, BKB, C::KCST, C::NT>(sKc, sKcs, a.kc_code + bhk * DQK * N,
                                           a.kc_scale + bhk * DQK * (N / 32), kb0, N);

  v16f dk[CK], dv[CV];
#pragma unroll
  for (int i = 0; i < CK; i++)
#pragma unroll
    for (int r = 0; r < 16; r++) dk[i][r] = 0.f;
#pragma unroll
  for (int i = 0; i < CV; i++)
#pragma unroll
    for (int r = 0; r < 16; r++) dv[i][r] = 0.f;

  const int nqt = (N + BQ - 1) / BQ, qt0 = kb0 / BQ, nq = nqt - qt0;
  const int total = G * nq;
  BwdStage<DQK, DV> st;
  bwd_load<DQK, DV>(st, bwd_head<DQK, DV>(a, (size_t)b * Hq + kh * G, N), qt0 * BQ, N, hot);
  bwd_store<DQK, DV>(st, sQ[0], sQs[0], sO[0], sOs[0], sQc[0], sQcs[0], sOc[0], sOcs[0], sRow[0], hot);
  __syncthreads();

  // dQ atomics: lane part of the offset into the [B, N, Hq, Dqk] workspace
  const uint32_t HqD = (uint32_t)Hq * DQK;
  const uint32_t dq_lane = (uint32_t)(4 * hf) * HqD + li;

  for (int it = 0; it < total; it++) {
    const int cur = C::NBUF == 2 ? (it & 1) : 0;   // staging buffer of this tile
    const int dsb = C::NDS == 2 ? (it & 1) : 0;
    const int h = kh * G + it / nq;
    const int i0 = (qt0 + it % nq) * BQ;
    {
      // next tile (the last iteration reloads the first one into the idle
      // buffer): loads are issued unconditionally so that no merge of old and
      // new register values forces a wait right here
      const int itn = it + 1 < total ? it + 1 : 0;
      bwd_load<DQK, DV>(st, bwd_head<DQK, DV>(a, (size_t)b * Hq + kh * G + itn / nq, N),
                        (qt0 + itn % nq) * BQ, N, hot);
    }

    const uint8_t* Q = sQ[cur];
    const uint8_t* Qs = sQs[cur];
    const uint8_t* O = sO[cur];
    const uint8_t* Os = sOs[cur];
    const float* Row = sRow[cur];
    v8i pa, da;          // P' and dS' codes: A operands of dV and dK (k = the tile's 64 queries)
    int dse[2] = {-127, -127};
    bool any = false;
    // tiles wholly after the workgroup's keys and inside the sequence: no
    // mask, no skipped sub-block
    const bool full = i0 >= kb0 + BKB && i0 + BQ <= N;

    auto subblock = [&](const int qs, auto edge_tag) {
      constexpr bool EDGE = decltype(edge_tag)::value;
      const int qb = i0 + 32 * qs;               // first query of the sub-block
      if (EDGE && (!live || qb < kw0 || qb >= N)) {
#pragma unroll
        for (int k = 0; k < 4; k++) { pa[4 * qs + k] = 0; da[4 * qs + k] = 0; }
        return;
      }
      any = true;
      v16f s, dp;
#pragma unroll
      for (int r = 0; r < 16; r++) { s[r] = 0.f; dp[r] = 0.f; }
#pragma unroll
      for (int t = 0; t < KS; t++)
        s = mfma_mx(frag_rows<C::QST>(Q, 32 * qs + li, t, hf), kf[t], s,
                    Qs[(32 * qs + li) * (DQK / 32) + 2 * t + hf], ksc[t]);
#pragma unroll
      for (int t = 0; t < VS; t++)
        dp = mfma_mx(frag_rows<C::OST>(O, 32 * qs + li, t, hf), vf[t], dp,
                     Os[(32 * qs + li) * (DV / 32) + 2 * t + hf], vsc[t]);
      // lane holds queries qb + 8 g + 4 hf + e (accumulator r = 4 g + e)
      float amax = 0.f;
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const int qo = 32 * qs + 8 * g + 4 * hf;
        const float4 Lg = *reinterpret_cast<const float4*>(&Row[qo]);
        const float4 Hg = *reinterpret_cast<const float4*>(&Row[BQ + qo]);
        const float4 Og = *reinterpret_cast<const float4*>(&Row[2 * BQ + qo]);
        const float4 Qg = *reinterpret_cast<const float4*>(&Row[3 * BQ + qo]);
        const float Lv[4] = {Lg.x, Lg.y, Lg.z, Lg.w}, Hv[4] = {Hg.x, Hg.y, Hg.z, Hg.w};
        const float Ov[4] = {Og.x, Og.y, Og.z, Og.w}, Qh[4] = {Qg.x, Qg.y, Qg.z, Qg.w};
#pragma unroll
        for (int e = 0; e < 4; e++) {
          const int r = 4 * g + e;
          float p = bwd_prob(__builtin_fmaf(Qh[e], khot, s[r]), c, Lv[e]);
          if (EDGE && qb == kw0) p = (li > 8 * g + 4 * hf + e) ? 0.f : p;   // diagonal block: key > query
          s[r] = p;
          dp[r] = p * ((dp[r] - Hv[e]) - Ov[e]);
          amax = fmaxf(amax, fabsf(dp[r]));
        }
      }
#pragma unroll
      for (int k = 0; k < 4; k++)
        pa[4 * qs + k] = (int)cvt4_div(s[4 * k], s[4 * k + 1], s[4 * k + 2], s[4 * k + 3], 0.00390625f);
      int e = pow2_exponent(wave_max_nonneg(amax));
      e = e < -126 ? -126 : e;
      const float sc = exp2i(e);
#pragma unroll
      for (int k = 0; k < 4; k++)
        da[4 * qs + k] = (int)cvt4_div(dp[4 * k], dp[4 * k + 1], dp[4 * k + 2], dp[4 * k + 3], sc);
      dse[qs] = e;
      if constexpr (STATS) {
        // per query row: FP64 sums over this wave's 32 keys, then atomics
#pragma unroll
        for (int r = 0; r < 16; r++) {
          const float cast = fp8_value((uint32_t)da[4 * qs + (r >> 2)], r & 3) * sc;
          const double s0 = half_sum_d((double)dp[r]);
          const double s1 = half_sum_d((double)fabsf(dp[r]));
          const double s2 = half_sum_d((double)cast);
          const float mx = half_max(fabsf(dp[r]));
          const int qi = qb + 8 * (r >> 2) + 4 * hf + (r & 3);
          if (li == 0) {
            double* sp = a.rowstats + (((size_t)b * Hq + h) * N + qi) * 4;
            atomicAdd(sp + 0, s0);
            atomicAdd(sp + 1, s1);
            atomicAdd(sp + 2, s2);
            atomicMax(reinterpret_cast<unsigned long long*>(sp + 3),
                      (unsigned long long)__double_as_longlong((double)mx));
          }
        }
      }
    };
    if (full) {
      subblock(0, std::false_type{});
      subblock(1, std::false_type{});
    } else {
      subblock(0, std::true_type{});
      subblock(1, std::true_type{});
    }
    if (any) {
      // dV += P'^T dO_col ; dK += dS'^T Q_col   (k = the 64 queries of the tile)
      const int dascale = (hf ? dse[1] : dse[0]) + 127;
      const uint8_t* Oc = sOc[cur];
      const uint8_t* Ocs = sOcs[cur];
      const uint8_t* Qc = sQc[cur];
      const uint8_t* Qcs = sQcs[cur];
#pragma unroll
      for (int i = 0; i < CV; i++)
        dv[i] = mfma_mx(pa, frag_cols<C::CST>(Oc, 32 * i + li, hf), dv[i], 127 - 8, Ocs[(32 * i + li) * 2 + hf]);
#pragma unroll
      for (int i = 0; i < CK; i++)
        dk[i] = mfma_mx(da, frag_cols<C::CST>(Qc, 32 * i + li, hf), dk[i], dascale, Qcs[(32 * i + li) * 2 + hf]);
    }
    // dS' codes to LDS: row = key (32 w + li), columns = the lane's queries
    uint8_t* dS_l = sdS[dsb];
#pragma unroll
    for (int qs = 0; qs < 2; qs++)
#pragma unroll
      for (int g = 0; g < 4; g++)
        *reinterpret_cast<int*>(dS_l + (32 * w + li) * C::DST + 32 * qs + 8 * g + 4 * hf) = da[4 * qs + g];
    if (lane == 0) {
      sdSs[dsb][w * 2] = (uint8_t)(dse[0] + 127);
      sdSs[dsb][w * 2 + 1] = (uint8_t)(dse[1] + 127);
    }
    // the next tile into the other staging buffer (nobody reads it this tile)
    if constexpr (C::NBUF == 2) {
      const int nb = cur ^ 1;
      bwd_store<DQK, DV>(st, sQ[nb], sQs[nb], sO[nb], sOs[nb], sQc[nb], sQcs[nb], sOc[nb], sOcs[nb], sRow[nb], hot);
    }
    __syncthreads();
    // dQ tile (64 queries x DQK) = dS'(64 x BKB) K_col(BKB x DQK): output blocks
    // m = qs * CK + i, distributed round-robin over the waves
    for (int m = w; m < 2 * CK; m += NWK) {
      const int qs = m / CK, i = m % CK;
      const int qb = i0 + 32 * qs;
      if (qb >= N) continue;
      v16f acc;
#pragma unroll
      for (int r = 0; r < 16; r++) acc[r] = 0.f;
      const int i16 = lane & 15;
      const int qbase = 32 * qs + 16 * ((lane >> 4) & 1);
#pragma unroll
      for (int ks = 0; ks < BKB / 64; ks++) {
        if (kb0 + 64 * ks > qb + 31) break;    // these keys are all in the future of the sub-block
        // A: rows = queries of sub-block qs, k = keys 64 ks .. 64 ks + 63 (natural order)
        v8i af;
#pragma unroll
        for (int part = 0; part < 4; part++) {
          const int kk = 64 * ks + 32 * (part >> 1) + 16 * hf + 8 * (part & 1);
          const uint8_t* addr = dS_l + (kk + (i16 >> 1)) * C::DST + qbase + 8 * (i16 & 1);
          const v2i t = __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) v2i*)(addr));
          af[2 * part] = t[0];
          af[2 * part + 1] = t[1];
        }
        acc = mfma_mx(af, frag_rows<C::KCST>(sKc, 32 * i + li, ks, hf), acc, sdSs[dsb][(2 * ks + hf) * 2 + qs],
                      sKcs[(32 * i + li) * (BKB / 32) + 2 * ks + hf]);
      }
      // lane holds channel 32 i + li, queries qb + 8 (r/4) + 4 hf + r % 4
      float* dqb = a.dq_acc + (((size_t)b * N + qb) * Hq + h) * DQK + 32 * i;
#pragma unroll
      for (int r = 0; r < 16; r++)
        atomicAdd(dqb + (uint32_t)(8 * (r >> 2) + (r & 3)) * HqD + dq_lane, acc[r]);
    }
    if constexpr (C::NDS == 1) __syncthreads();   // single dS buffer: reads done before the next writes
    if constexpr (C::NBUF == 1) {
      if (it + 1 < total) {
        if constexpr (C::NDS == 2) __syncthreads();
        bwd_store<DQK, DV>(st, sQ[0], sQs[0], sO[0], sOs[0], sQc[0], sQcs[0], sOc[0], sOcs[0], sRow[0], hot);
        __syncthreads();
      }
    }
  }
  if (!live) return;
  // dK (times tau) and dV: lane holds channel 32 i + li, keys kw0 + 8 (r/4) + 4 hf + r % 4
#pragma unroll
  for (int r = 0; r < 16; r++) {
    const int key = kw0 + 8 * (r >> 2) + 4 * hf + (r & 3);
    if (a.grad_bf16) {
      uint16_t* kd = reinterpret_cast<uint16_t*>(a.dk) + b * a.dks[0] + (int64_t)key * a.dks[1] + kh * a.dks[2];
      uint16_t* vd = reinterpret_cast<uint16_t*>(a.dv) + b * a.dvs[0] + (int64_t)key * a.dvs[1] + kh * a.dvs[2];
#pragma unroll
      for (int i = 0; i < CK; i++) kd[32 * i + li] = f32_to_bf16(dk[i][r] * a.tau);
#pragma unroll
      for (int i = 0; i < CV; i++) vd[32 * i + li] = f32_to_bf16(dv[i][r]);
    } else {
      float* kd = reinterpret_cast<float*>(a.dk) + b * a.dks[0] + (int64_t)key * a.dks[1] + kh * a.dks[2];
      float* vd = reinterpret_cast<float*>(a.dv) + b * a.dvs[0] + (int64_t)key * a.dvs[1] + kh * a.dvs[2];
#pragma unroll
      for (int i = 0; i < CK; i++) kd[32 * i + li] = dk[i][r] * a.tau;
#pragma unroll
      for (int i = 0; i < CV; i++) vd[32 * i + li] = dv[i][r];
    }
  }
}

template <int DQK, int DV>
static hipError_t bwd_dispatch(const AttnArgs& a, hipStream_t s) {
  using C = BwdCfg<DQK, DV>;
  const int64_t nkb = (a.N + C::BKB - 1) / C::BKB;
  dim3 grid((unsigned)nkb, (unsigned)a.Hkv, (unsigned)a.B);
  if (a.rowstats) hipLaunchKernelGGL((bwd_kernel<DQK, DV, true>), grid, dim3(C::NT), 0, s, a);
  else hipLaunchKernelGGL((bwd_kernel<DQK, DV, false>), grid, dim3(C::NT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_bwd(const AttnArgs& a, int dqk, int dv, hipStream_t s) {
  if (dqk == 64 && dv == 64) return bwd_dispatch<64, 64>(a, s);
  if (dqk == 128 && dv == 128) return bwd_dispatch<128, 128>(a, s);
  if (dqk == 256 && dv == 256) return bwd_dispatch<256, 256>(a, s);
  if (dqk == 192 && dv == 128) return bwd_dispatch<192, 128>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace afp8
