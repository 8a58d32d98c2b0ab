// Backward pass (Sec. 2.3; App. B.6.3 with power-of-two casts).
//
// Key-major: a workgroup owns BKB = 32*NWK keys of one (batch, KV head); wave
// w owns keys 32w..32w+31 of them.  The workgroup loops over the query heads
// of the KV group and over 64-query tiles from the causal diagonal to the end
// of the sequence.  dK and dV for its keys stay in registers (FP32) across
// the whole loop, which is the GQA group sum.
//
// Per wave, tile and 32-query sub-block qs:
//   S  = Q K^T, dP = dO V^T   MX MFMA (A = Q / dO row tiles in LDS, B = the
//                             wave's K / V row codes in registers); lane l
//                             owns key l % 32 and holds 16 queries.
//   P  = bwd_prob(S), zero for masked pairs;  dS = P ((dP - hi) - lo).
//   P' = C8(256 P) with scale 2^-8;  dS' = C8(dS / 2^e) with one exponent e
//        per aligned 32x32 block (the wave's 32 keys x 32 queries).
//   dV += P'^T dO_col,  dK += dS'^T Q_col   (A = codes straight from
//                             registers, B = col tiles in LDS permuted to the
//                             lane's queries).
// dQ: every wave writes its dS' codes to LDS ([key][query]); after a barrier
// the 64 x Dqk dQ tile = dS'(64 x BKB) K_col(BKB x Dqk) is split over the
// waves, the dS' operand read with the 8-bit LDS transpose, and added to the
// FP32 workspace with atomics (dQ = tau * workspace is stored by a second
// kernel).
#include "common.hpp"
#include "kernels.hpp"
#include "tiles.hpp"

namespace afp8 {

// Columns [k0, k0 + W) of a col-copy code matrix [D, N] into LDS [D][W]
// (natural order, row stride ST) and their scales into [D][W/32].
template <int D, int W, int ST, int NT>
__device__ __forceinline__ void stage_col_slice(uint8_t* lds, uint8_t* lds_scale, const uint8_t* code,
                                                const uint8_t* scale, int64_t k0, int64_t N) {
  constexpr int PER = W / 16;
  for (int u = threadIdx.x; u < D * PER; u += NT) {
    const int c = u / PER, q = u % PER;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (k0 + q * 16 < N) v = *reinterpret_cast<const uint4*>(code + (int64_t)c * N + k0 + q * 16);
    *reinterpret_cast<uint4*>(lds + c * ST + q * 16) = v;
  }
  for (int u = threadIdx.x; u < D * (W / 32); u += NT) {
    const int c = u / (W / 32), g = u % (W / 32);
    lds_scale[u] = (k0 + g * 32 < N) ? scale[(int64_t)c * (N / 32) + k0 / 32 + g] : (uint8_t)0;
  }
}

// max over the 64 lanes of a wave
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 1; m < 32; m <<= 1) v = fmaxf(v, __shfl_xor(v, m));
  return fmaxf(v, partner(v));
}

__device__ __forceinline__ float half_sum(float v) {
#pragma unroll
  for (int m = 1; m < 32; m <<= 1) v += __shfl_xor(v, m);
  return v;
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

template <int DQK, int DV, int NWK, bool STATS>
__global__ __launch_bounds__(64 * NWK) void bwd_kernel(AttnArgs a) {
  constexpr int BKB = 32 * NWK, BQ = 64;
  constexpr int KS = DQK / 64, VS = DV / 64, CK = DQK / 32, CV = DV / 32;
  constexpr int QST = DQK + 16, OST = DV + 16, CST = BQ + 16, KCST = BKB + 16, DST = BQ + 16;
  constexpr int NT = 64 * NWK;
  __shared__ __attribute__((aligned(16))) uint8_t sQ[BQ * QST];
  __shared__ __attribute__((aligned(16))) uint8_t sQs[BQ * DQK / 32];
  __shared__ __attribute__((aligned(16))) uint8_t sO[BQ * OST];
  __shared__ __attribute__((aligned(16))) uint8_t sOs[BQ * DV / 32];
  __shared__ __attribute__((aligned(16))) uint8_t sQc[DQK * CST];
  __shared__ __attribute__((aligned(16))) uint8_t sQcs[DQK * 2];
  __shared__ __attribute__((aligned(16))) uint8_t sOc[DV * CST];
  __shared__ __attribute__((aligned(16))) uint8_t sOcs[DV * 2];
  __shared__ __attribute__((aligned(16))) uint8_t sKc[DQK * KCST];
  __shared__ __attribute__((aligned(16))) uint8_t sKcs[DQK * BKB / 32];
  __shared__ __attribute__((aligned(16))) uint8_t sdS[BKB * DST];
  __shared__ __attribute__((aligned(16))) uint8_t sdSs[NWK * 2];
  __shared__ __attribute__((aligned(16))) float sL[BQ];
  __shared__ __attribute__((aligned(16))) float sD[BQ * 2];
  __shared__ __attribute__((aligned(16))) float sQh[BQ];
  __shared__ int hot_slot;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hf = lane >> 5, li = lane & 31;
  const int64_t kb0 = (int64_t)blockIdx.x * BKB;  // key block (block 0 has the most work)
  const int64_t kh = blockIdx.y, b = blockIdx.z;
  const int64_t kw0 = kb0 + 32 * w;                 // this wave's first key
  const bool live = kw0 < a.N;
  const int64_t kj = kw0 + li;                      // this lane's key
  const int hot = select_hot_channel<DQK>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, &hot_slot);

  // K and V row codes of this lane's key (B operands of S and dP)
  v8i kf[KS], vf[VS];
  int ksc[KS], vsc[VS];
#pragma unroll
  for (int s = 0; s < KS; s++) { kf[s] = v8i{0, 0, 0, 0, 0, 0, 0, 0}; ksc[s] = 0; }
#pragma unroll
  for (int s = 0; s < VS; s++) { vf[s] = v8i{0, 0, 0, 0, 0, 0, 0, 0}; vsc[s] = 0; }
  if (live) {
    const int64_t row = (b * a.Hkv + kh) * a.N + kj;
#pragma unroll
    for (int s = 0; s < KS; s++) {
      kf[s] = frag_rows_global(a.k_code + row * DQK, s, hf);
      clear_channel(kf[s], s, hf, hot);
      ksc[s] = a.k_scale[row * (DQK / 32) + 2 * s + hf];
    }
#pragma unroll
    for (int s = 0; s < VS; s++) {
      vf[s] = frag_rows_global(a.v_code + row * DV, s, hf);
      vsc[s] = a.v_scale[row * (DV / 32) + 2 * s + hf];
    }
  }
  const float khot = (live && hot >= 0) ? row_value<DQK>(a.k_code, a.k_scale, (b * a.Hkv + kh) * a.N + kj, hot) : 0.f;
  // K col codes of the workgroup's keys (B operand of dQ), once
  stage_col_slice<DQK, BKB, KCST, NT>(sKc, sKcs, a.kc_code + (b * a.Hkv + kh) * (int64_t)DQK * a.N,
                                      a.kc_scale + (b * a.Hkv + kh) * (int64_t)DQK * (a.N / 32), kb0, a.N);

  v16f dk[CK], dv[CV];
#pragma unroll
  for (int c = 0; c < CK; c++)
#pragma unroll
    for (int r = 0; r < 16; r++) dk[c][r] = 0.f;
#pragma unroll
  for (int c = 0; c < CV; c++)
#pragma unroll
    for (int r = 0; r < 16; r++) dv[c][r] = 0.f;

  const int64_t nqt = (a.N + BQ - 1) / BQ;
  const int64_t qt0 = kb0 / BQ;
  for (int64_t hh = 0; hh < a.G; hh++) {
    const int64_t h = kh * a.G + hh;
    const int64_t bh = b * a.Hq + h;
    for (int64_t qt = qt0; qt < nqt; qt++) {
      const int64_t i0 = qt * BQ;
      __syncthreads();
      stage_rows<BQ, DQK, QST, NT>(sQ, sQs, a.q_code + bh * a.N * DQK, a.q_scale + bh * a.N * (DQK / 32), i0, a.N,
                                   hot);
      stage_rows<BQ, DV, OST, NT>(sO, sOs, a.do_code + bh * a.N * DV, a.do_scale + bh * a.N * (DV / 32), i0, a.N);
      stage_cols_perm<DQK, CST, NT>(sQc, sQcs, a.qc_code + bh * (int64_t)DQK * a.N,
                                    a.qc_scale + bh * (int64_t)DQK * (a.N / 32), i0, a.N);
      stage_cols_perm<DV, CST, NT>(sOc, sOcs, a.doc_code + bh * (int64_t)DV * a.N,
                                   a.doc_scale + bh * (int64_t)DV * (a.N / 32), i0, a.N);
      for (int u = threadIdx.x; u < BQ; u += NT) {
        const bool ok = i0 + u < a.N;
        sL[u] = ok ? a.lse[bh * a.N + i0 + u] * kLog2e : 0.f;
        sD[2 * u] = ok ? a.delta[(bh * a.N + i0 + u) * 2] : 0.f;
        sD[2 * u + 1] = ok ? a.delta[(bh * a.N + i0 + u) * 2 + 1] : 0.f;
        sQh[u] = (ok && hot >= 0) ? row_value<DQK>(a.q_code, a.q_scale, bh * a.N + i0 + u, hot) : 0.f;
      }
      __syncthreads();

      // this wave has work unless every query of the tile precedes its keys
      const bool work = live && (i0 + BQ - 1 >= kw0);
      const bool needmask = (i0 < kw0 + 31) || (i0 + BQ > a.N);
      uint32_t dsc_codes[2][4];
      int dse[2] = {-127, -127};
      if (work) {
        uint32_t pc[2][4];
#pragma unroll
        for (int qs = 0; qs < 2; qs++) {
          v16f s, dp;
#pragma unroll
          for (int r = 0; r < 16; r++) { s[r] = 0.f; dp[r] = 0.f; }
#pragma unroll
          for (int st = 0; st < KS; st++)
            s = mfma_mx(frag_rows<QST>(sQ, 32 * qs + li, st, hf), kf[st], s,
                        sQs[(32 * qs + li) * (DQK / 32) + 2 * st + hf], ksc[st]);
#pragma unroll
          for (int st = 0; st < VS; st++)
            dp = mfma_mx(frag_rows<OST>(sO, 32 * qs + li, st, hf), vf[st], dp,
                         sOs[(32 * qs + li) * (DV / 32) + 2 * st + hf], vsc[st]);
          // lane holds queries 32 qs + 8 g + 4 hf + e (accumulator r = 4 g + e)
          float P[16], dS[16];
          float amax = 0.f;
#pragma unroll
          for (int g = 0; g < 4; g++) {
            const int qo = 32 * qs + 8 * g + 4 * hf;
            const float4 Lg = *reinterpret_cast<const float4*>(&sL[qo]);
            const float4 d01 = *reinterpret_cast<const float4*>(&sD[2 * qo]);
            const float4 d23 = *reinterpret_cast<const float4*>(&sD[2 * qo + 4]);
            const float4 qh = *reinterpret_cast<const float4*>(&sQh[qo]);
            const float Qh[4] = {qh.x, qh.y, qh.z, qh.w};
            const float Lv[4] = {Lg.x, Lg.y, Lg.z, Lg.w};
            const float Hv[4] = {d01.x, d01.z, d23.x, d23.z};
            const float Lo[4] = {d01.y, d01.w, d23.y, d23.w};
#pragma unroll
            for (int e = 0; e < 4; e++) {
              const int r = 4 * g + e;
              float p = bwd_prob(__builtin_fmaf(Qh[e], khot, s[r]), a.c, Lv[e]);
              if (needmask) {
                const int64_t qi = i0 + qo + e;
                p = (kj > qi || qi >= a.N) ? 0.f : p;
              }
              P[r] = p;
              dS[r] = p * ((dp[r] - Hv[e]) - Lo[e]);
              amax = fmaxf(amax, fabsf(dS[r]));
            }
          }
#pragma unroll
          for (int k = 0; k < 4; k++)
            pc[qs][k] = cvt4_div(P[4 * k], P[4 * k + 1], P[4 * k + 2], P[4 * k + 3], 0.00390625f);
          int e = pow2_exponent(wave_max(amax));
          e = e < -126 ? -126 : e;
          const float sc = exp2i(e);
#pragma unroll
          for (int k = 0; k < 4; k++)
            dsc_codes[qs][k] = cvt4_div(dS[4 * k], dS[4 * k + 1], dS[4 * k + 2], dS[4 * k + 3], sc);
          dse[qs] = e;
          if constexpr (STATS) {
            // per query row: FP64 sums over this wave's 32 keys, then atomics
#pragma unroll
            for (int r = 0; r < 16; r++) {
              const float cast = fp8_value(dsc_codes[qs][r >> 2], r & 3) * sc;
              const double s0 = half_sum_d((double)dS[r]);
              const double s1 = half_sum_d((double)fabsf(dS[r]));
              const double s2 = half_sum_d((double)cast);
              const float mx = half_max(fabsf(dS[r]));
              const int64_t qi = i0 + 32 * qs + 8 * (r >> 2) + 4 * hf + (r & 3);
              if (li == 0 && qi < a.N) {
                double* st = a.rowstats + (bh * a.N + qi) * 4;
                atomicAdd(st + 0, s0);
                atomicAdd(st + 1, s1);
                atomicAdd(st + 2, s2);
                atomicMax(reinterpret_cast<unsigned long long*>(st + 3),
                          (unsigned long long)__double_as_longlong((double)mx));
              }
            }
          }
        }
        // dV += P'^T dO_col ; dK += dS'^T Q_col   (k = the 64 queries of the tile)
        const v8i pa = v8i{(int)pc[0][0], (int)pc[0][1], (int)pc[0][2], (int)pc[0][3],
                           (int)pc[1][0], (int)pc[1][1], (int)pc[1][2], (int)pc[1][3]};
        const v8i da = v8i{(int)dsc_codes[0][0], (int)dsc_codes[0][1], (int)dsc_codes[0][2], (int)dsc_codes[0][3],
                           (int)dsc_codes[1][0], (int)dsc_codes[1][1], (int)dsc_codes[1][2], (int)dsc_codes[1][3]};
        const int dascale = (hf ? dse[1] : dse[0]) + 127;
#pragma unroll
        for (int c = 0; c < CV; c++)
          dv[c] = mfma_mx(pa, frag_cols<CST>(sOc, 32 * c + li, hf), dv[c], 127 - 8, sOcs[(32 * c + li) * 2 + hf]);
#pragma unroll
        for (int c = 0; c < CK; c++)
          dk[c] = mfma_mx(da, frag_cols<CST>(sQc, 32 * c + li, hf), dk[c], dascale, sQcs[(32 * c + li) * 2 + hf]);
      } else {
#pragma unroll
        for (int qs = 0; qs < 2; qs++)
#pragma unroll
          for (int k = 0; k < 4; k++) dsc_codes[qs][k] = 0u;
      }
      // dS' codes to LDS: row = key (32 w + li), columns = the lane's queries
#pragma unroll
      for (int qs = 0; qs < 2; qs++)
#pragma unroll
        for (int g = 0; g < 4; g++)
          *reinterpret_cast<uint32_t*>(sdS + (32 * w + li) * DST + 32 * qs + 8 * g + 4 * hf) = dsc_codes[qs][g];
      if (lane == 0) {
        sdSs[w * 2] = (uint8_t)(dse[0] + 127);
        sdSs[w * 2 + 1] = (uint8_t)(dse[1] + 127);
      }
      __syncthreads();
      // dQ tile (64 queries x DQK) = dS'(64 x BKB) K_col(BKB x DQK): output
      // blocks m = qs * CK + c, distributed round-robin over the waves
      for (int m = w; m < 2 * CK; m += NWK) {
        const int qs = m / CK, c = m % CK;
        v16f acc;
#pragma unroll
        for (int r = 0; r < 16; r++) acc[r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < BKB / 64; ks++) {
          // A: rows = queries of sub-block qs, k = keys 64 ks .. 64 ks + 63 (natural order)
          const int i16 = lane & 15;
          const int qbase = 32 * qs + 16 * ((lane >> 4) & 1);
          int words[8];
#pragma unroll
          for (int part = 0; part < 4; part++) {
            const int kk = 64 * ks + 32 * (part >> 1) + 16 * hf + 8 * (part & 1);
            const uint8_t* addr = sdS + (kk + (i16 >> 1)) * DST + qbase + 8 * (i16 & 1);
            const v2i t = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                (__attribute__((address_space(3))) v2i*)(addr));
            words[2 * part] = t[0];
            words[2 * part + 1] = t[1];
          }
          const v8i af = v8i{words[0], words[1], words[2], words[3], words[4], words[5], words[6], words[7]};
          const int as = sdSs[(2 * ks + hf) * 2 + qs];
          acc = mfma_mx(af, frag_rows<KCST>(sKc, 32 * c + li, ks, hf), acc, as,
                        sKcs[(32 * c + li) * (BKB / 32) + 2 * ks + hf]);
        }
        // lane holds channel 32 c + li, queries 32 qs + 8 (r/4) + 4 hf + r % 4
        float* base = a.dq_acc + (b * a.N * a.Hq + h) * DQK + 32 * c + li;
#pragma unroll
        for (int r = 0; r < 16; r++) {
          const int64_t qi = i0 + 32 * qs + 8 * (r >> 2) + 4 * hf + (r & 3);
          if (qi < a.N) atomicAdd(base + qi * a.Hq * DQK, acc[r]);
        }
      }
    }
  }
  if (!live) return;
  // dK (times tau) and dV: lane holds channel 32 c + li, keys kw0 + 8 (r/4) + 4 hf + r % 4
#pragma unroll
  for (int r = 0; r < 16; r++) {
    const int64_t key = kw0 + 8 * (r >> 2) + 4 * hf + (r & 3);
    if (key >= a.N) continue;
    if (a.grad_bf16) {
      uint16_t* kd = reinterpret_cast<uint16_t*>(a.dk) + b * a.dks[0] + key * a.dks[1] + kh * a.dks[2];
      uint16_t* vd = reinterpret_cast<uint16_t*>(a.dv) + b * a.dvs[0] + key * a.dvs[1] + kh * a.dvs[2];
#pragma unroll
      for (int c = 0; c < CK; c++) kd[32 * c + li] = f32_to_bf16(dk[c][r] * a.tau);
#pragma unroll
      for (int c = 0; c < CV; c++) vd[32 * c + li] = f32_to_bf16(dv[c][r]);
    } else {
      float* kd = reinterpret_cast<float*>(a.dk) + b * a.dks[0] + key * a.dks[1] + kh * a.dks[2];
      float* vd = reinterpret_cast<float*>(a.dv) + b * a.dvs[0] + key * a.dvs[1] + kh * a.dvs[2];
#pragma unroll
      for (int c = 0; c < CK; c++) kd[32 * c + li] = dk[c][r] * a.tau;
#pragma unroll
      for (int c = 0; c < CV; c++) vd[32 * c + li] = dv[c][r];
    }
  }
}

template <int DQK, int DV>
static hipError_t bwd_dispatch(const AttnArgs& a, hipStream_t s) {
  constexpr int NWK = 4;
  const int64_t nkb = (a.N + 32 * NWK - 1) / (32 * NWK);
  dim3 grid((unsigned)nkb, (unsigned)a.Hkv, (unsigned)a.B);
  if (a.rowstats) hipLaunchKernelGGL((bwd_kernel<DQK, DV, NWK, true>), grid, dim3(64 * NWK), 0, s, a);
  else hipLaunchKernelGGL((bwd_kernel<DQK, DV, NWK, false>), grid, dim3(64 * NWK), 0, s, a);
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
