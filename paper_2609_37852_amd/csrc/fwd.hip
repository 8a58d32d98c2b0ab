// Forward pass (Sec. 2.3; App. B.6.2 with power-of-two probability scales).
//
// Workgroup: NW waves, 32 queries each, one (batch, query head).  Key tiles of
// 64 are staged once in LDS and shared by the waves, visited from the causal
// diagonal down to key 0.
//
// Per wave and tile:
//   S^T = K Q^T       MX MFMA, A = K row tile (LDS), B = Q row codes (regs);
//                     lane l owns query l % 32 and holds 16 keys of each
//                     32-key half, so row reductions are in-lane plus one
//                     exchange with lane l ^ 32.
//   x = S * tau*log2e, masked keys -> -inf.
//   M = integer running max (ceil of the row max).  When it grows, O and l
//       are multiplied by 2^(M_old - M_new), an exact power of two.
//   p = 2^(x - M) (FP32, before any cast) feeds l.
//   per aligned 32-key group g: E_g = smallest integer with max_g p <= 448 * 2^E_g,
//       codes C8(p / 2^E_g) -- the group scale of the probability operand.
//   O^T += V^T P^T    MX MFMA, A = V col tile (LDS, permuted to the lane's
//                     keys), B = probability codes straight from registers.
// Epilogue: O = O_acc / l (bf16 or fp32), LSE = (M + log2 l) ln 2.
#include "common.hpp"
#include "kernels.hpp"
#include "tiles.hpp"

namespace afp8 {

template <int DQK, int DV, int NW>
__global__ __launch_bounds__(64 * NW) void fwd_kernel(AttnArgs a) {
  constexpr int BQ = 32 * NW, BK = 64;
  constexpr int KS = DQK / 64, CB = DV / 32;
  constexpr int KST = DQK + 16, VST = BK + 16;
  __shared__ __attribute__((aligned(16))) uint8_t sK[BK * KST];
  __shared__ __attribute__((aligned(16))) uint8_t sKs[BK * DQK / 32];
  __shared__ __attribute__((aligned(16))) uint8_t sV[DV * VST];
  __shared__ __attribute__((aligned(16))) uint8_t sVs[DV * 2];
  __shared__ __attribute__((aligned(16))) float sKh[BK];
  __shared__ int hot_slot;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hf = lane >> 5, li = lane & 31;
  const int64_t nqb = (a.N + BQ - 1) / BQ;
  const int64_t qb = nqb - 1 - (int64_t)blockIdx.x;  // longest causal rows first
  const int64_t h = blockIdx.y, b = blockIdx.z, kh = h / a.G;
  const int64_t q0 = qb * BQ + 32 * w;
  const bool live = q0 < a.N;
  const int64_t qi = q0 + li;
  const int hot = select_hot_channel<DQK>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, &hot_slot);

  v8i qf[KS];
  int qsc[KS];
#pragma unroll
  for (int s = 0; s < KS; s++) {
    qf[s] = v8i{0, 0, 0, 0, 0, 0, 0, 0};
    qsc[s] = 0;
  }
  if (live) {
    const int64_t row = (b * a.Hq + h) * a.N + qi;
#pragma unroll
    for (int s = 0; s < KS; s++) {
      qf[s] = frag_rows_global(a.q_code + row * DQK, s, hf);
      clear_channel(qf[s], s, hf, hot);
      qsc[s] = a.q_scale[row * (DQK / 32) + 2 * s + hf];
    }
  }
  // the isolated channel's query value (0 without isolation)
  const float qhot = (live && hot >= 0) ? row_value<DQK>(a.q_code, a.q_scale, (b * a.Hq + h) * a.N + qi, hot) : 0.f;

  v16f oacc[CB];
#pragma unroll
  for (int cb = 0; cb < CB; cb++)
#pragma unroll
    for (int r = 0; r < 16; r++) oacc[cb][r] = 0.f;
  float M = -__builtin_inff();
  float lsum = 0.f;

  const int64_t qend = ((qb + 1) * BQ < a.N) ? (qb + 1) * BQ : a.N;
  const int ntiles = (int)((qend + BK - 1) / BK);
  const uint8_t* kcode = a.k_code + (b * a.Hkv + kh) * a.N * DQK;
  const uint8_t* kscale = a.k_scale + (b * a.Hkv + kh) * a.N * (DQK / 32);
  const uint8_t* vcode = a.vc_code + (b * a.Hkv + kh) * (int64_t)DV * a.N;
  const uint8_t* vscale = a.vc_scale + (b * a.Hkv + kh) * (int64_t)DV * (a.N / 32);

  for (int t = ntiles - 1; t >= 0; t--) {
    const int64_t j0 = (int64_t)t * BK;
    __syncthreads();
    stage_rows<BK, DQK, KST, 64 * NW>(sK, sKs, kcode, kscale, j0, a.N, hot);
    stage_cols_perm<DV, VST, 64 * NW>(sV, sVs, vcode, vscale, j0, a.N);
    if (threadIdx.x < BK)
      sKh[threadIdx.x] = (hot >= 0 && j0 + threadIdx.x < a.N) ? row_value<DQK>(kcode, kscale, j0 + threadIdx.x, hot) : 0.f;
    __syncthreads();
    if (!live || j0 > q0) continue;  // every key of the tile is in this wave's future

    v16f s[2];
#pragma unroll
    for (int kb = 0; kb < 2; kb++) {
#pragma unroll
      for (int r = 0; r < 16; r++) s[kb][r] = 0.f;
#pragma unroll
      for (int st = 0; st < KS; st++) {
        const v8i kf = frag_rows<KST>(sK, 32 * kb + li, st, hf);
        const int ksc = sKs[(32 * kb + li) * (DQK / 32) + 2 * st + hf];
        s[kb] = mfma_mx(kf, qf[st], s[kb], ksc, qsc[st]);
      }
    }
    const bool diag = j0 + BK - 1 > q0;
    float gmax[2];
#pragma unroll
    for (int kb = 0; kb < 2; kb++) {
      float m = -__builtin_inff();
      float kh4[16];
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const float4 v4 = *reinterpret_cast<const float4*>(&sKh[32 * kb + 8 * g + 4 * hf]);
        kh4[4 * g] = v4.x; kh4[4 * g + 1] = v4.y; kh4[4 * g + 2] = v4.z; kh4[4 * g + 3] = v4.w;
      }
#pragma unroll
      for (int r = 0; r < 16; r++) {
        float x = __builtin_fmaf(qhot, kh4[r], s[kb][r]) * a.c;
        if (diag) {
          const int64_t key = j0 + 32 * kb + 8 * (r >> 2) + 4 * hf + (r & 3);
          x = key > qi ? -__builtin_inff() : x;
        }
        s[kb][r] = x;
        m = fmaxf(m, x);
      }
      gmax[kb] = m;
    }
    // full group maxima in every lane (two exchanges with lane l ^ 32)
    const Pair p1 = permlane32_swap(gmax[0], gmax[1]);
    const float gown = fmaxf(p1.lo, p1.hi);
    const Pair p2 = permlane32_swap(gown, gown);
    const float g0 = p2.lo, g1 = p2.hi;

    const float mnew = fmaxf(M, __builtin_ceilf(fmaxf(g0, g1)));
    if (mnew > M) {
      float alpha = 0.f;  // first visible tile: nothing accumulated yet
      if (M != -__builtin_inff()) {
        const int d = (int)(M - mnew);
        alpha = d < -126 ? 0.f : exp2i(d);
      }
      lsum *= alpha;
#pragma unroll
      for (int cb = 0; cb < CB; cb++)
#pragma unroll
        for (int r = 0; r < 16; r++) oacc[cb][r] *= alpha;
      M = mnew;
    }
    float ls = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; kb++)
#pragma unroll
      for (int r = 0; r < 16; r++) {
        const float p = __builtin_amdgcn_exp2f(s[kb][r] - M);
        s[kb][r] = p;
        ls += p;
      }
    lsum += ls;
    int e0 = pow2_exponent(__builtin_amdgcn_exp2f(g0 - M));
    int e1 = pow2_exponent(__builtin_amdgcn_exp2f(g1 - M));
    e0 = e0 < -126 ? -126 : e0;
    e1 = e1 < -126 ? -126 : e1;
    const float sc0 = exp2i(e0), sc1 = exp2i(e1);
    v8i pf;
#pragma unroll
    for (int k = 0; k < 4; k++) {
      pf[k] = (int)cvt4_div(s[0][4 * k], s[0][4 * k + 1], s[0][4 * k + 2], s[0][4 * k + 3], sc0);
      pf[4 + k] = (int)cvt4_div(s[1][4 * k], s[1][4 * k + 1], s[1][4 * k + 2], s[1][4 * k + 3], sc1);
    }
    const int psc = (hf ? e1 : e0) + 127;
#pragma unroll
    for (int cb = 0; cb < CB; cb++) {
      const v8i vf = frag_cols<VST>(sV, 32 * cb + li, hf);
      const int vsc = sVs[(32 * cb + li) * 2 + hf];
      oacc[cb] = mfma_mx(vf, pf, oacc[cb], vsc, psc);
    }
  }
  if (!live) return;
  const float l = lsum + partner(lsum);
  const float inv = 1.0f / l;
  // lane (query qi, half hf) holds channels 32 cb + 8 (r/4) + 4 hf + r % 4
  if (a.o_bf16) {
    uint16_t* orow = reinterpret_cast<uint16_t*>(a.o) + b * a.os[0] + qi * a.os[1] + h * a.os[2];
#pragma unroll
    for (int cb = 0; cb < CB; cb++)
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const int ch = 32 * cb + 8 * g + 4 * hf;
        uint2 v;
        v.x = (uint32_t)f32_to_bf16(oacc[cb][4 * g] * inv) | ((uint32_t)f32_to_bf16(oacc[cb][4 * g + 1] * inv) << 16);
        v.y = (uint32_t)f32_to_bf16(oacc[cb][4 * g + 2] * inv) | ((uint32_t)f32_to_bf16(oacc[cb][4 * g + 3] * inv) << 16);
        *reinterpret_cast<uint2*>(orow + ch) = v;
      }
  } else {
    float* orow = reinterpret_cast<float*>(a.o) + b * a.os[0] + qi * a.os[1] + h * a.os[2];
#pragma unroll
    for (int cb = 0; cb < CB; cb++)
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const int ch = 32 * cb + 8 * g + 4 * hf;
        *reinterpret_cast<float4*>(orow + ch) =
            make_float4(oacc[cb][4 * g] * inv, oacc[cb][4 * g + 1] * inv, oacc[cb][4 * g + 2] * inv,
                        oacc[cb][4 * g + 3] * inv);
      }
  }
  if (hf == 0) a.lse_out[(b * a.Hq + h) * a.N + qi] = (M + __builtin_amdgcn_logf(l)) * kLn2;
}

template <int DQK, int DV>
static hipError_t fwd_dispatch(const AttnArgs& a, hipStream_t s) {
  constexpr int NW = 4;
  const int64_t nqb = (a.N + 32 * NW - 1) / (32 * NW);
  dim3 grid((unsigned)nqb, (unsigned)a.Hq, (unsigned)a.B);
  hipLaunchKernelGGL((fwd_kernel<DQK, DV, NW>), grid, dim3(64 * NW), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_fwd(const AttnArgs& a, int dqk, int dv, hipStream_t s) {
  if (dqk == 64 && dv == 64) return fwd_dispatch<64, 64>(a, s);
  if (dqk == 128 && dv == 128) return fwd_dispatch<128, 128>(a, s);
  if (dqk == 256 && dv == 256) return fwd_dispatch<256, 256>(a, s);
  if (dqk == 192 && dv == 128) return fwd_dispatch<192, 128>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace afp8
