// Forward pass (Sec. 2.3; App. B.6.2 with power-of-two probability scales).
//
// Workgroup: NW waves, 32 queries each, one (batch, query head).  Key tiles of
// BK = 128 keys (64 for wide heads without the mask; K row codes [BK][Dqk], V
// col codes [Dv][BK], their scales) reach
// LDS by direct loads, double-buffered: the next tile streams in while the
// current one is computed, one barrier per tile.  Tiles run from key 0 up to
// the causal diagonal (to the last key without the mask), so the workgroups
// of one KV head that run together read the same tiles.
//
// Per wave and tile (aligned 32-key groups, taken in 64-key halves):
//   S^T = K Q^T       MX MFMA, A = K row tile (LDS), B = Q row codes (regs);
//                     lane l owns query l % 32 and holds 16 keys of each
//                     group, so row reductions are in-lane plus one exchange
//                     with lane l ^ 32.  The isolated score channel (if any)
//                     is cleared in Q and its exact product added by one
//                     FP32 rank-1 MFMA update.
//   M = integer running reference for x = S tau log2e (ceil of the row max,
//       raised lazily).  When it is raised, O and l are multiplied by
//       2^(M_old - M_new), an exact power of two (decided per wave).
//   p = 2^(x - M) (FP32, before any cast) feeds l.
//   group g: E_g = smallest integer with 2^(x_g - M) <= 448 * 2^E_g (x_g the
//       group max), codes C8(p / 2^E_g) -- the group's probability scale.
//       Since M is an integer the codes equal C8(2^(x - E)) with E the
//       group's absolute exponent, whatever the running max was.
//   O^T += V^T P^T    MX MFMA, A = V col tile (LDS), B = probability codes
//                     from registers, put in natural key order by one
//                     v_permlane32_swap per dword pair.
// Only the group holding the diagonal needs a mask; groups wholly in a wave's
// future (causal) or past the last key skip their MFMA and exponentials.
// Epilogue: O = O_acc / l (bf16 or fp32), LSE = (M + log2 l) ln 2.
#include <type_traits>

#include "common.hpp"
#include "dma.hpp"
#include "kernels.hpp"
#include "tiles.hpp"

namespace afp8 {

constexpr float kLog2_448 = 8.807354922057604f;
// The reference M is raised only once some row's maximum exceeds it by more
// than this many powers of two: until then p = 2^(x - M) <= 2^16 simply
// accumulates larger, which FP32 holds exactly in range.  Rescales are exact
// powers of two and the codes do not depend on M, so O and l come out the
// same whenever the rescales happen.
constexpr float kLazyRescale = 16.0f;

// NH: isolated score channels (1, or 3 with ATTN_FP8_FLAG_ISOLATE3)
template <int DQK, int DV, int NH = 1, bool CAUSAL = true>
struct FwdCfg {
  static constexpr int NW = 4, NT = 64 * NW, BQ = 32 * NW;
  static constexpr int al16(int x) { return (x + 15) & ~15; }
  static constexpr int stage_bytes(int bk) {
    return al16(al16(bk * (DQK + DV) + bk * DQK / 32) + DV * 4) + bk * 4 * NH;
  }
  // Workgroups per CU.  At dv = 256 each wave holds 128 VGPRs of O
  // accumulators: with two workgroups (two waves a SIMD, 256 VGPRs each) the
  // causal kernel spilled inside its tile loop, and every spill reload waited
  // for the tile loads in flight, so it runs one workgroup per CU (no spills,
  // 128-key tiles: 0.53 against 0.61 ms on B = 2, N = 8192, 8 / 2 heads).
  // Without the mask it spills less and two workgroups stay faster (0.82
  // against 0.97 ms).
  static constexpr int WGS = CAUSAL && DV > 128 ? 1 : 2;
  // 128-key tiles where the double-buffered workgroups fit a CU's LDS (two
  // in 80 KB each, or one), else 64-key tiles (wide heads)
  static constexpr int BK = WGS == 1 || 2 * stage_bytes(128) <= 80 * 1024 ? 128 : 64;
  static constexpr int K_OFF = 0;                               // K row codes [BK][DQK], swizzled
  static constexpr int V_OFF = K_OFF + BK * DQK;                // V col codes [DV][BK], swizzled
  static constexpr int KS_OFF = V_OFF + DV * BK;                // K row scales [BK][DQK/32]
  static constexpr int VS_OFF = al16(KS_OFF + BK * DQK / 32);   // V col scales [DV][4] (BK/32 used)
  static constexpr int KH_OFF = al16(VS_OFF + DV * 4);          // isolated-channel key values [NH][BK] FP32
  static constexpr int STAGE = KH_OFF + BK * 4 * NH;
  static_assert(STAGE == stage_bytes(BK), "stage layout");
  static_assert(DV <= NT, "one V scale word per thread");
  static_assert(BQ % BK == 0, "a query block's diagonal starts a key tile");
  static_assert(WGS * 2 * STAGE <= 160 * 1024, "LDS of the forward");
};

// CAUSAL: the mask (key length = query length) or every key of Nk; a
// template parameter, so the causal kernel carries no key-length arithmetic.
// NH: isolated score channels; with 3, the first two share one rank-2 FP32
// MFMA (its two k slots) and the third takes a second one.
template <int DQK, int DV, bool CAUSAL, int NH = 1>
__global__ __launch_bounds__(256, (FwdCfg<DQK, DV, NH, CAUSAL>::WGS)) void fwd_kernel(AttnArgs a) {
  using C = FwdCfg<DQK, DV, NH, CAUSAL>;
  constexpr int NW = C::NW, BQ = C::BQ, BK = C::BK;
  constexpr int KS = DQK / 64, CB = DV / 32;
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
  // keys j0 .. visible to the wave's queries start groups before klim (a
  // multiple of 32): the diagonal group's end when causal, else the key length
  const int klim = causal ? q0 + 32 : L.k;
  int hots[NH];
  if constexpr (NH == 1) hots[0] = select_hot_channel<DQK>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, hot_slot);
  else select_hot_channels<DQK, NH>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, hot_slot, hots);
  const int hot = hots[0];

  const size_t bhq = (size_t)b * a.Hq + h, bhk = (size_t)b * a.Hkv + kh;
  const uint8_t* kcode = a.k_code + bhk * Nk * DQK;
  const uint8_t* kscale = a.k_scale + bhk * Nk * (DQK / 32);
  const uint8_t* vcode = a.vc_code + bhk * DV * Nk;
  const uint8_t* vscale = a.vc_scale + bhk * DV * (Nk / 32);

  v8i qf[KS];
  int qsc[KS];
  float qv = 0.f;     // B operand of the isolated channel's rank-1 update (lanes < 32)
  float qv2 = 0.f;    // NH = 3: qv holds channel 0 (lanes < 32) and 1 (lanes >= 32), qv2 channel 2
  {
    const size_t row = bhq * N + (live ? qi : 0);
#pragma unroll
    for (int s = 0; s < KS; s++) {
      qf[s] = frag_rows_global(a.q_code + row * DQK, s, hf);
      qsc[s] = a.q_scale[row * (DQK / 32) + 2 * s + hf];
#pragma unroll
      for (int i = 0; i < NH; i++) clear_channel(qf[s], s, hf, hots[i]);
    }
    if constexpr (NH == 1) {
      if (hot >= 0 && hf == 0) qv = row_value<DQK>(a.q_code, a.q_scale, (int64_t)row, hot);
    } else if (hot >= 0) {
      qv = row_value<DQK>(a.q_code, a.q_scale, (int64_t)row, hf ? hots[1] : hots[0]);
      if (hf == 0) qv2 = row_value<DQK>(a.q_code, a.q_scale, (int64_t)row, hots[2]);
    }
  }

  v16f oacc[CB];
#pragma unroll
  for (int cb = 0; cb < CB; cb++)
#pragma unroll
    for (int r = 0; r < 16; r++) oacc[cb][r] = 0.f;
  float M = -__builtin_inff();
  float lsum = 0.f;
  const float c = a.c;
  // key tiles up to the block's diagonal, or over all keys
  const int ktiles = (L.k + BK - 1) / BK;
  const int ntiles = causal && (qb + 1) * (BQ / BK) < ktiles ? (qb + 1) * (BQ / BK) : ktiles;

  // Loads of tile j0: codes and K scales straight to LDS; the V col scales
  // (4 strided bytes per channel) and the isolated-channel bytes of each key
  // through registers, written by finish().
  uint32_t vsr[BK / 32] = {};
  uint32_t khc[NH] = {}, khs[NH] = {};
  RowLoads<DQK, NW, BK> kload;
  ColLoads<DV, NW, BK> vload;
  kload.init(w, lane);
  vload.init(w, lane, Nk);
  auto issue = [&](lds8* st, int j0) __attribute__((always_inline)) {
    // keys past the sequence are clamped to its last ones (never the padding)
    kload.issue(st + C::K_OFF, kcode, j0, L.k, w, lane);
    vload.issue(st + C::V_OFF, vcode, j0, Nk, L.k, w, lane);
    dma_row_scales<DQK, NW, BK>(st + C::KS_OFF, kscale, j0, L.k, w, lane, 0);
    if (threadIdx.x < DV) {
#pragma unroll
      for (int g = 0; g < BK / 32; g++) {
        const int grp = (j0 + 32 * g < L.k ? j0 + 32 * g : L.k - 32) / 32;
        vsr[g] = vscale[threadIdx.x * (Nk / 32) + grp];
      }
    }
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
    if (threadIdx.x < DV) {
      if constexpr (BK == 128)
        *reinterpret_cast<uint32_t*>(st + C::VS_OFF + 4 * threadIdx.x) =
            vsr[0] | (vsr[1] << 8) | (vsr[2] << 16) | (vsr[3] << 24);
      else
        *reinterpret_cast<uint16_t*>(st + C::VS_OFF + 4 * threadIdx.x) = (uint16_t)(vsr[0] | (vsr[1] << 8));
    }
    if (threadIdx.x < BK) {
#pragma unroll
      for (int i = 0; i < NH; i++)
        reinterpret_cast<float*>(st + C::KH_OFF)[i * BK + threadIdx.x] = hot >= 0 ? scaled_value(khc[i], khs[i]) : 0.f;
    }
  };

  // FULL: every key of the tile is visible to every query of the wave (no
  // mask, no skipped group, no branch between groups, so one half's MFMAs
  // can overlap the other's vector work)
  auto tile_body = [&](const uint8_t* st, int j0, auto full_tag) __attribute__((always_inline)) {
    constexpr bool FULL = decltype(full_tag)::value;
    const uint8_t* K = st + C::K_OFF;
    const uint8_t* Ks = st + C::KS_OFF;
    const uint8_t* V = st + C::V_OFF;
    const uint8_t* Vs = st + C::VS_OFF;
    const float* Kh = reinterpret_cast<const float*>(st + C::KH_OFF);
#pragma unroll
    for (int hk = 0; hk < BK / 64; hk++) {
      if (!FULL && j0 + 64 * hk >= klim) break;   // both groups of this half are invisible
      v16f s[2];
      float gm[2];
#pragma unroll
      for (int g2 = 0; g2 < 2; g2++) {
        const int kb = 2 * hk + g2;
        const int g0 = j0 + 32 * kb;           // first key of the group
        if (!FULL && g0 >= klim) {             // whole group invisible to this wave
          gm[g2] = -__builtin_inff();
          continue;
        }
#pragma unroll
        for (int r = 0; r < 16; r++) s[g2][r] = 0.f;
#pragma unroll
        for (int t = 0; t < KS; t++)
          s[g2] = mfma_mx(frag_rows_swz<DQK>(K, 32 * kb + li, t, hf), qf[t], s[g2],
                          Ks[(32 * kb + li) * (DQK / 32) + 2 * t + hf], qsc[t]);
        // + k_c* q_c*: rank-1 update, A = isolated-channel key value
        // (lanes < 32), B = qv; lanes >= 32 contribute 0 * 0
        if constexpr (NH == 1) {
          if (hot >= 0) s[g2] = rank2_update(hf ? 0.f : Kh[32 * kb + li], qv, s[g2]);
        } else if (hot >= 0) {
          s[g2] = rank2_update(Kh[(hf ? BK : 0) + 32 * kb + li], qv, s[g2]);
          s[g2] = rank2_update(hf ? 0.f : Kh[2 * BK + 32 * kb + li], qv2, s[g2]);
        }
        // lane holds keys g0 + 8 (r/4) + 4 hf + r % 4 of query qi
        float m = -__builtin_inff();
        if (!FULL && causal && g0 == q0) {     // the diagonal group: keys after the query are masked
#pragma unroll
          for (int r = 0; r < 16; r++) {
            s[g2][r] = (8 * (r >> 2) + 4 * hf + (r & 3)) > li ? -__builtin_inff() : s[g2][r];
            m = fmaxf(m, s[g2][r]);
          }
        } else {
#pragma unroll
          for (int r = 0; r < 16; r++) m = fmaxf(m, s[g2][r]);
        }
        gm[g2] = m;
      }
      // full group maxima (raw score units) in every lane
      gm[0] = fmaxf(gm[0], partner(gm[0]));
      gm[1] = fmaxf(gm[1], partner(gm[1]));
      const float mnew = fmaxf(M, __builtin_ceilf(fmaxf(gm[0], gm[1]) * c));
      if (M == -__builtin_inff()) {
        M = mnew;                              // first visible keys: nothing accumulated yet
      } else if (__any(mnew > M + kLazyRescale)) {
        const int d = (int)(M - mnew);         // 0 for lanes whose max did not move
        const float alpha = d < -126 ? 0.f : exp2i(d);
        lsum *= alpha;
#pragma unroll
        for (int cb = 0; cb < CB; cb++)
#pragma unroll
          for (int r = 0; r < 16; r++) oacc[cb][r] *= alpha;
        M = mnew;
      }
      const float nM = -M;
      v4i codes[2];
      int eg[2];
#pragma unroll
      for (int g2 = 0; g2 < 2; g2++) {
        if (!FULL && j0 + 32 * (2 * hk + g2) >= klim) {
          codes[g2] = v4i{0, 0, 0, 0};
          eg[g2] = -126;
          continue;
        }
        // smallest E with 2^(x_g - M) <= 448 * 2^E, kept in the normal FP32 range
        int e = (int)__builtin_ceilf(__builtin_fmaf(gm[g2], c, nM) - kLog2_448);
        e = e < -126 ? -126 : e;
        eg[g2] = e;
        const float sc = exp2i(e);
        float p[16];
#pragma unroll
        for (int r = 0; r < 16; r++) {
          p[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[g2][r], c, nM));
          lsum += p[r];
        }
#pragma unroll
        for (int k = 0; k < 4; k++)
          codes[g2][k] = (int)cvt4_div(p[4 * k], p[4 * k + 1], p[4 * k + 2], p[4 * k + 3], sc);
        codes[g2] = to_natural4(codes[g2]);    // lane half hf: keys 16 hf .. 16 hf + 15 of the group
      }
      // B operand of the 64-key step: group 2 hk in bytes 0-15, group 2 hk + 1
      // in bytes 16-31; lane half hf carries the scale of group 2 hk + hf
      const v8i pfr = v8i{codes[0][0], codes[0][1], codes[0][2], codes[0][3],
                          codes[1][0], codes[1][1], codes[1][2], codes[1][3]};
      const int psc = (hf ? eg[1] : eg[0]) + 127;
#pragma unroll
      for (int cb = 0; cb < CB; cb++)
        oacc[cb] = mfma_mx(frag_rows_swz<BK>(V, 32 * cb + li, hk, hf), pfr, oacc[cb],
                           Vs[(32 * cb + li) * 4 + 2 * hk + hf], psc);
    }
  };
  auto tile = [&](const uint8_t* st, int j0) __attribute__((always_inline)) {
    if (!live || j0 >= klim) return;
    if constexpr (CAUSAL) {
      if (j0 + BK <= q0) tile_body(st, j0, std::true_type{});
      else tile_body(st, j0, std::false_type{});
    } else {
      // one body (its group tests pass on every tile but the last): the
      // second body of the masked kernel does not fit the registers here
      tile_body(st, j0, std::false_type{});
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
  if (!live) return;
  const float l = lsum + partner(lsum);
  const float inv = 1.0f / l;
  // lane (query qi, half hf) holds channels 32 cb + 8 (r/4) + 4 hf + r % 4
  if (a.o_bf16) {
    uint16_t* orow = reinterpret_cast<uint16_t*>(a.o) + b * a.os[0] + (int64_t)qi * a.os[1] + h * a.os[2];
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
    float* orow = reinterpret_cast<float*>(a.o) + b * a.os[0] + (int64_t)qi * a.os[1] + h * a.os[2];
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
  if (hf == 0) a.lse_out[bhq * N + qi] = (M + __builtin_amdgcn_logf(l)) * kLn2;
}

template <int DQK, int DV>
static hipError_t fwd_dispatch(const AttnArgs& a, hipStream_t s) {
  using C = FwdCfg<DQK, DV>;
  const int64_t nqb = (a.N + C::BQ - 1) / C::BQ;
  const dim3 grid((unsigned)(nqb * a.Hq * a.B));
  if (a.iso3) {
    if (a.causal) hipLaunchKernelGGL((fwd_kernel<DQK, DV, true, 3>), grid, dim3(C::NT), 0, s, a);
    else hipLaunchKernelGGL((fwd_kernel<DQK, DV, false, 3>), grid, dim3(C::NT), 0, s, a);
  } else {
    if (a.causal) hipLaunchKernelGGL((fwd_kernel<DQK, DV, true>), grid, dim3(C::NT), 0, s, a);
    else hipLaunchKernelGGL((fwd_kernel<DQK, DV, false>), grid, dim3(C::NT), 0, s, a);
  }
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
