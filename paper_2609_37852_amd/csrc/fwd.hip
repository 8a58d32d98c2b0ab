// Forward pass (Sec. 2.3; App. B.6.2 with power-of-two probability scales).
//
// Workgroup: NW waves, 32 queries each, one (batch, query head).  Key tiles of
// BK = 128 are double-buffered in LDS (global loads for the next tile are in
// flight while the current one is computed; one barrier per tile) and visited
// from the causal diagonal down to key 0.
//
// Per wave and tile (4 aligned 32-key groups):
//   S^T = K Q^T       MX MFMA, A = K row tile (LDS), B = Q row codes (regs);
//                     lane l owns query l % 32 and holds 16 keys of each
//                     group, so row reductions are in-lane plus one exchange
//                     with lane l ^ 32.  The isolated score channel (if any)
//                     is added with one FMA.
//   M = integer running max of x = S tau log2e (ceil of the row max).  When it
//       grows, O and l are multiplied by 2^(M_old - M_new), an exact power of
//       two (decided per wave; at most a few times per row).
//   p = 2^(x - M) (FP32, before any cast) feeds l.
//   group g: E_g = smallest integer with 2^(x_g - M) <= 448 * 2^E_g (x_g the
//       group max), codes C8(p / 2^E_g) -- the group's probability scale.
//   O^T += V^T P^T    MX MFMA, A = V col tile (LDS, permuted to the lane's
//                     keys), B = probability codes straight from registers.
// Only the group holding the diagonal needs a mask; groups wholly in a wave's
// future skip their MFMA and exponentials.
// Epilogue: O = O_acc / l (bf16 or fp32), LSE = (M + log2 l) ln 2.
#include "common.hpp"
#include "kernels.hpp"
#include "tiles.hpp"

namespace afp8 {

constexpr float kLog2_448 = 8.807354922057604f;

template <int DQK, int DV, int NW>
struct FwdTile {
  static constexpr int BK = 128, NT = 64 * NW;
  static constexpr int KST = DQK + 16, VST = BK + 16;
  static constexpr int KU = BK * DQK / 16 / NT;   // uint4 of K codes per thread
  static constexpr int VU = DV * BK / 16 / NT;    // uint4 of V codes per thread
  static_assert(KU * NT * 16 == BK * DQK && VU * NT * 16 == DV * BK, "tile split");
  static_assert(DQK <= NT && DV <= NT && BK <= NT, "one scale word / hot value per thread");
};

// Registers holding one tile in flight from global memory.
template <int DQK, int DV, int NW>
struct FwdPrefetch {
  using T = FwdTile<DQK, DV, NW>;
  uint4 k[T::KU];
  uint4 v[T::VU];
  uint32_t ks;     // 4 K scale bytes (thread < DQK)
  uint32_t vs[4];  // V scale bytes of one channel, one per 32-key group (thread < DV)
  uint32_t khc, khs;  // isolated-channel code and scale byte of one key (thread < BK)
};
// Only loads are issued here; everything that needs the loaded values waits
// for fwd_store, so the loads stay in flight while the current tile is computed.

template <int DQK, int DV, int NW>
__device__ __forceinline__ void fwd_load(FwdPrefetch<DQK, DV, NW>& f, const uint8_t* kcode, const uint8_t* kscale,
                                         const uint8_t* vcode, const uint8_t* vscale, int j0, int N, int hot) {
  using T = FwdTile<DQK, DV, NW>;
  const int tid = threadIdx.x;
  // K rows [j0, j0 + BK): contiguous; rows past N read the last valid bytes
  // (finite codes whose scores the causal mask removes)
  const int klim = (N - j0) * DQK - 16;
#pragma unroll
  for (int i = 0; i < T::KU; i++) {
    const int off = (tid + i * T::NT) * 16;
    f.k[i] = *reinterpret_cast<const uint4*>(kcode + (size_t)j0 * DQK + (off < klim ? off : klim));
  }
  // V col rows: channel c, keys [j0, j0 + BK) in 16-byte pieces
#pragma unroll
  for (int i = 0; i < T::VU; i++) {
    const int u = tid + i * T::NT, c = u / (T::BK / 16), q = u % (T::BK / 16);
    const int col = j0 + q * 16 < N - 16 ? j0 + q * 16 : N - 16;
    f.v[i] = *reinterpret_cast<const uint4*>(vcode + (size_t)c * N + col);
  }
  if (tid < DQK) {  // K scales: BK rows x DQK/32 bytes = DQK dwords, clamped to the head's array
    const int off = j0 * (DQK / 32) + tid * 4, lim = N * (DQK / 32) - 4;
    f.ks = *reinterpret_cast<const uint32_t*>(kscale + (off < lim ? off : lim));
  }
  if (tid < DV) {   // V scales: 4 groups of channel tid
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const int grp = (j0 + 32 * g < N ? j0 + 32 * g : N - 32) / 32;
      f.vs[g] = vscale[tid * (N / 32) + grp];
    }
  }
  if (tid < T::BK && hot >= 0) {
    const int r = j0 + tid < N ? j0 + tid : N - 1;
    f.khc = kcode[r * DQK + hot];
    f.khs = kscale[r * (DQK / 32) + hot / 32];
  }
}

template <int DQK, int DV, int NW>
__device__ __forceinline__ void fwd_store(const FwdPrefetch<DQK, DV, NW>& f, uint8_t* sK, uint8_t* sKs, uint8_t* sV,
                                          uint8_t* sVs, float* sKh, int hot) {
  using T = FwdTile<DQK, DV, NW>;
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < T::KU; i++) {
    const int off = (tid + i * T::NT) * 16;
    const int r = off / DQK, c = off % DQK;
    uint4 val = f.k[i];
    if (hot >= c && hot < c + 16) clear_byte(val, hot - c);
    *reinterpret_cast<uint4*>(sK + r * T::KST + c) = val;
  }
#pragma unroll
  for (int i = 0; i < T::VU; i++) {
    const int u = tid + i * T::NT, c = u / (T::BK / 16), q = u % (T::BK / 16);
    // 16 keys 16q..16q+15: group q/2; within the group, 4-key chunks go to
    // position 16 * (chunk & 1) + 4 * (chunk >> 1) (see stage_cols_perm)
    // (32-bit stores: a 64-bit store of {x, z} would make the compiler pair
    // the registers right after the load and wait for it there)
    uint32_t* base = reinterpret_cast<uint32_t*>(sV + c * T::VST + (q >> 1) * 32 + (q & 1) * 8);
    base[0] = f.v[i].x;
    base[1] = f.v[i].z;
    base[4] = f.v[i].y;
    base[5] = f.v[i].w;
  }
  if (tid < DQK) *reinterpret_cast<uint32_t*>(sKs + tid * 4) = f.ks;
  if (tid < DV)
    *reinterpret_cast<uint32_t*>(sVs + tid * 4) = f.vs[0] | (f.vs[1] << 8) | (f.vs[2] << 16) | (f.vs[3] << 24);
  if (tid < T::BK) sKh[tid] = hot >= 0 ? scaled_value(f.khc, f.khs) : 0.f;
}

template <int DQK, int DV, int NW>
__global__ __launch_bounds__(64 * NW, 2) void fwd_kernel(AttnArgs a) {
  using T = FwdTile<DQK, DV, NW>;
  constexpr int BQ = 32 * NW, BK = T::BK;
  constexpr int KS = DQK / 64, CB = DV / 32;
  __shared__ __attribute__((aligned(16))) uint8_t sK[2][BK * T::KST];
  __shared__ __attribute__((aligned(16))) uint8_t sKs[2][BK * DQK / 32];
  __shared__ __attribute__((aligned(16))) uint8_t sV[2][DV * T::VST];
  __shared__ __attribute__((aligned(16))) uint8_t sVs[2][DV * 4];
  __shared__ __attribute__((aligned(16))) float sKh[2][BK];
  __shared__ int hot_slot;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hf = lane >> 5, li = lane & 31;
  const int N = (int)a.N;
  const int nqb = (N + BQ - 1) / BQ;
  const WgCoord wc = query_major_coord((int)blockIdx.x, (int)a.B, (int)a.Hq, (int)a.Hkv);
  const int qb = nqb - 1 - wc.r;              // longest causal rows first
  const int h = wc.h, b = wc.b, kh = h / (int)a.G;
  const int q0 = qb * BQ + 32 * w;
  const bool live = q0 < N;
  const int qi = q0 + li;
  const int hot = select_hot_channel<DQK>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, &hot_slot);

  const size_t bhq = (size_t)b * a.Hq + h, bhk = (size_t)b * a.Hkv + kh;
  const uint8_t* kcode = a.k_code + bhk * N * DQK;
  const uint8_t* kscale = a.k_scale + bhk * N * (DQK / 32);
  const uint8_t* vcode = a.vc_code + bhk * DV * N;
  const uint8_t* vscale = a.vc_scale + bhk * DV * (N / 32);

  v8i qf[KS];
  int qsc[KS];
  float qhot = 0.f;
  {
    const int row = live ? qi : 0;
    const uint8_t* qrow = a.q_code + (bhq * N + row) * DQK;
#pragma unroll
    for (int s = 0; s < KS; s++) {
      qf[s] = frag_rows_global(qrow, s, hf);
      clear_channel(qf[s], s, hf, hot);
      qsc[s] = a.q_scale[(bhq * N + row) * (DQK / 32) + 2 * s + hf];
    }
    if (hot >= 0) qhot = row_value<DQK>(a.q_code + bhq * N * DQK, a.q_scale + bhq * N * (DQK / 32), row, hot);
  }

  v16f oacc[CB];
#pragma unroll
  for (int cb = 0; cb < CB; cb++)
#pragma unroll
    for (int r = 0; r < 16; r++) oacc[cb][r] = 0.f;
  float M = -__builtin_inff();
  float lsum = 0.f;
  const float c = a.c;

  const int qend = (qb + 1) * BQ < N ? (qb + 1) * BQ : N;
  const int ntiles = (qend + BK - 1) / BK;
  FwdPrefetch<DQK, DV, NW> pf;
  fwd_load<DQK, DV, NW>(pf, kcode, kscale, vcode, vscale, (ntiles - 1) * BK, N, hot);
  fwd_store<DQK, DV, NW>(pf, sK[0], sKs[0], sV[0], sVs[0], sKh[0], hot);
  __syncthreads();

  for (int it = 0; it < ntiles; it++) {
    const int cur = it & 1;
    const int j0 = (ntiles - 1 - it) * BK;
    // always issue the next tile's loads (the last iteration reloads tile 0
    // into the idle buffer): a conditional load would merge old and new
    // register values after the branch and wait for the loads right there
    fwd_load<DQK, DV, NW>(pf, kcode, kscale, vcode, vscale, j0 >= BK ? j0 - BK : 0, N, hot);

    if (live && j0 <= q0) {
      const uint8_t* K = sK[cur];
      const uint8_t* Ks = sKs[cur];
      const float* Kh = sKh[cur];
      const uint8_t* V = sV[cur];
      const uint8_t* Vs = sVs[cur];
      // two 64-key halves, each: scores -> max -> rescale -> exponentials -> P V
#pragma unroll
      for (int hk = 0; hk < 2; hk++) {
        if (j0 + 64 * hk > q0) break;          // both groups of this half are in the wave's future
        v16f s[2];
        float gm[2];
#pragma unroll
        for (int g2 = 0; g2 < 2; g2++) {
          const int kb = 2 * hk + g2;
          const int g0 = j0 + 32 * kb;         // first key of the group
          if (g0 > q0) {                       // whole group in this wave's future
            gm[g2] = -__builtin_inff();
            continue;
          }
#pragma unroll
          for (int r = 0; r < 16; r++) s[g2][r] = 0.f;
#pragma unroll
          for (int st = 0; st < KS; st++)
            s[g2] = mfma_mx(frag_rows<T::KST>(K, 32 * kb + li, st, hf), qf[st], s[g2],
                            Ks[(32 * kb + li) * (DQK / 32) + 2 * st + hf], qsc[st]);
          float kh16[16];
#pragma unroll
          for (int g = 0; g < 4; g++) {
            const float4 v4 = *reinterpret_cast<const float4*>(&Kh[32 * kb + 8 * g + 4 * hf]);
            kh16[4 * g] = v4.x; kh16[4 * g + 1] = v4.y; kh16[4 * g + 2] = v4.z; kh16[4 * g + 3] = v4.w;
          }
          float m = -__builtin_inff();
          if (g0 == q0) {                      // the diagonal group: key offset > query offset is masked
#pragma unroll
            for (int r = 0; r < 16; r++) {
              const float t = __builtin_fmaf(qhot, kh16[r], s[g2][r]);
              s[g2][r] = (8 * (r >> 2) + 4 * hf + (r & 3)) > li ? -__builtin_inff() : t;
              m = fmaxf(m, s[g2][r]);
            }
          } else {
#pragma unroll
            for (int r = 0; r < 16; r++) {
              s[g2][r] = __builtin_fmaf(qhot, kh16[r], s[g2][r]);
              m = fmaxf(m, s[g2][r]);
            }
          }
          gm[g2] = m;
        }
        // full group maxima (raw score units) in every lane
        gm[0] = fmaxf(gm[0], partner(gm[0]));
        gm[1] = fmaxf(gm[1], partner(gm[1]));
        const float mnew = fmaxf(M, __builtin_ceilf(fmaxf(gm[0], gm[1]) * c));
        if (M == -__builtin_inff()) {
          M = mnew;                            // first visible keys: nothing accumulated yet
        } else if (__any(mnew > M)) {
          const int d = (int)(M - mnew);       // 0 for lanes whose max did not move
          const float alpha = d < -126 ? 0.f : exp2i(d);
          lsum *= alpha;
#pragma unroll
          for (int cb = 0; cb < CB; cb++)
#pragma unroll
            for (int r = 0; r < 16; r++) oacc[cb][r] *= alpha;
          M = mnew;
        }
        const float nM = -M;
        uint32_t codes[2][4];
        int eg[2];
#pragma unroll
        for (int g2 = 0; g2 < 2; g2++) {
          if (j0 + 32 * (2 * hk + g2) > q0) {
#pragma unroll
            for (int k = 0; k < 4; k++) codes[g2][k] = 0u;
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
          for (int k = 0; k < 4; k++) codes[g2][k] = cvt4_div(p[4 * k], p[4 * k + 1], p[4 * k + 2], p[4 * k + 3], sc);
        }
        const v8i pfr = v8i{(int)codes[0][0], (int)codes[0][1], (int)codes[0][2], (int)codes[0][3],
                            (int)codes[1][0], (int)codes[1][1], (int)codes[1][2], (int)codes[1][3]};
        const int psc = (hf ? eg[1] : eg[0]) + 127;
#pragma unroll
        for (int cb = 0; cb < CB; cb++) {
          const uint8_t* vp = V + (32 * cb + li) * T::VST + 64 * hk + 16 * hf;
          const uint4 lo = *reinterpret_cast<const uint4*>(vp);
          const uint4 hi = *reinterpret_cast<const uint4*>(vp + 32);
          const v8i vf = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
          oacc[cb] = mfma_mx(vf, pfr, oacc[cb], Vs[(32 * cb + li) * 4 + 2 * hk + hf], psc);
        }
      }
    }
    fwd_store<DQK, DV, NW>(pf, sK[cur ^ 1], sKs[cur ^ 1], sV[cur ^ 1], sVs[cur ^ 1], sKh[cur ^ 1], hot);
    __syncthreads();
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
  constexpr int NW = 4;
  const int64_t nqb = (a.N + 32 * NW - 1) / (32 * NW);
  const dim3 grid((unsigned)(nqb * a.Hq * a.B));
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
