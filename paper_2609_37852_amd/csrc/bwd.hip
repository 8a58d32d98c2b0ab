// Backward pass, host side and the passes around the main kernel (Sec. 2.3;
// App. B.6.3): the preparation kernel that packs the per-query values and
// col scales the main kernel streams, the query-major dQ pass over the stored
// dS' units, and the launch sequencing.  The main kernel is in bwd_main.hpp.
#include "bwd_main.hpp"

namespace afp8 {

// Query-side data the tile loop streams besides the code tiles:
//   rows    [B, Hq, ceil(N/64)] x 1 KB: per 64-query tile, the pairs
//           {isolated-channel query value, -LSE / tau} of its queries (8 B
//           each), then -delta_hi of each (4 B; delta rounded to FP32), then
//           -delta_lo (4 B; read by the compensated formation), zero past the
//           end of the sequence;
//   tile_cs [B, Hq, ceil(N/64)] x 2 (Dqk + Dv) B: for each 64-query tile, the
//           col-copy scales of Q then dO for the tile's two 32-query groups
//           ([channel][group]), the second clamped to the first past the end;
//   tile_kcs [B, Hkv, ceil(Nk/64)] x 2 Dqk B: the same for K per 64-key step
//           (dq_kernel).
// Workgroup x covers the PT = 4 tiles of queries and keys 64 PT x ..
// 64 PT x + 64 PT - 1 (any may lie past its sequence; "the end" is the
// sequence's own length, the layouts have N and Nk rows), with one
// isolated-channel choice per workgroup, made once every load that does not
// depend on it is in flight.
constexpr int kPrepTiles = 4;
template <int DQK, int DV>
__global__ __launch_bounds__(256) void bwd_prep_kernel(AttnArgs a) {
  constexpr int PT = kPrepTiles;
  static_assert(PT * 64 == 256, "one query per thread");
  __shared__ int hot_slot;
  const int N = (int)a.N, Nk = (int)a.Nk;
  const int h = blockIdx.y, b = blockIdx.z, kh = h / (int)a.G;
  const SeqLens L = a.causal ? seq_lens<true>(a, b, N, Nk) : seq_lens<false>(a, b, N, Nk);
  const size_t bh = (size_t)b * a.Hq + h;
  const int x0 = blockIdx.x * PT, t = threadIdx.x;
  const int nq = (N + 63) / 64, nk = (Nk + 63) / 64;
  // every load that does not depend on the isolated channel is issued before
  // its choice (which ends in a barrier)
  // records: thread t holds query t % 64 of tile x0 + t / 64
  const int xr = x0 + t / 64, r = t % 64, i = 64 * xr + r;
  const bool rec = xr < nq, inseq = rec && i < L.q;
  const size_t row = bh * N + (inseq ? i : 0);
  float2 d = make_float2(0.f, 0.f);
  float lse = 0.f;
  if (inseq) {
    d = *reinterpret_cast<const float2*>(a.delta + row * 2);
    lse = a.lse[row];
  }
  // col scales of Q and dO for the tiles' two 32-query groups: where all PT
  // tiles lie inside the sequence, one 8-byte load per channel (its 2 PT
  // consecutive groups), else one byte at a time
  constexpr int NU = (DQK + DV + 255) / 256;
  uint8_t v[NU][PT][2];
  const bool whole = 64 * (x0 + PT) <= L.q && (N / 32) % (2 * PT) == 0;
#pragma unroll
  for (int k = 0; k < NU; k++) {
    const int u = t + 256 * k;
    if (u >= DQK + DV) continue;
    const uint8_t* src = u < DQK ? a.qc_scale + (bh * DQK + u) * (N / 32)
                                 : a.doc_scale + (bh * DV + (u - DQK)) * (N / 32);
    if (whole) {
      const uint2 w = *reinterpret_cast<const uint2*>(src + 2 * x0);
#pragma unroll
      for (int j = 0; j < PT; j++) {
        const uint32_t q = j < 2 ? w.x : w.y;
        v[k][j][0] = (uint8_t)(q >> (16 * (j & 1)));
        v[k][j][1] = (uint8_t)(q >> (16 * (j & 1) + 8));
      }
      continue;
    }
#pragma unroll
    for (int j = 0; j < PT; j++) {
      const int i0 = 64 * (x0 + j);
      if (i0 < L.q) {
        const int g0 = i0 / 32, g1 = (i0 + 32 < L.q ? i0 + 32 : i0) / 32;
        v[k][j][0] = src[g0];
        v[k][j][1] = src[g1];
      }
    }
  }
  // the K col scales of keys 64 (x0 + j) .., once per KV head (for dq_kernel)
  constexpr int NK = (DQK + 255) / 256;
  uint8_t kv[NK][PT][2];
  const size_t bk = (size_t)b * a.Hkv + (h < a.Hkv ? h : 0);
  if (h < a.Hkv) {
    const bool kwhole = 64 * (x0 + PT) <= L.k && (Nk / 32) % (2 * PT) == 0;
#pragma unroll
    for (int k = 0; k < NK; k++) {
      const int u = t + 256 * k;
      if (u >= DQK) continue;
      const uint8_t* src = a.kc_scale + (bk * DQK + u) * (Nk / 32);
      if (kwhole) {
        const uint2 w = *reinterpret_cast<const uint2*>(src + 2 * x0);
#pragma unroll
        for (int j = 0; j < PT; j++) {
          const uint32_t q = j < 2 ? w.x : w.y;
          kv[k][j][0] = (uint8_t)(q >> (16 * (j & 1)));
          kv[k][j][1] = (uint8_t)(q >> (16 * (j & 1) + 8));
        }
        continue;
      }
#pragma unroll
      for (int j = 0; j < PT; j++) {
        const int i0 = 64 * (x0 + j);
        if (i0 < L.k) {
          const int g0 = i0 / 32, g1 = (i0 + 32 < L.k ? i0 + 32 : i0) / 32;
          kv[k][j][0] = src[g0];
          kv[k][j][1] = src[g1];
        }
      }
    }
  }

  const int hot = select_hot_channel<DQK>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, &hot_slot);
  if (rec) {
    uint8_t* blk = reinterpret_cast<uint8_t*>(a.rows) + (bh * nq + xr) * 1024;
    float2 pr = make_float2(0.f, 0.f);
    if (inseq) {
      const float qh = hot >= 0 ? row_value<DQK>(a.q_code, a.q_scale, (int64_t)row, hot) : 0.f;
      pr = make_float2(qh, neg_lse_over_tau(lse, a.tau));
    }
    reinterpret_cast<float2*>(blk)[r] = pr;
    reinterpret_cast<float*>(blk + 512)[r] = inseq ? -d.x : 0.f;
    reinterpret_cast<float*>(blk + 768)[r] = inseq ? -d.y : 0.f;
  }
#pragma unroll
  for (int k = 0; k < NU; k++) {
    const int u = t + 256 * k;
#pragma unroll
    for (int j = 0; j < PT; j++) {
      if (u < DQK + DV && 64 * (x0 + j) < L.q) {
        uint8_t* dst = a.tile_cs + (bh * nq + x0 + j) * (2 * (DQK + DV));
        *reinterpret_cast<uint16_t*>(dst + 2 * u) = (uint16_t)(v[k][j][0] | (v[k][j][1] << 8));
      }
    }
  }
  if (h < a.Hkv) {
#pragma unroll
    for (int k = 0; k < NK; k++) {
      const int u = t + 256 * k;
#pragma unroll
      for (int j = 0; j < PT; j++) {
        if (u < DQK && 64 * (x0 + j) < L.k) {
          uint8_t* dk = a.tile_kcs + (bk * nk + x0 + j) * (2 * DQK);
          *reinterpret_cast<uint16_t*>(dk + 2 * u) = (uint16_t)(kv[k][j][0] | (kv[k][j][1] << 8));
        }
      }
    }
  }
}

// dQ = tau dS' K_col, query-major: a workgroup of 4 waves owns 128 queries
// of one (batch, query head), wave w one 32-query block and all Dqk channels
// (small workgroups: several per CU keep more unit loads in flight).
// The keys are taken SB 64-key steps at a time between two barriers: per
// 64-key step up to the diagonal (over all keys without the mask) the A
// operand is the stored unit (32 bytes per lane in operand order, as two
// 1 KB halves, loaded into registers during the previous interval); the K col
// tile of the step [Dqk][64] and its scales reach LDS by direct loads,
// double-buffered and shared by the 4 waves.  Every barrier waits for all
// loads in flight, so the loads of a wave between two barriers are what
// hides the memory latency: SB steps of them per interval.  Keys past the
// sequence meet zero dS' codes (their K loads are clamped to the sequence's
// last keys).
template <int DQK>
__global__ __launch_bounds__(256, DQK <= 128 ? 4 : 1) void dq_kernel(AttnArgs a) {
  constexpr int CQ = DQK / 32, NW = 4, SB = 2;
  constexpr int KT = DQK * 64, KSB = 2 * DQK;       // K tile and scale bytes per step
  constexpr int KST = KT + KSB;
  __shared__ __attribute__((aligned(16))) uint8_t kA[SB * KST];
  __shared__ __attribute__((aligned(16))) uint8_t kB[SB * KST];
  const int lane = threadIdx.x & 63, w = wave_id(), hf = lane >> 5, li = lane & 31;
  const int N = (int)a.N, Nk = (int)a.Nk, nqb = N / 32;
  const bool causal = a.causal != 0;
  const int nks = (Nk + 63) / 64;                    // 64-key steps over the keys (unit layout)
  const int ntile = (nqb + NW - 1) / NW;
  const WgCoord wc = query_major_coord((int)blockIdx.x, (int)a.B, (int)a.Hq, (int)a.Hkv, a.lens_q != nullptr);
  const int tile = ntile - 1 - wc.r;                 // longest rows first
  const int h = wc.h, b = wc.b, kh = h / (int)a.G;
  // the sequence's own lengths bound the work
  const SeqLens L = causal ? seq_lens<true>(a, b, N, Nk) : seq_lens<false>(a, b, N, Nk);
  const int nqs = L.q / 32, nkss = (L.k + 63) / 64;
  if (NW * tile >= nqs) return;                      // the whole tile is past the sequence
  const int qb = NW * tile + w;                      // this wave's 32-query block
  const int qlast = NW * tile + NW - 1 < nqs - 1 ? NW * tile + NW - 1 : nqs - 1;
  const int nk = qb < nqs ? (causal ? qb / 2 + 1 : nkss) : 0;   // this wave's 64-key steps
  const int nkw = causal ? qlast / 2 + 1 : nkss;                 // the workgroup's
  const int64_t bh = (int64_t)b * a.Hq + h;
  const int64_t unit0 = bh * units_before(nqb, nks, causal) + units_before(qb < nqs ? qb : 0, nks, causal);
  const uint8_t* units = a.ds_units + unit0 * 2048 + 16 * lane;
  const uint8_t* ex = a.ds_exp + unit0 * 2;
  const int64_t bk = (int64_t)b * a.Hkv + kh;
  const uint8_t* kc = a.kc_code + bk * DQK * Nk;
  const uint8_t* tk = a.tile_kcs + bk * nks * KSB;

  const Buf tkb = make_buf(tk, (uint32_t)nks * KSB);
  // K col tiles and scales of steps ks0 .. ks0 + SB - 1 (those before nkw)
  auto issue = [&](lds8* dst, int ks0) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < SB; s++) {
      const int ks = ks0 + s;
      if (ks >= nkw) break;
      dma_cols<DQK, NW>(dst + s * KST, kc, 64 * ks, Nk, L.k, w, lane);
      constexpr int NI = (KSB + 255) / 256;
      for (int k = 0; k < NI; k++) {
        if ((NW - 1 - k) != w) continue;
        const int off = 256 * k + 4 * lane;
        if (off < KSB) dma4(tkb, (uint32_t)(ks * KSB + off), dst + s * KST + KT + 256 * k);
      }
    }
  };
  struct Aop { uint4 lo, hi; uint32_t e; };
  // the wave's units of steps ks0 .. ks0 + SB - 1 (those before nk)
  auto load_a = [&](Aop (&op)[SB], int ks0) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < SB; s++) {
      const int ks = ks0 + s;
      if (ks >= nk) break;
      // read once: streamed past the caches, which keep the K tiles
      const v4i lo = __builtin_nontemporal_load(reinterpret_cast<const v4i*>(units + ks * 2048));
      const v4i hi = __builtin_nontemporal_load(reinterpret_cast<const v4i*>(units + ks * 2048 + 1024));
      op[s].lo = make_uint4((uint32_t)lo[0], (uint32_t)lo[1], (uint32_t)lo[2], (uint32_t)lo[3]);
      op[s].hi = make_uint4((uint32_t)hi[0], (uint32_t)hi[1], (uint32_t)hi[2], (uint32_t)hi[3]);
      op[s].e = ex[2 * ks + hf];
    }
  };
  v16f acc[CQ];
#pragma unroll
  for (int i = 0; i < CQ; i++)
#pragma unroll
    for (int r = 0; r < 16; r++) acc[i][r] = 0.f;
  auto compute = [&](const uint8_t* kt0, const Aop (&op)[SB], int ks0) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < SB; s++) {
      if (ks0 + s >= nk) break;
      const uint8_t* kt = kt0 + s * KST;
      const v8i af = v8i{(int)op[s].lo.x, (int)op[s].lo.y, (int)op[s].lo.z, (int)op[s].lo.w,
                         (int)op[s].hi.x, (int)op[s].hi.y, (int)op[s].hi.z, (int)op[s].hi.w};
#pragma unroll
      for (int i = 0; i < CQ; i++) {
        const int ch = 32 * i + li;
        acc[i] = mfma_mx(af, frag_cols_swz(kt, ch, hf), acc[i], (int)op[s].e, kt[KT + 2 * ch + hf]);
      }
    }
  };
  // one register set: the units of the next interval are loaded after the
  // MFMAs that read the current ones (the loads are in flight across the
  // barrier wait, which the short MFMA work barely shortens)
  Aop op[SB];
  load_a(op, 0);
  issue((lds8*)kA, 0);
  lds_barrier();
  for (int ks = 0; ks < nkw; ks += 2 * SB) {
    if (ks + SB < nkw) issue((lds8*)kB, ks + SB);
    compute(kA, op, ks);
    load_a(op, ks + SB);
    lds_barrier();
    if (ks + SB >= nkw) break;
    if (ks + 2 * SB < nkw) issue((lds8*)kA, ks + 2 * SB);
    compute(kB, op, ks + SB);
    load_a(op, ks + 2 * SB);
    lds_barrier();
  }
  if (qb >= nqs) return;
  // lane holds channel 32 i + li, queries 32 qb + 8 (r/4) + 4 hf + r % 4
#pragma unroll
  for (int r = 0; r < 16; r++) {
    const int q = 32 * qb + 8 * (r >> 2) + 4 * hf + (r & 3);
    if (a.grad_bf16) {
      uint16_t* d = reinterpret_cast<uint16_t*>(a.dq) + b * a.dqs[0] + (int64_t)q * a.dqs[1] + h * a.dqs[2];
#pragma unroll
      for (int i = 0; i < CQ; i++) d[32 * i + li] = f32_to_bf16(acc[i][r] * a.tau);
    } else {
      float* d = reinterpret_cast<float*>(a.dq) + b * a.dqs[0] + (int64_t)q * a.dqs[1] + h * a.dqs[2];
#pragma unroll
      for (int i = 0; i < CQ; i++) d[32 * i + li] = acc[i][r] * a.tau;
    }
  }
}

// BF16 copies of dO and V for the protected-dP backward: x [B, N, H, D] of
// FP32 or BF16 with element strides {sb, sn, sh} -> out [B, H, N, D] BF16
// (round to nearest even), head-major like the FP8 row copies.  A thread
// converts 8 channels (one 16-byte store); rows past a sequence's length
// (lens, clamped and rounded down as in seq_lens) are not read.
template <typename T>
__global__ __launch_bounds__(256) void pack_bf16_kernel(const T* x, int64_t sb, int64_t sn, int64_t sh, int64_t B,
                                                        int64_t N, int64_t H, int D, const int32_t* lens,
                                                        uint16_t* out) {
  const int64_t c8n = D / 8, total = B * N * H * c8n;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int64_t c8 = i % c8n, r = i / c8n, h = r % H, n = (r / H) % N, b = r / (H * N);
    if (lens) {
      const int64_t v = lens[b];
      if (n >= ((v < 0 ? 0 : v > N ? N : v) & ~int64_t(31))) continue;
    }
    const T* src = x + b * sb + n * sn + h * sh + 8 * c8;
    uint32_t w[4];
    if constexpr (sizeof(T) == 2) {
      const uint4 u = *reinterpret_cast<const uint4*>(src);
      w[0] = u.x; w[1] = u.y; w[2] = u.z; w[3] = u.w;
    } else {
      const float4 f0 = reinterpret_cast<const float4*>(src)[0], f1 = reinterpret_cast<const float4*>(src)[1];
      const float f[8] = {f0.x, f0.y, f0.z, f0.w, f1.x, f1.y, f1.z, f1.w};
#pragma unroll
      for (int k = 0; k < 4; k++)
        w[k] = (uint32_t)f32_to_bf16(f[2 * k]) | ((uint32_t)f32_to_bf16(f[2 * k + 1]) << 16);
    }
    *reinterpret_cast<uint4*>(out + ((b * H + h) * N + n) * D + 8 * c8) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

hipError_t launch_pack_bf16(const void* x, int bf16, const int64_t st[3], int64_t B, int64_t N, int64_t H, int D,
                            const int32_t* lens, uint16_t* out, hipStream_t s) {
  const int64_t total = B * N * H * (D / 8);
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks == 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(pack_bf16_kernel<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, s,
                       reinterpret_cast<const uint16_t*>(x), st[0], st[1], st[2], B, N, H, D, lens, out);
  else
    hipLaunchKernelGGL(pack_bf16_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, s,
                       reinterpret_cast<const float*>(x), st[0], st[1], st[2], B, N, H, D, lens, out);
  return hipGetLastError();
}

hipError_t launch_dq(const AttnArgs& a, int dqk, hipStream_t s) {
  const dim3 grid((unsigned)((a.N / 32 + 3) / 4 * a.Hq * a.B));
  switch (dqk) {
    case 64: hipLaunchKernelGGL((dq_kernel<64>), grid, dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL((dq_kernel<128>), grid, dim3(256), 0, s, a); break;
    case 192: hipLaunchKernelGGL((dq_kernel<192>), grid, dim3(256), 0, s, a); break;
    case 256: hipLaunchKernelGGL((dq_kernel<256>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

int64_t dq_units_per_head(int64_t nq, int64_t nk, bool causal) { return units_before(nq / 32, (nk + 63) / 64, causal); }

template <int DQK, int DV>
static hipError_t bwd_dispatch(const AttnArgs& a0, hipStream_t s) {
  using C = BwdCfg<DQK, DV>;
  const int64_t nkb = (a0.Nk + C::BKB - 1) / C::BKB;
  const dim3 grid((unsigned)(nkb * a0.Hkv * a0.B));
  // workgroups of one KV head that run at once: one per compute unit (the
  // kernel's LDS allows one), the units shared by the B Hkv heads
  static int cu_count[64];   // per device, queried once
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  int cus = __atomic_load_n(&cu_count[dev], __ATOMIC_RELAXED);
  if (cus <= 0) {
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      return hipErrorInvalidDevice;
    __atomic_store_n(&cu_count[dev], cus, __ATOMIC_RELAXED);
  }
  AttnArgs a = a0;
  const int64_t per_head = cus / (a.B * a.Hkv);
  a.bwd_cohort = (int)(per_head > 1 ? per_head : 1);
  if (a.pdp) return a.causal ? launch_bwd_main<true, 4>(a, DQK, DV, grid, s) : launch_bwd_main<false, 4>(a, DQK, DV, grid, s);
  if (a.iso3) return a.causal ? launch_bwd_main<true, 8>(a, DQK, DV, grid, s) : launch_bwd_main<false, 8>(a, DQK, DV, grid, s);
  switch ((a.causal ? 4 : 0) | (a.pmx ? 2 : 0) | (a.comp ? 1 : 0)) {
    case 0: return launch_bwd_main<false, 0>(a, DQK, DV, grid, s);
    case 1: return launch_bwd_main<false, 1>(a, DQK, DV, grid, s);
    case 2: return launch_bwd_main<false, 2>(a, DQK, DV, grid, s);
    case 3: return launch_bwd_main<false, 3>(a, DQK, DV, grid, s);
    case 4: return launch_bwd_main<true, 0>(a, DQK, DV, grid, s);
    case 5: return launch_bwd_main<true, 1>(a, DQK, DV, grid, s);
    case 6: return launch_bwd_main<true, 2>(a, DQK, DV, grid, s);
    default: return launch_bwd_main<true, 3>(a, DQK, DV, grid, s);
  }
}

hipError_t launch_bwd_prep(const AttnArgs& a, int dqk, int dv, hipStream_t s) {
  const int64_t L = a.N > a.Nk ? a.N : a.Nk;
  const dim3 grid((unsigned)(((L + 63) / 64 + kPrepTiles - 1) / kPrepTiles), (unsigned)a.Hq, (unsigned)a.B);
  if (dqk == 64 && dv == 64) hipLaunchKernelGGL((bwd_prep_kernel<64, 64>), grid, dim3(256), 0, s, a);
  else if (dqk == 128 && dv == 128) hipLaunchKernelGGL((bwd_prep_kernel<128, 128>), grid, dim3(256), 0, s, a);
  else if (dqk == 256 && dv == 256) hipLaunchKernelGGL((bwd_prep_kernel<256, 256>), grid, dim3(256), 0, s, a);
  else if (dqk == 192 && dv == 128) hipLaunchKernelGGL((bwd_prep_kernel<192, 128>), grid, dim3(256), 0, s, a);
  else return hipErrorInvalidValue;
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
