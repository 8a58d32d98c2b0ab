// Backward pass (Sec. 2.3; App. B.6.3 with power-of-two casts).
//
// Key-major: a workgroup owns BKB = 32*NWK keys of one (batch, KV head); wave
// w owns keys 32w..32w+31 of them.  The workgroup loops over the query heads
// of the KV group and over 64-query tiles from the causal diagonal (the first
// tile, without the mask) to the end of the sequence.  dK and dV for its keys stay in MFMA accumulators (FP32)
// across the whole loop, which is the GQA group sum.
//
// Query tiles reach LDS by direct global->LDS loads (no registers): while
// tile t is computed, tile t+1 streams into the other stage buffer.  Tile
// layouts are unpadded with an XOR swizzle of the 16-byte chunks, chosen so
// that the 16-byte fragment reads of 16 consecutive lanes hit distinct banks.
//
// Per wave, tile and 32-query sub-block qs (near the diagonal a sub-block is
// skipped when it lies wholly before the wave's keys or past the sequence,
// and masked when it holds them; tiles wholly after the workgroup's keys, or
// any tile inside both sequences without the mask, take a path without
// either):
//   S  = Q K^T, dP = dO V^T   MX MFMA (A = Q / dO row tiles in LDS, B = the
//                             wave's K / V row codes in registers); lane l
//                             owns key l % 32 and holds 16 queries.
//   S' = S + q_c* k_c* - LSE / tau by one FP32 rank-2 MFMA (the per-query
//        values come from the records);
//   P  = bwd_prob(S') = 2^(tau log2e S'), dS = fma(P, dP, fl(P (-delta))):
//        P dP enters exactly and every rounding is of its own element.  (The
//        shift dP - delta taken first, as the definition reads, rounds every
//        dP of one binade by the same amount, since they share one FP32
//        grid; on long flat rows those equal errors add up, weighted by P,
//        to more than the row's whole zero-sum budget.)  COMP (compensated
//        formation): the rounding error of fl(P (-delta_hi)), recovered
//        exactly by an fma, and P (-delta_lo) are added back, so the error of
//        dS scales with dS itself rather than with P |dP|.
//   P' = C8(256 P) with scale 2^-8 (PMX: C8(P / 2^ep), one exponent ep per
//        aligned 32x32 block from its largest P);  dS' = C8(dS / 2^e) with one
//        exponent e per aligned 32x32 block (the wave's 32 keys x 32 queries).
//   dV += P'^T dO_col,  dK += dS'^T Q_col   (A = the codes after one
//                             v_permlane32_swap per dword pair puts each
//                             lane's 16 queries in natural order).
// dQ: every wave writes its dS' codes to LDS ([key][query]); after the
// tile's barrier, at the start of the next iteration, the waves read them
// back with the 8-bit LDS transpose read as the A operands of dQ = dS' K_col
// (32 queries x 64 keys each, the "units") and store those to HBM, in the
// register order of the MFMA operand, with their two block exponents (the
// paper also stores FP8 dS between passes).  dq_kernel then computes
// dQ = tau dS' K_col query-major, without atomics.
//
// A preparation kernel packs what the tile loop needs besides the code tiles
// into arrays it can stream with the same direct loads: per 64-query tile a
// 1 KB block of per-query values (the pair {isolated-channel query value,
// -LSE / tau} at 8 q, the A operands of the score's rank-2 update, a lane of
// half hf reading the value at 8 q + 4 hf; -delta_hi at 512 + 4 q,
// -delta_lo at 768 + 4 q) and the col-copy scales of Q and dO.
#pragma once

#include <type_traits>

#include "common.hpp"
#include "dma.hpp"
#include "kernels.hpp"
#include "tiles.hpp"

namespace afp8 {

// PDP: the protected-dP variant, dP = dO V^T from BF16 operands (the dO row
// part of a query tile holds BF16 values, the workgroup's V rows sit in LDS
// as BF16); every other product keeps its FP8 operands.
template <int DQK, int DV, bool PDP = false>
struct BwdCfg {
  // 8 waves: 4 blocks of 32 keys x 2 query halves.  The two waves of a key
  // block (w and w + KBW) each compute S, dP, P and dS for one 32-query half
  // of the tile; after exchanging codes through LDS the first accumulates dV
  // and the second dK for all channels of their keys.  Wide heads (dqk + dv
  // > 256) take 2 key blocks (4 waves): with 4 the accumulators and the K / V
  // fragments of 8 waves do not fit the registers and the LDS together.
  static constexpr int KBW = DQK + DV > 256 ? 2 : 4, NWK = 2 * KBW;
  // the direct loads of the query tiles are issued by the first wave of each
  // key block only (one wave per SIMD; these also store the dQ units), so the
  // other four issue no vector memory instructions: spread over all eight,
  // every wave stalls behind the burst of load instructions at the start of
  // a tile
  static constexpr int NLD = KBW;
  static constexpr int NT = 64 * NWK, BKB = 32 * KBW, BQ = 64;
  static constexpr int DST = BQ + 16;   // row stride of the dS' tile [key][query]
  static constexpr int al16(int x) { return (x + 15) & ~15; }
  // row part of a query tile (operands of S and dP, the per-query records)
  static constexpr int OB = PDP ? 2 : 1;                            // bytes per dO row element
  static constexpr int Q_OFF = 0;                                   // Q row codes [BQ][DQK], swizzled
  static constexpr int O_OFF = Q_OFF + BQ * DQK;                    // dO row codes [BQ][DV] (PDP: BF16), swizzled
  static constexpr int QS_OFF = O_OFF + BQ * DV * OB;               // Q row scales [BQ][DQK/32]
  static constexpr int OS_OFF = al16(QS_OFF + BQ * DQK / 32);       // dO row scales [BQ][DV/32] (not with PDP)
  static constexpr int ROW_OFF = al16(OS_OFF + (PDP ? 0 : BQ * DV / 32));   // the tile's 1 KB block of per-query values
  static constexpr int RSTAGE = ROW_OFF + BQ * 16;
  // col part (operands of dV and dK)
  static constexpr int QC_OFF = 0;                                  // Q col codes [DQK][BQ], swizzled
  static constexpr int OC_OFF = QC_OFF + DQK * BQ;                  // dO col codes [DV][BQ], swizzled
  static constexpr int QCS_OFF = OC_OFF + DV * BQ;                  // Q col scales [DQK][2]
  static constexpr int OCS_OFF = QCS_OFF + DQK * 2;                 // dO col scales [DV][2]
  static constexpr int CS_BYTES = 2 * (DQK + DV);                   // both, as packed per tile by bwd_prep
  static constexpr int CSTAGE = al16(QCS_OFF + CS_BYTES);
  // dS' tiles, exponents and code exchange, two of each
  static constexpr int FIXED = 2 * (BKB * DST + KBW * 2 + 2 * KBW * 64 * 16);
  // the workgroup's K and V row codes [BKB][DQK + DV] (swizzled), read as
  // MFMA operands from LDS at wide heads; up to d = 128 each lane keeps its
  // key's fragments in registers (no LDS traffic for them).  PDP: the V rows
  // are BF16 [BKB][DV] in LDS at every head dim, the K codes as above.
  static constexpr int KV = BKB * (DQK + (PDP ? 0 : DV));
  static constexpr int VB = PDP ? BKB * DV * 2 : 0;
  static constexpr int LIM = 156 * 1024;
  // row parts are double-buffered; col parts too and K / V are kept in LDS
  // where the LDS allows, preferring K / V in LDS over a second col buffer
  static constexpr bool KV_LDS = DQK + DV > 256 && 2 * RSTAGE + CSTAGE + FIXED + KV + VB <= LIM;
  static constexpr int NCB = 2 * RSTAGE + 2 * CSTAGE + FIXED + (KV_LDS ? KV : 0) + VB <= LIM ? 2 : 1;
  static_assert(2 * RSTAGE + NCB * CSTAGE + FIXED + (KV_LDS ? KV : 0) + VB <= LIM, "LDS of the backward");
};

// dQ operand units of one head before 32-query block q.  Causal: block q has
// q/2 + 1 units of 64 keys up to the diagonal, sum_{i<q} (floor(i/2) + 1);
// without the mask every block has nks = ceil(Nk / 64).
__host__ __device__ __forceinline__ int64_t units_before(int64_t q, int64_t nks, bool causal) {
  if (!causal) return q * nks;
  const int64_t m = q >> 1;
  return (q & 1) ? (m + 1) * (m + 1) : m * (m + 1);
}

// Query-side operands of one (batch, KV group): the bases of its first query
// head (the G heads of a group are adjacent in every layout); a loading wave
// builds a buffer over the group's heads at each load and adds the head and
// tile offsets as scalar offsets to loop-invariant lane offsets.
struct BwdGroup {
  const uint8_t *qrow, *qsc, *orow, *osc, *qcol, *ocol, *tcs, *rows;
};

template <int DQK, int DV, bool PDP = false>
struct BwdStrides {   // bytes from one query head to the next
  int N;
  __device__ __forceinline__ uint32_t q() const { return (uint32_t)N * DQK; }
  __device__ __forceinline__ uint32_t qs() const { return (uint32_t)N * (DQK / 32); }
  __device__ __forceinline__ uint32_t o() const { return (uint32_t)N * DV * (PDP ? 2 : 1); }   // row part of dO
  __device__ __forceinline__ uint32_t oc() const { return (uint32_t)N * DV; }                  // col codes of dO
  __device__ __forceinline__ uint32_t os() const { return (uint32_t)N * (DV / 32); }
  __device__ __forceinline__ uint32_t tcs() const { return (uint32_t)((N + 63) / 64) * (2 * (DQK + DV)); }
  __device__ __forceinline__ uint32_t rows() const { return (uint32_t)((N + 63) / 64) * 1024; }
};

template <int DQK, int DV, bool PDP>
__device__ __forceinline__ BwdGroup bwd_group(const AttnArgs& a, size_t bh0, int N) {
  const BwdStrides<DQK, DV, PDP> S{N};
  BwdGroup g;
  g.qrow = a.q_code + bh0 * S.q();
  g.qsc = a.q_scale + bh0 * S.qs();
  g.orow = PDP ? reinterpret_cast<const uint8_t*>(a.do_bf16) + bh0 * S.o() : a.do_code + bh0 * S.o();
  g.osc = PDP ? nullptr : a.do_scale + bh0 * S.os();
  g.qcol = a.qc_code + bh0 * S.q();
  g.ocol = a.doc_code + bh0 * S.oc();
  g.tcs = a.tile_cs + bh0 * S.tcs();
  g.rows = reinterpret_cast<const uint8_t*>(a.rows) + bh0 * S.rows();
  return g;
}

// Load plans of one loading wave (index w among the NLD) for the code tiles
// of a query tile.
template <int DQK, int DV, bool PDP>
struct BwdLoads {
  static constexpr int NL = BwdCfg<DQK, DV>::NLD;
  RowLoads<DQK, NL, 64> q;
  RowLoads<DV * (PDP ? 2 : 1), NL, 64> o;   // PDP: BF16 rows of 2 DV bytes
  ColLoads<DQK, NL> qc;
  ColLoads<DV, NL> oc;
  __device__ __forceinline__ void init(int w, int lane, int N) {
    q.init(w, lane);
    o.init(w, lane);
    qc.init(w, lane, N);
    oc.init(w, lane, N);
  }
};

// Index of this wave among the loading waves (the first NLD), or -1.
template <int DQK, int DV>
__device__ __forceinline__ int loader_index() {
  using C = BwdCfg<DQK, DV>;
  const int w = wave_id();
  return w < C::NLD ? w : -1;
}

// Direct-to-LDS loads of the row part of one query tile (head hi of the
// group, queries i0..): codes, row scales and the per-query records.  N is
// the layouts' query length, lim the sequence's (queries at or past it are
// clamped to its last ones).
template <int DQK, int DV, bool PDP>
__device__ __forceinline__ void stage_rows(lds8* st, const BwdLoads<DQK, DV, PDP>& L, const BwdGroup& g, int G,
                                           int hi, int i0, int N, int lim) {
  using C = BwdCfg<DQK, DV, PDP>;
  constexpr int NWK = C::NLD;
  const int lane = threadIdx.x & 63, w = loader_index<DQK, DV>();
  if (w < 0) return;
  const BwdStrides<DQK, DV, PDP> S{N};
  L.q.issue_s(st + C::Q_OFF, make_buf(g.qrow, G * S.q()), hi * S.q(), i0, lim, w, lane);
  L.o.issue_s(st + C::O_OFF, make_buf(g.orow, G * S.o()), hi * S.o(), i0, lim, w, lane);
  dma_row_scales_s<DQK, NWK>(st + C::QS_OFF, make_buf(g.qsc, G * S.qs()), hi * S.qs(), i0, lim, w, lane, 0);
  if constexpr (!PDP)
    dma_row_scales_s<DV, NWK>(st + C::OS_OFF, make_buf(g.osc, G * S.os()), hi * S.os(), i0, lim, w, lane, 1);
  if (w == (3 % NWK)) {
    dma16s(make_buf(g.rows, G * S.rows()), (uint32_t)lane * 16, hi * S.rows() + (uint32_t)(i0 / 64) * 1024,
           st + C::ROW_OFF);
  }
}

// ... and of its col part: codes and the col scales packed by bwd_prep.
template <int DQK, int DV, bool PDP>
__device__ __forceinline__ void stage_cols(lds8* st, const BwdLoads<DQK, DV, PDP>& L, const BwdGroup& g, int G,
                                           int hi, int i0, int N, int lim) {
  using C = BwdCfg<DQK, DV, PDP>;
  constexpr int NWK = C::NLD;
  const int lane = threadIdx.x & 63, w = loader_index<DQK, DV>();
  if (w < 0) return;
  const BwdStrides<DQK, DV, PDP> S{N};
  L.qc.issue_s(st + C::QC_OFF, make_buf(g.qcol, G * S.q()), hi * S.q(), i0, N, lim, w, lane);
  L.oc.issue_s(st + C::OC_OFF, make_buf(g.ocol, G * S.oc()), hi * S.oc(), i0, N, lim, w, lane);
  constexpr int NCI = (C::CS_BYTES + 255) / 256;
  for (int k = 0; k < NCI; k++) {
    if ((2 + k) % NWK != w) continue;   // loaders 2, 3, ...: 0 and 1 take the row scales
    // the piece's offset in the scalar part, the lane's 4 bytes in the vector part
    if (4 * lane < C::CS_BYTES - 256 * k)
      dma4s(make_buf(g.tcs, G * S.tcs()), (uint32_t)(4 * lane),
            hi * S.tcs() + (uint32_t)(i0 / 64) * C::CS_BYTES + 256 * k, st + C::QCS_OFF + 256 * k);
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

// Order of the key blocks in the grid (slot s = workgroup id / (B Hkv)).  The
// blocks pair up as j and nkb - 1 - j (the pair's tile counts add to the same
// total for every j).  In cohorts of P pairs, P the number of workgroups of
// one KV head that run at once: first the long blocks j of the cohort, their
// query tiles visited downwards from the end of the sequence, then the
// partners, upwards from their diagonal, in the order the long blocks finish
// (workgroups start in id order as earlier ones end, so each partner takes
// the place of its own long block); a middle block (odd nkb) last.  With
// nqt = 2 nkb query tiles, the workgroups of a cohort then stand at tile
// nqt - 1 - t or t - 2 at step t, whichever block they hold: they read at
// most two distinct tiles at a time and share them in the L2 (the workgroups
// of one KV head run on one XCD).
struct KeyBlock {
  int kb;
  bool up;
};
__device__ __forceinline__ KeyBlock key_block_of(int s, int nkb, int P) {
  const int npair = nkb / 2, F = npair / P;
  int cohort, o, m;
  if (s < 2 * P * F) {
    cohort = s / (2 * P);
    o = s % (2 * P);
    m = P;
  } else {
    cohort = F;
    o = s - 2 * P * F;
    m = npair - F * P;
  }
  const int j0 = cohort * P;
  if (o < m) return KeyBlock{j0 + o, false};
  if (o < 2 * m) return KeyBlock{nkb - 1 - (j0 + m - 1 - (o - m)), true};
  return KeyBlock{npair, false};
}

// Position of a query tile in the workgroup's loop: query head kh G + hi,
// step r along the sequence (the G query heads of a step are consecutive);
// its 64 queries start at (nqt - 1 - r) * 64 when the tiles are visited
// downwards from the end of the sequence, at (qt0 + r) * 64 when upwards
// from the key block's diagonal tile qt0.
struct TilePos {
  int hi, r;
};
__device__ __forceinline__ TilePos next_pos(TilePos p, int G) {
  return p.hi + 1 < G ? TilePos{p.hi + 1, p.r} : TilePos{0, p.r + 1};
}

// CAUSAL: the mask (key length = query length) or every key of Nk; VAR:
// numerics variant, bit 0 compensated dS formation (COMP), bit 1 block-scaled
// backward probability operand (PMX), bit 2 dP from BF16 operands (PDP),
// bit 3 three isolated score channels (ISO3: channels 1 and 2 take a second
// rank-2 FP32 MFMA after the one that adds channel 0 and the shift, as in the
// correction pass, so both form S identically)
template <int DQK, int DV, bool STATS, bool CAUSAL, int VAR>
__global__ __launch_bounds__((BwdCfg<DQK, DV>::NT)) void bwd_kernel(AttnArgs a) {
  constexpr bool PDP = (VAR & 4) != 0, ISO3 = (VAR & 8) != 0;
  constexpr int NH = ISO3 ? 3 : 1;
  using C = BwdCfg<DQK, DV, PDP>;
  constexpr int KBW = C::KBW, BKB = C::BKB, BQ = C::BQ, NCB = C::NCB;
  constexpr int KS = DQK / 64, VS = DV / 64, CK = DQK / 32, CV = DV / 32;
  constexpr int CMAX = CK > CV ? CK : CV;
  // every buffer that alternates between tiles is two distinct objects, so
  // the compiler can tell loads into one from reads of the other
  __shared__ __attribute__((aligned(16))) uint8_t rA[C::RSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t rB[C::RSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t cA[C::CSTAGE];
  __shared__ __attribute__((aligned(16))) uint8_t cB[NCB == 2 ? C::CSTAGE : 16];
  __shared__ __attribute__((aligned(16))) uint8_t dsA[BKB * C::DST];
  __shared__ __attribute__((aligned(16))) uint8_t dsB[BKB * C::DST];
  constexpr bool COMP = (VAR & 1) != 0, PMX = (VAR & 2) != 0;
  // block exponents + 127 of the two query halves: dS' at [half][kbw], P'
  // (PMX) at 2 KBW + [half][kbw]
  __shared__ __attribute__((aligned(16))) uint8_t esA[KBW * 4];
  __shared__ __attribute__((aligned(16))) uint8_t esB[KBW * 4];
  // code exchange within a key block, 16 bytes per lane in natural query
  // order: [0] dS' of the first half (for dK), [1] P' of the second (for dV)
  __shared__ __attribute__((aligned(16))) uint4 xA[2][KBW * 64];
  __shared__ __attribute__((aligned(16))) uint4 xB[2][KBW * 64];
  __shared__ int hot_slot[NH];

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, hf = lane >> 5, li = lane & 31;
  const int kbw = w % KBW;                      // this wave's 32-key block within the workgroup
  const int qs = w / KBW;                       // and its 32-query half of every tile
  constexpr bool causal = CAUSAL;
  const int N = (int)a.N, Nk = CAUSAL ? N : (int)a.Nk;
  // workgroup id -> key block (slowest, in the order of key_block_of) and
  // (batch, KV head) (fastest: the key blocks of one KV head get ids equal
  // mod 16, hence one XCD and its L2 when B * Hkv % 8 == 0)
  // (with sequences of their own lengths the groups rotate over the XCDs
  // from one slot to the next, as in query_major_coord)
  const int GI = (int)(a.B * a.Hkv), slot = (int)blockIdx.x / GI;
  const KeyBlock kbk = key_block_of(slot, (Nk + BKB - 1) / BKB, a.bwd_cohort);
  const int kb0 = kbk.kb * BKB;
  const bool up = kbk.up;
  const int gi = a.lens_q ? ((int)blockIdx.x % GI + slot) % GI : (int)blockIdx.x % GI;
  const int kh = gi % (int)a.Hkv, b = gi / (int)a.Hkv;
  // the sequence's own lengths bound the work; N and Nk remain the strides
  const SeqLens L = seq_lens<CAUSAL>(a, b, N, Nk);
  if (kb0 >= L.k) return;                       // the whole key block is past the sequence
  const int kw0 = kb0 + 32 * kbw;               // this wave's first key
  const bool live = kw0 < L.k;
  const int kj = kw0 + li;                      // this lane's key
  int hots[NH];
  if constexpr (NH == 1) hots[0] = select_hot_channel<DQK>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, hot_slot);
  else select_hot_channels<DQK, NH>(a.q_amax, a.k_amax, b, kh, a.Hq, a.Hkv, a.G, hot_slot, hots);
  const int hot = hots[0];
  const size_t bhk = (size_t)b * a.Hkv + kh;
  const int Hq = (int)a.Hq, G = (int)a.G;
  const float c = a.c;

  // K and V row codes of this lane's key (B operands of S and dP); kb: B
  // operand of the score's rank-2 update (isolated-channel key value, or 1 in
  // lanes >= 32)
  v8i kf[KS], vf[VS];
  int ksc[KS], vsc[VS];
  float kb = 1.0f;
  float kb12 = 0.f;   // ISO3: the key's channel 1 (lanes < 32) and 2 (lanes >= 32) values
  constexpr bool KVL = C::KV_LDS;
  __shared__ __attribute__((aligned(16))) uint8_t kL[KVL ? BKB * DQK : 16];
  __shared__ __attribute__((aligned(16))) uint8_t vL[KVL && !PDP ? BKB * DV : 16];
  // PDP: the keys' BF16 V rows [BKB][2 DV bytes], 16-byte chunks swizzled as
  // in a row tile
  __shared__ __attribute__((aligned(16))) uint8_t vB[PDP ? C::VB : 16];
  {
    const int row = live ? kj : 0;
    const uint8_t* kr = a.k_code + (bhk * Nk + row) * DQK;
    const uint8_t* vr = a.v_code + (bhk * Nk + row) * DV;
#pragma unroll
    for (int s = 0; s < KS; s++) {
      kf[s] = frag_rows_global(kr, s, hf);
#pragma unroll
      for (int i = 0; i < NH; i++) clear_channel(kf[s], s, hf, hots[i]);
      ksc[s] = a.k_scale[(bhk * Nk + row) * (DQK / 32) + 2 * s + hf];
    }
    if constexpr (!PDP) {
#pragma unroll
      for (int s = 0; s < VS; s++) {
        vf[s] = frag_rows_global(vr, s, hf);
        vsc[s] = a.v_scale[(bhk * Nk + row) * (DV / 32) + 2 * s + hf];
      }
    } else {
      // the second wave of each key block stores its keys' BF16 V rows, the
      // two lane halves alternate chunks (visible after the prologue's barrier)
      if (qs == 1) {
        const uint4* src = reinterpret_cast<const uint4*>(a.v_bf16 + (bhk * Nk + row) * DV);
        const int kr2 = 32 * kbw + li;
#pragma unroll
        for (int ch = hf; ch < DV / 8; ch += 2)
          *reinterpret_cast<uint4*>(vB + kr2 * (2 * DV) + 16 * (ch ^ swz_row<2 * DV>(kr2))) = src[ch];
      }
    }
    if (hf == 0)
      kb = hot >= 0 ? row_value<DQK>(a.k_code + bhk * Nk * DQK, a.k_scale + bhk * Nk * (DQK / 32), row, hot) : 0.f;
    if constexpr (ISO3) {
      if (hot >= 0)
        kb12 = row_value<DQK>(a.k_code + bhk * Nk * DQK, a.k_scale + bhk * Nk * (DQK / 32), row, hf ? hots[2] : hots[1]);
    }
    if constexpr (KVL) {
      // the first wave of each key block stores the K fragments, the second
      // the V fragments, where frag_rows_swz reads them (visible after the
      // prologue's barrier)
      const int kr2 = 32 * kbw + li;
      if (qs == 0) {
#pragma unroll
        for (int t = 0; t < KS; t++) kv_store<DQK>(kL, kr2, t, hf, kf[t]);
      } else if constexpr (!PDP) {
#pragma unroll
        for (int t = 0; t < VS; t++) kv_store<DV>(vL, kr2, t, hf, vf[t]);
      }
    }
  }
  // operand fragments of k-step t of this lane's key
  auto kfrag = [&](int t) __attribute__((always_inline)) {
    if constexpr (KVL) return frag_rows_swz<DQK>(kL, 32 * kbw + li, t, hf);
    else return kf[t];
  };
  auto vfrag = [&](int t) __attribute__((always_inline)) {
    if constexpr (KVL) return frag_rows_swz<DV>(vL, 32 * kbw + li, t, hf);
    else return vf[t];
  };

  // dV (first half, CV blocks) or dK (second half, CK blocks) of the wave's keys
  v16f acc[CMAX];
#pragma unroll
  for (int i = 0; i < CMAX; i++)
#pragma unroll
    for (int r = 0; r < 16; r++) acc[i][r] = 0.f;

  const int nqt = (L.q + BQ - 1) / BQ, qt0 = causal ? kb0 / BQ : 0, nq = nqt - qt0;
  const int total = G * nq;                     // 0 only for a sequence without queries
  const size_t bh0 = (size_t)b * Hq + (size_t)kh * G;   // first query head of the group
  const int nks = (Nk + 63) / 64;               // 64-key steps of the dQ units
  const int64_t units_per_head = units_before(N / 32, nks, causal);
  auto q0_of = [&](TilePos p) __attribute__((always_inline)) { return (up ? qt0 + p.r : nqt - 1 - p.r) * BQ; };
  BwdLoads<DQK, DV, PDP> ld;
  ld.init(loader_index<DQK, DV>() >= 0 ? loader_index<DQK, DV>() : 0, lane, N);
  auto row_rec = [&](const uint8_t* R) __attribute__((always_inline)) {
    return *reinterpret_cast<const float*>(R + C::ROW_OFF + (32 * qs + li) * 8 + 4 * hf);
  };
  const BwdGroup grp = bwd_group<DQK, DV, PDP>(a, bh0, N);

  // Pipeline, per tile i (each step a function of the buffers it touches):
  //   barrier (codes of tile i exchanged, loads of rows i+1 and cols i landed)
  //   loads: rows of tile i+2, cols of tile i+1
  //   MFMA:  S, dP of tile i+1;  dV or dK of tile i
  //   store: dQ units of tile i
  //   VALU:  P, dS and codes of tile i+1 (overlapping the MFMAs above)
  v16f s, dp;
  v4i pn = v4i{0, 0, 0, 0}, dn = v4i{0, 0, 0, 0};   // this half's P' / dS' codes, natural query order
  int e = -127;                                      // and the dS' block exponent
  int ep = -8;                                       // and the P' block exponent (PMX)
  v4i mine = v4i{0, 0, 0, 0};                        // this wave's operand codes for dV (P') or dK (dS')

  // P, dS and their codes from the shifted s, dp; EDGE tiles may skip the
  // half or hold the diagonal block (masked)
  auto probs = [&](auto edge_tag, int qb, bool skip, int h, const uint8_t* R) __attribute__((always_inline)) {
    constexpr bool EDGE = decltype(edge_tag)::value;
    v4i pc, dc;
    e = -127;
    ep = -8;
    if (EDGE && skip) {
      pn = v4i{0, 0, 0, 0};
      dn = v4i{0, 0, 0, 0};
      return;
    }
    // lane holds queries qb + 8 g + 4 hf + e4 (accumulator r = 4 g + e4)
    float amax = 0.f;
    [[maybe_unused]] float pmax = 0.f;
    float pdp[16];   // |P dP| (row statistics only)
#pragma unroll
    for (int g = 0; g < 4; g++) {
      // -delta of the lane's four queries 8 g + 4 hf .. + 3 of the half
      const float4 nd = *reinterpret_cast<const float4*>(R + C::ROW_OFF + 512 + 4 * (32 * qs + 8 * g + 4 * hf));
      const float ndv[4] = {nd.x, nd.y, nd.z, nd.w};
      float ndl[4] = {0.f, 0.f, 0.f, 0.f};   // -delta_lo (COMP)
      if constexpr (COMP) {
        const float4 l = *reinterpret_cast<const float4*>(R + C::ROW_OFF + 768 + 4 * (32 * qs + 8 * g + 4 * hf));
        ndl[0] = l.x;
        ndl[1] = l.y;
        ndl[2] = l.z;
        ndl[3] = l.w;
      }
#pragma unroll
      for (int e4 = 0; e4 < 4; e4++) {
        const int r = 4 * g + e4;
        float p = bwd_prob(s[r], c);
        if (EDGE && causal && qb == kw0) p = (li > 8 * g + 4 * hf + e4) ? 0.f : p;   // diagonal block: key > query
        s[r] = p;
        if constexpr (PMX) pmax = fmaxf(pmax, p);
        if constexpr (STATS) pdp[r] = fabsf(p * dp[r]);
        if constexpr (COMP) {
          const float pd = p * ndv[e4];                        // fl(P (-delta_hi))
          const float e1 = __builtin_fmaf(p, ndv[e4], -pd);    // its rounding error, exact
          const float t = __builtin_fmaf(p, dp[r], pd);
          dp[r] = t + __builtin_fmaf(p, ndl[e4], e1);
        } else {
          dp[r] = __builtin_fmaf(p, dp[r], p * ndv[e4]);
        }
        amax = fmaxf(amax, fabsf(dp[r]));
      }
    }
    float scp = 0.00390625f;   // the P' scale: 2^-8, or the block's (PMX)
    if constexpr (PMX) {
      ep = pow2_exponent(wave_max_nonneg(pmax));
      ep = ep < -126 ? -126 : ep;
      scp = exp2i(ep);
    }
#pragma unroll
    for (int k = 0; k < 4; k++)
      pc[k] = (int)cvt4_div(s[4 * k], s[4 * k + 1], s[4 * k + 2], s[4 * k + 3], scp);
    e = pow2_exponent(wave_max_nonneg(amax));
    e = e < -126 ? -126 : e;
    const float sc = exp2i(e);
#pragma unroll
    for (int k = 0; k < 4; k++)
      dc[k] = (int)cvt4_div(dp[4 * k], dp[4 * k + 1], dp[4 * k + 2], dp[4 * k + 3], sc);
    if constexpr (STATS) {
      // per query row: FP64 sums over this wave's 32 keys, then atomics
      // (non-negative maxima as the integer maximum of their bit patterns)
#pragma unroll
      for (int r = 0; r < 16; r++) {
        const float cast = fp8_value((uint32_t)dc[r >> 2], r & 3) * sc;
        const float pcast = fp8_value((uint32_t)pc[r >> 2], r & 3) * scp;
        const double s0 = half_sum_d((double)dp[r]);
        const double s1 = half_sum_d((double)fabsf(dp[r]));
        const double s2 = half_sum_d((double)cast);
        const double s3 = half_sum_d((double)fabsf(cast));
        const double s6 = half_sum_d((double)pcast);
        const float mx = half_max(fabsf(dp[r]));
        const float mpdp = half_max(pdp[r]);
        const int qi = qb + 8 * (r >> 2) + 4 * hf + (r & 3);
        if (li == 0) {
          double* sp = a.rowstats + (((size_t)b * Hq + h) * N + qi) * kRowStats;
          atomicAdd(sp + 0, s0);
          atomicAdd(sp + 1, s1);
          atomicAdd(sp + 2, s2);
          atomicMax(reinterpret_cast<unsigned long long*>(sp + 3),
                    (unsigned long long)__double_as_longlong((double)mx));
          atomicAdd(sp + 4, s3);
          atomicMax(reinterpret_cast<unsigned long long*>(sp + 5),
                    (unsigned long long)__double_as_longlong((double)mpdp));
          atomicAdd(sp + 6, s6);
        }
      }
    }
    if constexpr (STATS) {
      // the cast dump: pre-cast P and dS of the lane's 16 pairs, their codes,
      // and the block exponents
      if (a.cast_dump) {
        const size_t S = (size_t)a.B * Hq * N * Nk, bhq = (size_t)b * Hq + h;
        float* Pd = reinterpret_cast<float*>(a.cast_dump);
        float* Dd = Pd + S;
        uint8_t* Pcd = reinterpret_cast<uint8_t*>(Dd + S);
        uint8_t* Dcd = Pcd + S;
        uint8_t* Ed = Dcd + S;
#pragma unroll
        for (int r = 0; r < 16; r++) {
          const size_t idx = (bhq * N + qb + 8 * (r >> 2) + 4 * hf + (r & 3)) * Nk + kj;
          Pd[idx] = s[r];
          Dd[idx] = dp[r];
          Pcd[idx] = (uint8_t)((uint32_t)pc[r >> 2] >> (8 * (r & 3)));
          Dcd[idx] = (uint8_t)((uint32_t)dc[r >> 2] >> (8 * (r & 3)));
        }
        if (lane == 0) {
          const size_t bi = (bhq * (N / 32) + qb / 32) * (Nk / 32) + kw0 / 32;
          Ed[bi] = (uint8_t)(e + 127);
          if constexpr (PMX) Ed[(size_t)a.B * Hq * (N / 32) * (Nk / 32) + bi] = (uint8_t)(ep + 127);
        }
      }
    }
    // natural query order: lane hf holds queries 16 hf .. 16 hf + 15 of the half
    pn = to_natural4(pc);
    dn = to_natural4(dc);
  };

  // P, dS and codes of the tile at p for this wave's half, written to ds / es / x
  auto front_vals = [&](TilePos p, const uint8_t* R, uint8_t* ds, uint8_t* es, uint4 (*x)[KBW * 64])
      __attribute__((always_inline)) {
    const int i0 = q0_of(p);
    const int qb = i0 + 32 * qs;
    const bool full = (causal ? i0 >= kb0 + BKB : kb0 + BKB <= L.k) && i0 + BQ <= L.q;
    const bool skip = !full && (!live || (causal && qb < kw0) || qb >= L.q);
    const int h = kh * G + p.hi;
    if (full) probs(std::false_type{}, qb, skip, h, R);
    else probs(std::true_type{}, qb, skip, h, R);
    // dS' codes for the dQ units and the exchange with the other half
    *reinterpret_cast<uint4*>(ds + (32 * kbw + li) * C::DST + 32 * qs + 16 * hf) =
        make_uint4((uint32_t)dn[0], (uint32_t)dn[1], (uint32_t)dn[2], (uint32_t)dn[3]);
    if (lane == 0) {
      es[qs * KBW + kbw] = (uint8_t)(e + 127);
      if constexpr (PMX) es[2 * KBW + qs * KBW + kbw] = (uint8_t)(ep + 127);
    }
    const v4i xv = qs == 0 ? dn : pn;
    x[qs][kbw * 64 + lane] = make_uint4((uint32_t)xv[0], (uint32_t)xv[1], (uint32_t)xv[2], (uint32_t)xv[3]);
    mine = qs == 0 ? pn : dn;
  };
  auto front_skip = [&](TilePos p) __attribute__((always_inline)) {
    const int i0 = q0_of(p);
    const int qb = i0 + 32 * qs;
    const bool full = (causal ? i0 >= kb0 + BKB : kb0 + BKB <= L.k) && i0 + BQ <= L.q;
    return !full && (!live || (causal && qb < kw0) || qb >= L.q);
  };

  // The MFMAs of one pipeline step, as one straight sequence: S and dP of the
  // next tile's half (skipped halves: none; zero codes later), the rank-2
  // update of S (per-query shifts: S += q_c* k_c*, then -LSE / tau), and
  // dV += P'^T dO_col (first wave of a key block) or dK +=
  // dS'^T Q_col (second).  The LDS operands of each MFMA are read one MFMA
  // ahead and a scheduling fence keeps them there, so each MFMA waits only
  // for its own reads while the next ones are in flight.
  // dV / dK: k = the tile's 64 queries.  The first wave's A holds its own P'
  // codes (queries 0..31 of the tile) in bytes 0..15 and the second half's
  // in bytes 16..31; the second wave's A holds its own dS' codes (queries
  // 32..63) in bytes 0..15 and the first half's in bytes 16..31, so both
  // build A from the same registers without a branch; the second wave's B
  // fragments and the scale bytes of both operands swap the two 32-query
  // blocks to match (the sum over k does not depend on the block order).
  struct Opnd {
    v8i a, b;
    int sa, sb;
  };
  auto mfmas = [&](const uint8_t* R, bool skip, float rec, const uint8_t* Cc, const uint8_t* es,
                   uint4 (*x)[KBW * 64], auto back_tag) __attribute__((always_inline)) {
    // ISO3: the lane's query's channel 1 (lanes < 32) or 2 value, decoded
    // from the staged Q row tile
    [[maybe_unused]] float rec12 = 0.f;
    if constexpr (ISO3) {
      if (hot >= 0) {
        const int row = 32 * qs + li, c = hf ? hots[2] : hots[1];
        const uint32_t code = R[C::Q_OFF + row * DQK + 16 * ((c >> 4) ^ swz_row<DQK>(row)) + (c & 15)];
        rec12 = scaled_value(code, R[C::QS_OFF + row * (DQK / 32) + c / 32]);
      }
    }
    const uint8_t* Q = R + C::Q_OFF;
    const uint8_t* Qs = R + C::QS_OFF;
    const uint8_t* O = R + C::O_OFF;
    const uint8_t* Os = R + C::OS_OFF;
    const int qrow = 32 * qs + li;
    const uint4 o = x[1 - qs][kbw * 64 + lane];
    const v8i A = v8i{mine[0], mine[1], mine[2], mine[3], (int)o.x, (int)o.y, (int)o.z, (int)o.w};
    // A scale of the lane half: own block (hf = 0) or the other half's
    int ascale;
    if constexpr (PMX) ascale = hf ? (int)es[(qs == 0 ? 3 * KBW : 0) + kbw] : (qs == 0 ? ep : e) + 127;
    else ascale = qs == 0 ? 127 - 8 : (hf ? (int)es[kbw] : e + 127);
    const uint8_t* Bt = Cc + (qs ? C::QC_OFF : C::OC_OFF);
    const uint8_t* Bs = Cc + (qs ? C::QCS_OFF : C::OCS_OFF);
    const int nb = qs ? CK : CV;
    const int clo = hf + 2 * qs, chi = hf + 2 - 2 * qs, sbk = hf ^ qs;
    // S and dP operations interleaved while both last (independent chains);
    // PDP: dP in DV / 16 BF16 MFMAs of 16 channels each
    constexpr int VSD = PDP ? DV / 16 : VS;
    constexpr int NSD = KS + VSD, NI2 = KS < VSD ? KS : VSD;
    auto sd_is_s = [](int m) { return m < 2 * NI2 ? (m & 1) == 0 : KS > VSD; };
    auto sd_t = [](int m) { return m < 2 * NI2 ? m >> 1 : m - NI2; };
    auto load = [&](int m) __attribute__((always_inline)) {
      Opnd r;
      if (m < NSD) {
        const int t = sd_t(m);
        if (sd_is_s(m)) {
          r.a = frag_rows_swz<DQK>(Q, qrow, t, hf);
          r.b = kfrag(t);
          r.sa = Qs[qrow * (DQK / 32) + 2 * t + hf];
          r.sb = ksc[t];
        } else if constexpr (PDP) {
          // BF16 fragments of channels 16 t + 8 hf .. + 7 of the query's dO
          // row and the key's V row (both operands pair the same channels)
          const int kr2 = 32 * kbw + li;
          const v4i av = *reinterpret_cast<const v4i*>(O + qrow * (2 * DV) + 16 * ((2 * t + hf) ^ swz_row<2 * DV>(qrow)));
          const v4i bv = *reinterpret_cast<const v4i*>(vB + kr2 * (2 * DV) + 16 * ((2 * t + hf) ^ swz_row<2 * DV>(kr2)));
          r.a = v8i{av[0], av[1], av[2], av[3], 0, 0, 0, 0};
          r.b = v8i{bv[0], bv[1], bv[2], bv[3], 0, 0, 0, 0};
          r.sa = 0;
          r.sb = 0;
        } else {
          r.a = frag_rows_swz<DV>(O, qrow, t, hf);
          r.b = vfrag(t);
          r.sa = Os[qrow * (DV / 32) + 2 * t + hf];
          r.sb = vsc[t];
        }
      } else {
        const int ch = 32 * (m - NSD) + li;
        r.a = A;
        r.b = frag_cols_chunks(Bt, ch, clo, chi);
        r.sa = ascale;
        r.sb = Bs[ch * 2 + sbk];
      }
      return r;
    };
    auto exec = [&](int m, const Opnd& r) __attribute__((always_inline)) {
      if (m < NSD) {
        if (sd_is_s(m)) s = mfma_mx(r.a, r.b, s, r.sa, r.sb);
        else if constexpr (PDP) dp = mfma_bf16(r.a, r.b, dp);
        else dp = mfma_mx(r.a, r.b, dp, r.sa, r.sb);
      } else {
        const int i = m - NSD;
        acc[i] = mfma_mx(r.a, r.b, acc[i], r.sa, r.sb);
      }
    };
    // operations M0 .. M1 - 1 of the sequence; the rank-2 update follows the
    // second dV / dK MFMA (the S chain has finished by then), or the last
    // S / dP MFMA when there is no dV / dK work
    auto run = [&](auto from_tag, auto with_back) __attribute__((always_inline)) {
      constexpr int M0 = decltype(from_tag)::value;
      constexpr int M1 = decltype(with_back)::value ? NSD + CMAX : NSD;
      constexpr int R2 = M1 > NSD ? NSD + (CMAX > 1 ? 1 : 0) : NSD - 1;
      if (M0 == 0) {
#pragma unroll
        for (int r = 0; r < 16; r++) { s[r] = 0.f; dp[r] = 0.f; }
      }
      Opnd cur = load(M0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int m = M0; m < M1; m++) {
        // past the last dV MFMA of the first wave (dqk > dv): the second
        // wave's remaining dK MFMAs only
        const bool act = m < NSD || m - NSD < (CK < CV ? CK : CV) || m - NSD < nb;
        Opnd nxt;
        if (m + 1 < M1 && (m + 1 < NSD || m + 1 - NSD < (CK < CV ? CK : CV) || m + 1 - NSD < nb)) nxt = load(m + 1);
        if (act) exec(m, cur);
        if (M0 == 0 && m == R2) {
          s = rank2_update(rec, kb, s);
          if constexpr (ISO3) s = rank2_update(rec12, kb12, s);
        }
        __builtin_amdgcn_sched_group_barrier(0x100, 16, 0);   // the reads of the next MFMA
        __builtin_amdgcn_sched_group_barrier(0x008, 3, 0);    // then this step's MFMAs
        __builtin_amdgcn_sched_barrier(0);
        cur = nxt;
      }
    };
    if constexpr (decltype(back_tag)::value) {
      if (skip) run(std::integral_constant<int, NSD>{}, std::true_type{});
      else run(std::integral_constant<int, 0>{}, std::true_type{});
    } else {
      // S and dP only (the first tile, before any dV / dK work)
      if (!skip) run(std::integral_constant<int, 0>{}, std::false_type{});
    }
  };

  // dQ operand units of the tile at p (its dS' codes and exponents in ds /
  // es): unit (query half uq, key step ks) holds 32 queries x 64 keys; units
  // wholly in the future of their queries (causal) or past the last key do
  // not exist
  auto ds_store = [&](TilePos p, const uint8_t* ds, const uint8_t* es) __attribute__((always_inline)) {
    constexpr int KSN = BKB / 64;
    const int h = kh * G + p.hi;
    const int i0 = q0_of(p);
    if (w >= 2 * KSN) return;
    const int uq = w / KSN, ks = w % KSN;
    const int qb = i0 + 32 * uq;
    if (qb >= L.q || (CAUSAL ? kb0 + 64 * ks > qb + 31 : kb0 + 64 * ks >= L.k)) return;
    uint32_t ex2 = *reinterpret_cast<const uint16_t*>(es + uq * KBW + 2 * ks);
    asm volatile("" : "+v"(ex2));
    const int i16 = lane & 15;
    const int qbase = 32 * uq + 16 * ((lane >> 4) & 1);
    // A: rows = queries of half uq, k = keys 64 ks .. 64 ks + 63 (natural order)
    v8i af;
#pragma unroll
    for (int part = 0; part < 4; part++) {
      const int kk = 64 * ks + 32 * (part >> 1) + 16 * hf + 8 * (part & 1);
      const uint8_t* addr = ds + (kk + (i16 >> 1)) * C::DST + qbase + 8 * (i16 & 1);
      const v2i tv = __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) v2i*)(addr));
      af[2 * part] = tv[0];
      af[2 * part + 1] = tv[1];
    }
    const int64_t unit = ((int64_t)b * Hq + h) * units_per_head + units_before(qb / 32, nks, causal) + (kb0 + 64 * ks) / 64;
    // streamed past the caches: the units are read once, by dq_kernel, and
    // must not evict the query tiles the workgroups share
    // (a unit is two 1 KB halves, operand bytes 0..15 then 16..31 of every
    // lane, so each store covers 1 KB contiguously)
    uint8_t* dst = a.ds_units + unit * 2048 + 16 * lane;
    __builtin_nontemporal_store(v4i{af[0], af[1], af[2], af[3]}, reinterpret_cast<v4i*>(dst));
    __builtin_nontemporal_store(v4i{af[4], af[5], af[6], af[7]}, reinterpret_cast<v4i*>(dst + 1024));
    if (lane == 0) *reinterpret_cast<uint16_t*>(a.ds_exp + unit * 2) = (uint16_t)ex2;
  };

  // one step of the pipeline for tile i at position p (p1, p2: tiles i+1,
  // i+2); R1: rows of tile i+1, Rl: buffer for the rows of tile i+2, Cc:
  // cols of tile i, Cl: buffer for the cols of tile i+1 (Cc itself with one
  // col buffer, after a barrier)
  auto body = [&](int i, TilePos p, TilePos p1, TilePos p2, const uint8_t* R1, lds8* Rl, const uint8_t* Cc, lds8* Cl,
                  const uint8_t* ds, const uint8_t* es, uint4 (*x)[KBW * 64], uint8_t* ds1, uint8_t* es1,
                  uint4 (*x1)[KBW * 64]) __attribute__((always_inline)) {
    lds_barrier();
    const bool more = i + 1 < total;
    // LDS reads the compiler cannot attribute to one buffer come first, before
    // any load into LDS is in flight: the dQ units of tile i and the records
    // of tile i+1
    ds_store(p, ds, es);
    const float rec = row_rec(R1);
    if constexpr (NCB == 2) {
      if (more) stage_cols<DQK, DV, PDP>(Cl, ld, grp, G, p1.hi, q0_of(p1), N, L.q);
    }
    if (i + 2 < total) stage_rows<DQK, DV, PDP>(Rl, ld, grp, G, p2.hi, q0_of(p2), N, L.q);
    const bool skip1 = !more || front_skip(p1);
    mfmas(R1, skip1, rec, Cc, es, x, std::true_type{});
    __builtin_amdgcn_sched_barrier(0);   // every MFMA issues before the VALU work below
    if constexpr (NCB == 1) {
      lds_sync();                          // every wave has read the col operands of tile i
      if (more) stage_cols<DQK, DV, PDP>(Cl, ld, grp, G, p1.hi, q0_of(p1), N, L.q);
    }
    if (more) front_vals(p1, R1, ds1, es1, x1);
  };

  // prologue: rows of tiles 0 and 1, cols of tile 0; S, dP, P, dS of tile 0
  // (none without queries: the key gradients are then zero)
  const TilePos p0 = TilePos{0, 0};
  if (total > 0) {
    stage_rows<DQK, DV, PDP>((lds8*)rA, ld, grp, G, p0.hi, q0_of(p0), N, L.q);
    stage_cols<DQK, DV, PDP>((lds8*)cA, ld, grp, G, p0.hi, q0_of(p0), N, L.q);
    TilePos pa = next_pos(p0, G);
    if (total > 1) stage_rows<DQK, DV, PDP>((lds8*)rB, ld, grp, G, pa.hi, q0_of(pa), N, L.q);
    lds_barrier();
    mfmas(rA, front_skip(p0), row_rec(rA), cA, esA, xA, std::false_type{});
    front_vals(p0, rA, dsA, esA, xA);
  }

  TilePos p = p0;
  for (int i = 0; i < total; i += 2) {
    const TilePos q1 = next_pos(p, G), q2 = next_pos(q1, G);
    if constexpr (NCB == 2) {
      body(i, p, q1, q2, rB, (lds8*)rA, cA, (lds8*)cB, dsA, esA, xA, dsB, esB, xB);
    } else {
      body(i, p, q1, q2, rB, (lds8*)rA, cA, (lds8*)cA, dsA, esA, xA, dsB, esB, xB);
    }
    if (i + 1 >= total) break;
    const TilePos q3 = next_pos(q2, G);
    if constexpr (NCB == 2) {
      body(i + 1, q1, q2, q3, rA, (lds8*)rB, cB, (lds8*)cA, dsB, esB, xB, dsA, esA, xA);
    } else {
      body(i + 1, q1, q2, q3, rA, (lds8*)rB, cA, (lds8*)cA, dsB, esB, xB, dsA, esA, xA);
    }
    p = q2;
  }

  if (!live) return;
  // dV (first half) or dK times tau (second half): lane holds channel
  // 32 i + li, keys kw0 + 8 (r/4) + 4 hf + r % 4
#pragma unroll
  for (int r = 0; r < 16; r++) {
    const int key = kw0 + 8 * (r >> 2) + 4 * hf + (r & 3);
    if (qs == 0) {
      if (a.grad_bf16) {
        uint16_t* vd = reinterpret_cast<uint16_t*>(a.dv) + b * a.dvs[0] + (int64_t)key * a.dvs[1] + kh * a.dvs[2];
#pragma unroll
        for (int i = 0; i < CV; i++) vd[32 * i + li] = f32_to_bf16(acc[i][r]);
      } else {
        float* vd = reinterpret_cast<float*>(a.dv) + b * a.dvs[0] + (int64_t)key * a.dvs[1] + kh * a.dvs[2];
#pragma unroll
        for (int i = 0; i < CV; i++) vd[32 * i + li] = acc[i][r];
      }
    } else {
      if (a.grad_bf16) {
        uint16_t* kd = reinterpret_cast<uint16_t*>(a.dk) + b * a.dks[0] + (int64_t)key * a.dks[1] + kh * a.dks[2];
#pragma unroll
        for (int i = 0; i < CK; i++) kd[32 * i + li] = f32_to_bf16(acc[i][r] * a.tau);
      } else {
        float* kd = reinterpret_cast<float*>(a.dk) + b * a.dks[0] + (int64_t)key * a.dks[1] + kh * a.dks[2];
#pragma unroll
        for (int i = 0; i < CK; i++) kd[32 * i + li] = acc[i][r] * a.tau;
      }
    }
  }
}

// Launch of the main backward kernel for one (mask, numerics) variant; each
// variant is instantiated in a translation unit of its own (they compile in
// parallel), the row statistics and the head dims at run time.
template <bool CAUSAL, int VAR>
hipError_t launch_bwd_main(const AttnArgs& a, int dqk, int dv, dim3 grid, hipStream_t s) {
#define AFP8_BWD_GO(Q, V)                                                                                   \
  if (dqk == Q && dv == V) {                                                                                \
    if (a.rowstats)                                                                                         \
      hipLaunchKernelGGL((bwd_kernel<Q, V, true, CAUSAL, VAR>), grid, dim3(BwdCfg<Q, V>::NT), 0, s, a);     \
    else                                                                                                    \
      hipLaunchKernelGGL((bwd_kernel<Q, V, false, CAUSAL, VAR>), grid, dim3(BwdCfg<Q, V>::NT), 0, s, a);    \
    return hipGetLastError();                                                                               \
  }
  AFP8_BWD_GO(64, 64)
  AFP8_BWD_GO(128, 128)
  // the protected-dP variant's BF16 dO and V tiles do not fit the LDS at d = 256
  if constexpr ((VAR & 4) == 0) {
    AFP8_BWD_GO(256, 256)
  }
  AFP8_BWD_GO(192, 128)
#undef AFP8_BWD_GO
  return hipErrorInvalidValue;
}

#define AFP8_BWD_EXTERN(C, V) extern template hipError_t launch_bwd_main<C, V>(const AttnArgs&, int, int, dim3, hipStream_t);
AFP8_BWD_EXTERN(true, 0)
AFP8_BWD_EXTERN(true, 1)
AFP8_BWD_EXTERN(true, 2)
AFP8_BWD_EXTERN(true, 3)
AFP8_BWD_EXTERN(true, 4)
AFP8_BWD_EXTERN(true, 8)
AFP8_BWD_EXTERN(false, 0)
AFP8_BWD_EXTERN(false, 1)
AFP8_BWD_EXTERN(false, 2)
AFP8_BWD_EXTERN(false, 3)
AFP8_BWD_EXTERN(false, 4)
AFP8_BWD_EXTERN(false, 8)
#undef AFP8_BWD_EXTERN

}  // namespace afp8
