// LDS staging of FP8 operand tiles shared by the forward, correction and
// backward kernels.  All loads are 16-byte vector loads; rows past the end of
// the sequence are zero-filled (zero codes, scale byte 0) so the MFMA sees
// exact zeros there.
#pragma once

#include "common.hpp"

namespace afp8 {

// Clears byte `pos` (0..15) of a 16-byte vector.
__device__ __forceinline__ void clear_byte(uint4& v, int pos) {
  const uint32_t m = ~(0xffu << (8 * (pos & 3)));
  const int d = pos >> 2;
  v.x &= d == 0 ? m : 0xffffffffu;
  v.y &= d == 1 ? m : 0xffffffffu;
  v.z &= d == 2 ? m : 0xffffffffu;
  v.w &= d == 3 ? m : 0xffffffffu;
}

// Rows [r0, r0 + ROWS) of a row-major [N, D] code matrix (one batch/head)
// into LDS with row stride ST bytes; the block's E8M0 bytes [N, D/32] into
// a dense [ROWS][D/32] LDS array.  zcol >= 0: that column's codes are stored
// as zero (the isolated score channel).
template <int ROWS, int D, int ST, int NT>
__device__ __forceinline__ void stage_rows(uint8_t* lds, uint8_t* lds_scale, const uint8_t* code,
                                           const uint8_t* scale, int64_t r0, int64_t N, int zcol = -1) {
  constexpr int V = ROWS * D / 16;  // uint4 per tile
  for (int u = threadIdx.x; u < V; u += NT) {
    const int r = u / (D / 16), c = (u % (D / 16)) * 16;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (r0 + r < N) val = *reinterpret_cast<const uint4*>(code + (r0 + r) * D + c);
    if (zcol >= c && zcol < c + 16) clear_byte(val, zcol - c);
    *reinterpret_cast<uint4*>(lds + r * ST + c) = val;
  }
  constexpr int S = ROWS * D / 32;  // scale bytes
  static_assert(S % 4 == 0, "scale tile is whole dwords");
  for (int u = threadIdx.x; u < S / 4; u += NT) {
    const int r = (u * 4) / (D / 32);
    uint32_t val = 0;
    if (r0 + r < N) val = *reinterpret_cast<const uint32_t*>(scale + r0 * (D / 32) + u * 4);
    *reinterpret_cast<uint32_t*>(lds_scale + u * 4) = val;
  }
}

// Columns [j0, j0 + 64) of a col-copy code matrix [D, N] (one batch/head)
// into LDS as [D][64] with row stride ST, permuted inside each 32-wide group
// so that the 16 sequence positions an MFMA lane of half hf holds in the
// "C layout" (positions 8a + 4hf + b, a, b in 0..3) are contiguous:
//   LDS position 16 hf + 4 a + b  <-  sequence position 8 a + 4 hf + b.
// Scales [D, N/32] -> LDS [D][2].
template <int D, int ST, int NT>
__device__ __forceinline__ void stage_cols_perm(uint8_t* lds, uint8_t* lds_scale, const uint8_t* code,
                                                const uint8_t* scale, int64_t j0, int64_t N) {
  constexpr int V = D * 4;  // 4 uint4 per 64-wide row
  for (int u = threadIdx.x; u < V; u += NT) {
    const int c = u >> 2, q = u & 3;  // q: 16-position quarter of the 64-wide row
    uint4 val = make_uint4(0, 0, 0, 0);
    if (j0 + q * 16 < N) val = *reinterpret_cast<const uint4*>(code + (int64_t)c * N + j0 + q * 16);
    uint8_t* base = lds + c * ST + (q >> 1) * 32 + (q & 1) * 8;
    *reinterpret_cast<uint2*>(base) = make_uint2(val.x, val.z);
    *reinterpret_cast<uint2*>(base + 16) = make_uint2(val.y, val.w);
  }
  for (int u = threadIdx.x; u < D; u += NT) {
    const int64_t g = j0 / 32;
    const uint8_t s0 = (j0 < N) ? scale[(int64_t)u * (N / 32) + g] : 0;
    const uint8_t s1 = (j0 + 32 < N) ? scale[(int64_t)u * (N / 32) + g + 1] : 0;
    lds_scale[u * 2] = s0;
    lds_scale[u * 2 + 1] = s1;
  }
}

// A/B fragment of a row-staged tile: lane (row li, half hf), k-step s.
template <int ST>
__device__ __forceinline__ v8i frag_rows(const uint8_t* lds, int row, int s, int hf) {
  const uint8_t* p = lds + row * ST + 64 * s + 16 * hf;
  const uint4 lo = *reinterpret_cast<const uint4*>(p);
  const uint4 hi = *reinterpret_cast<const uint4*>(p + 32);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// Same fragment straight from global memory (row-major [*, D] codes).
__device__ __forceinline__ v8i frag_rows_global(const uint8_t* row_ptr, int s, int hf) {
  const uint8_t* p = row_ptr + 64 * s + 16 * hf;
  const uint4 lo = *reinterpret_cast<const uint4*>(p);
  const uint4 hi = *reinterpret_cast<const uint4*>(p + 32);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// Fragment of a permuted col-staged tile (stage_cols_perm): lane (row li of
// the D dimension, half hf); bytes 0..15 cover group 0, 16..31 group 1.
template <int ST>
__device__ __forceinline__ v8i frag_cols(const uint8_t* lds, int row, int hf) {
  const uint8_t* p = lds + row * ST + 16 * hf;
  const uint4 lo = *reinterpret_cast<const uint4*>(p);
  const uint4 hi = *reinterpret_cast<const uint4*>(p + 32);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// Same fragment with the isolated channel `hot` (if it falls in k-step s and
// this lane's half) cleared.
__device__ __forceinline__ void clear_channel(v8i& f, int s, int hf, int hot) {
  const int cl = hot - 64 * s;
  if (hot < 0 || cl < 0 || cl >= 64 || ((cl & 31) >> 4) != hf) return;
  const int t = (cl < 32 ? 0 : 16) + (cl & 15);  // byte of the fragment holding channel `hot`
  const uint32_t m = ~(0xffu << (8 * (t & 3)));
#pragma unroll
  for (int d = 0; d < 8; d++) f[d] = (int)((uint32_t)f[d] & (d == (t >> 2) ? m : 0xffffffffu));
}

// Value of one E4M3 code (low byte of `code`) with its E8M0 scale byte.
__device__ __forceinline__ float scaled_value(uint32_t code, uint32_t scale) {
  return __builtin_ldexpf(fp8_value(code, 0), (int)(scale & 0xff) - 127);
}

// The isolated channel `hot` alone: the lane's fragment of k-step s with
// every byte but that channel's cleared (all zero when the channel is not in
// this k-step or not in this lane's half).  An MFMA with this operand and the
// other operand's fragment of the same k-step adds exactly the one product
// of the channel to each score.
__device__ __forceinline__ v8i keep_channel(const v8i& f, int s, int hf, int hot) {
  const int cl = hot - 64 * s;
  v8i z = v8i{0, 0, 0, 0, 0, 0, 0, 0};
  if (hot < 0 || cl < 0 || cl >= 64 || ((cl & 31) >> 4) != hf) return z;
  const int t = (cl < 32 ? 0 : 16) + (cl & 15);  // byte of the fragment holding channel `hot`
  const uint32_t m = 0xffu << (8 * (t & 3));
#pragma unroll
  for (int d = 0; d < 8; d++) z[d] = d == (t >> 2) ? (int)((uint32_t)f[d] & m) : 0;
  return z;
}

// Decoded value of the element in column `col` of row `row` of a row copy.
template <int D>
__device__ __forceinline__ float row_value(const uint8_t* code, const uint8_t* scale, int64_t row, int col) {
  const float v = fp8_value(code[row * D + col], 0);
  return __builtin_ldexpf(v, (int)scale[row * (D / 32) + col / 32] - 127);
}

// The isolated score channel of KV head kh (see attn_fp8.h): argmax over c of
// max_{h in group} q_amax[b,h,c] * k_amax[b,kh,c], lowest index on ties, or
// -1 without the per-channel maxima.  Computed by wave 0; every thread of the
// block returns the same value (contains a barrier).
template <int D>
__device__ __forceinline__ int select_hot_channel(const float* q_amax, const float* k_amax, int64_t b, int64_t kh,
                                                  int64_t Hq, int64_t Hkv, int64_t G, int* slot) {
  if (!q_amax || !k_amax) return -1;
  if (threadIdx.x < 64) {
    float best = -1.f;
    int bi = D;
    for (int c = threadIdx.x; c < D; c += 64) {
      float qm = 0.f;
      for (int64_t g = 0; g < G; g++) qm = fmaxf(qm, q_amax[(b * Hq + kh * G + g) * D + c]);
      const float sc = qm * k_amax[(b * Hkv + kh) * D + c];
      if (sc > best) { best = sc; bi = c; }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float ob = __shfl_xor(best, m);
      const int oi = __shfl_xor(bi, m);
      if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
    }
    if (threadIdx.x == 0) *slot = bi < D ? bi : -1;
  }
  __syncthreads();
  return *slot;
}

// The NH isolated score channels of KV head kh (ATTN_FP8_FLAG_ISOLATE3):
// the channels with the NH largest max_{h in group} q_amax[b,h,c] *
// k_amax[b,kh,c], in decreasing order (lowest index first on ties), chosen
// one at a time by select_hot_channel's rule over the channels not yet
// taken; all -1 without the per-channel maxima.  Computed by wave 0; every
// thread of the block gets the same values (contains a barrier).
template <int D, int NH>
__device__ __forceinline__ void select_hot_channels(const float* q_amax, const float* k_amax, int64_t b,
                                                    int64_t kh, int64_t Hq, int64_t Hkv, int64_t G, int* slots,
                                                    int (&hot)[NH]) {
  if (!q_amax || !k_amax) {
#pragma unroll
    for (int i = 0; i < NH; i++) hot[i] = -1;
    return;
  }
  if (threadIdx.x < 64) {
    constexpr int PER = D / 64;       // channels per lane: threadIdx.x + 64 u
    float sc[PER];
#pragma unroll
    for (int u = 0; u < PER; u++) {
      const int c = threadIdx.x + 64 * u;
      float qm = 0.f;
      for (int64_t g = 0; g < G; g++) qm = fmaxf(qm, q_amax[(b * Hq + kh * G + g) * D + c]);
      sc[u] = qm * k_amax[(b * Hkv + kh) * D + c];
    }
#pragma unroll
    for (int i = 0; i < NH; i++) {
      float best = -1.f;
      int bi = D;
#pragma unroll
      for (int u = 0; u < PER; u++)
        if (sc[u] > best) { best = sc[u]; bi = threadIdx.x + 64 * u; }
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        const float ob = __shfl_xor(best, m);
        const int oi = __shfl_xor(bi, m);
        if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
      }
      // the chosen channel is out of the next rounds
#pragma unroll
      for (int u = 0; u < PER; u++)
        if ((int)threadIdx.x + 64 * u == bi) sc[u] = -2.f;
      if (threadIdx.x == 0) slots[i] = bi < D ? bi : -1;
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < NH; i++) hot[i] = slots[i];
}

typedef int v4i __attribute__((ext_vector_type(4)));

// The four code dwords a lane holds for one 32-wide block of an MFMA result
// (rows 8 g + 4 hf + e in dword g, e < 4) put in natural order (rows
// 16 hf + 4 d + e in dword d), as an MFMA operand wants them: lane l < 32
// receives {x_g, partner's x_g} for g = 0, 1; lane l >= 32 {partner's x_g, x_g}
// for g = 2, 3.
__device__ __forceinline__ v4i to_natural4(const v4i& x) {
  const auto r0 = __builtin_amdgcn_permlane32_swap((uint32_t)x[0], (uint32_t)x[2], false, false);
  const auto r1 = __builtin_amdgcn_permlane32_swap((uint32_t)x[1], (uint32_t)x[3], false, false);
  return v4i{(int)r0[0], (int)r0[1], (int)r1[0], (int)r1[1]};
}

}  // namespace afp8
