// Device helpers shared by the gfx950 kernels: FP8/E8M0 arithmetic and the
// MX-scaled 32x32x64 MFMA.
//
// Register layout of v_mfma_scale_f32_32x32x64_f8f6f4 with E4M3 operands
// (measured on gfx950; lane l, half hf = l / 32):
//   A (32 x 64):  lane l holds row l % 32; its bytes 0..15 are k = 16 hf + t,
//                 bytes 16..31 are k = 32 + 16 hf + (t - 16).
//   B (64 x 32):  lane l holds column l % 32 with the same k mapping.
//   scales:       lane l's scale byte is the E8M0 scale of row (A) / column (B)
//                 l % 32 for the 32-wide k block hf (k in [32 hf, 32 hf + 32)).
//   C (32 x 32):  lane l, accumulator r holds row 8 (r / 4) + 4 hf + r % 4,
//                 column l % 32.
// Within one 32-wide k block the hardware sums products in chunks with an
// aligned fixed-point adder (about 2^-13 of the largest product of a chunk);
// chunk sums and the accumulator are FP32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace afp8 {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef short v2s __attribute__((ext_vector_type(2)));
typedef int v2i __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ v16f mfma_mx(const v8i& a, const v8i& b, const v16f& c, int scale_a,
                                        int scale_b) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, scale_a, 0, scale_b);
}

// BF16 32x32x16 MFMA with FP32 accumulation: lane l gives 8 BF16 values of
// row (A) / column (B) l % 32 in the low four dwords of a / b, lane half hf
// the k values 8 hf .. 8 hf + 7 (the same mapping for both operands, so
// loading both with the same channels pairs them); C as above.
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
__device__ __forceinline__ v16f mfma_bf16(const v8i& a, const v8i& b, const v16f& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, __builtin_shufflevector(a, a, 0, 1, 2, 3)),
                                                 __builtin_bit_cast(v8bf, __builtin_shufflevector(b, b, 0, 1, 2, 3)),
                                                 c, 0, 0, 0);
}

// Smallest integer e with amax <= 448 * 2^e (448 = 1.75 * 2^8), clamped to the
// E8M0 range [-127, 127]; zero and FP32-subnormal amax give -127.  Pure
// integer arithmetic on the FP32 bit pattern.
__device__ __forceinline__ int pow2_exponent(float amax) {
  const uint32_t u = __float_as_uint(amax) & 0x7fffffffu;
  const int be = (int)(u >> 23);
  int e = be - 135 + ((u & 0x7fffffu) > 0x600000u ? 1 : 0);
  e = be == 0 ? -127 : e;
  e = be == 255 ? 127 : e;
  return e < -127 ? -127 : (e > 127 ? 127 : e);
}

// 2^e as an FP32 value for e in [-126, 127].
__device__ __forceinline__ float exp2i(int e) { return __uint_as_float((uint32_t)(e + 127) << 23); }

// Four E4M3 codes of a/scale .. d/scale (scale a power of two, normal FP32),
// round to nearest even, packed little-endian into one dword.
// (the first convert's unused high half comes from a's register, which the
// second overwrites, so no zeroed destination is needed)
__device__ __forceinline__ uint32_t cvt4_div(float a, float b, float c, float d, float scale) {
  v2s r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(__builtin_bit_cast(v2s, a), a, b, scale, false);
  r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(r, c, d, scale, true);
  return __builtin_bit_cast(uint32_t, r);
}

// Four E4M3 codes of already-scaled values (no saturation: |x| <= 448 by
// construction at every call site).
__device__ __forceinline__ uint32_t cvt4(float a, float b, float c, float d) {
  uint32_t r = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, __builtin_bit_cast(uint32_t, a), false);
  return __builtin_amdgcn_cvt_pk_fp8_f32(c, d, r, true);
}

// Decode byte `sel` (0..3) of a packed dword of E4M3 codes.
__device__ __forceinline__ float fp8_value(uint32_t packed, int sel) {
  switch (sel & 3) {
    case 0: return __builtin_amdgcn_cvt_f32_fp8((int)packed, 0);
    case 1: return __builtin_amdgcn_cvt_f32_fp8((int)packed, 1);
    case 2: return __builtin_amdgcn_cvt_f32_fp8((int)packed, 2);
    default: return __builtin_amdgcn_cvt_f32_fp8((int)packed, 3);
  }
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// FP32 -> bfloat16 bits, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// v_permlane32_swap: for lanes < 32 returns {a[l], a[l + 32]}, for lanes >= 32
// returns {b[l - 32], b[l]}.  With a = value of group 0, b = value of group 1,
// each half of the wave receives both halves' values of "its" group.
struct Pair { float lo, hi; };
__device__ __forceinline__ Pair permlane32_swap(float a, float b) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  return Pair{__uint_as_float(r[0]), __uint_as_float(r[1])};
}

// Maximum over the 64 lanes of a wave of a non-negative value (FP32 order of
// non-negative values is the integer order of their bit patterns): DPP within
// rows of 16 lanes, then the row and half swaps of gfx950.
__device__ __forceinline__ float wave_max_nonneg(float v) {
  uint32_t u = __float_as_uint(v);
  u = max(u, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)u, 0xB1, 0xf, 0xf, false));   // quad_perm 1,0,3,2
  u = max(u, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)u, 0x4E, 0xf, 0xf, false));   // quad_perm 2,3,0,1
  u = max(u, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)u, 0x124, 0xf, 0xf, false));  // row_ror 4
  u = max(u, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)u, 0x128, 0xf, 0xf, false));  // row_ror 8
  auto r16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);                        // rows 2k <-> 2k+1
  u = max((uint32_t)r16[0], (uint32_t)r16[1]);
  auto r32 = __builtin_amdgcn_permlane32_swap(u, u, false, false);                        // halves
  u = max((uint32_t)r32[0], (uint32_t)r32[1]);
  return __uint_as_float(u);
}

// Workgroup order of the attention kernels (one-dimensional grids; the
// hardware hands out workgroups in index order, round-robin over the 8 XCDs):
// the heaviest work items come first (longest-processing-time order), and the
// workgroups that share a KV head land on the same XCD, i.e. the same L2.
//   query-major kernels: id -> (rank r of the query block, heaviest first,
//   batch b, query head h); within a rank, the query heads of one KV group
//   get ids that are equal mod 8 whenever B * Hkv is a multiple of 8.
//   rotate (sequences of their own lengths): the groups move to the next
//   XCD from one rank to the next, so that no XCD holds only long sequences
//   (with equal lengths every group weighs the same and stays on its XCD).
struct WgCoord { int r, b, h; };
__device__ __forceinline__ WgCoord query_major_coord(int id, int B, int Hq, int Hkv, bool rotate = false) {
  const int BH = B * Hq, G = Hq / Hkv, GI = B * Hkv;
  WgCoord c;
  c.r = id / BH;
  const int u = id % BH;
  if (GI % 8 == 0) {
    const int xcd = u % 8, j = u / 8;
    int gi = (j / G) * 8 + xcd;                 // (batch, KV head) group
    if (rotate) gi = (gi + c.r) % GI;
    c.b = gi / Hkv;
    c.h = (gi % Hkv) * G + j % G;
  } else {
    c.b = u / Hq;
    c.h = u % Hq;
  }
  return c;
}

// Index of the calling wave in its workgroup, as a wave-uniform (scalar)
// value: taken from threadIdx.x directly the compiler treats it as varying
// per lane, so every branch on it (which waves load, store or skip) would be
// compiled as a divergent branch with exec-mask bookkeeping.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }

// Value of `v` in the partner lane l ^ 32.
__device__ __forceinline__ float partner(float v) {
  Pair p = permlane32_swap(v, v);
  return (threadIdx.x & 32) ? p.lo : p.hi;
}

}  // namespace afp8

namespace afp8 {
// Two rank-1 updates of a 32x32 FP32 accumulator in one MFMA:
// C[i][j] += a0_i b0_j, then += a1_i b1_j, where lane l < 32 supplies a0_l
// (row l) and b0_l (column l) and lane l >= 32 supplies a1, b1 of row / column
// l - 32.  Each addition is rounded to nearest even in that order (a property
// of v_mfma_f32_32x32x2_f32 measured on the hardware), so with exact products
// the result is exactly fl(fl(C + a0 b0) + a1 b1), whichever operand holds
// the rows.
__device__ __forceinline__ v16f rank2_update(float a, float b, const v16f& c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Per-query shift of the raw score S (no tau) that makes P = 2^(c (S + shift))
// with c = tau log2e equal exp(tau S - LSE) (App. B.6.3).  Every kernel that
// recomputes P derives it from LSE with this one expression.
__device__ __forceinline__ float neg_lse_over_tau(float lse, float tau) { return -(lse / tau); }

// Backward probability from the shifted score: 2^(c s), clamped to [0, 1]
// (the clamp is a free modifier of the exponential and keeps 256 P inside
// the E4M3 range whatever LSE the caller passed).
__device__ __forceinline__ float bwd_prob(float s, float c) {
  return __builtin_amdgcn_fmed3f(__builtin_amdgcn_exp2f(s * c), 0.f, 1.f);
}
}  // namespace afp8
