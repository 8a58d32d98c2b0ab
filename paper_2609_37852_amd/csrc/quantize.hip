// Input quantizer: E4M3 codes with power-of-two (E8M0) scales, two copies
// (App. B.6.1 with 1x32 / 32x1 blocks).  HBM-bound: one pass reads x once and
// writes both copies.
//
// One workgroup = 64 tokens (2 blocks of 32) x D channels of one (batch,
// head), 2*D threads (two loads in flight per thread; 4 blocks measured
// slower).
//   row copy: thread t owns tokens 32 u + t / (D/16), 16 channels each; a
//             1x32 block spans the thread and its neighbour t ^ 1.
//   col copy: the tile is transposed through LDS (BF16 inputs kept BF16);
//             thread t owns channel t / 2 and the whole 32x1 block t % 2 of
//             that channel.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace afp8 {

template <typename T>
__device__ __forceinline__ void load16(const T* p, float (&v)[16]);

template <>
__device__ __forceinline__ void load16<float>(const float* p, float (&v)[16]) {
  const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
  for (int k = 0; k < 4; k++) {
    float4 f = q[k];
    v[4 * k] = f.x; v[4 * k + 1] = f.y; v[4 * k + 2] = f.z; v[4 * k + 3] = f.w;
  }
}

template <>
__device__ __forceinline__ void load16<uint16_t>(const uint16_t* p, float (&v)[16]) {
  const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
  for (int k = 0; k < 2; k++) {
    uint4 u = q[k];
    uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int m = 0; m < 4; m++) {
      v[8 * k + 2 * m] = __uint_as_float(w[m] << 16);
      v[8 * k + 2 * m + 1] = __uint_as_float(w[m] & 0xffff0000u);
    }
  }
}

// Codes of 16 values for one block exponent e: x * 2^-e is exact (power-of-two
// scaling; |x * 2^-e| <= 448 by the choice of e), then rounded to E4M3.
__device__ __forceinline__ uint4 encode16(const float (&v)[16], int e) {
  uint32_t w[4];
#pragma unroll
  for (int k = 0; k < 4; k++)
    w[k] = cvt4(__builtin_ldexpf(v[4 * k], -e), __builtin_ldexpf(v[4 * k + 1], -e),
                __builtin_ldexpf(v[4 * k + 2], -e), __builtin_ldexpf(v[4 * k + 3], -e));
  return make_uint4(w[0], w[1], w[2], w[3]);
}

__device__ __forceinline__ float amax16(const float (&v)[16]) {
  float m = 0.f;
#pragma unroll
  for (int k = 0; k < 16; k++) m = fmaxf(m, fabsf(v[k]));
  return m;
}

// Input values as kept in the transpose tile: BF16 inputs stay BF16 (exact).
template <typename T> struct TileOf { typedef float type; };
template <> struct TileOf<uint16_t> { typedef uint16_t type; };
__device__ __forceinline__ float tile_get(float x) { return x; }
__device__ __forceinline__ float tile_get(uint16_t x) { return __uint_as_float((uint32_t)x << 16); }
__device__ __forceinline__ void tile_put(float& d, float x) { d = x; }
__device__ __forceinline__ void tile_put(uint16_t& d, float x) { d = (uint16_t)(__float_as_uint(x) >> 16); }

// Codes of 32 values for one block exponent e.
__device__ __forceinline__ void encode32(const float (&v)[32], int e, uint4& lo, uint4& hi) {
  uint32_t w[8];
#pragma unroll
  for (int k = 0; k < 8; k++)
    w[k] = cvt4(__builtin_ldexpf(v[4 * k], -e), __builtin_ldexpf(v[4 * k + 1], -e),
                __builtin_ldexpf(v[4 * k + 2], -e), __builtin_ldexpf(v[4 * k + 3], -e));
  lo = make_uint4(w[0], w[1], w[2], w[3]);
  hi = make_uint4(w[4], w[5], w[6], w[7]);
}

// FP32 multiply and subtract, each rounded once: the pragma keeps the
// compiler from contracting a product and a following subtraction into one
// FMA (HIP compiles with contraction on).
__device__ __forceinline__ float mul_rn(float x, float y) {
#pragma clang fp contract(off)
  return x * y;
}
__device__ __forceinline__ float sub_rn(float x, float y) {
#pragma clang fp contract(off)
  return x - y;
}
__device__ __forceinline__ float add_rn(float x, float y) {
#pragma clang fp contract(off)
  return x + y;
}

// One rotated channel of the fused rotary embedding: the first of a pair
// gives x cos - p sin, the second x cos + p sin (x this channel's value, p
// the pair partner's), every product and the sum rounded to FP32, the result
// rounded to BF16.
//
// Rounding to BF16 uses the hardware conversion (v_cvt_pk_bf16_f32, round to
// nearest even; it agrees with the integer rounding rule on every finite
// FP32 value, subnormals included, which an in-bounds probe checked on 4M
// values).
__device__ __forceinline__ float round_bf16(float x) { return (float)(__bf16)x; }

__device__ __forceinline__ float rope_rotate(float x, float p, float2 cs, bool first) {
  const float a = mul_rn(x, cs.x), b = mul_rn(p, cs.y);
  return round_bf16(first ? sub_rn(a, b) : add_rn(a, b));
}

// One channel of the QK normalization: x times the row's reciprocal RMS,
// times the channel gain, each product rounded to FP32, rounded to BF16.
__device__ __forceinline__ float qk_norm(float x, float r, float g) {
  return round_bf16(mul_rn(mul_rn(x, r), g));
}

// One workgroup = 32 NB tokens (NB 32-token blocks; the last ones may lie
// past the end of the sequence) x D channels of one (batch, head), 2*D threads.
// PROD: the input producer's transform is applied to every value first
// (FP32 multiply by the prescale, then FP32 subtraction of the channel mean,
// each rounded once: no contraction into an FMA); the transposed tile then
// holds FP32 values.
template <int D, typename T, int NB, bool PROD>
__global__ __launch_bounds__(2 * D) void quantize_kernel(QuantArgs a) {
  constexpr int CH = D / 16;  // 16-channel chunks per token
  typedef typename std::conditional<PROD, float, typename TileOf<T>::type>::type TT;
  __shared__ TT tile[32 * NB][D + (sizeof(TT) == 2 ? 2 : 1)];
  const int t = threadIdx.x;
  const int64_t n0 = (int64_t)blockIdx.x * 32 * NB, h = blockIdx.y, b = blockIdx.z;
  const int64_t bh = b * a.H + h;
  const int nb = (int)((a.N - n0) / 32 < NB ? (a.N - n0) / 32 : NB);   // blocks inside the sequence
  const int tok = t / CH, ch = (t % CH) * 16;
  const T* src = reinterpret_cast<const T*>(a.x) + b * a.sb + h * a.sh + ch;
  float v[NB][16];
#pragma unroll
  for (int u = 0; u < NB; u++) {
    if (u < nb) load16<T>(src + (n0 + 32 * u + tok) * a.sn, v[u]);
    else {
#pragma unroll
      for (int k = 0; k < 16; k++) v[u][k] = 0.f;
    }
  }
  // the producer's other inputs, loaded together with the tokens: row
  // scales, gains, rotary table entries and the channel means (gain, table
  // and mean are 16-byte aligned, ch a multiple of 16)
  [[maybe_unused]] float rsc[NB], gn[16], mu[16];
  [[maybe_unused]] float4 cs[NB][8];
  [[maybe_unused]] const int h2 = a.rope_dim >> 1, rel = ch - a.rope_lo;
  [[maybe_unused]] const bool rot = a.rope && rel >= 0 && rel < a.rope_dim, first = rel < h2;
  [[maybe_unused]] const int pch = first ? ch + h2 : ch - h2, c0 = first ? rel : rel - h2;
  if constexpr (PROD) {
#pragma unroll
    for (int u = 0; u < NB; u++) rsc[u] = a.gain && u < nb ? a.rscale[((b * a.N) + n0 + 32 * u + tok) * a.H + h] : 1.f;
#pragma unroll
    for (int k = 0; k < 4; k++) {
      const float4 g4 = a.gain ? reinterpret_cast<const float4*>(a.gain + ch)[k] : make_float4(1.f, 1.f, 1.f, 1.f);
      const float4 m4 = a.mean ? reinterpret_cast<const float4*>(a.mean + bh * D + ch)[k] : make_float4(0.f, 0.f, 0.f, 0.f);
      gn[4 * k] = g4.x; gn[4 * k + 1] = g4.y; gn[4 * k + 2] = g4.z; gn[4 * k + 3] = g4.w;
      mu[4 * k] = m4.x; mu[4 * k + 1] = m4.y; mu[4 * k + 2] = m4.z; mu[4 * k + 3] = m4.w;
    }
#pragma unroll
    for (int u = 0; u < NB; u++) {
      if (rot && u < nb) {
        const float4* cs4 = reinterpret_cast<const float4*>(
            reinterpret_cast<const float2*>(a.rope) + (n0 + 32 * u + tok) * h2 + c0);
#pragma unroll
        for (int k = 0; k < 8; k++) cs[u][k] = cs4[k];
      }
    }
  }

  if (a.nonfinite) {
    uint32_t bad = 0;
#pragma unroll
    for (int u = 0; u < NB; u++)
#pragma unroll
      for (int k = 0; k < 16; k++) bad += __builtin_isfinite(v[u][k]) ? 0u : 1u;
    if (bad) atomicAdd(a.nonfinite, bad);
  }
  if constexpr (PROD) {
    if (a.gain) {
#pragma unroll
      for (int u = 0; u < NB; u++) {
        if (u >= nb) break;
#pragma unroll
        for (int k = 0; k < 16; k++) v[u][k] = qk_norm(v[u][k], rsc[u], gn[k]);
      }
    }
    if (a.rope) {
      // fused rotary embedding: the pair partner's 16 values come from the
      // lane h2 / 16 further along the token (a token's CH lanes are
      // consecutive), or through the tile where a token's chunks may lie in
      // two waves (64 % CH != 0)
      if constexpr (64 % CH == 0) {
        const int plane = (t & 63) + (rot ? (pch - ch) / 16 : 0);
#pragma unroll
        for (int u = 0; u < NB; u++) {
          float pv[16];
#pragma unroll
          for (int k = 0; k < 16; k++) pv[k] = __shfl(v[u][k], plane);
          if (rot && u < nb) {
#pragma unroll
            for (int k = 0; k < 8; k++) {
              v[u][2 * k] = rope_rotate(v[u][2 * k], pv[2 * k], make_float2(cs[u][k].x, cs[u][k].y), first);
              v[u][2 * k + 1] = rope_rotate(v[u][2 * k + 1], pv[2 * k + 1], make_float2(cs[u][k].z, cs[u][k].w), first);
            }
          }
        }
      } else {
#pragma unroll
        for (int u = 0; u < NB; u++)
#pragma unroll
          for (int k = 0; k < 16; k++) tile[32 * u + tok][ch + k] = v[u][k];
        __syncthreads();
        if (rot) {
#pragma unroll
          for (int u = 0; u < NB; u++) {
            if (u >= nb) break;
#pragma unroll
            for (int k = 0; k < 8; k++) {
              v[u][2 * k] = rope_rotate(v[u][2 * k], tile[32 * u + tok][pch + 2 * k], make_float2(cs[u][k].x, cs[u][k].y), first);
              v[u][2 * k + 1] = rope_rotate(v[u][2 * k + 1], tile[32 * u + tok][pch + 2 * k + 1],
                                            make_float2(cs[u][k].z, cs[u][k].w), first);
            }
          }
        }
        __syncthreads();   // the tile is written again below
      }
    }
#pragma unroll
    for (int u = 0; u < NB; u++)
#pragma unroll
      for (int k = 0; k < 16; k++) {
        const float xs = mul_rn(v[u][k], a.prescale);
        v[u][k] = a.mean ? sub_rn(xs, mu[k]) : xs;
      }
  }
  if (a.which & 1) {
#pragma unroll
    for (int u = 0; u < NB; u++) {
      if (u >= nb) break;
      const int64_t n = n0 + 32 * u + tok;
      float am = amax16(v[u]);
      am = fmaxf(am, __shfl_xor(am, 1));
      const int e = pow2_exponent(am);
      *reinterpret_cast<uint4*>(a.code_row + (bh * a.N + n) * D + ch) = encode16(v[u], e);
      if ((t & 1) == 0) a.scale_row[(bh * a.N + n) * (D / 32) + ch / 32] = (uint8_t)(e + 127);
    }
  }
  if (a.which & 2) {
#pragma unroll
    for (int u = 0; u < NB; u++)
#pragma unroll
      for (int k = 0; k < 16; k++) tile_put(tile[32 * u + tok][ch + k], v[u][k]);
    __syncthreads();
    // thread (channel c, parity u0): the 32 tokens of col blocks u0, u0 + 2, ..
    const int c = t >> 1, u0 = t & 1;
    float cam = 0.f;
#pragma unroll
    for (int u = u0; u < NB; u += 2) {
      const bool valid = u < nb;
      float w[32];
#pragma unroll
      for (int k = 0; k < 32; k++) w[k] = tile_get(tile[32 * u + k][c]);
      float am = 0.f;
#pragma unroll
      for (int k = 0; k < 32; k++) am = fmaxf(am, fabsf(w[k]));
      am = valid ? am : 0.f;
      cam = fmaxf(cam, am);
      if (valid) {
        const int e = pow2_exponent(am);
        uint4 lo, hi;
        encode32(w, e, lo, hi);
        uint4* dst = reinterpret_cast<uint4*>(a.code_col + (bh * D + c) * a.N + n0 + 32 * u);
        dst[0] = lo;
        dst[1] = hi;
        a.scale_col[(bh * D + c) * (a.N / 32) + n0 / 32 + u] = (uint8_t)(e + 127);
      }
    }
    // non-negative FP32 values order like their bit patterns
    if (a.chan_amax) {
      const float am2 = fmaxf(cam, __shfl_xor(cam, 1));   // every block of the channel
      if (u0 == 0) atomicMax(reinterpret_cast<unsigned int*>(a.chan_amax + bh * D + c), __float_as_uint(am2));
    }
  }
}

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s);

// Key mean of the input producer (reading R13): FP64 sums of the prescaled
// values over aligned 32-token blocks, tokens ascending (one thread per 8
// channels and block), then the block sums ascending (one thread per
// channel: grid (H, B)), divided by N in FP64 and rounded once to FP32.  The
// fixed order makes the mean independent of scheduling.
// Eight consecutive channels of one token as FP32, from their raw bytes
// (one 16-byte word for BF16, two for FP32).
template <typename T>
__device__ __forceinline__ void unpack8(const uint4 (&u)[sizeof(T) / 2], float (&v)[8]) {
  if constexpr (sizeof(T) == 2) {
    const uint32_t w[4] = {u[0].x, u[0].y, u[0].z, u[0].w};
#pragma unroll
    for (int m = 0; m < 4; m++) {
      v[2 * m] = __uint_as_float(w[m] << 16);
      v[2 * m + 1] = __uint_as_float(w[m] & 0xffff0000u);
    }
  } else {
    const uint32_t w[8] = {u[0].x, u[0].y, u[0].z, u[0].w, u[1].x, u[1].y, u[1].z, u[1].w};
#pragma unroll
    for (int m = 0; m < 8; m++) v[m] = __uint_as_float(w[m]);
  }
}

// Key-mean partial sums: a thread owns channels c .. c + 7 of one aligned
// 32-token block of one (batch, head) and sums the transformed values of
// each in FP64 over the block's tokens in ascending order; a workgroup of
// D / 2 threads takes kPartialBlocks blocks (D / 8 threads each).  Partials
// are laid out [B, H, N/32, D] so that the mean pass reads them coalesced.
// The transform (norm, rotation, prescale) is the quantizer's; the eight
// channels of a thread are all rotary or all not, and all first or all
// second of their pairs (the rotary range and its halves are multiples of
// 16 channels), so their partners are consecutive as well.
// With sequence lengths, the mean's tokens of batch entry b: its first L_b
// (clamped into [0, N], rounded down to a multiple of 32, as the attention
// kernels take it).
constexpr int kPartialBlocks = 4;

__device__ __forceinline__ int64_t mean_tokens(const QuantArgs& a, int64_t b) {
  if (!a.lens) return a.N;
  const int64_t v = a.lens[b];
  return (v < 0 ? 0 : v > a.N ? a.N : v) & ~int64_t(31);
}

template <typename T>
__global__ __launch_bounds__(128) void producer_partials_kernel(QuantArgs a, int D) {
  const int cpr = D / 8, c = 8 * ((int)threadIdx.x % cpr);
  const int64_t nblk = a.N / 32, t = (int64_t)blockIdx.x * kPartialBlocks + threadIdx.x / cpr;
  const int64_t h = blockIdx.y, b = blockIdx.z;
  if (t >= nblk) return;
  double2* out = reinterpret_cast<double2*>(a.partials + ((b * a.H + h) * nblk + t) * D + c);
  if (32 * t >= mean_tokens(a, b)) {
    // a block past the sequence adds nothing to its mean
#pragma unroll
    for (int m = 0; m < 4; m++) out[m] = make_double2(0.0, 0.0);
    return;
  }
  const T* src = reinterpret_cast<const T*>(a.x) + b * a.sb + h * a.sh + c;
  const int h2 = a.rope_dim >> 1, rel = c - a.rope_lo;
  const bool rot = a.rope && rel >= 0 && rel < a.rope_dim, first = rel < h2;
  const int poff = first ? h2 : -h2, c0 = first ? rel : rel - h2;
  float g[8], pg[8];
#pragma unroll
  for (int m = 0; m < 8; m++) {
    g[m] = a.gain ? a.gain[c + m] : 1.f;
    pg[m] = a.gain && rot ? a.gain[c + poff + m] : 1.f;
  }
  double part[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
  // KC tokens' loads issued ahead of their arithmetic (c is a multiple of 8
  // and every stride a multiple of 16 bytes, so the words are aligned)
  constexpr int KC = 8, W = sizeof(T) / 2;
  for (int k0 = 0; k0 < 32; k0 += KC) {
    uint4 xr[KC][W], pr[KC][W];
    float4 cs[KC][4];
    float rs[KC];
#pragma unroll
    for (int k = 0; k < KC; k++) {
      const int64_t n = 32 * t + k0 + k;
      const uint4* x4 = reinterpret_cast<const uint4*>(src + n * a.sn);
#pragma unroll
      for (int m = 0; m < W; m++) xr[k][m] = x4[m];
      if (rot) {
        const uint4* p4 = reinterpret_cast<const uint4*>(src + n * a.sn + poff);
        const float4* c4 = reinterpret_cast<const float4*>(a.rope + 2 * (n * h2 + c0));
#pragma unroll
        for (int m = 0; m < W; m++) pr[k][m] = p4[m];
#pragma unroll
        for (int m = 0; m < 4; m++) cs[k][m] = c4[m];
      }
      rs[k] = a.gain ? a.rscale[(b * a.N + n) * a.H + h] : 1.f;
    }
#pragma unroll
    for (int k = 0; k < KC; k++) {
      float f[8], p[8];
      unpack8<T>(xr[k], f);
      if (rot) unpack8<T>(pr[k], p);
      if (a.gain) {
#pragma unroll
        for (int m = 0; m < 8; m++) {
          f[m] = qk_norm(f[m], rs[k], g[m]);
          if (rot) p[m] = qk_norm(p[m], rs[k], pg[m]);
        }
      }
      if (rot) {
#pragma unroll
        for (int m = 0; m < 4; m++) {
          f[2 * m] = rope_rotate(f[2 * m], p[2 * m], make_float2(cs[k][m].x, cs[k][m].y), first);
          f[2 * m + 1] = rope_rotate(f[2 * m + 1], p[2 * m + 1], make_float2(cs[k][m].z, cs[k][m].w), first);
        }
      }
#pragma unroll
      for (int m = 0; m < 8; m++) part[m] += (double)mul_rn(f[m], a.prescale);
    }
  }
#pragma unroll
  for (int m = 0; m < 4; m++) out[m] = make_double2(part[2 * m], part[2 * m + 1]);
}

// Reciprocal RMS of every (token, head) row for the QK normalization: the
// squares summed in FP64 over the channels in ascending order, divided by D,
// eps added, 1 / sqrt in FP64 (each rounded to nearest), rounded once to
// FP32.  A workgroup of 256 threads takes 256 rows: 32-channel slices of
// them reach LDS with coalesced loads (rows in (b, n, h) order, h fastest),
// then each thread continues its own row's sum over the slice.
template <typename T>
__global__ __launch_bounds__(256) void producer_rscale_kernel(QuantArgs a, int D) {
  constexpr int RS = 33;                                   // padded row of a slice (floats)
  __shared__ float sl[256 * RS];
  const int64_t rows = a.B * a.N * a.H, row0 = (int64_t)blockIdx.x * 256;
  const int t = threadIdx.x, q = t & 3;
  // thread t loads the 8-channel piece q = t % 4 of rows t / 4 + 64 j
  const T* base[4];
#pragma unroll
  for (int j = 0; j < 4; j++) {
    const int64_t rr = row0 + (t >> 2) + 64 * j, row = rr < rows ? rr : rows - 1;
    const int64_t h = row % a.H, n = (row / a.H) % a.N, b = row / (a.H * a.N);
    base[j] = reinterpret_cast<const T*>(a.x) + b * a.sb + n * a.sn + h * a.sh + 8 * q;
  }
  double ss = 0.0;
  for (int c0 = 0; c0 < D; c0 += 32) {
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int r = (t >> 2) + 64 * j;
      const T* src = base[j] + c0;
      float v[8];
      if constexpr (sizeof(T) == 2) {
        const uint4 u = *reinterpret_cast<const uint4*>(src);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int m = 0; m < 4; m++) {
          v[2 * m] = __uint_as_float(w[m] << 16);
          v[2 * m + 1] = __uint_as_float(w[m] & 0xffff0000u);
        }
      } else {
        const float4 x0 = reinterpret_cast<const float4*>(src)[0], x1 = reinterpret_cast<const float4*>(src)[1];
        v[0] = x0.x; v[1] = x0.y; v[2] = x0.z; v[3] = x0.w; v[4] = x1.x; v[5] = x1.y; v[6] = x1.z; v[7] = x1.w;
      }
#pragma unroll
      for (int k = 0; k < 8; k++) sl[r * RS + 8 * q + k] = v[k];
    }
    __syncthreads();
#pragma unroll 8
    for (int k = 0; k < 32; k++) {
      const double x = (double)sl[t * RS + k];
      ss += x * x;                                          // exact products
    }
    __syncthreads();
  }
  if (row0 + t < rows) a.rscale[row0 + t] = (float)(1.0 / __builtin_sqrt(ss / (double)D + a.eps));
}

// The key mean: FP64 sum of the block partial sums in block order (coalesced
// over the channels), divided by the token count (N, or the sequence's
// length) in FP64, rounded once to FP32; 0 for a sequence without tokens.
__global__ __launch_bounds__(256) void producer_mean_kernel(QuantArgs a, int D) {
  const int c = threadIdx.x;
  if (c >= D) return;
  const int64_t h = blockIdx.x, b = blockIdx.y, nblk = a.N / 32, n = mean_tokens(a, b);
  const double* p = a.partials + (b * a.H + h) * nblk * D + c;
  // 64 block sums loaded at a time, then added in order
  double total = 0.0;
  const int64_t nb = n / 32;
  int64_t t0 = 0;
  for (; t0 + 64 <= nb; t0 += 64) {
    double v[64];
#pragma unroll
    for (int k = 0; k < 64; k++) v[k] = p[(t0 + k) * D];
#pragma unroll
    for (int k = 0; k < 64; k++) total += v[k];
  }
  for (; t0 < nb; t0++) total += p[t0 * D];
  a.mean[(b * a.H + h) * D + c] = n > 0 ? (float)(total / (double)n) : 0.f;
}

hipError_t launch_quantize(const QuantArgs& a, int D, int dtype_bf16, hipStream_t s) {
  constexpr int NB = 2;
  dim3 grid((unsigned)((a.N + 32 * NB - 1) / (32 * NB)), (unsigned)a.H, (unsigned)a.B);
  if (a.chan_amax) {
    const hipError_t e = launch_fill_zero(a.chan_amax, a.B * a.H * D, s);
    if (e != hipSuccess) return e;
  }
  const bool prod = a.prescale != 1.0f || a.mean || a.rope || a.gain;
  if (a.gain) {
    const dim3 g0((unsigned)((a.B * a.N * a.H + 255) / 256));
    if (dtype_bf16) hipLaunchKernelGGL(producer_rscale_kernel<uint16_t>, g0, dim3(256), 0, s, a, D);
    else hipLaunchKernelGGL(producer_rscale_kernel<float>, g0, dim3(256), 0, s, a, D);
  }
  if (a.mean) {
    const dim3 g1((unsigned)((a.N / 32 + kPartialBlocks - 1) / kPartialBlocks), (unsigned)a.H, (unsigned)a.B),
        g2((unsigned)a.H, (unsigned)a.B);
    if (dtype_bf16) hipLaunchKernelGGL(producer_partials_kernel<uint16_t>, g1, dim3(D / 2), 0, s, a, D);
    else hipLaunchKernelGGL(producer_partials_kernel<float>, g1, dim3(D / 2), 0, s, a, D);
    hipLaunchKernelGGL(producer_mean_kernel, g2, dim3(256), 0, s, a, D);
  }
#define AFP8_Q(DD)                                                                                      \
  if (D == DD) {                                                                                        \
    if (prod) {                                                                                         \
      if (dtype_bf16) hipLaunchKernelGGL((quantize_kernel<DD, uint16_t, NB, true>), grid, dim3(2 * DD), 0, s, a); \
      else hipLaunchKernelGGL((quantize_kernel<DD, float, NB, true>), grid, dim3(2 * DD), 0, s, a);     \
    } else {                                                                                            \
      if (dtype_bf16) hipLaunchKernelGGL((quantize_kernel<DD, uint16_t, NB, false>), grid, dim3(2 * DD), 0, s, a); \
      else hipLaunchKernelGGL((quantize_kernel<DD, float, NB, false>), grid, dim3(2 * DD), 0, s, a);    \
    }                                                                                                   \
    return hipGetLastError();                                                                           \
  }
  AFP8_Q(64)
  AFP8_Q(128)
  AFP8_Q(192)
  AFP8_Q(256)
#undef AFP8_Q
  return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// Saved-output corrections, delta_i = sum_c dO_ic O_ic in FP32 with the
// stored O: stale (Sec. 3.2) from the raw dO; consistent dO (Sec. 3.4,
// QDO) from the dequantized row copy of dO, the operand of dP (E4M3 code
// times the block's power-of-two scale, both exact in FP32).
//
// HBM-bound (4 bytes per channel read for BF16 dO and O, 8 bytes per row
// written).  A lane owns 8 consecutive channels of a row: one 16-byte load
// of each BF16 operand (two for FP32), 8 FMAs in channel order, then a
// butterfly sum over the DV / 8 lanes of the row.  A workgroup of 256 lanes
// holds 2048 / DV rows at a time and each lane takes RPT rows (the rows of
// one workgroup are consecutive (b, n, h) positions, so with the usual
// [B, N, H, D] layout its loads cover one contiguous range); the grid
// strides over the rows beyond that.
template <typename T>
__device__ __forceinline__ void load8(const T* p, float (&v)[8]);
template <>
__device__ __forceinline__ void load8<uint16_t>(const uint16_t* p, float (&v)[8]) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int m = 0; m < 4; m++) {
    v[2 * m] = __uint_as_float(w[m] << 16);
    v[2 * m + 1] = __uint_as_float(w[m] & 0xffff0000u);
  }
}
template <>
__device__ __forceinline__ void load8<float>(const float* p, float (&v)[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// Whether (b, n, h) row `row` lies inside its sequence (per-sequence lengths
// clamped and rounded down to a multiple of 32, a sequence without keys
// empty, as the attention kernels take them); rows past it are neither read
// nor written.
__device__ __forceinline__ bool row_in_sequence(const StaleArgs& a, int64_t row) {
  if (!a.lens_q && !a.lens_k) return true;
  const int64_t n = (row / a.Hq) % a.N, b = row / (a.Hq * a.N);
  if (a.lens_k) {
    const int64_t k = a.lens_k[b];
    if (((k < 0 ? 0 : k > a.Nk ? a.Nk : k) & ~int64_t(31)) == 0) return false;
  }
  if (!a.lens_q) return true;
  const int64_t v = a.lens_q[b];
  return n < ((v < 0 ? 0 : v > a.N ? a.N : v) & ~int64_t(31));
}

template <int DV, typename TD, typename TO, bool QDO>
__global__ __launch_bounds__(256) void stale_rowsum_kernel(StaleArgs a) {
  constexpr int LPR = DV / 8;            // lanes per row
  constexpr int RPW = 256 / LPR;         // rows per workgroup pass
  constexpr int RPT = 2;                 // rows per lane (loads in flight)
  const int t = threadIdx.x, sub = t % LPR, c0 = 8 * sub;
  const int64_t nrows = a.B * a.N * a.Hq;
  for (int64_t base = (int64_t)blockIdx.x * RPW * RPT; base < nrows; base += (int64_t)gridDim.x * RPW * RPT) {
    float acc[RPT];
    int64_t rr[RPT];
#pragma unroll
    for (int u = 0; u < RPT; u++) {
      const int64_t row = base + u * RPW + t / LPR;   // (b, n, h) position
      rr[u] = row;
      acc[u] = 0.f;
      if (row >= nrows || !row_in_sequence(a, row)) continue;
      const int64_t h = row % a.Hq, n = (row / a.Hq) % a.N, b = row / (a.Hq * a.N);
      float dv[8], ov[8];
      if constexpr (QDO) {
        const int64_t r = (b * a.Hq + h) * a.N + n;
        const uint2 cw = *reinterpret_cast<const uint2*>(a.do_code + r * DV + c0);
        const int e = (int)a.do_scale[r * (DV / 32) + c0 / 32] - 127;
#pragma unroll
        for (int k = 0; k < 8; k++) dv[k] = __builtin_ldexpf(fp8_value(k < 4 ? cw.x : cw.y, k & 3), e);
      } else {
        load8<TD>(reinterpret_cast<const TD*>(a.dout) + b * a.ds[0] + n * a.ds[1] + h * a.ds[2] + c0, dv);
      }
      load8<TO>(reinterpret_cast<const TO*>(a.o) + b * a.os[0] + n * a.os[1] + h * a.os[2] + c0, ov);
#pragma unroll
      for (int k = 0; k < 8; k++) acc[u] = __builtin_fmaf(dv[k], ov[k], acc[u]);
    }
#pragma unroll
    for (int u = 0; u < RPT; u++) {
#pragma unroll
      for (int m = LPR / 2; m >= 1; m >>= 1) acc[u] += __shfl_xor(acc[u], m);
      const int64_t row = rr[u];
      if (sub == 0 && row < nrows && row_in_sequence(a, row)) {
        const int64_t h = row % a.Hq, n = (row / a.Hq) % a.N, b = row / (a.Hq * a.N);
        *reinterpret_cast<float2*>(a.delta + ((b * a.Hq + h) * a.N + n) * 2) = make_float2(acc[u], 0.f);
      }
    }
  }
}

template <int DV>
static void launch_rowsum_dv(const StaleArgs& a, dim3 grid, int dout_bf16, int o_bf16, bool qdo, hipStream_t s) {
  if (qdo) {
    if (o_bf16) hipLaunchKernelGGL((stale_rowsum_kernel<DV, uint16_t, uint16_t, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((stale_rowsum_kernel<DV, uint16_t, float, true>), grid, dim3(256), 0, s, a);
  } else if (dout_bf16 && o_bf16) {
    hipLaunchKernelGGL((stale_rowsum_kernel<DV, uint16_t, uint16_t, false>), grid, dim3(256), 0, s, a);
  } else if (dout_bf16) {
    hipLaunchKernelGGL((stale_rowsum_kernel<DV, uint16_t, float, false>), grid, dim3(256), 0, s, a);
  } else if (o_bf16) {
    hipLaunchKernelGGL((stale_rowsum_kernel<DV, float, uint16_t, false>), grid, dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL((stale_rowsum_kernel<DV, float, float, false>), grid, dim3(256), 0, s, a);
  }
}

static hipError_t launch_rowsum(const StaleArgs& a, int dout_bf16, int o_bf16, bool qdo, hipStream_t s) {
  const int64_t nrows = a.B * a.N * a.Hq;
  const int64_t per_wg = 2 * (2048 / a.Dv), wgs = (nrows + per_wg - 1) / per_wg;
  const dim3 grid((unsigned)(wgs < (int64_t(1) << 20) ? wgs : (int64_t(1) << 20)));
  switch (a.Dv) {
    case 64: launch_rowsum_dv<64>(a, grid, dout_bf16, o_bf16, qdo, s); break;
    case 128: launch_rowsum_dv<128>(a, grid, dout_bf16, o_bf16, qdo, s); break;
    case 256: launch_rowsum_dv<256>(a, grid, dout_bf16, o_bf16, qdo, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_stale_rowsum(const StaleArgs& a, int dout_bf16, int o_bf16, hipStream_t s) {
  return launch_rowsum(a, dout_bf16, o_bf16, false, s);
}

hipError_t launch_consistent_rowsum(const StaleArgs& a, int o_bf16, hipStream_t s) {
  return launch_rowsum(a, 1, o_bf16, true, s);
}

// ---------------------------------------------------------------------------
// Buffer clear (a fill kernel rather than a memset node, so callers may
// capture the calls in a graph).
__global__ __launch_bounds__(256) void fill_zero_kernel(float4* p, int64_t n4) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256)
    p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
}

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s) {
  const int64_t n4 = n / 4;  // n is a multiple of 4 at every call site
  if (n4 == 0) return hipSuccess;
  int64_t blocks = (n4 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, reinterpret_cast<float4*>(p), n4);
  return hipGetLastError();
}

}  // namespace afp8
