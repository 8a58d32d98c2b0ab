// Direct global -> LDS staging (global_load_lds, gfx950) shared by the
// attention kernels: swizzled unpadded tile layouts, the loads that fill
// them, the fragment reads, and the barriers that go with them.
#pragma once

#include "common.hpp"

namespace afp8 {

// XOR swizzle of the 16-byte chunks of a row-major tile with D-byte rows
// (16 consecutive rows read at one logical chunk land on distinct banks).
template <int D>
__device__ __forceinline__ int swz_row(int r) {
  if constexpr (D == 64) return (r >> 2) & 3;
  else if constexpr (D == 128) return (r >> 1) & 7;
  else if constexpr (D == 192) return (r >> 2) & 3;
  else return r & 15;
}
// col tiles have 64-byte rows (one channel, 64 queries)
__device__ __forceinline__ int swz_col(int c) { return (c >> 2) & 3; }

// LDS byte pointer; direct-to-LDS loads take their destination in this form
// (pointers derived from the __shared__ arrays themselves, never from a
// generic pointer)
typedef __attribute__((address_space(3))) uint8_t lds8;

// Direct loads are MUBUF buffer loads with the LDS bit, over a buffer
// resource of a wave-uniform base address: the FLAT-encoded global_load_lds
// form makes the compiler treat every LDS access as completing out of order
// while one is in flight, so each LDS wait would drain all outstanding reads
// (lgkmcnt(0)); buffer loads count in vmcnt only, so operand reads for the
// next MFMA can stay in flight while the current one waits.  `off` is the
// lane's byte offset from the base; offsets at or past `bytes` read as zero.
struct Buf {
  __amdgpu_buffer_rsrc_t r;
};
__device__ __forceinline__ Buf make_buf(const void* base, uint32_t bytes) {
  // 0x00020000: raw (untyped) buffer, 32-bit data format (gfx9 family)
  return Buf{__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000)};
}
__device__ __forceinline__ void dma16(const Buf& b, uint32_t off, lds8* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(b.r, (__attribute__((address_space(3))) void*)lds_base, 16, (int)off, 0, 0, 0);
}
__device__ __forceinline__ void dma4(const Buf& b, uint32_t off, lds8* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(b.r, (__attribute__((address_space(3))) void*)lds_base, 4, (int)off, 0, 0, 0);
}
// The same with a wave-uniform part of the offset in a scalar register
// (address = base + soff + voff): the per-lane part can stay in a long-lived
// register while the head and tile offsets change.  The buffer's range check
// covers voff only, so callers keep soff + voff inside the buffer themselves.
__device__ __forceinline__ void dma16s(const Buf& b, uint32_t voff, uint32_t soff, lds8* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(b.r, (__attribute__((address_space(3))) void*)lds_base, 16, (int)voff,
                                           (int)soff, 0, 0);
}
__device__ __forceinline__ void dma4s(const Buf& b, uint32_t voff, uint32_t soff, lds8* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(b.r, (__attribute__((address_space(3))) void*)lds_base, 4, (int)voff,
                                           (int)soff, 0, 0);
}

// Waits for this wave's LDS writes and direct-to-LDS loads (and any other
// vector memory operation), then a workgroup barrier ordered for LDS only.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0x0070);   // vmcnt(0) lgkmcnt(0)
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Workgroup barrier after this wave's LDS writes only: direct-to-LDS loads
// in flight stay in flight (an LDS release fence would wait for them, since
// they write LDS), so the ordering of the surrounding LDS accesses is kept
// by compiler barriers instead.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Row-major code tile [ROWS][D] (rows i0.., clamped to the sequence) into
// LDS, swizzled; wave w issues instructions w, w + NWK, ...
template <int D, int NWK, int ROWS = 64>
__device__ __forceinline__ void dma_rows(lds8* lds, const uint8_t* code, int i0, int N, int w, int lane) {
  constexpr int NI = ROWS * D / 1024;
  const Buf b = make_buf(code, (uint32_t)N * D);
  for (int k = w; k < NI; k += NWK) {
    const int off = 1024 * k + 16 * lane;
    const int r = off / D, p = (off % D) / 16;
    const int row = i0 + r < N ? i0 + r : N - 1;
    dma16(b, (uint32_t)(row * D + 16 * (p ^ swz_row<D>(r))), lds + 1024 * k);
  }
}
// Col-copy code tile: channels [0, D), queries [i0, i0 + 64) of a [D][N]
// matrix, clamped to the first lim (<= N, >= 16) -> [D][64].
template <int D, int NWK>
__device__ __forceinline__ void dma_cols(lds8* lds, const uint8_t* code, int i0, int N, int lim, int w, int lane) {
  constexpr int NI = D * 64 / 1024;
  const Buf b = make_buf(code, (uint32_t)D * N);
  for (int k = w; k < NI; k += NWK) {
    const int off = 1024 * k + 16 * lane;
    const int c = off / 64, p = (off % 64) / 16;
    const int q = p ^ swz_col(c);
    const int col = i0 + 16 * q < lim - 16 ? i0 + 16 * q : lim - 16;
    dma16(b, (uint32_t)(c * N + col), lds + 1024 * k);
  }
}
// Row-copy scales of ROWS rows: ROWS * D / 32 contiguous bytes (clamped).
template <int D, int NWK, int ROWS = 64>
__device__ __forceinline__ void dma_row_scales(lds8* lds, const uint8_t* scale, int i0, int N, int w, int lane,
                                               int first_wave) {
  constexpr int BYTES = ROWS * D / 32, NI = (BYTES + 255) / 256;
  const Buf b = make_buf(scale, (uint32_t)N * (D / 32));
  for (int k = 0; k < NI; k++) {
    if ((first_wave + k) % NWK != w) continue;
    const int off = 256 * k + 4 * lane;
    if (off < BYTES) {
      const int g = i0 * (D / 32) + off, lim = N * (D / 32) - 4;
      dma4(b, (uint32_t)(g < lim ? g : lim), lds + 256 * k);
    }
  }
}

// dma_row_scales for a scale matrix at byte offset `head` inside buffer b.
template <int D, int NWK, int ROWS = 64>
__device__ __forceinline__ void dma_row_scales_s(lds8* lds, const Buf& b, uint32_t head, int i0, int N, int w,
                                                 int lane, int first_wave) {
  constexpr int BYTES = ROWS * D / 32, NI = (BYTES + 255) / 256;
  for (int k = 0; k < NI; k++) {
    if ((first_wave + k) % NWK != w) continue;
    const int off = 256 * k + 4 * lane;
    if (off < BYTES) {
      const int g = i0 * (D / 32) + off, lim = N * (D / 32) - 4;
      dma4s(b, (uint32_t)(g < lim ? g : lim), head, lds + 256 * k);
    }
  }
}

// A/B fragment (row `row`, k-step t, half hf) of a swizzled row-major tile.
template <int D>
__device__ __forceinline__ v8i frag_rows_swz(const uint8_t* tile, int row, int t, int hf) {
  const int s = swz_row<D>(row), c = 4 * t + hf;
  const uint8_t* base = tile + row * D;
  const uint4 lo = *reinterpret_cast<const uint4*>(base + 16 * (c ^ s));
  const uint4 hi = *reinterpret_cast<const uint4*>(base + 16 * ((c + 2) ^ s));
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}
// Stores a fragment where frag_rows_swz<D>(tile, row, t, hf) reads it.
template <int D>
__device__ __forceinline__ void kv_store(uint8_t* tile, int row, int t, int hf, const v8i& f) {
  const int s = swz_row<D>(row), c = 4 * t + hf;
  uint8_t* base = tile + row * D;
  *reinterpret_cast<uint4*>(base + 16 * (c ^ s)) = make_uint4((uint32_t)f[0], (uint32_t)f[1], (uint32_t)f[2], (uint32_t)f[3]);
  *reinterpret_cast<uint4*>(base + 16 * ((c + 2) ^ s)) = make_uint4((uint32_t)f[4], (uint32_t)f[5], (uint32_t)f[6], (uint32_t)f[7]);
}
// B fragment of a swizzled col tile: channel ch, queries 16 hf.. and 32 + 16 hf..
__device__ __forceinline__ v8i frag_cols_swz(const uint8_t* tile, int ch, int hf) {
  const int s = swz_col(ch);
  const uint8_t* base = tile + ch * 64;
  const uint4 lo = *reinterpret_cast<const uint4*>(base + 16 * (hf ^ s));
  const uint4 hi = *reinterpret_cast<const uint4*>(base + 16 * ((hf + 2) ^ s));
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}
// The same with explicit chunk indices (clo: bytes 0..15, chi: 16..31, each
// before the swizzle).
__device__ __forceinline__ v8i frag_cols_chunks(const uint8_t* tile, int ch, int clo, int chi) {
  const int s = swz_col(ch);
  const uint8_t* base = tile + ch * 64;
  const uint4 lo = *reinterpret_cast<const uint4*>(base + 16 * (clo ^ s));
  const uint4 hi = *reinterpret_cast<const uint4*>(base + 16 * (chi ^ s));
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// Precomputed plans for the tile loads of one wave: the lane's byte offset in
// the source matrix for its first load instruction (k = w); the later ones
// (k = w + NWK j) sit a fixed stride further wherever the swizzle repeats
// with that stride, so a whole tile costs one address add per load.  A tile
// that reaches past the sequence end takes the clamping loaders above.
//
// Row tile: rows [i0, i0 + ROWS) of a [N][D] code matrix -> LDS [ROWS][D].
template <int D, int NWK, int ROWS>
struct RowLoads {
  static constexpr int NI = ROWS * D / 1024, NS = (NI + NWK - 1) / NWK;
  // the instructions of one wave are 1024 NWK / D rows apart; the swizzle
  // repeats every 16 rows for every D but 192
  static constexpr bool STRIDED = (1024 * NWK) % D == 0 && ((1024 * NWK) / D) % 16 == 0;
  uint32_t off[STRIDED ? 1 : NS];   // r D + 16 (swizzled chunk), r the lane's row in the tile
  __device__ __forceinline__ void init(int w, int lane) {
#pragma unroll
    for (int j = 0; j < (STRIDED ? 1 : NS); j++) {
      const int o = 1024 * (w + NWK * j) + 16 * lane;
      const int r = o / D, p = (o % D) / 16;
      off[j] = (uint32_t)(r * D + 16 * (p ^ swz_row<D>(r)));
    }
  }
  __device__ __forceinline__ void issue(lds8* lds, const uint8_t* code, int i0, int N, int w, int lane) const {
    if (i0 + ROWS > N) {
      dma_rows<D, NWK, ROWS>(lds, code, i0, N, w, lane);
      return;
    }
    const Buf b = make_buf(code, (uint32_t)N * D);
    const uint32_t base = (uint32_t)i0 * D;
#pragma unroll
    for (int j = 0; j < NS; j++) {
      const int k = w + NWK * j;
      if (k < NI) dma16(b, base + (STRIDED ? off[0] + 1024 * NWK * j : off[j]), lds + 1024 * k);
    }
  }
  // Rows of a matrix at byte offset `head` inside buffer b (head: wave-uniform).
  __device__ __forceinline__ void issue_s(lds8* lds, const Buf& b, uint32_t head, int i0, int N, int w,
                                          int lane) const {
    if (i0 + ROWS > N) {
      for (int k = w; k < NI; k += NWK) {
        const int o = 1024 * k + 16 * lane;
        const int r = o / D, p = (o % D) / 16;
        const int row = i0 + r < N ? i0 + r : N - 1;
        dma16s(b, (uint32_t)(row * D + 16 * (p ^ swz_row<D>(r))), head, lds + 1024 * k);
      }
      return;
    }
    const uint32_t sb = head + (uint32_t)i0 * D;
#pragma unroll
    for (int j = 0; j < NS; j++) {
      const int k = w + NWK * j;
      if (k < NI) dma16s(b, STRIDED ? off[0] + 1024 * NWK * j : off[j], sb, lds + 1024 * k);
    }
  }
};

// Col tile: channels [0, D), sequence positions [i0, i0 + COLS) of a [D][N]
// code matrix -> LDS [D][COLS] (COLS = 64: the col-tile swizzle; 128: the
// 128-byte row swizzle; both repeat with the channel step of one wave's
// instructions).  Positions at or past lim (<= N, >= 16) are clamped to the
// last 16 before it.
template <int D, int NWK, int COLS = 64>
struct ColLoads {
  static_assert(COLS == 64 || COLS == 128, "col tile width");
  static constexpr int NI = D * COLS / 1024, NS = (NI + NWK - 1) / NWK;
  static constexpr int CSTEP = 1024 * NWK / COLS;   // channels between a wave's instructions
  static_assert(CSTEP % 16 == 0, "swizzle period");
  uint32_t off;   // c N + 16 q of the first instruction (q the swizzled chunk)
  int cstride;    // CSTEP N
  __device__ __forceinline__ void init(int w, int lane, int N) {
    const int o = 1024 * w + 16 * lane;
    const int c = o / COLS, p = (o % COLS) / 16;
    const int q = COLS == 64 ? (p ^ swz_col(c)) : (p ^ swz_row<128>(c));
    off = (uint32_t)(c * N + 16 * q);
    cstride = CSTEP * N;
  }
  __device__ __forceinline__ void issue(lds8* lds, const uint8_t* code, int i0, int N, int lim, int w,
                                        int lane) const {
    const Buf b = make_buf(code, (uint32_t)D * N);
    if (i0 + COLS > lim) {
      // ragged tile: clamp every 16-byte piece into its row
#pragma unroll
      for (int j = 0; j < NS; j++) {
        const int k = w + NWK * j;
        if (k >= NI) break;
        const int o = 1024 * k + 16 * lane;
        const int c = o / COLS, p = (o % COLS) / 16;
        const int q = COLS == 64 ? (p ^ swz_col(c)) : (p ^ swz_row<128>(c));
        const int col = i0 + 16 * q < lim - 16 ? i0 + 16 * q : lim - 16;
        dma16(b, (uint32_t)(c * N + col), lds + 1024 * k);
      }
      return;
    }
    const uint32_t base = (uint32_t)i0 + off;
#pragma unroll
    for (int j = 0; j < NS; j++) {
      const int k = w + NWK * j;
      if (k < NI) dma16(b, base + (uint32_t)(j * cstride), lds + 1024 * k);
    }
  }
  // The same for a matrix at byte offset `head` inside buffer b.
  __device__ __forceinline__ void issue_s(lds8* lds, const Buf& b, uint32_t head, int i0, int N, int lim, int w,
                                          int lane) const {
    if (i0 + COLS > lim) {
#pragma unroll
      for (int j = 0; j < NS; j++) {
        const int k = w + NWK * j;
        if (k >= NI) break;
        const int o = 1024 * k + 16 * lane;
        const int c = o / COLS, p = (o % COLS) / 16;
        const int q = COLS == 64 ? (p ^ swz_col(c)) : (p ^ swz_row<128>(c));
        const int col = i0 + 16 * q < lim - 16 ? i0 + 16 * q : lim - 16;
        dma16s(b, (uint32_t)(c * N + col), head, lds + 1024 * k);
      }
      return;
    }
    const uint32_t sb = head + (uint32_t)i0;
#pragma unroll
    for (int j = 0; j < NS; j++) {
      const int k = w + NWK * j;
      if (k < NI) dma16s(b, off + (uint32_t)(j * cstride), sb, lds + 1024 * k);
    }
  }
};

}  // namespace afp8
