// Kernel argument blocks and launchers (internal to the library; the public
// interface is include/attn_fp8.h).  Host code validates every argument
// before a launcher is called; kernels assume the geometry checked there.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace afp8 {

// Per-row statistics of the instrumented backward (FP64, per query row over
// all keys): sum dS, sum |dS|, sum dS', max |dS|, sum |dS'|, max P |dP|,
// sum P' (dS, P, dP the FP32 values before the cast; dS', P' the decoded
// FP8 operands).
constexpr int kRowStats = 7;

struct QuantArgs {
  const void* x;
  int64_t sb, sn, sh;        // element strides of x (channel stride 1)
  int64_t B, N, H;
  uint8_t *code_row, *scale_row, *code_col, *scale_col;
  int which;                 // bit 0 row copy, bit 1 col copy
  uint32_t* nonfinite;       // nullable
  float* chan_amax;          // nullable [B, H, D]: max over tokens of |x| (zeroed before the launch)
  // input producer (all optional): x' = fl32(x * prescale), then
  // fl32(x' - mean[b, h, c]) when mean is given; partials: [B, H, N/32, D]
  // FP64 block sums of x' the mean is formed from
  float prescale;            // 1 for none
  float* mean;               // nullable [B, H, D]
  double* partials;          // required with mean
  const int32_t* lens;       // nullable [B]: each sequence's length for the mean
  // fused rotary embedding before the prescale (nullable): channels
  // rope_lo .. rope_lo + rope_dim - 1 rotated in pairs (c, c + rope_dim/2)
  // by rope[n][c][{cos, sin}] ([N, rope_dim/2, 2] FP32) and rounded to BF16
  const float* rope;
  int rope_lo, rope_dim;
  // QK normalization before the rotary embedding (nullable gain [D]): each
  // (token, head) row times rscale[b, n, h] (FP32, from FP64 statistics,
  // written by producer_rscale_kernel), times the gain, rounded to BF16
  const float* gain;
  double eps;
  float* rscale;             // workspace [B, N, H], with gain
};

struct StaleArgs {
  const void* dout;                    // raw dO (stale), or NULL when the row copy below is read
  const uint8_t* do_code;              // consistent dO: row codes [B,Hq,N,Dv]
  const uint8_t* do_scale;             //                and scales [B,Hq,N,Dv/32]
  int64_t ds[3];
  const void* o;
  int64_t os[3];
  float* delta;              // [B, Hq, N, 2]
  int64_t B, N, Hq;
  int Dv;
  // nullable [B]: query and key length of each sequence (rows past the
  // query length, and every row of a sequence without keys, are skipped)
  const int32_t* lens_q;
  const int32_t* lens_k;
  int64_t Nk;
};

// Shared by the forward, the matched-correction pass and the backward.
// Query-side arrays have the query length N, key-side arrays (K, V, dK, dV,
// the K col scales per 64-key step) the key length Nk (equal when causal).
struct AttnArgs {
  int64_t B, N, Hq, Hkv, G;  // G = Hq / Hkv
  int64_t Nk;                // key / value length
  int causal;                // 1: key j visible to query i iff j <= i; 0: every key
  int comp;                  // compensated correction: FP64 products in the correction pass,
                             // compensated dS formation in the backward
  int pmx;                   // block-scaled backward probability operand (one scale per 32x32 block)
  int pdp;                   // protected dP: dP = dO V^T from the BF16 copies below
  int iso3;                  // three isolated score channels instead of one
  float c;                   // tau * log2(e), applied to the score accumulator
  float tau;
  const uint8_t *q_code, *q_scale;     // row copy of Q      [B,Hq,N,Dqk], [B,Hq,N,Dqk/32]
  const uint8_t *k_code, *k_scale;     // row copy of K      [B,Hkv,Nk,Dqk]
  const uint8_t *v_code, *v_scale;     // row copy of V      [B,Hkv,Nk,Dv]
  const uint8_t *do_code, *do_scale;   // row copy of dO     [B,Hq,N,Dv]
  const uint8_t *qc_code, *qc_scale;   // col copy of Q      [B,Hq,Dqk,N], [B,Hq,Dqk,N/32]
  const uint8_t *kc_code, *kc_scale;   // col copy of K      [B,Hkv,Dqk,Nk]
  const uint8_t *vc_code, *vc_scale;   // col copy of V      [B,Hkv,Dv,Nk]
  const uint8_t *doc_code, *doc_scale; // col copy of dO     [B,Hq,Dv,N]
  const uint16_t* do_bf16;             // protected dP: dO   [B,Hq,N,Dv] BF16 (workspace)
  const uint16_t* v_bf16;              //               V    [B,Hkv,Nk,Dv] BF16 (workspace)
  const float* q_amax;                 // nullable [B,Hq,Dqk] per-channel max |q|
  const float* k_amax;                 // nullable [B,Hkv,Dqk] per-channel max |k|
  const float* lse;                    // [B,Hq,N]
  float* lse_out;
  const float* delta;                  // [B,Hq,N,2]
  float* delta_out;
  float* rows;                         // [B,Hq,ceil(N/64)] x 1 KB backward per-query values (workspace)
  uint8_t* tile_cs;                    // [B,Hq,ceil(N/64),2(Dqk+Dv)] backward per-tile col scales (workspace)
  uint8_t* tile_kcs;                   // [B,Hkv,ceil(Nk/64),2 Dqk] K col scales per 64-key step (workspace)
  void* o;  int64_t os[3]; int o_bf16;
  uint8_t* ds_units;                   // dQ operand units (workspace): 2048 B per (head, 32 queries, 64 keys)
  uint8_t* ds_exp;                     // their block exponents, 2 B per unit
  void* dq; int64_t dqs[3];
  void* dk; int64_t dks[3];
  void* dv; int64_t dvs[3];
  int grad_bf16;
  int bwd_cohort;                      // backward: workgroups of one KV head that run at once (set at launch)
  double* rowstats;                    // nullable [B,Hq,N,kRowStats]
  void* cast_dump;                     // nullable, with rowstats: pre-cast P, dS and their codes
  // Padded batch of sequences of their own lengths (nullable [B] each):
  // sequence b has lens_q[b] queries and lens_k[b] keys, at the first
  // positions of the N / Nk of the layouts above; NULL: N and Nk
  const int32_t* lens_q;
  const int32_t* lens_k;
};

// Query and key length of sequence b as the kernels use them: the given
// length clamped into [0, N] / [0, Nk] and rounded down to a multiple of 32
// (so no access leaves the arrays), the key length equal to the query length
// under the mask, and no queries where there are no keys.
struct SeqLens {
  int q, k;
};
template <bool CAUSAL>
__device__ __forceinline__ SeqLens seq_lens(const AttnArgs& a, int b, int N, int Nk) {
  int q = N, k = Nk;
  if (a.lens_q) {
    const int v = a.lens_q[b];
    q = (v < 0 ? 0 : v > N ? N : v) & ~31;
  }
  if (CAUSAL) {
    k = q;
  } else if (a.lens_k) {
    const int v = a.lens_k[b];
    k = (v < 0 ? 0 : v > Nk ? Nk : v) & ~31;
  }
  if (k == 0) q = 0;
  return SeqLens{q, k};
}

hipError_t launch_quantize(const QuantArgs& a, int D, int dtype_bf16, hipStream_t s);
hipError_t launch_stale_rowsum(const StaleArgs& a, int dout_bf16, int o_bf16, hipStream_t s);
hipError_t launch_consistent_rowsum(const StaleArgs& a, int o_bf16, hipStream_t s);
hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t s);
hipError_t launch_fwd(const AttnArgs& a, int dqk, int dv, hipStream_t s);
hipError_t launch_delta_matching(const AttnArgs& a, int dqk, int dv, hipStream_t s);
hipError_t launch_bwd_prep(const AttnArgs& a, int dqk, int dv, hipStream_t s);
hipError_t launch_bwd(const AttnArgs& a, int dqk, int dv, hipStream_t s);
hipError_t launch_dq(const AttnArgs& a, int dqk, hipStream_t s);
hipError_t launch_pack_bf16(const void* x, int bf16, const int64_t st[3], int64_t B, int64_t N, int64_t H, int D,
                            const int32_t* lens, uint16_t* out, hipStream_t s);
// stored dQ operand units of one head: one per (32-query block, 64-key
// step) that holds a visible key
int64_t dq_units_per_head(int64_t nq, int64_t nk, bool causal);

}  // namespace afp8
