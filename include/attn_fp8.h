/*
 * attn_fp8.h -- C ABI of the gfx950 (MI355X) block-scaled FP8 attention
 * library with Delta-Matching.
 *
 * Method: "Delta-Matching: Closing the Final Gap of Native 8-bit Training for
 * LLMs".  Softmax attention (Sec. 2.3), causal or not, whose seven matrix products all
 * take FP8 (E4M3) operands with power-of-two (E8M0) block scales, and whose
 * backward row correction is the matched correction
 *     delta_i = sum_j P_ij dP_ij            (Sec. 3.4)
 * computed from the unquantized probabilities and the FP32 products of the
 * FP8 backward operands, in place of the saved-output shortcut
 * sum_c dO_ic O_ic (Sec. 3.2, still available as DELTA_STALE_ROWSUM).
 * Kernel numerics follow App. B.6, with power-of-two block scales:
 *   - FP8 is OCP E4M3FN, round to nearest even; a block's scale is 2^e with e
 *     the smallest integer such that max|x| <= 448 * 2^e (e in [-127, 127]).
 *   - Every input X in {Q, K, V, dO} has two MX copies made from its source
 *     values: a "row" copy in 1x32 blocks along head_dim (operand of the
 *     products that contract head_dim: S = Q K^T, dP = dO V^T) and a "col"
 *     copy in 32x1 blocks along the sequence (operand of the products that
 *     contract the sequence: O = P V, dV = P^T dO, dK = dS^T Q, dQ = dS K).
 *   - Forward probabilities are cast per query row and aligned 32-key group
 *     with a power-of-two scale; the normalizer uses the values before the
 *     cast.  Backward probabilities for dV use the fixed scale 2^-8; dS is
 *     cast in aligned 32x32 (query x key) blocks shared by dQ and dK.
 *
 * Conventions (all entry points):
 *   - Every pointer argument named as device memory is a device (HBM)
 *     address owned by the caller; the library never allocates or frees
 *     device memory.  Between calls it keeps only the thread-local error
 *     text and, per device, the compute-unit count it queries once (the
 *     backward sizes its key-block order by it); attn_fp8_bwd_noalloc
 *     alone uses device memory of the library's own (see there).
 *   - Work is enqueued on `stream` and the call returns without
 *     synchronizing; faults inside a kernel surface at the caller's next
 *     synchronization.
 *   - Return value 0 on success, else a negative attn_fp8_status; on error
 *     nothing is launched and attn_fp8_last_error() describes the problem.
 *   - Causal masking is top-left aligned: key j is visible to query i iff
 *     j <= i (equal query and key lengths).  Without the mask (causal = 0)
 *     every query sees all seqlen_kv keys, which may differ from seqlen:
 *     K, V, dK and dV then have length seqlen_kv.  GQA: query head h reads
 *     KV head floor(h / (heads_q / heads_kv)).  MLA-style problems use
 *     dim_qk != dim_v with heads_q == heads_kv.
 *   - Supported geometry: seqlen % 32 == 0 and seqlen_kv % 32 == 0 (seqlen
 *     may be 0; then seqlen_kv must be too), dim_qk in
 *     {64, 128, 192, 256}, dim_v in {64, 128, 256} with (dim_qk, dim_v) in
 *     {(64,64), (128,128), (256,256), (192,128)}, heads_q % heads_kv == 0.
 *     Batch or head counts of 0 are valid empty problems.  Launch limits
 *     (ATTN_FP8_EUNSUPPORTED beyond them): batch and heads <= 65535,
 *     seqlen, seqlen_kv <= 2^30, batch * heads_q * seqlen < 2^31,
 *     batch * heads_kv * seqlen_kv < 2^30 and max((heads_q / heads_kv) *
 *     seqlen, seqlen_kv) * max(dim_qk, dim_v) < 2^32 (one GQA group's
 *     operands are addressed with 32-bit offsets).
 *   - Strides are in elements; the last (channel) dimension is contiguous.
 *     Device pointers must be 16-byte aligned, and every stride times the
 *     element size must be a multiple of 16 bytes.
 */
#ifndef ATTN_FP8_H
#define ATTN_FP8_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ATTN_FP8_OK = 0,
  ATTN_FP8_EINVAL = -1,        /* NULL pointer, bad shape, stride or dtype */
  ATTN_FP8_EUNSUPPORTED = -2,  /* valid request outside the supported geometry */
  ATTN_FP8_EALIGN = -3,        /* pointer or stride not 16-byte aligned */
  ATTN_FP8_EWORKSPACE = -4,    /* workspace missing or smaller than required */
  ATTN_FP8_EHIP = -5           /* the HIP runtime rejected a launch */
} attn_fp8_status;

typedef enum { ATTN_FP8_DTYPE_F32 = 0, ATTN_FP8_DTYPE_BF16 = 1 } attn_fp8_dtype;

typedef enum {
  ATTN_FP8_DELTA_MATCHING = 0,      /* delta_i = sum_j P_ij dP_ij / sum_j P_ij (Sec. 3.4) */
  ATTN_FP8_DELTA_STALE_ROWSUM = 1,  /* delta_i = sum_c dO_ic O_ic (Sec. 3.2)            */
  ATTN_FP8_DELTA_CONSISTENT_DO = 2, /* delta_i = sum_c dO^_ic O_ic, dO^ the dequantized
                                       row copy of dO (Sec. 3.4, App. B.6)           */
  ATTN_FP8_DELTA_MATCHING_COMPENSATED = 3
                                    /* the matched correction, with every product
                                       P_ij dP_ij formed exactly and summed in FP64, and
                                       the backward's dS formed with the rounding error
                                       of P (-delta_hi) and P (-delta_lo) added back
                                       (an opt-in refinement, not from the paper): the
                                       pre-cast row sums then meet 1e-5 max_j |dS_ij|
                                       down to max|dS| / max P|dP| = 2^-31 (2^-5 with
                                       the plain formation), for about 17 % more time
                                       in the correction pass and 8 % in the main
                                       backward kernel (d = 128, 8K)                  */
} attn_fp8_delta_mode;

enum { ATTN_FP8_QUANT_ROW = 1, ATTN_FP8_QUANT_COL = 2, ATTN_FP8_QUANT_BOTH = 3 };

/* Numerics options of a problem (attn_fp8_problem.flags). */
enum {
  /* Backward probability operand of dV cast with one power-of-two scale per
   * aligned 32x32 (query x key) block, chosen from the block's largest P as
   * for dS', instead of the fixed scale 2^-8 of App. B.6.3.  A variant, not
   * the paper's kernel: the fixed scale keeps probabilities below 2^-14 in
   * E4M3's subnormal range (one or two significant bits, zero below 2^-17),
   * the block scale keeps three mantissa bits at any magnitude. */
  ATTN_FP8_FLAG_PBWD_BLOCK_SCALED = 1,
  /* The protected-dP variant (App. B.6.3, correction variants; App. C.4.2):
   * the backward computes dP = dO V^T from BF16 operands with FP32
   * accumulation and keeps every other product in FP8, with the stale
   * correction.  Its backward is attn_fp8_bwd_protected_dp (attn_fp8_bwd and
   * attn_fp8_bwd_noalloc refuse the flag, attn_fp8_delta refuses the matched
   * modes); attn_fp8_bwd_workspace_size counts its BF16 copies.  Not with
   * ATTN_FP8_FLAG_PBWD_BLOCK_SCALED, nor at head dims (256, 256). */
  ATTN_FP8_FLAG_PROTECTED_DP = 2,
  /* Three isolated score channels instead of one (see the score-precision
   * note at attn_fp8_mx): the channels with the three largest
   * max_h amax_q[b,h,c] * amax_k[b,kv,c] are taken out of the FP8 MFMA and
   * their exact products added in FP32, for inputs with several outlier
   * channels.  An opt-in instantiation of the forward, the matched
   * correction and the backward (one more rank-2 FP32 MFMA per 32 x 32
   * score block); not with ATTN_FP8_FLAG_PBWD_BLOCK_SCALED,
   * ATTN_FP8_FLAG_PROTECTED_DP or the compensated correction. */
  ATTN_FP8_FLAG_ISOLATE3 = 4
};

/* Problem geometry, read-only.  softmax_scale (tau, e.g. 1/sqrt(dim_qk))
 * multiplies the FP32 score accumulator S = Q K^T.
 *
 * Sequences of their own lengths (a padded batch): with seqlens_q (and,
 * without the mask, seqlens_kv) every batch entry b is its own attention
 * problem over its first Lq_b = seqlens_q[b] queries and Lk_b =
 * seqlens_kv[b] keys (Lk_b = Lq_b under the mask); seqlen and seqlen_kv stay
 * the lengths of every array's layout.  Both are nullable device int32 [B]
 * arrays, 4-byte aligned, read by the kernels (the host never reads them).
 * Each length must lie in [0, seqlen] / [0, seqlen_kv] and be a multiple of
 * 32; a length outside that is clamped into it and rounded down to a
 * multiple of 32, so no access ever leaves the arrays (the results are then
 * those of the rounded length).  Positions at or past a sequence's length
 * are padding: the attention kernels never read them and leave their rows
 * of O, LSE, delta and dQ (queries) and dK, dV (keys) unwritten.  A sequence
 * with keys and no queries gets zero dK, dV; one with queries and no keys
 * counts as empty.  The channel maxima of Q and K (channel_amax) come from
 * the quantizer over the whole layout, padding included: keep the padding
 * finite (e.g. zero) for them to describe the sequences. */
typedef struct {
  int64_t batch, seqlen, heads_q, heads_kv, dim_qk, dim_v;
  int32_t causal;          /* 1: top-left causal mask (seqlen_kv == seqlen); 0: no mask */
  float softmax_scale;
  int64_t seqlen_kv;       /* key / value length; 0 stands for seqlen */
  int32_t flags;           /* ATTN_FP8_FLAG_* (0: the paper's numerics) */
  const int32_t* seqlens_q;   /* nullable device [B]: query length of each sequence */
  const int32_t* seqlens_kv;  /* nullable device [B]: key length of each sequence (NULL
                                 under the mask, where it equals the query length) */
  void* cast_dump;            /* nullable device buffer, test instrumentation read by
                                 the instrumented backward only (rowstats given): see
                                 ATTN_FP8_CAST_DUMP_BYTES */
} attn_fp8_problem;

/* Cast dump of the instrumented backward (App. B.6.3's in-kernel casts, for
 * checking them code by code against a reference codec): with
 * problem.cast_dump and rowstats, attn_fp8_bwd also writes, for every
 * (query, key) pair of every 32 x 32 block it computes (blocks it skips are
 * left as they were), with S = B Hq N Nk:
 *   float   P[S]        the backward probability, pre-cast (0 where masked)
 *   float   dS[S]       the score gradient, pre-cast
 *   uint8_t Pc[S]       the code of P' (scale 2^-8, or the block's with
 *                       ATTN_FP8_FLAG_PBWD_BLOCK_SCALED)
 *   uint8_t dSc[S]      the code of dS' in its 32 x 32 block
 *   uint8_t eS[B Hq (N/32) (Nk/32)]  dS' block exponents + 127
 *   uint8_t eP[B Hq (N/32) (Nk/32)]  P' block exponents + 127 (with the flag)
 * each array [b, h, query, key] / [b, h, query block, key block], one after
 * the other in this order, the buffer 16-byte aligned (EALIGN otherwise).
 * For small problems only (about 10 bytes per pair); EINVAL without
 * rowstats. */
#define ATTN_FP8_CAST_DUMP_BYTES(B, Hq, N, Nk) \
  (10 * (size_t)(B) * (Hq) * (N) * (Nk) + 2 * (size_t)(B) * (Hq) * ((N) / 32) * ((Nk) / 32))

/* One MX-quantized operand X of shape [B, N, H, D]; device memory, caller-owned.
 *   code_row  [B, H, N, D]     E4M3FN codes, 1x32 blocks along D
 *   scale_row [B, H, N, D/32]  E8M0 bytes (value 2^(byte-127))
 *   code_col  [B, H, D, N]     E4M3FN codes, 32x1 blocks along N
 *   scale_col [B, H, D, N/32]  E8M0 bytes
 *   channel_amax [B, H, D] float, nullable: max over n of |x[b, n, h, c]|.
 * A copy that an entry point does not read may be NULL.
 *
 * Score precision (all kernels that form S = Q K^T): the gfx950 FP8 MFMA sums
 * each group of 8 consecutive products on a fixed-point grid set by the
 * group's largest exponent (about 11-13 fraction bits), so one outlier
 * channel (a large q_c k_c) rounds away the other products of its group.
 * When both q and k carry channel_amax, the channel c* maximizing
 * max_h amax_q[b,h,c] * amax_k[b,kv,c] (per batch and KV head; lowest index
 * on ties) is taken out of the MFMA (its codes are zeroed in one operand)
 * and its exact product q^_c* k^_c* is added to the FP32 score; with
 * ATTN_FP8_FLAG_ISOLATE3 the three channels with the largest products. */
typedef struct {
  uint8_t* code_row;
  uint8_t* scale_row;
  uint8_t* code_col;
  uint8_t* scale_col;
  float* channel_amax;
} attn_fp8_mx;

/* Input quantizer (App. B.6.1 with power-of-two 1x32 / 32x1 blocks).
 *   x        device, [B, N, H, D] of x_dtype with element strides
 *            strides = {stride_b, stride_n, stride_h}; channel stride 1.
 *   out      receives the copies selected by `which` (ATTN_FP8_QUANT_*).
 *   nonfinite_count  nullable device uint32: incremented by the number of
 *            non-finite inputs seen (codes for them are NaN codes).  The
 *            caller zeroes it.
 *   out->channel_amax, when non-NULL, receives max_n |x| per (b, h, c)
 *            (requires which to include the col copy).
 * D must be one of 64, 128, 192, 256; N % 32 == 0. */
int attn_fp8_quantize(const void* x, int x_dtype, int64_t B, int64_t N, int64_t H, int64_t D,
                      const int64_t strides[3], const attn_fp8_mx* out, int which,
                      uint32_t* nonfinite_count, hipStream_t stream);

/* Options of the input producer (App. B.6.1, Operands, Scaling, and
 * Accumulation; App. B.4 and B.2 for the QK normalization).  Applied in this
 * order to every (token n, head h) row x of D channels:
 *   u  = x, or with rms_gain: the QK normalization (RMSNorm)
 *        r_nh = fl32(1 / sqrt(sum_c x_c^2 / D + rms_eps)), the sum of the
 *        squares taken in FP64 over c ascending and divided, offset (by the
 *        FP32 eps) and inverted in FP64, each step rounded to nearest, then
 *        u_c = bf16(fl32(fl32(x_c r_nh) g_c)), g = rms_gain
 *   r  = u, with channels rope_lo .. rope_lo + rope_dim - 1 rotated (the
 *        fused rotary embedding) when rope_dim > 0: pairs (c, c + rope_dim/2)
 *        of that range, first r_c = u_c cos - u_{c+h} sin, second
 *        r_{c+h} = u_{c+h} cos + u_c sin with h = rope_dim/2 and (cos, sin) =
 *        rope_cs[n][c - rope_lo] of token n; each product and sum rounded to
 *        FP32, the rotated channels then rounded to BF16 (RNE)
 *   x' = fl32(r * prescale)                     (e.g. the query times tau,
 *                                                 with softmax_scale 1 later)
 *   y  = fl32(x' - mean[b, h, c])   if center   (e.g. the key minus its mean
 *                                                 over sequence positions,
 *                                                 per channel and KV head)
 * each rounded once to FP32 (no fused multiply-add).  The mean is the FP64
 * sum of FP64 sums over aligned 32-token blocks (tokens ascending, blocks
 * ascending), divided by N in FP64 and rounded to FP32, so it does not depend
 * on scheduling.  With seqlens (a padded batch, as in attn_fp8_problem) the
 * mean of batch entry b runs over its first L_b tokens only, L_b =
 * seqlens[b] clamped into [0, N] and rounded down to a multiple of 32 (the
 * length the attention kernels take), and is 0 where L_b = 0; every row is
 * still transformed and quantized (the padding's codes are never read).
 *   prescale      finite, nonzero (1 for none)
 *   center        0 or 1
 *   channel_mean  device float [B, H, D], written when center (else unused)
 *   rms_gain      nullable device float [D], 16-byte aligned: the norm's
 *                 per-channel gain; NULL for no normalization
 *   rms_eps       finite, >= 0 (read with rms_gain)
 *   rope_cs       device float [N, rope_dim/2, 2] (cos, sin of token n's
 *                 angle for each pair; the caller's table, so positions and
 *                 frequencies are the caller's), 16-byte aligned; read when
 *                 rope_dim > 0
 *   rope_lo, rope_dim  multiples of 32 with rope_lo + rope_dim <= D
 *                 (EUNSUPPORTED otherwise); rope_dim 0 for no rotation
 *   seqlens       nullable device int32 [B], 4-byte aligned: the sequence
 *                 length of each batch entry for the key mean (read when
 *                 center) */
typedef struct attn_fp8_producer {
  float prescale;
  int32_t center;
  float* channel_mean;
  const float* rms_gain;
  float rms_eps;
  const float* rope_cs;
  int64_t rope_lo;
  int64_t rope_dim;
  const int32_t* seqlens;
} attn_fp8_producer;

/* Workspace bytes attn_fp8_quantize_producer needs with these options: the
 * key-mean partial sums (FP64 [B, H, N/32, D]) when center, then the norm's
 * row scales (FP32 [B, N, H]) when rms_gain, each rounded up to 256 bytes;
 * 0 when neither.  Checks the options and sizes as the producer does.
 * Returns 0 / negative status. */
int attn_fp8_producer_workspace_size(int64_t B, int64_t N, int64_t H, int64_t D,
                                     const attn_fp8_producer* opt, size_t* bytes);

/* Input producer + quantizer: the quantizer above applied to the values y
 * that the options (attn_fp8_producer) define.  The backward takes the
 * resulting codes as given: gradients are those of the transformed operands
 * (straight-through, App. B.6.3; the key gradient is not re-centered and
 * refers to the normalized, rotated key).
 *   opt        the options (not NULL)
 *   workspace  device, at least attn_fp8_producer_workspace_size() bytes,
 *              256-byte aligned (may be NULL when that size is 0); its
 *              contents on entry do not matter and on return are unspecified
 * Other arguments, checks and outputs as attn_fp8_quantize (channel_amax,
 * when requested, is of the transformed values).  The input is read once
 * more for the norm's row scales and once more for the key mean. */
int attn_fp8_quantize_producer(const void* x, int x_dtype, int64_t B, int64_t N, int64_t H,
                               int64_t D, const int64_t strides[3], const attn_fp8_producer* opt,
                               void* workspace, size_t workspace_bytes, const attn_fp8_mx* out,
                               int which, uint32_t* nonfinite_count, hipStream_t stream);

/* Forward (Sec. 2.3; App. B.6.2): S = tau * Q K^T, online softmax with
 * power-of-two rescaling, FP8 probabilities per 32-key group, O = P V / l.
 *   q, k     row copies used;  v  col copy used.
 *   o        device, [B, N, Hq, Dv] of o_dtype, strides o_strides {b, n, h}.
 *   lse      device float [B, Hq, N]: natural-log LSE_i = m_i + ln l_i. */
int attn_fp8_fwd(const attn_fp8_problem* p, const attn_fp8_mx* q, const attn_fp8_mx* k,
                 const attn_fp8_mx* v, void* o, int o_dtype, const int64_t o_strides[3],
                 float* lse, hipStream_t stream);

/* Row correction (Sec. 3.4 / Sec. 3.2; App. B.6.3 "Matched correction").
 *   MATCHING:     reads q, k, v, dout row copies and lse; recomputes
 *                 P = 2^(S log2 e - LSE log2 e) and dP = dO_q V_q^T in FP32,
 *                 reduces sum P dP and sum P in FP32 per 32-key group, then
 *                 in FP64, and stores delta = num / den.
 *   STALE_ROWSUM: reads dout_raw [B,N,Hq,Dv] (dout_dtype, strides
 *                 dout_strides) and the stored output o (o_dtype,
 *                 o_strides); delta = sum_c dO_ic O_ic in FP32.
 *   CONSISTENT_DO: reads the row copy of dout (code_row, scale_row) and o;
 *                 delta = sum_c dO^_ic O_ic in FP32 with dO^ = E4M3 code
 *                 times the block's E8M0 scale (exact in FP32).
 * Pointers the mode does not read may be NULL.
 *   delta    device float [B, Hq, N, 2]: (hi, lo) with delta ~= hi + lo
 *            (lo = 0 for STALE_ROWSUM and CONSISTENT_DO). */
int attn_fp8_delta(const attn_fp8_problem* p, int delta_mode, const attn_fp8_mx* q,
                   const attn_fp8_mx* k, const attn_fp8_mx* v, const attn_fp8_mx* dout,
                   const float* lse, const void* dout_raw, int dout_dtype,
                   const int64_t dout_strides[3], const void* o, int o_dtype,
                   const int64_t o_strides[3], float* delta, hipStream_t stream);

/* Workspace bytes attn_fp8_bwd needs for this problem: the FP8 dS' operand
 * units (per query head, 2048 code bytes + 2 exponent bytes for every
 * 32-query block x 64-key step at or before the diagonal), the internal delta
 * buffer [B,Hq,N,2], 16-byte per-query records [B,Hq,N] that the main kernel
 * streams with its query tiles, and per-tile packed col scales (Q and dO per
 * 64-query tile, K per 64-key tile).  Returns 0 / negative status. */
int attn_fp8_bwd_workspace_size(const attn_fp8_problem* p, size_t* bytes);

/* Backward (Sec. 2.3; App. B.6.3).  Key-major pass: recompute S, P, dP;
 * dS = P (dP - delta) formed as fma(P, dP, fl(P * (-d))) with d the
 * correction rounded to FP32 (the hi part; P dP enters exactly and every
 * rounding is of its own element); P' = C8(256 P) 2^-8 (P clamped to
 * [0, 1]); dS' cast per 32x32 block; dV += P'^T dO_col, dK += dS'^T Q_col (summed over the
 * KV group in FP32), dS' stored in the workspace; then a query-major pass
 * computes dQ = dS' K_col.  dQ and dK are multiplied by tau and stored.
 *   delta_in nullable device float [B, Hq, N, 2]: when given, used as the
 *            correction (and delta_mode is ignored); else the correction is
 *            computed first per delta_mode, exactly as attn_fp8_delta does.
 *   dq [B,N,Hq,Dqk], dk [B,N,Hkv,Dqk], dv [B,N,Hkv,Dv]: device, grad_dtype,
 *            element strides {b, n, h} in dq_strides / dk_strides / dv_strides.
 *   workspace device, at least attn_fp8_bwd_workspace_size() bytes, 256-byte
 *            aligned; contents on entry are ignored.
 *   rowstats nullable device double [B, Hq, N, 7], zeroed by the caller:
 *            accumulates, per query row and over all keys, sum dS, sum |dS|,
 *            sum dS', max |dS|, sum |dS'|, max P |dP| and sum P' (FP64 sums
 *            of the FP32 values before the cast, dS and P dP, and of the
 *            decoded FP8 operands dS' and P'; debug instrumentation of
 *            App. C.1; a separate, slower kernel instantiation whose
 *            gradients are bitwise those of the plain one).
 *   main_events nullable pointer to two events: recorded on `stream`
 *            immediately before and after the main backward kernel, so a
 *            caller can time that kernel alone. */
int attn_fp8_bwd(const attn_fp8_problem* p, int delta_mode, const attn_fp8_mx* q,
                 const attn_fp8_mx* k, const attn_fp8_mx* v, const attn_fp8_mx* dout,
                 const float* lse, const void* dout_raw, int dout_dtype,
                 const int64_t dout_strides[3], const void* o, int o_dtype,
                 const int64_t o_strides[3], const float* delta_in, void* dq, void* dk, void* dv,
                 int grad_dtype, const int64_t dq_strides[3], const int64_t dk_strides[3],
                 const int64_t dv_strides[3], void* workspace, size_t workspace_bytes,
                 double* rowstats, const hipEvent_t* main_events, hipStream_t stream);

/* Protected-dP backward (App. B.6.3, correction variants; App. C.4.2, the
 * SageBwd-style precision split): attn_fp8_bwd's passes with dP = dO V^T
 * formed from BF16 operands (dout_raw and v_raw rounded to BF16, nearest
 * even, products exact, FP32 MFMA accumulation) instead of the FP8 row
 * copies, and the stale correction delta_i = sum_c dO_ic O_ic (or delta_in).
 * S, P', dS', dV, dK and dQ keep their FP8 operands and casts.
 *   p        flags must hold ATTN_FP8_FLAG_PROTECTED_DP (so that
 *            attn_fp8_bwd_workspace_size counts the BF16 copies of dO and V
 *            the call packs into the workspace); head dims (64, 64),
 *            (128, 128) or (192, 128)
 *   q, k     row and col copies;  dout  col copy (the operand of dV)
 *   dout_raw device [B, N, Hq, Dv] of dout_dtype with dout_strides: the
 *            operand of dP and of the stale correction
 *   v_raw    device [B, Nk, Hkv, Dv] of v_dtype with v_strides, 16-byte
 *            aligned rows: the operand of dP
 *   o        the stored output (stale correction; unused with delta_in)
 * Other arguments, outputs and errors as attn_fp8_bwd. */
int attn_fp8_bwd_protected_dp(const attn_fp8_problem* p, const attn_fp8_mx* q,
                              const attn_fp8_mx* k, const attn_fp8_mx* dout, const float* lse,
                              const void* dout_raw, int dout_dtype, const int64_t dout_strides[3],
                              const void* v_raw, int v_dtype, const int64_t v_strides[3],
                              const void* o, int o_dtype, const int64_t o_strides[3],
                              const float* delta_in, void* dq, void* dk, void* dv, int grad_dtype,
                              const int64_t dq_strides[3], const int64_t dk_strides[3],
                              const int64_t dv_strides[3], void* workspace, size_t workspace_bytes,
                              double* rowstats, hipStream_t stream);

/* Backward without any device allocation, for callers that cannot allocate
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation).  Same arguments, checks and results as attn_fp8_bwd, whose
 * kernels it runs, except that the workspace is the library's own scratch:
 * ATTN_FP8_NOALLOC_SCRATCH_BYTES of device memory per device, held from the
 * call that first uses a device until the process ends (its device address
 * is looked up once per device with that device current).
 *   - Problems whose attn_fp8_bwd_workspace_size exceeds the scratch are
 *     rejected with ATTN_FP8_EUNSUPPORTED before anything is launched.
 *   - The call allocates and frees nothing (no hipMalloc/hipFree, no
 *     allocating library routine).
 *   - All calls on one device share its scratch and leave their contents
 *     there; nothing in it needs to start at zero.  Calls that overlap on one
 *     device (other streams, other threads) race on it: serialize them. */
#define ATTN_FP8_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int attn_fp8_bwd_noalloc(const attn_fp8_problem* p, int delta_mode, const attn_fp8_mx* q,
                         const attn_fp8_mx* k, const attn_fp8_mx* v, const attn_fp8_mx* dout,
                         const float* lse, const void* dout_raw, int dout_dtype,
                         const int64_t dout_strides[3], const void* o, int o_dtype,
                         const int64_t o_strides[3], const float* delta_in, void* dq, void* dk,
                         void* dv, int grad_dtype, const int64_t dq_strides[3],
                         const int64_t dk_strides[3], const int64_t dv_strides[3], double* rowstats,
                         const hipEvent_t* main_events, hipStream_t stream);

/* Thread-local text describing the last error returned on this thread. */
const char* attn_fp8_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* ATTN_FP8_H */
