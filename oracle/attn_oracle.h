/*
 * attn_oracle.h -- reference oracle for block-scaled FP8 attention with
 * Delta-Matching.  TEST INFRASTRUCTURE ONLY: the product path never links,
 * loads or calls this library; only the tests, the smoke check and the CPU
 * baseline leg of the benchmark do.
 *
 * Plain, slow, FP64.  Every function states the passage of the paper
 * ("Delta-Matching: Closing the Final Gap of Native 8-bit Training for LLMs")
 * it follows.  Where the paper leaves a choice open, the reading taken is
 * stated at the function.
 *
 * Layouts (all arrays dense, row-major, caller-owned):
 *   raw inputs          x[B, N, H, D]
 *   row copy  codes     [B, H, N, D]      scales [B, H, N, D/32]   (1x32 blocks along D)
 *   col copy  codes     [B, H, D, N]      scales [B, H, D, N/32]   (32x1 blocks along N)
 *   dequantized operand [B, H, N, D]      (both copies are returned in this layout)
 *   O, dQ               [B, N, Hq, D]     LSE, delta [B, Hq, N]
 *   dK, dV              [B, Nk, Hkv, D]
 * (K and V have the key length Nk, equal to N for causal problems.)
 */
#ifndef ATTN_ORACLE_H
#define ATTN_ORACLE_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

/* ---- FP8 E4M3FN codec and E8M0 block exponents (App. B.6.1, the input
 *      quantizer; OCP 8-bit float formats) ---- */
double  orc_e4m3_value(uint8_t code);          /* decode; NaN for 0x7F/0xFF */
uint8_t orc_e4m3_round(double y);              /* C8: RNE, saturating to +-448 */
int     orc_pow2_exponent(double amax);        /* smallest e with amax <= 448*2^e, in [-127,127] */
double  orc_bf16_round(double x);              /* RNE to bfloat16, returned as double */

void orc_e4m3_round_array(const double* y, int64_t n, uint8_t* out);
void orc_e4m3_value_array(const uint8_t* c, int64_t n, double* out);
void orc_pow2_exponent_array(const double* a, int64_t n, int32_t* out);
void orc_bf16_round_array(const double* x, int64_t n, double* out);

/* Quantize x[B,N,H,D] into row (1x32 along D) and col (32x1 along N) MX copies.
 * Returns the number of non-finite inputs (the copies are then meaningless). */
int64_t orc_quantize(const double* x, int64_t B, int64_t N, int64_t H, int64_t D,
                     uint8_t* code_row, uint8_t* scale_row,
                     uint8_t* code_col, uint8_t* scale_col);

/* Input producer (App. B.6.1): y = fl32(fl32(x * prescale) - mean), the
 * mean over tokens per (b, h, c) as reading R13 defines it when center != 0
 * (else 0).  x, y [B,N,H,D]; mean [B,H,D].  N % 32 == 0. */
void orc_producer(const double* x, int64_t B, int64_t N, int64_t H, int64_t D, double prescale, int center,
                  double* y, double* mean);

/* Input producer with the fused rotary embedding (App. B.6.1, reading R16):
 * channels lo .. lo + R - 1 of every (token n, head) are rotated in pairs
 * (lo + c, lo + c + R/2), c < R/2, by the angle whose cosine and sine are
 * rope[(n * R/2 + c) * 2 + {0, 1}] (FP32 values):
 *   y_c      = fl32(fl32(x_c cos) - fl32(x_{c+R/2} sin))
 *   y_{c+R/2} = fl32(fl32(x_{c+R/2} cos) + fl32(x_c sin)),
 * each rounded to BF16 (RNE); other channels pass unchanged.  Then the
 * producer above (prescale, mean) runs on the result.  R = 0 (or rope NULL):
 * no rotation. */
void orc_producer_rope(const double* x, int64_t B, int64_t N, int64_t H, int64_t D, const double* rope,
                       int64_t lo, int64_t R, double prescale, int center, double* y, double* mean);

/* The producer with the QK normalization in front (reading R17): when gain
 * (FP32 values, [D], shared by the heads) is given, every (token, head) row
 * becomes bf16(fl32(fl32(x_c r) g_c)) with r = fl32(1 / sqrt(ss / D + eps))
 * in FP64, ss the FP64 sum of x_c^2 over c ascending (the key RMSNorm of
 * App. B.4; eps 1e-6 in App. B.2); then orc_producer_rope. */
void orc_producer_ext(const double* x, int64_t B, int64_t N, int64_t H, int64_t D, const double* gain, double eps,
                      const double* rope, int64_t lo, int64_t R, double prescale, int center, double* y,
                      double* mean);

/* Decode both copies into [B,H,N,D] doubles (either output may be NULL). */
void orc_dequantize(const uint8_t* code_row, const uint8_t* scale_row,
                    const uint8_t* code_col, const uint8_t* scale_col,
                    int64_t B, int64_t N, int64_t H, int64_t D,
                    double* x_row, double* x_col);

typedef struct {
  int64_t B, N, Hq, Hkv, Dqk, Dv;
  double tau;                 /* softmax scale, applied to the score accumulator */
  int64_t Nk;                 /* key / value length (== N when causal) */
  int32_t causal;             /* 1: top-left causal mask; 0: every query sees all Nk keys */
} orc_problem;

enum { ORC_EXACT_PFWD = 1,    /* forward probabilities are not cast to FP8 */
       ORC_EXACT_PBWD = 2,    /* backward (dV) probabilities are not cast */
       ORC_EXACT_DS   = 4,    /* dS is not cast */
       ORC_MX_PBWD    = 8 };  /* backward probabilities cast with one power-of-two
                                 scale per aligned 32x32 block (a variant, R15)
                                 instead of the fixed 2^-8 */
enum { ORC_DELTA_MATCHING = 0, ORC_DELTA_STALE_ROWSUM = 1, ORC_DELTA_CONSISTENT_DO = 2 };
enum { ORC_ROUND_NONE = 0, ORC_ROUND_F32 = 1, ORC_ROUND_BF16 = 2 };

/* per-row statistics written when rowstats != NULL, [B, Hq, N, ORC_NSTAT] */
enum { ORC_ST_SUM_DS = 0,      /* sum_j dS_ij (pre-cast)            */
       ORC_ST_SUMABS_DS,       /* sum_j |dS_ij|                      */
       ORC_ST_MAXABS_DS,       /* max_j |dS_ij|                      */
       ORC_ST_MAX_PDP,         /* max_j P_ij |dP_ij|                  */
       ORC_ST_SUM_DSCAST,      /* sum_j dS'_ij (after the FP8 cast)  */
       ORC_ST_SUMABS_DSCAST,   /* sum_j |dS'_ij|                     */
       ORC_ST_SUM_P,           /* sum_j P_ij                          */
       ORC_ST_SUM_PDP,         /* sum_j P_ij dP_ij                    */
       ORC_ST_SUM_PCAST,       /* sum_j P'_ij (decoded dV operand)    */
       ORC_ST_SUM_P_ABSTERMS,  /* sum_j P_ij sum_c |dO_ic V_jc| (the
                                  magnitude of dP's terms, weighted by P) */
       ORC_NSTAT };

/* Forward + correction + backward of softmax attention on dequantized
 * operands (row copies feed the contractions over head_dim, col copies the
 * contractions over the sequence).  See attn_oracle.c for the steps.
 * O receives the stored output (rounded per o_round); gradients are rounded
 * per grad_round.  delta_in (nullable) replaces the computed correction;
 * lse_in (nullable, [B,Hq,N]) replaces the stored LSE in the correction and
 * gradient passes (the forward is unchanged).
 * row_lo (a multiple of 32, 0 for the whole problem; causal problems only)
 * restricts the work to
 * query rows i >= row_lo (O, LSE, delta, dQ, row statistics) and keys
 * j >= row_lo (dK, dV): by causality those depend on no other rows or keys'
 * outputs, so they come out exactly as in the whole problem; the rest of
 * the outputs are left untouched.
 * phat / dsraw / dshat / pbhat (nullable, [B,Hq,N,Nk]) receive the
 * normalized forward probabilities actually used for O, dS before and after
 * the FP8 cast, and the backward probability operand P' of dV (tiny problems
 * only).
 * Returns 0, or -1 on invalid geometry. */
int orc_attention(const orc_problem* p, int flags, int delta_mode,
                  int o_round, int grad_round,
                  const double* Qr, const double* Kr, const double* Vr, const double* dOr,
                  const double* Qc, const double* Kc, const double* Vc, const double* dOc,
                  const double* dO_raw, const double* delta_in, const double* lse_in,
                  double* O, double* O_unrounded, double* LSE, double* delta,
                  double* dQ, double* dK, double* dV,
                  double* rowstats, double* phat, double* dsraw, double* dshat, double* pbhat,
                  int64_t row_lo, int nthreads);

#ifdef __cplusplus
}
#endif
#endif
