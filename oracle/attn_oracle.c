/*
 * attn_oracle.c -- reference oracle for block-scaled FP8 attention with
 * Delta-Matching.  TEST INFRASTRUCTURE ONLY (see attn_oracle.h).
 *
 * Written from the paper "Delta-Matching: Closing the Final Gap of Native
 * 8-bit Training for LLMs":
 *   - softmax attention forward/backward ............ Sec. 2.3
 *   - zero-row-sum invariant .......................... Sec. 3.1
 *   - matched correction delta = sum_j P_ij dP_ij ..... Sec. 3.4
 *   - stale (saved-output) correction ................. Sec. 3.2, App. A.3
 *   - consistent-dO correction ........................ Sec. 3.4, App. B.6
 *   - kernel numerics (quantizer, probability codes,
 *     correction pass, dS cast, GQA sums) ............. App. B.6.1-B.6.3
 * adapted to power-of-two (E8M0) block scales as follows (readings of the
 * paper; each is listed with its reason in the design notes):
 *   R1 FP8 is OCP E4M3FN, round to nearest even, saturating at +-448.
 *   R2 a block's scale is 2^e with e the smallest integer such that
 *      amax <= 448*2^e, clamped to [-127,127]; amax = 0 gives e = -127.
 *   R3 each of Q, K, V, dO is quantized twice from its source values: a
 *      "row" copy in 1x32 blocks along head_dim (feeds S = QK^T and
 *      dP = dO V^T) and a "col" copy in 32x1 blocks along the sequence
 *      (feeds O = PV, dV = P^T dO, dK = dS^T Q, dQ = dS K).
 *   R4 the softmax scale tau multiplies the score accumulator.
 *   R5 forward probability codes: per query row and aligned 32-key group g,
 *      E_g is the smallest integer with 2^{x_g} <= 448*2^{E_g} (x = S log2 e,
 *      x_g the group max over visible keys); code = C8(2^{x - E_g}); the
 *      normalizer uses the exponentials before the cast.
 *   R6 backward probability codes for dV: C8(256 P) with fixed scale 2^-8;
 *      the recomputed P is clamped to at most 1.  The paper clamps the
 *      base-two exponent of 256 P at 12 (P <= 16).  The two clamps differ
 *      only when the LSE handed to the backward is below the row's largest
 *      score, which the forward's own LSE never is; lse_in reaches it.
 *   R7 dS codes: aligned 32x32 blocks (query x key), one power-of-two scale
 *      per block, shared by dQ and dK.
 *   R8 matched correction: (sum_j P_ij dP_ij) / (sum_j P_ij) from the
 *      unquantized P and the products of the FP8 backward operands.
 *   R9 stale correction: sum_c dO_ic O_ic from the raw dO and stored O.
 *   R11 consistent-dO correction: the stale correction with the raw dO
 *      replaced by its dequantized row copy (the operand of dP), the stored
 *      O unchanged: sum_c dO^_ic O_ic.
 *   R15 (a variant, not the paper's kernel; ORC_MX_PBWD): the backward
 *      probability operand cast like dS' (R7), one power-of-two scale per
 *      aligned 32x32 block from its largest P, instead of the fixed 2^-8.
 *   R16 fused rotary producer: rotated channels in half-split pairs
 *      (lo + c, lo + c + R/2) with the caller's FP32 cosine/sine table,
 *      each product and sum rounded to FP32, then to BF16, before the
 *      prescale (orc_producer_rope).
 *   R17 QK normalization in the producer: the row statistic in FP64,
 *      rounded once to FP32; x r and the gain product in FP32; BF16 result
 *      (orc_producer_ext).
 *   R10 causal mask is top-left aligned (key j visible to query i iff j <= i,
 *      equal query and key lengths); without the mask (causal == 0) every
 *      query sees all Nk keys and the key length may differ from the query
 *      length; query head h reads KV head floor(h / (Hq/Hkv)); dK and dV are
 *      summed over the query heads of a KV group before rounding.
 */
#include "attn_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_MAXD 512  /* largest head dimension handled */

/* ------------------------------------------------------------------ */
/* FP8 E4M3FN: 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits.  */
/* Exponent field 0 holds subnormals m * 2^-9; field 15 with mantissa  */
/* 7 is NaN; there is no infinity; the largest finite value is 448.    */
/* ------------------------------------------------------------------ */
double orc_e4m3_value(uint8_t code) {
  int sign = code >> 7, e = (code >> 3) & 15, m = code & 7;
  if (e == 15 && m == 7) return NAN;
  double mag = (e == 0) ? ldexp((double)m, -9)          /* m/8 * 2^-6   */
                        : ldexp((double)(8 + m), e - 10); /* (1+m/8) 2^(e-7) */
  return sign ? -mag : mag;
}

/* C8 of App. B.6.1: round to nearest, ties to the even code, and saturate
 * magnitudes at or above 448 to +-448.  The 127 finite non-negative codes
 * 0x00..0x7E are increasing in value, so the rounding finds the bracketing
 * pair of codes by binary search and compares distances (both differences
 * are exact in double by Sterbenz' lemma: neighbours differ by at most 2x). */
static double e4m3_table[127];         /* values of codes 0x00..0x7E, increasing */
__attribute__((constructor)) static void e4m3_table_init(void) {
  for (int c = 0; c < 127; c++) e4m3_table[c] = orc_e4m3_value((uint8_t)c);
}

uint8_t orc_e4m3_round(double y) {
  const double* table = e4m3_table;
  if (isnan(y)) return 0x7F;
  uint8_t sign = signbit(y) ? 0x80 : 0x00;
  double a = fabs(y);
  if (a >= 448.0) return sign | 0x7E;
  /* lo = largest code with table[lo] <= a (binary search; table[0] = 0 <= a) */
  int lo = 0, hi = 126;
  while (lo < hi) {
    int mid = (lo + hi + 1) / 2;
    if (table[mid] <= a) lo = mid; else hi = mid - 1;
  }
  if (table[lo] == a) return sign | (uint8_t)lo;
  const int up = lo + 1;               /* exists: a < 448 = table[126] */
  const double dlo = a - table[lo], dhi = table[up] - a;
  int pick;
  if (dlo < dhi) pick = lo;
  else if (dhi < dlo) pick = up;
  else pick = (lo % 2 == 0) ? lo : up; /* tie: even mantissa LSB */
  return sign | (uint8_t)pick;
}

/* Reading R2: smallest integer e with amax <= 448 * 2^e, clamped to
 * [-127, 127] (the E8M0 range); amax == 0 gives -127. */
int orc_pow2_exponent(double amax) {
  if (!(amax > 0.0)) return -127;
  if (isinf(amax)) return 127;
  int e = ilogb(amax) - 9;
  while (ldexp(448.0, e) < amax) e++;
  while (ldexp(448.0, e - 1) >= amax) e--;
  if (e < -127) e = -127;
  if (e > 127) e = 127;
  return e;
}

/* bfloat16 (8 significant bits, FP32 exponent range), round to nearest even,
 * applied directly to the double (no intermediate float rounding). */
double orc_bf16_round(double x) {
  if (!isfinite(x) || x == 0.0) return x;
  double a = fabs(x);
  double r;
  if (a < ldexp(1.0, -126)) {
    r = nearbyint(ldexp(a, 133)) ; r = ldexp(r, -133);      /* subnormal grid 2^-133 */
  } else {
    int ex;
    double fr = frexp(a, &ex);                               /* a = fr 2^ex, fr in [0.5,1) */
    r = ldexp(nearbyint(ldexp(fr, 8)), ex - 8);              /* 8 significant bits */
  }
  return x < 0 ? -r : r;
}

void orc_e4m3_round_array(const double* y, int64_t n, uint8_t* out) {
  for (int64_t i = 0; i < n; i++) out[i] = orc_e4m3_round(y[i]);
}
void orc_e4m3_value_array(const uint8_t* c, int64_t n, double* out) {
  for (int64_t i = 0; i < n; i++) out[i] = orc_e4m3_value(c[i]);
}
void orc_pow2_exponent_array(const double* a, int64_t n, int32_t* out) {
  for (int64_t i = 0; i < n; i++) out[i] = orc_pow2_exponent(a[i]);
}
void orc_bf16_round_array(const double* x, int64_t n, double* out) {
  for (int64_t i = 0; i < n; i++) out[i] = orc_bf16_round(x[i]);
}

/* One MX block (reading R2): scale exponent from the block amax, codes
 * C8(v * 2^-e).  vals[k*stride], k < n.  Returns the scale byte e + 127. */
static uint8_t mx_block(const double* vals, int64_t n, int64_t stride, uint8_t* codes,
                        int64_t cstride) {
  double amax = 0.0;
  for (int64_t k = 0; k < n; k++) {
    double a = fabs(vals[k * stride]);
    if (a > amax) amax = a;
  }
  int e = orc_pow2_exponent(amax);
  for (int64_t k = 0; k < n; k++) codes[k * cstride] = orc_e4m3_round(ldexp(vals[k * stride], -e));
  return (uint8_t)(e + 127);
}

/* Input quantizer (App. B.6.1, with readings R1-R3): both copies from the
 * source values.  Blocks are separate per batch and head. */
int64_t orc_quantize(const double* x, int64_t B, int64_t N, int64_t H, int64_t D,
                     uint8_t* code_row, uint8_t* scale_row,
                     uint8_t* code_col, uint8_t* scale_col) {
  int64_t nonfinite = 0;
  for (int64_t i = 0; i < B * N * H * D; i++)
    if (!isfinite(x[i])) nonfinite++;
  for (int64_t b = 0; b < B; b++)
    for (int64_t h = 0; h < H; h++) {
      /* row copy: for each token n, blocks of 32 consecutive channels */
      for (int64_t n = 0; n < N; n++)
        for (int64_t c0 = 0; c0 < D; c0 += 32) {
          const double* src = x + ((b * N + n) * H + h) * D + c0;
          uint8_t* dst = code_row + ((b * H + h) * N + n) * D + c0;
          scale_row[((b * H + h) * N + n) * (D / 32) + c0 / 32] = mx_block(src, 32, 1, dst, 1);
        }
      /* col copy: for each channel c, blocks of 32 consecutive tokens */
      for (int64_t c = 0; c < D; c++)
        for (int64_t n0 = 0; n0 < N; n0 += 32) {
          const double* src = x + ((b * N + n0) * H + h) * D + c;
          uint8_t* dst = code_col + ((b * H + h) * D + c) * N + n0;
          scale_col[((b * H + h) * D + c) * (N / 32) + n0 / 32] =
              mx_block(src, 32, H * D, dst, 1);
        }
    }
  return nonfinite;
}

/* Input producer (App. B.6.1, Operands, Scaling, and Accumulation): before
 * quantization the query is multiplied by the attention scale in FP32, and
 * the key has its FP32 mean over sequence positions subtracted, separately
 * for each channel and KV head.  Reading R13 (the paper does not fix the
 * mean's summation): x' = fl32(x * prescale); the mean is the FP64 sum of
 * the FP64 sums of aligned 32-token blocks (tokens ascending within a
 * block, blocks ascending), divided by N in FP64 and rounded once to FP32;
 * y = fl32(x' - mean) (center != 0) or y = x' (center == 0).  x, y
 * [B,N,H,D]; mean [B,H,D] (zero without centering).  N % 32 == 0. */
static double fl32(double v) { return (double)(float)v; }

void orc_producer(const double* x, int64_t B, int64_t N, int64_t H, int64_t D, double prescale, int center,
                  double* y, double* mean) {
  for (int64_t b = 0; b < B; b++)
    for (int64_t h = 0; h < H; h++)
      for (int64_t c = 0; c < D; c++) {
        double m = 0.0;
        if (center) {
          double total = 0.0;
          for (int64_t n0 = 0; n0 < N; n0 += 32) {
            double part = 0.0;
            for (int64_t n = n0; n < n0 + 32; n++) part += fl32(x[((b * N + n) * H + h) * D + c] * prescale);
            total += part;
          }
          m = fl32(total / (double)N);
        }
        mean[(b * H + h) * D + c] = m;
        for (int64_t n = 0; n < N; n++) {
          const int64_t o = ((b * N + n) * H + h) * D + c;
          y[o] = fl32(fl32(x[o] * prescale) - m);
        }
      }
}

/* Reading R16 (the rotation's arithmetic; the paper fixes only that the
 * rotated channels are rounded to BF16 before the prescale): products and
 * the sum of each rotated channel rounded to FP32, pairs (lo + c,
 * lo + c + R/2), the caller's cosine/sine table per token. */
/* Reading R17 (the QK normalization's arithmetic; App. B.4 gives the key
 * RMSNorm, App. B.2 its eps and FP32 computation): the row statistic in
 * FP64 (squares summed over channels ascending, divided by D, eps added, the
 * reciprocal square root), rounded once to FP32; then two FP32 products and
 * the rounding to BF16 of the normalized activation. */
void orc_producer_ext(const double* x, int64_t B, int64_t N, int64_t H, int64_t D, const double* gain, double eps,
                      const double* rope, int64_t lo, int64_t R, double prescale, int center, double* y,
                      double* mean) {
  const int64_t n_el = B * N * H * D;
  double* t = (double*)malloc(sizeof(double) * (size_t)(n_el > 0 ? n_el : 1));
  memcpy(t, x, sizeof(double) * (size_t)n_el);
  if (gain) {
    for (int64_t row = 0; row < B * N * H; row++) {
      double* v = t + row * D;
      double ss = 0.0;
      for (int64_t c = 0; c < D; c++) ss += v[c] * v[c];
      const double r = fl32(1.0 / sqrt(ss / (double)D + eps));
      for (int64_t c = 0; c < D; c++) v[c] = orc_bf16_round(fl32(fl32(v[c] * r) * gain[c]));
    }
  }
  orc_producer_rope(t, B, N, H, D, rope, lo, R, prescale, center, y, mean);
  free(t);
}

void orc_producer_rope(const double* x, int64_t B, int64_t N, int64_t H, int64_t D, const double* rope,
                       int64_t lo, int64_t R, double prescale, int center, double* y, double* mean) {
  const int64_t n_el = B * N * H * D, h2 = R / 2;
  double* r = (double*)malloc(sizeof(double) * (size_t)(n_el > 0 ? n_el : 1));
  memcpy(r, x, sizeof(double) * (size_t)n_el);
  if (rope && R > 0) {
    for (int64_t b = 0; b < B; b++)
      for (int64_t n = 0; n < N; n++)
        for (int64_t h = 0; h < H; h++) {
          const double* src = x + ((b * N + n) * H + h) * D;
          double* dst = r + ((b * N + n) * H + h) * D;
          for (int64_t c = 0; c < h2; c++) {
            const double cs = rope[(n * h2 + c) * 2], sn = rope[(n * h2 + c) * 2 + 1];
            const double a = src[lo + c], p = src[lo + c + h2];
            dst[lo + c] = orc_bf16_round(fl32(fl32(a * cs) - fl32(p * sn)));
            dst[lo + c + h2] = orc_bf16_round(fl32(fl32(p * cs) + fl32(a * sn)));
          }
        }
  }
  orc_producer(r, B, N, H, D, prescale, center, y, mean);
  free(r);
}

void orc_dequantize(const uint8_t* code_row, const uint8_t* scale_row,
                    const uint8_t* code_col, const uint8_t* scale_col,
                    int64_t B, int64_t N, int64_t H, int64_t D,
                    double* x_row, double* x_col) {
  for (int64_t b = 0; b < B; b++)
    for (int64_t h = 0; h < H; h++)
      for (int64_t n = 0; n < N; n++)
        for (int64_t c = 0; c < D; c++) {
          int64_t o = ((b * H + h) * N + n) * D + c;
          if (x_row) {
            int e = (int)scale_row[((b * H + h) * N + n) * (D / 32) + c / 32] - 127;
            x_row[o] = ldexp(orc_e4m3_value(code_row[o]), e);
          }
          if (x_col) {
            int e = (int)scale_col[((b * H + h) * D + c) * (N / 32) + n / 32] - 127;
            x_col[o] = ldexp(orc_e4m3_value(code_col[((b * H + h) * D + c) * N + n]), e);
          }
        }
}

/* ------------------------------------------------------------------ */
/* attention                                                           */
/* ------------------------------------------------------------------ */
static double dot(const double* a, const double* b, int64_t n) {
  /* four partial sums in a fixed order (k mod 4), then combined */
  double s0 = 0, s1 = 0, s2 = 0, s3 = 0;
  int64_t k = 0;
  for (; k + 4 <= n; k += 4) {
    s0 += a[k] * b[k];
    s1 += a[k + 1] * b[k + 1];
    s2 += a[k + 2] * b[k + 2];
    s3 += a[k + 3] * b[k + 3];
  }
  for (; k < n; k++) s0 += a[k] * b[k];
  return (s0 + s1) + (s2 + s3);
}

/* sum_k |a_k b_k|: the magnitude scale of a dot product's terms */
static double dot_abs(const double* a, const double* b, int64_t n) {
  double s = 0.0;
  for (int64_t k = 0; k < n; k++) s += fabs(a[k] * b[k]);
  return s;
}

static double round_to(double v, int mode) {
  if (mode == ORC_ROUND_F32) return (double)(float)v;
  if (mode == ORC_ROUND_BF16) return orc_bf16_round(v);
  return v;
}

/* Reading R5: the smallest integer E with 2^{xg} <= 448 * 2^E. */
static int group_exponent(double xg) {
  int E = (int)ceil(xg - log2(448.0));
  while (exp2(xg - (E - 1)) <= 448.0) E--;
  while (exp2(xg - E) > 448.0) E++;
  return E;
}

/* P_ij = exp(S_ij - LSE_i) with the score S_ij = tau <q_i, k_j> (App. B.6.3),
 * clamped to at most 1 (R6): with the LSE of the same scores P <= 1 already;
 * the clamp only matters for an inconsistent LSE. */
static double probability(double tau, const double* q, const double* k, int64_t d, double lse) {
  double pij = exp(tau * dot(q, k, d) - lse);
  return pij > 1.0 ? 1.0 : pij;
}

typedef struct {
  int64_t B, N, Nk, Hq, Hkv, Dqk, Dv, G;
  int causal;
  double tau;
  int flags;
  const double *Qr, *Kr, *Vr, *dOr, *LSE, *delta;
} tile_ctx;

/* One aligned 32x32 tile of the backward (query rows i0.., keys j0..):
 * P and dS = P (dP - delta) before any cast (zero for masked j > i when
 * causal), the backward probability operand P' = C8(256 P) 2^-8 (R6; with
 * ORC_MX_PBWD, R15: C8(P 2^-e) 2^e with e from the tile's largest P by R2's
 * rule) and the dS operand dS' cast with one power-of-two scale for the whole
 * tile (R7). */
static void tile(const tile_ctx* c, int64_t b, int64_t h, int64_t i0, int64_t nr, int64_t j0,
                 int64_t nc, double P[32][32], double dS[32][32], double Pb[32][32], double dSh[32][32]) {
  const int64_t kh = h / c->G;
  double amax = 0.0, pmax = 0.0;
  for (int64_t r = 0; r < 32; r++)
    for (int64_t t = 0; t < 32; t++) {
      const int64_t i = i0 + r, j = j0 + t;
      if (r >= nr || t >= nc || (c->causal && j > i)) { P[r][t] = 0.0; dS[r][t] = 0.0; continue; }
      const double lse = c->LSE[(b * c->Hq + h) * c->N + i];
      const double pij = probability(c->tau, c->Qr + ((b * c->Hq + h) * c->N + i) * c->Dqk,
                                     c->Kr + ((b * c->Hkv + kh) * c->Nk + j) * c->Dqk, c->Dqk, lse);
      const double dpij = dot(c->dOr + ((b * c->Hq + h) * c->N + i) * c->Dv,
                              c->Vr + ((b * c->Hkv + kh) * c->Nk + j) * c->Dv, c->Dv);
      P[r][t] = pij;
      dS[r][t] = pij * (dpij - c->delta[(b * c->Hq + h) * c->N + i]);
      if (fabs(dS[r][t]) > amax) amax = fabs(dS[r][t]);
      if (pij > pmax) pmax = pij;
    }
  const int e = orc_pow2_exponent(amax);
  const int ep = (c->flags & ORC_MX_PBWD) ? orc_pow2_exponent(pmax) : -8;
  for (int64_t r = 0; r < 32; r++)
    for (int64_t t = 0; t < 32; t++) {
      Pb[r][t] = (c->flags & ORC_EXACT_PBWD) ? P[r][t]
                                             : ldexp(orc_e4m3_value(orc_e4m3_round(ldexp(P[r][t], -ep))), ep);
      dSh[r][t] = (c->flags & ORC_EXACT_DS) ? dS[r][t]
                                            : ldexp(orc_e4m3_value(orc_e4m3_round(ldexp(dS[r][t], -e))), e);
    }
}

int orc_attention(const orc_problem* p, int flags, int delta_mode,
                  int o_round, int grad_round,
                  const double* Qr, const double* Kr, const double* Vr, const double* dOr,
                  const double* Qc, const double* Kc, const double* Vc, const double* dOc,
                  const double* dO_raw, const double* delta_in, const double* lse_in,
                  double* O, double* O_unrounded, double* LSE, double* delta,
                  double* dQ, double* dK, double* dV,
                  double* rowstats, double* phat, double* dsraw, double* dshat, double* pbhat,
                  int64_t row_lo, int nthreads) {
  const int64_t B = p->B, N = p->N, Nk = p->Nk, Hq = p->Hq, Hkv = p->Hkv, Dqk = p->Dqk, Dv = p->Dv;
  const int causal = p->causal;
  const double tau = p->tau;
  if (B < 0 || N < 0 || Nk < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || Dqk <= 0 || Dv <= 0 ||
      Dqk > ORC_MAXD || Dv > ORC_MAXD || row_lo < 0 || row_lo % 32 != 0 || (N > 0 && row_lo >= N))
    return -1;
  /* causal: equal lengths (R10); row_lo restricts a causal problem only; a
   * query needs at least one key */
  if ((causal != 0 && causal != 1) || (causal && Nk != N) || (!causal && row_lo != 0) || (N > 0 && Nk == 0))
    return -1;
  const int64_t G = Hq / Hkv;
  const double LOG2E = 1.4426950408889634074;
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
  if (phat) memset(phat, 0, sizeof(double) * (size_t)(B * Hq * N * Nk));
  if (dshat) memset(dshat, 0, sizeof(double) * (size_t)(B * Hq * N * Nk));
  if (dsraw) memset(dsraw, 0, sizeof(double) * (size_t)(B * Hq * N * Nk));
  if (pbhat) memset(pbhat, 0, sizeof(double) * (size_t)(B * Hq * N * Nk));

  /* ---- forward (Sec. 2.3; App. B.6.2 with reading R5) ---- */
#pragma omp parallel
  {
    double* x = (double*)malloc(sizeof(double) * (size_t)(Nk > 0 ? Nk : 1));
    double* w = (double*)malloc(sizeof(double) * (size_t)(Nk > 0 ? Nk : 1));
#pragma omp for collapse(3) schedule(dynamic, 16)
    for (int64_t b = 0; b < B; b++)
      for (int64_t h = 0; h < Hq; h++)
        for (int64_t i = row_lo; i < N; i++) {
          const int64_t kh = h / G;
          const double* q = Qr + ((b * Hq + h) * N + i) * Dqk;
          /* scores over the visible keys j < je (j <= i when causal), base-2
           * exponent x = S log2 e */
          const int64_t je = causal ? i + 1 : Nk;
          double smax = -INFINITY;
          for (int64_t j = 0; j < je; j++) {
            double s = tau * dot(q, Kr + ((b * Hkv + kh) * Nk + j) * Dqk, Dqk);
            x[j] = s;
            if (s > smax) smax = s;
          }
          double se = 0.0;
          for (int64_t j = 0; j < je; j++) se += exp(x[j] - smax);
          LSE[(b * Hq + h) * N + i] = smax + log(se);
          for (int64_t j = 0; j < je; j++) x[j] *= LOG2E;
          /* integer reference Mi: every weight below is relative to 2^Mi */
          const double Mi = ceil(smax * LOG2E);
          double ell = 0.0;                      /* normalizer from pre-cast exponentials */
          for (int64_t j = 0; j < je; j++) ell += exp2(x[j] - Mi);
          for (int64_t g0 = 0; g0 < je; g0 += 32) {
            const int64_t g1 = (g0 + 32 < je) ? g0 + 32 : je;
            if (flags & ORC_EXACT_PFWD) {
              for (int64_t j = g0; j < g1; j++) w[j] = exp2(x[j] - Mi);
            } else {
              double xg = -INFINITY;
              for (int64_t j = g0; j < g1; j++) if (x[j] > xg) xg = x[j];
              const int Eg = group_exponent(xg);
              for (int64_t j = g0; j < g1; j++)
                w[j] = orc_e4m3_value(orc_e4m3_round(exp2(x[j] - Eg))) * exp2((double)Eg - Mi);
            }
          }
          for (int64_t c = 0; c < Dv; c++) {
            double acc = 0.0;
            for (int64_t j = 0; j < je; j++) acc += w[j] * Vc[((b * Hkv + kh) * Nk + j) * Dv + c];
            const double o = acc / ell;
            const int64_t oi = ((b * N + i) * Hq + h) * Dv + c;
            if (O_unrounded) O_unrounded[oi] = o;
            O[oi] = round_to(o, o_round);
          }
          if (phat)
            for (int64_t j = 0; j < je; j++) phat[((b * Hq + h) * N + i) * Nk + j] = w[j] / ell;
        }
    free(x);
    free(w);
  }

  /* ---- correction pass (Sec. 3.4; App. B.6.3 with readings R8, R9) ----
   * P_ij = exp(S_ij - LSE_i) recomputed from the scores, dP_ij = <dOr_i, Vr_j>.
   * The backward reads the LSE the forward stored, or lse_in when given (a
   * caller-supplied LSE, e.g. an inconsistent one that exercises R6's clamp). */
  const double* LB = lse_in ? lse_in : LSE;
#pragma omp parallel for collapse(3) schedule(dynamic, 16)
  for (int64_t b = 0; b < B; b++)
    for (int64_t h = 0; h < Hq; h++)
      for (int64_t i = row_lo; i < N; i++) {
        const int64_t kh = h / G;
        const double lse = LB[(b * Hq + h) * N + i];
        const double* q = Qr + ((b * Hq + h) * N + i) * Dqk;
        const double* go = dOr + ((b * Hq + h) * N + i) * Dv;
        double num = 0.0, den = 0.0, maxpdp = 0.0, tabs = 0.0;
        const int64_t je = causal ? i + 1 : Nk;
        for (int64_t j = 0; j < je; j++) {
          const double pij = probability(tau, q, Kr + ((b * Hkv + kh) * Nk + j) * Dqk, Dqk, lse);
          const double dpij = dot(go, Vr + ((b * Hkv + kh) * Nk + j) * Dv, Dv);
          num += pij * dpij;
          den += pij;
          if (rowstats) tabs += pij * dot_abs(go, Vr + ((b * Hkv + kh) * Nk + j) * Dv, Dv);
          if (fabs(pij * dpij) > maxpdp) maxpdp = fabs(pij * dpij);
        }
        double d;
        if (delta_in) d = delta_in[(b * Hq + h) * N + i];
        else if (delta_mode == ORC_DELTA_MATCHING) d = num / den;
        else if (delta_mode == ORC_DELTA_CONSISTENT_DO) {
          d = 0.0;
          for (int64_t c = 0; c < Dv; c++) d += go[c] * O[((b * N + i) * Hq + h) * Dv + c];
        } else {
          d = 0.0;
          for (int64_t c = 0; c < Dv; c++)
            d += dO_raw[((b * N + i) * Hq + h) * Dv + c] * O[((b * N + i) * Hq + h) * Dv + c];
        }
        delta[(b * Hq + h) * N + i] = d;
        if (rowstats) {
          double* st = rowstats + ((b * Hq + h) * N + i) * ORC_NSTAT;
          st[ORC_ST_MAX_PDP] = maxpdp;
          st[ORC_ST_SUM_P] = den;
          st[ORC_ST_SUM_PDP] = num;
          st[ORC_ST_SUM_P_ABSTERMS] = tabs;
        }
      }

  /* ---- gradient passes (Sec. 2.3; App. B.6.3 with readings R6, R7, R10) ----
   * Both passes rebuild the same aligned 32x32 tiles (query block rb, key
   * block jb) with tile(), so the dQ pass (one query block at a time) and the
   * dK/dV pass (one key block at a time, looping the query heads of its KV
   * group) see identical dS' and P' values, and every sum has a fixed order. */
  const int64_t nrb = (N + 31) / 32, nkb = (Nk + 31) / 32;
  tile_ctx ctx = {B, N, Nk, Hq, Hkv, Dqk, Dv, G, causal, tau, flags, Qr, Kr, Vr, dOr, LB, delta};
#pragma omp parallel for collapse(3) schedule(dynamic, 1)
  for (int64_t b = 0; b < B; b++)
    for (int64_t h = 0; h < Hq; h++)
      for (int64_t rb = row_lo / 32; rb < nrb; rb++) {
        const int64_t kh = h / G;
        double P[32][32], dS[32][32], Pb[32][32], dSh[32][32];
        double sds[32] = {0}, sads[32] = {0}, mads[32] = {0}, sdc[32] = {0}, sadc[32] = {0}, spc[32] = {0};
        double dq[32][ORC_MAXD];
        memset(dq, 0, sizeof dq);
        const int64_t i0 = rb * 32, nr = (i0 + 32 <= N) ? 32 : N - i0;
        const int64_t jb_end = causal ? rb + 1 : nkb;
        for (int64_t jb = 0; jb < jb_end; jb++) {
          const int64_t j0 = jb * 32, nc = (j0 + 32 <= Nk) ? 32 : Nk - j0;
          tile(&ctx, b, h, i0, nr, j0, nc, P, dS, Pb, dSh);
          for (int64_t r = 0; r < nr; r++) {
            const int64_t i = i0 + r;
            for (int64_t t = 0; t < nc; t++) {
              const int64_t j = j0 + t;
              if (causal && j > i) break;
              const double g = dSh[r][t];
              sds[r] += dS[r][t];
              sads[r] += fabs(dS[r][t]);
              if (fabs(dS[r][t]) > mads[r]) mads[r] = fabs(dS[r][t]);
              sdc[r] += g;
              sadc[r] += fabs(g);
              spc[r] += Pb[r][t];
              if (dsraw) dsraw[((b * Hq + h) * N + i) * Nk + j] = dS[r][t];
              if (dshat) dshat[((b * Hq + h) * N + i) * Nk + j] = g;
              if (pbhat) pbhat[((b * Hq + h) * N + i) * Nk + j] = Pb[r][t];
              const double* kc = Kc + ((b * Hkv + kh) * Nk + j) * Dqk;
              for (int64_t c = 0; c < Dqk; c++) dq[r][c] += g * kc[c];
            }
          }
        }
        for (int64_t r = 0; r < nr; r++) {
          const int64_t i = i0 + r;
          for (int64_t c = 0; c < Dqk; c++) dQ[((b * N + i) * Hq + h) * Dqk + c] = tau * dq[r][c];
          if (rowstats) {
            double* st = rowstats + ((b * Hq + h) * N + i) * ORC_NSTAT;
            st[ORC_ST_SUM_DS] = sds[r];
            st[ORC_ST_SUMABS_DS] = sads[r];
            st[ORC_ST_MAXABS_DS] = mads[r];
            st[ORC_ST_SUM_DSCAST] = sdc[r];
            st[ORC_ST_SUMABS_DSCAST] = sadc[r];
            st[ORC_ST_SUM_PCAST] = spc[r];
          }
        }
      }
#pragma omp parallel for collapse(3) schedule(dynamic, 1)
  for (int64_t b = 0; b < B; b++)
    for (int64_t kh = 0; kh < Hkv; kh++)
      for (int64_t jb = row_lo / 32; jb < nkb; jb++) {
        double P[32][32], dS[32][32], Pb[32][32], dSh[32][32];
        double dk[32][ORC_MAXD], dv[32][ORC_MAXD];
        memset(dk, 0, sizeof dk);
        memset(dv, 0, sizeof dv);
        const int64_t j0 = jb * 32, nc = (j0 + 32 <= Nk) ? 32 : Nk - j0;
        for (int64_t h = kh * G; h < (kh + 1) * G; h++)
          for (int64_t rb = causal ? jb : 0; rb < nrb; rb++) {
            const int64_t i0 = rb * 32, nr = (i0 + 32 <= N) ? 32 : N - i0;
            tile(&ctx, b, h, i0, nr, j0, nc, P, dS, Pb, dSh);
            for (int64_t r = 0; r < nr; r++) {
              const int64_t i = i0 + r;
              const double* qc = Qc + ((b * Hq + h) * N + i) * Dqk;
              const double* gc = dOc + ((b * Hq + h) * N + i) * Dv;
              for (int64_t t = 0; t < nc; t++) {
                if (causal && j0 + t > i) break;
                const double g = dSh[r][t], pb = Pb[r][t];
                for (int64_t c = 0; c < Dqk; c++) dk[t][c] += g * qc[c];
                for (int64_t c = 0; c < Dv; c++) dv[t][c] += pb * gc[c];
              }
            }
          }
        for (int64_t t = 0; t < nc; t++) {
          const int64_t j = j0 + t;
          for (int64_t c = 0; c < Dqk; c++) dK[((b * Nk + j) * Hkv + kh) * Dqk + c] = tau * dk[t][c];
          for (int64_t c = 0; c < Dv; c++) dV[((b * Nk + j) * Hkv + kh) * Dv + c] = dv[t][c];
        }
      }
  for (int64_t k = 0; k < B * N * Hq * Dqk; k++) dQ[k] = round_to(dQ[k], grad_round);
  for (int64_t k = 0; k < B * Nk * Hkv * Dqk; k++) dK[k] = round_to(dK[k], grad_round);
  for (int64_t k = 0; k < B * Nk * Hkv * Dv; k++) dV[k] = round_to(dV[k], grad_round);
  return 0;
}
