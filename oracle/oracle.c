/*
 * oracle.c -- plain, slow, single-threaded CPU reference of the HiLoRe hot path.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the
 * benchmark's CPU-baseline leg; never by the GPU product path.  It shares no
 * code, header, table or constant generator with the GPU library.
 *
 * Everything here is written for a reader holding the paper: each routine is
 * the definition the paper gives (or the reading stated next to it), with no
 * blocking, fusion or reordering beyond what that definition states.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

static float f32_from_bits(uint32_t u) { float f; memcpy(&f, &u, sizeof f); return f; }
static uint32_t bits_from_f32(float f) { uint32_t u; memcpy(&u, &f, sizeof u); return u; }

/* ======================================================================= */
/* Number formats                                                          */
/* ======================================================================= */

/* bf16 is the upper half of a binary32 word: widening is exact. */
float orc_bf16_to_f32(uint16_t h) { return f32_from_bits((uint32_t)h << 16); }

/* fp32 -> bf16 with round-to-nearest, ties to even, written as the rule
 * itself: find the two bf16 neighbours of v, keep the nearer one, and on a
 * tie keep the one whose last mantissa bit is 0.  Overflow past the largest
 * bf16 goes to infinity exactly as IEEE rounding with an unbounded exponent
 * would (the would-be next value is 2^128).  NaN inputs are out of contract. */
uint16_t orc_bf16_rne(float v) {
  uint32_t u = bits_from_f32(v);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)(u >> 16); /* +-inf */
  uint32_t down = u & 0xFFFF0000u;              /* toward zero, same sign */
  uint32_t up = down + 0x10000u;                /* next magnitude */
  double mag = fabs((double)v);
  double lo = fabs((double)f32_from_bits(down));
  double hi = ((up & 0x7F800000u) == 0x7F800000u) ? ldexp(1.0, 128)
                                                  : fabs((double)f32_from_bits(up));
  double dl = mag - lo, dh = hi - mag;          /* exact in double */
  if (dl < dh) return (uint16_t)(down >> 16);
  if (dh < dl) return (uint16_t)(up >> 16);
  return (uint16_t)((((down >> 16) & 1u) == 0u) ? (down >> 16) : (up >> 16));
}

/* Exact value of an OCP E4M3FN code: 1 sign bit, 4 exponent bits (bias 7),
 * 3 mantissa bits; exponent field 0 holds subnormals m * 2^-9; S.1111.111 is
 * NaN and there are no infinities.  This is the format torch.float8_e4m3fn
 * names (App. B.1, Eq. fp8-roundtrip). */
double orc_e4m3fn_decode(uint8_t c) {
  int s = (c >> 7) & 1, e = (c >> 3) & 15, m = c & 7;
  if (e == 15 && m == 7) return NAN;
  double mag = (e == 0) ? ldexp((double)m, -9) : ldexp(1.0 + m / 8.0, e - 7);
  return s ? -mag : mag;
}

/* |v| rounded to nearest, ties to even, on the E4M3FN grid continued past
 * its top (448, 480, 512, ...): exact arithmetic in double.  The grid spacing
 * in the binade of |v| is 2^(max(e,-6)-3); round |v| / spacing to the nearest
 * integer (ties to the even integer) and multiply back. */
static double e4m3fn_round_mag(double a) {
  if (a == 0.0) return 0.0;
  int ex;
  frexp(a, &ex);                                /* a = f * 2^ex, f in [0.5,1) */
  int e = ex - 1;                               /* a in [2^e, 2^(e+1)) */
  int qe = (e < -6 ? -6 : e) - 3;               /* spacing exponent */
  double n = ldexp(a, -qe);                     /* exact */
  double fl = floor(n), frac = n - fl;
  double k;
  if (frac > 0.5) k = fl + 1.0;
  else if (frac < 0.5) k = fl;
  else k = (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;
  return ldexp(k, qe);
}

/* Code bits of a grid value g in [0, 448]. */
static uint8_t e4m3fn_encode_mag(double g) {
  if (g < ldexp(1.0, -6)) return (uint8_t)ldexp(g, 9); /* subnormal: g = m * 2^-9 */
  int gx;
  frexp(g, &gx);
  int ge = gx - 1;                              /* g in [2^ge, 2^(ge+1)) */
  int mant = (int)ldexp(g, 3 - ge) - 8;         /* 3-bit mantissa */
  return (uint8_t)(((ge + 7) << 3) | mant);
}

/* fp32 -> E4M3FN, round to nearest with ties to even on the E4M3FN grid,
 * saturating at +-448, keeping the sign of zero. */
uint8_t orc_e4m3fn_rne(float v) {
  uint8_t sign = (bits_from_f32(v) >> 31) ? 0x80 : 0x00;
  double g = e4m3fn_round_mag(fabs((double)v));
  if (g > 448.0) g = 448.0;                     /* saturate */
  return (uint8_t)(sign | e4m3fn_encode_mag(g));
}

/* The paper's literal codec (App. B.1, Eq. fp8-roundtrip: a torch.float8_e4m3fn
 * cast, no scale): the same rounding without saturation.  A value whose
 * rounded magnitude passes 448 (|v| > 464), an infinity or a NaN has no
 * E4M3FN encoding and becomes NaN, S.1111.111, keeping the sign. */
uint8_t orc_e4m3fn_cast(float v) {
  uint8_t sign = (bits_from_f32(v) >> 31) ? 0x80 : 0x00;
  if (isnan(v) || isinf(v)) return (uint8_t)(sign | 0x7F);
  double g = e4m3fn_round_mag(fabs((double)v));
  if (g > 448.0) return (uint8_t)(sign | 0x7F);
  return (uint8_t)(sign | e4m3fn_encode_mag(g));
}

/* The cast back to bf16 of Eq. fp8-roundtrip: every finite E4M3FN value is a
 * bf16 value, so the conversion is exact; a NaN code becomes the canonical
 * bf16 NaN 0x7FC0, whatever its sign (torch's float8 -> bfloat16 conversion). */
uint16_t orc_e4m3fn_cast_to_bf16(uint8_t c) {
  if ((c & 0x7F) == 0x7F) return 0x7FC0;
  return orc_bf16_rne((float)orc_e4m3fn_decode(c));
}

void orc_bf16_rne_array(const float *v, int64_t n, uint16_t *out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_bf16_rne(v[i]);
}

void orc_e4m3fn_rne_array(const float *v, int64_t n, uint8_t *out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_e4m3fn_rne(v[i]);
}

void orc_e4m3fn_cast_array(const float *v, int64_t n, uint8_t *out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_e4m3fn_cast(v[i]);
}

float orc_code_value(int code, uint8_t c) {
  if (code == ORC_INT8) return (float)(int8_t)c;   /* E4M3FN and the literal cast decode alike */
  return (float)orc_e4m3fn_decode(c);
}

/* ======================================================================= */
/* GRPO                                                                    */
/* ======================================================================= */

/* Pairwise sum: the values padded with +0 to a power-of-two count, then
 * summed as (first half) + (second half), recursively, in fp32. */
static float pairsum_rec(const float *v, int lo, int len, int n) {
  if (len == 1) return lo < n ? v[lo] : 0.0f;
  int h = len / 2;
  return pairsum_rec(v, lo, h, n) + pairsum_rec(v, lo + h, h, n);
}
static float pairsum(const float *v, int n) {
  int p2 = 1;
  while (p2 < n) p2 *= 2;
  return pairsum_rec(v, 0, p2, n);
}

/* Group-relative advantages (Sec. 3.1; App. D.1.1 "GRPO and optimization"):
 * for each prompt, over its G responses, A = (R - mean) / (population std +
 * adv_eps); a group whose rewards are all equal gets A = 0.  fp32, with the
 * pairwise sums above so that the GPU can reproduce every bit. */
void orc_grpo_advantages(const float *rewards, int P, int G, float adv_eps, float *adv) {
  float *d = (float *)malloc(sizeof(float) * (size_t)(G > 0 ? G : 1));
  float *sq = (float *)malloc(sizeof(float) * (size_t)(G > 0 ? G : 1));
  for (int i = 0; i < P; ++i) {
    const float *r = rewards + (size_t)i * G;
    float mu = pairsum(r, G) / (float)G;
    for (int j = 0; j < G; ++j) { d[j] = r[j] - mu; sq[j] = d[j] * d[j]; }
    float sigma = sqrtf(pairsum(sq, G) / (float)G);
    for (int j = 0; j < G; ++j) adv[(size_t)i * G + j] = d[j] / (sigma + adv_eps);
  }
  free(d);
  free(sq);
}

static double count_valid(const uint8_t *mask, int64_t n) {
  if (!mask) return (double)n;
  int64_t c = 0;
  for (int64_t i = 0; i < n; ++i) c += mask[i] != 0;
  return (double)c;
}

/* Per-token quantities of the GRPO update for responses laid out
 * response-major, T slots each (slot j*T + t is token t of response j):
 *   ratio  r_t = exp(s_t - s_t^old)                        (Sec. 3.1)
 *   chi_t  = [(A >= 0 and r <= 1+eps) or (A < 0 and r >= 1-eps)]
 *                                                          (Eq. update-coefficient)
 *   flags  bit0 = m and chi (policy term active)
 *          bit1 = m and A != 0 and not chi (clipped, Eq. diagnostic-clipping)
 *   coeff  omega_t = dL/ds_t = -(m/N) chi r A + beta (m/N) [1 - exp(s_ref - s)]
 *          (Eq. update-coefficient; K3 derivative in the proof of Prop. 1)
 * Readings: chi is decided in log-ratio space, delta = s - s_old in fp32
 * against the fp32 thresholds log1p(+-eps) (the paper leaves the boundary to
 * the implementation); N is n_norm when positive (the whole rollout batch,
 * App. D.1.1), else the count of valid slots in this call; N = 0 gives
 * omega = 0.  Masked slots (mask byte 0) have omega = 0 and flags = 0.
 * adv/flags are the fp32/integer values the GPU must match exactly; ratio and
 * coeff are fp64 truth. */
void orc_grpo_coeffs(const float *rewards, const float *logp_new, const float *logp_old,
                     const float *logp_ref, const uint8_t *mask, int P, int G, int T,
                     float clip_eps, float adv_eps, double beta, double n_norm,
                     float *adv, double *ratio, uint8_t *flags, double *coeff) {
  const int64_t R = (int64_t)P * G;
  const int64_t n = R * (int64_t)T;
  orc_grpo_advantages(rewards, P, G, adv_eps, adv);
  const float hi = (float)log1p((double)clip_eps);
  const float lo = (float)log1p(-(double)clip_eps);
  const double N = n_norm > 0.0 ? n_norm : count_valid(mask, n);
  for (int64_t j = 0; j < R; ++j) {
    const float A = adv[j];
    for (int64_t t = 0; t < T; ++t) {
      const int64_t i = j * T + t;
      const int m = mask ? (mask[i] != 0) : 1;
      const float delta = logp_new[i] - logp_old[i];
      const int chi = (A >= 0.0f) ? (delta <= hi) : (delta >= lo);
      flags[i] = (uint8_t)((m && chi ? 1 : 0) | (m && A != 0.0f && !chi ? 2 : 0));
      const double r = exp((double)logp_new[i] - (double)logp_old[i]);
      if (ratio) ratio[i] = r;
      double w = 0.0;
      if (m && N > 0.0) {
        const double pol = chi ? r * (double)A : 0.0;
        const double kl = (beta != 0.0)
            ? beta * expm1((double)logp_ref[i] - (double)logp_new[i]) : 0.0;
        w = (-pol - kl) / N;
      }
      coeff[i] = w;
    }
  }
}

/* The GRPO objective itself (Sec. 3.1, Eq. grpo-objective, with the K3 KL of
 * the proof of Prop. 1), in fp64, as a function of the current log-probs, for
 * finite-difference checks of the coefficients:
 *   L = -(1/N) sum m min(r A, clip(r, 1-eps, 1+eps) A)
 *       + beta (1/N) sum m [exp(s_ref - s) - (s_ref - s) - 1].          */
double orc_grpo_loss(const float *adv, const double *logp_new, const float *logp_old,
                     const float *logp_ref, const uint8_t *mask, int R, int T,
                     double clip_eps, double beta, double n_norm) {
  const int64_t n = (int64_t)R * T;
  const double N = n_norm > 0.0 ? n_norm : count_valid(mask, n);
  if (N <= 0.0) return 0.0;
  double L = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    if (mask && !mask[i]) continue;
    const double A = (double)adv[i / T];
    const double r = exp(logp_new[i] - (double)logp_old[i]);
    double rc = r;
    if (rc < 1.0 - clip_eps) rc = 1.0 - clip_eps;
    if (rc > 1.0 + clip_eps) rc = 1.0 + clip_eps;
    const double a = r * A, b = rc * A;
    L -= (a < b ? a : b);
    if (beta != 0.0) {
      const double x = (double)logp_ref[i] - logp_new[i];
      L += beta * (exp(x) - x - 1.0);
    }
  }
  return L / N;
}

/* ======================================================================= */
/* Blockwise absmax codec                                                  */
/* ======================================================================= */

/* The paper's low-precision action stores an FP8 E4M3FN copy of a bf16
 * activation and casts it back for backward (App. B.1, Eq. fp8-roundtrip).
 * The scaled reading of that codec is the one used here: every run of `block`
 * consecutive elements of a row gets one fp32 scale.  Step by step, with
 * Q = 127 (int8) or 448 (E4M3FN):
 *   amax = max |x_j| over the block (exact: bf16 widens to fp32 exactly);
 *   if amax < 2^-64 (zero or negligible block): scale = 0, codes = 0;
 *   else  s = amax / Q  and  r = Q / amax   (IEEE fp32 divisions),
 *         v_j = x_j * r                      (fp32 multiply),
 *         int8:   q_j = clamp(nearest-even integer of v_j, -127, 127),
 *         E4M3FN: q_j = orc_e4m3fn_rne(v_j). */
void orc_quantize(const uint16_t *x, int64_t rows, int64_t cols, int64_t ld, int code,
                  int block, uint8_t *codes, float *scales) {
  if (code == ORC_E4M3FN_CAST) {                /* literal codec: no blocks, no scales */
    for (int64_t row = 0; row < rows; ++row)
      for (int64_t c = 0; c < cols; ++c)
        codes[row * cols + c] = orc_e4m3fn_cast(orc_bf16_to_f32(x[row * ld + c]));
    return;
  }
  const float Q = (code == ORC_INT8) ? 127.0f : 448.0f;
  const float tiny = ldexpf(1.0f, -64);
  const int64_t nb = cols / block;
  for (int64_t row = 0; row < rows; ++row) {
    for (int64_t b = 0; b < nb; ++b) {
      const uint16_t *xb = x + row * ld + b * block;
      uint8_t *cb = codes + row * cols + b * block;
      float amax = 0.0f;
      for (int j = 0; j < block; ++j) {
        const float a = fabsf(orc_bf16_to_f32(xb[j]));
        if (a > amax) amax = a;
      }
      if (!(amax >= tiny)) {
        scales[row * nb + b] = 0.0f;
        for (int j = 0; j < block; ++j) cb[j] = 0;
        continue;
      }
      const float s = amax / Q;
      const float r = Q / amax;
      scales[row * nb + b] = s;
      for (int j = 0; j < block; ++j) {
        const float v = orc_bf16_to_f32(xb[j]) * r;
        if (code == ORC_INT8) {
          float q = nearbyintf(v);              /* default mode: nearest, ties even */
          if (q > 127.0f) q = 127.0f;
          if (q < -127.0f) q = -127.0f;
          cb[j] = (uint8_t)(int8_t)(int)q;
        } else {
          cb[j] = orc_e4m3fn_rne(v);
        }
      }
    }
  }
}

/* Reconstruction (App. B.1, Eq. fp8-roundtrip, the cast back to BF16):
 * xhat = bf16_rne( value(q) * s ), the product an fp32 multiply. */
void orc_dequantize(const uint8_t *codes, const float *scales, int64_t rows, int64_t cols,
                    int code, int block, uint16_t *xhat) {
  if (code == ORC_E4M3FN_CAST) {                /* literal codec: cast back, no scale */
    for (int64_t i = 0; i < rows * cols; ++i) xhat[i] = orc_e4m3fn_cast_to_bf16(codes[i]);
    return;
  }
  const int64_t nb = cols / block;
  for (int64_t row = 0; row < rows; ++row)
    for (int64_t c = 0; c < cols; ++c) {
      const float q = orc_code_value(code, codes[row * cols + c]);
      const float s = scales[row * nb + c / block];
      xhat[row * cols + c] = orc_bf16_rne(q * s);
    }
}

/* Per-row sums in fp64: ss_x = sum x^2 (for the token RMS a_t of Eq.
 * activation-token-weights) and ss_err = sum (xhat - x)^2 (for the
 * reconstruction error of Eq. app-calibration-error). */
void orc_row_stats(const uint16_t *x, int64_t ld, const uint16_t *xhat, int64_t rows,
                   int64_t cols, double *ss_x, double *ss_err) {
  for (int64_t row = 0; row < rows; ++row) {
    double sx = 0.0, se = 0.0;
    for (int64_t c = 0; c < cols; ++c) {
      const double xv = (double)orc_bf16_to_f32(x[row * ld + c]);
      const double hv = (double)orc_bf16_to_f32(xhat[row * cols + c]);
      sx += xv * xv;
      se += (hv - xv) * (hv - xv);
    }
    if (ss_x) ss_x[row] = sx;
    if (ss_err) ss_err[row] = se;
  }
}

/* ======================================================================= */
/* Exposure and risk of one unit                                           */
/* ======================================================================= */

/* For one unit of width d_u over the rows (tokens) of a microbatch, with
 * T = rows whose mask byte is nonzero (all rows if mask is NULL):
 *   a_t      = sqrt(ss_x_t / d_u)                       (Eq. activation-token-weights)
 *   alpha_t  = (a_t + eps_a) / (mean_{s in T} a_s + eps_a)
 *   exposure = sum_{t in T} |omega_t| alpha_t            (Eq. mlp-weighted-exposure)
 *   risk     = sum_{t in T} |omega_t| sqrt(ss_err_t)     (token-weighted reconstruction
 *              error, the first-order bound of Thm. 1 for a linear consumer)
 *   rel_err  = sqrt(sum_t ss_err_t) / (sqrt(sum_t ss_x_t) + eps_rel) over all rows
 *                                                        (Eq. app-calibration-error)
 * An empty T gives exposure = risk = 0. */
void orc_unit_exposure_risk(const double *coeff, const uint8_t *mask, int64_t rows,
                            const double *ss_x, const double *ss_err, int64_t d_u,
                            double eps_alpha, double eps_rel,
                            double *exposure, double *risk, double *rel_err) {
  double sum_a = 0.0, cnt = 0.0, sx = 0.0, se = 0.0;
  for (int64_t t = 0; t < rows; ++t) {
    sx += ss_x[t];
    se += ss_err[t];
    if (mask && !mask[t]) continue;
    sum_a += sqrt(ss_x[t] / (double)d_u);
    cnt += 1.0;
  }
  double e = 0.0, k = 0.0;
  if (cnt > 0.0) {
    const double mean_a = sum_a / cnt;
    for (int64_t t = 0; t < rows; ++t) {
      if (mask && !mask[t]) continue;
      const double a = sqrt(ss_x[t] / (double)d_u);
      const double alpha = (a + eps_alpha) / (mean_a + eps_alpha);
      e += fabs(coeff[t]) * alpha;
      k += fabs(coeff[t]) * sqrt(ss_err[t]);
    }
  }
  *exposure = e;
  *risk = k;
  *rel_err = sqrt(se) / (sqrt(sx) + eps_rel);
}

/* ======================================================================= */
/* Weight gradient on reconstructed activations                            */
/* ======================================================================= */

static double deq_value(const uint8_t *codes, const float *scales, int code, int block,
                        int64_t M, int64_t t, int64_t i, int variant) {
  const uint8_t c = codes[t * M + i];
  if (code == ORC_E4M3FN_CAST)                  /* exact in bf16: both variants agree */
    return (double)orc_bf16_to_f32(orc_e4m3fn_cast_to_bf16(c));
  const float s = scales[t * (M / block) + i / block];
  if (variant == 0) {
    const double q = (code == ORC_INT8) ? (double)(int8_t)c : orc_e4m3fn_decode(c);
    return q * (double)s;
  }
  return (double)orc_bf16_to_f32(orc_bf16_rne(orc_code_value(code, c) * s));
}

/* dW[i][j] = sum_t Xtilde[t][i] * dY[t][j] in fp64 (the full-parameter weight
 * gradient of a linear layer whose saved input was recovered from its
 * low-precision copy; its relative Frobenius error against this is the
 * measure of Eq. measured-gradient-error). */
void orc_wgrad(const uint8_t *codes, const float *scales, int code, int block,
               const uint16_t *dy, int64_t K, int64_t M, int64_t N,
               int64_t i0, int64_t i1, int64_t j0, int64_t j1, int variant, double *out) {
  const int64_t w = j1 - j0;
  for (int64_t i = 0; i < (i1 - i0) * w; ++i) out[i] = 0.0;
  double *xcol = (double *)malloc(sizeof(double) * (size_t)(i1 - i0 > 0 ? i1 - i0 : 1));
  for (int64_t t = 0; t < K; ++t) {
    for (int64_t i = i0; i < i1; ++i)
      xcol[i - i0] = deq_value(codes, scales, code, block, M, t, i, variant);
    for (int64_t i = i0; i < i1; ++i) {
      const double xv = xcol[i - i0];
      double *o = out + (i - i0) * w;
      const uint16_t *dr = dy + t * N;
      for (int64_t j = j0; j < j1; ++j) o[j - j0] += xv * (double)orc_bf16_to_f32(dr[j]);
    }
  }
  free(xcol);
}

void orc_wgrad_entries(const uint8_t *codes, const float *scales, int code, int block,
                       const uint16_t *dy, int64_t K, int64_t M, int64_t N,
                       const int64_t *ii, const int64_t *jj, int64_t n, int variant,
                       double *out) {
  for (int64_t e = 0; e < n; ++e) {
    double acc = 0.0;
    for (int64_t t = 0; t < K; ++t)
      acc += deq_value(codes, scales, code, block, M, t, ii[e], variant) *
             (double)orc_bf16_to_f32(dy[t * N + jj[e]]);
    out[e] = acc;
  }
}

/* ======================================================================= */
/* Recovery allocation                                                     */
/* ======================================================================= */

/* Sec. 3.4 Eq. joint-allocation, solved as in App. B.2: each unit u takes one
 * action a in A_u(q_u) from {R, H, L}; R is the baseline with zero utility,
 * memory and risk; H has risk 0; L has risk psi_u.  Maximise the summed
 * utility subject to  sum dm <= m_res  and  sum risk <= delta_b.
 *
 * Available actions (App. B.3 Eq. available-recovery-actions): the verified
 * set of the unit intersected with {H,L,R} if the retained representation q_u
 * is H, {L,R} if it is L, {R} if it is R.  Non-R actions with non-positive
 * utility are excluded (App. B.2, utility profiling); so are actions whose
 * inputs are not finite or negative.  A zero risk budget disables L; a zero
 * memory budget admits only actions with zero memory cost. */
static int action_ok(int act, uint8_t q, uint8_t verified, double tau, double dm, double risk) {
  if (!((verified >> act) & 1u)) return 0;
  if (q == ORC_ACT_L && act == ORC_ACT_H) return 0;  /* an L copy cannot give H */
  if (q != ORC_ACT_H && q != ORC_ACT_L) return 0;    /* R (or unknown): only R */
  if (!(tau > 0.0) || !isfinite(tau)) return 0;
  if (!(dm >= 0.0) || !isfinite(dm)) return 0;
  if (!(risk >= 0.0) || !isfinite(risk)) return 0;
  return 1;
}

/* Integer cost of one action on a grid of n intervals of width h (Eq.
 * allocation-integer-costs): ceil(cost / h), or n + 1 (does not fit) when
 * that exceeds n.  With a zero budget (h unused) only a zero cost fits. */
static int64_t grid_cost(double cost, double budget, int n) {
  if (!(budget > 0.0)) return cost == 0.0 ? 0 : (int64_t)n + 1;
  const double h = budget / (double)n;
  const double c = ceil(cost / h);
  return c > (double)n ? (int64_t)n + 1 : (int64_t)c;
}

typedef struct {
  int ok_h, ok_l;
  int64_t b_h, b_l, r_l;
  double tau_h, tau_l;
} unit_costs;

static void costs_of(int u, const uint8_t *q, const uint8_t *verified, const double *tau_h,
                     const double *tau_l, const double *dm_h, const double *dm_l,
                     const double *psi, double m_res, double delta_b, int n_b, int n_d,
                     unit_costs *c) {
  c->ok_h = action_ok(ORC_ACT_H, q[u], verified[u], tau_h[u], dm_h[u], 0.0);
  c->ok_l = action_ok(ORC_ACT_L, q[u], verified[u], tau_l[u], dm_l[u], psi[u]) && delta_b > 0.0;
  c->b_h = c->ok_h ? grid_cost(dm_h[u], m_res, n_b) : 0;
  c->b_l = c->ok_l ? grid_cost(dm_l[u], m_res, n_b) : 0;
  c->r_l = c->ok_l ? grid_cost(psi[u], delta_b, n_d) : 0;
  if (c->b_h > n_b) c->ok_h = 0;
  if (c->b_l > n_b || c->r_l > n_d) c->ok_l = 0;
  c->tau_h = tau_h[u];
  c->tau_l = tau_l[u];
}

/* Grid sizes of Eq. allocation-grid: N + 1 states per axis, or a single state
 * when the budget on that axis is zero. */
static void grid_sizes(double m_res, double delta_b, int n_b, int n_d, int64_t *KB, int64_t *KD) {
  *KB = m_res > 0.0 ? (int64_t)n_b + 1 : 1;
  *KD = delta_b > 0.0 ? (int64_t)n_d + 1 : 1;
}

/* The dynamic programme of Eq. allocation-dp: F_i(j, k) is the largest
 * utility of units 1..i with integer memory cost exactly j and risk cost
 * exactly k; F_0(0,0) = 0, every other F_0 entry -inf;
 *   F_i(j,k) = max over available a with b_i(a) <= j, r_i(a) <= k of
 *              F_{i-1}(j - b_i(a), k - r_i(a)) + utility_i(a),
 * actions tried in the order R, H, L and replaced only by a strictly larger
 * value (the within-state tie rule).  The answer is the best terminal state,
 * ties to lower risk, then lower memory; the actions are recovered by
 * backtracking.  Outputs: action[u] in {0 = R, 1 = H, 2 = L}; totals = {summed
 * utility, memory, risk} (sums in unit order); jk = the terminal integer costs.
 * Returns 0, or -1 on invalid scalars. */
int orc_allocate(int U, const uint8_t *q, const uint8_t *verified, const double *tau_h,
                 const double *tau_l, const double *dm_h, const double *dm_l, const double *psi,
                 double m_res, double delta_b, int n_b, int n_d, uint8_t *action,
                 double *totals, int64_t *jk) {
  if (U < 0 || n_b < 1 || n_d < 1 || !(m_res >= 0.0) || !isfinite(m_res) ||
      !(delta_b >= 0.0) || !isfinite(delta_b))
    return -1;
  int64_t KB, KD;
  grid_sizes(m_res, delta_b, n_b, n_d, &KB, &KD);
  const int64_t cells = KB * KD;
  double *prev = (double *)malloc(sizeof(double) * (size_t)cells);
  double *cur = (double *)malloc(sizeof(double) * (size_t)cells);
  uint8_t *pred = (uint8_t *)malloc((size_t)(U > 0 ? U : 1) * (size_t)cells);
  unit_costs *uc = (unit_costs *)malloc(sizeof(unit_costs) * (size_t)(U > 0 ? U : 1));
  for (int64_t c = 0; c < cells; ++c) prev[c] = -INFINITY;
  prev[0] = 0.0;                                  /* F_0(0,0) = 0, cell index k * KB + j */
  for (int i = 0; i < U; ++i) {
    costs_of(i, q, verified, tau_h, tau_l, dm_h, dm_l, psi, m_res, delta_b, n_b, n_d, &uc[i]);
    const unit_costs *c = &uc[i];
    for (int64_t k = 0; k < KD; ++k)
      for (int64_t j = 0; j < KB; ++j) {
        double best = prev[k * KB + j];           /* R */
        uint8_t a = ORC_ACT_R;
        if (c->ok_h && c->b_h <= j) {
          const double v = prev[k * KB + (j - c->b_h)] + c->tau_h;
          if (v > best) { best = v; a = ORC_ACT_H; }
        }
        if (c->ok_l && c->b_l <= j && c->r_l <= k) {
          const double v = prev[(k - c->r_l) * KB + (j - c->b_l)] + c->tau_l;
          if (v > best) { best = v; a = ORC_ACT_L; }
        }
        cur[k * KB + j] = best;
        pred[(int64_t)i * cells + k * KB + j] = a;
      }
    double *t = prev; prev = cur; cur = t;
  }
  /* best terminal state: scanning risk, then memory, upward keeps the first */
  int64_t bj = 0, bk = 0;
  double bv = prev[0];
  for (int64_t k = 0; k < KD; ++k)
    for (int64_t j = 0; j < KB; ++j)
      if (prev[k * KB + j] > bv) { bv = prev[k * KB + j]; bj = j; bk = k; }
  jk[0] = bj;
  jk[1] = bk;
  totals[0] = bv;
  int64_t j = bj, k = bk;
  for (int i = U - 1; i >= 0; --i) {
    const uint8_t a = pred[(int64_t)i * cells + k * KB + j];
    action[i] = a;
    if (a == ORC_ACT_H) j -= uc[i].b_h;
    if (a == ORC_ACT_L) { j -= uc[i].b_l; k -= uc[i].r_l; }
  }
  double mem = 0.0, risk = 0.0;
  for (int i = 0; i < U; ++i) {
    if (action[i] == ORC_ACT_H) mem += dm_h[i];
    if (action[i] == ORC_ACT_L) { mem += dm_l[i]; risk += psi[i]; }
  }
  totals[1] = mem;
  totals[2] = risk;
  free(prev); free(cur); free(pred); free(uc);
  return 0;
}

/* Brute force over all 3^U assignments of the same discretised problem
 * (U <= 16): the utility of an assignment is its non-R utilities added in
 * unit order; feasible when every action is available and the integer costs
 * sum to at most n_b and n_d.  Best value first, then lower risk cost, then
 * lower memory cost, then the assignment that is smallest when compared from
 * the last unit backwards (R < H < L).  Same outputs as orc_allocate. */
int orc_allocate_brute(int U, const uint8_t *q, const uint8_t *verified, const double *tau_h,
                       const double *tau_l, const double *dm_h, const double *dm_l,
                       const double *psi, double m_res, double delta_b, int n_b, int n_d,
                       uint8_t *action, double *totals, int64_t *jk) {
  if (U < 0 || U > 16 || n_b < 1 || n_d < 1 || !(m_res >= 0.0) || !isfinite(m_res) ||
      !(delta_b >= 0.0) || !isfinite(delta_b))
    return -1;
  unit_costs uc[16];
  for (int i = 0; i < U; ++i)
    costs_of(i, q, verified, tau_h, tau_l, dm_h, dm_l, psi, m_res, delta_b, n_b, n_d, &uc[i]);
  int64_t total = 1;
  for (int i = 0; i < U; ++i) total *= 3;
  int have = 0;
  double bv = 0.0;
  int64_t bj = 0, bk = 0;
  uint8_t best[16] = {0}, a[16];
  for (int64_t code = 0; code < total; ++code) {
    int64_t x = code, j = 0, k = 0;
    double v = 0.0;
    int ok = 1;
    for (int i = 0; i < U; ++i) {
      a[i] = (uint8_t)(x % 3);
      x /= 3;
      if (a[i] == ORC_ACT_H) {
        if (!uc[i].ok_h) { ok = 0; break; }
        j += uc[i].b_h;
        v += uc[i].tau_h;
      } else if (a[i] == ORC_ACT_L) {
        if (!uc[i].ok_l) { ok = 0; break; }
        j += uc[i].b_l;
        k += uc[i].r_l;
        v += uc[i].tau_l;
      }
    }
    if (!ok || j > n_b || k > n_d) continue;
    int better = !have || v > bv || (v == bv && (k < bk || (k == bk && j < bj)));
    if (!better && v == bv && k == bk && j == bj) {
      for (int i = U - 1; i >= 0; --i)
        if (a[i] != best[i]) { better = a[i] < best[i]; break; }
    }
    if (better) {
      have = 1; bv = v; bj = j; bk = k;
      memcpy(best, a, (size_t)U);
    }
  }
  memcpy(action, best, (size_t)U);
  jk[0] = bj;
  jk[1] = bk;
  totals[0] = bv;
  double mem = 0.0, risk = 0.0;
  for (int i = 0; i < U; ++i) {
    if (action[i] == ORC_ACT_H) mem += dm_h[i];
    if (action[i] == ORC_ACT_L) { mem += dm_l[i]; risk += psi[i]; }
  }
  totals[1] = mem;
  totals[2] = risk;
  return 0;
}

/* ======================================================================= */
/* Calibration scalars and update diagnostics                              */
/* ======================================================================= */

/* Relative gradient error of one single-unit L intervention (App. B.1 Eq.
 * app-calibration-error, the y of Sec. 3.4 Eq. calibration-metrics): both
 * gradients are taken as fp32 values, the norms in fp64,
 *   y = sqrt( ||g_l - g_ex||^2 / max(||g_ex||^2, eps_num) ). */
double orc_grad_rel_err(const float *g_l, const float *g_ex, int64_t n, double eps_num) {
  double num = 0.0, den = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    const double d = (double)g_l[i] - (double)g_ex[i];
    num += d * d;
    den += (double)g_ex[i] * (double)g_ex[i];
  }
  return sqrt(num / (den > eps_num ? den : eps_num));
}

/* Susceptibility and mean reconstruction error from calibration passes
 * (App. B.1 Eqs. app-kappa, app-risk-score; Sec. 3.4 Eq. susceptibility).
 * Per calibration microbatch b and unit u the inputs hold the exposure E, the
 * reconstruction error e^L and the measured gradient error y, row b of each
 * [n_batches][n_units] array.  With x = E * e^L, the class-c least-squares fit
 * of y = kappa x over kappa >= 0 has the closed form
 *   kappa_c = max(0, sum x y / sum x^2)   (0 when sum x^2 = 0),
 * the sums running over the (u, b) with class(u) = c; units whose class is
 * outside [0, n_classes) take no part.  ebar_u = (1/n_batches) sum_b e^L_{u,b}. */
void orc_calibrate(int n_units, int n_batches, int n_classes, const int32_t *unit_class,
                   const float *exposure, const float *rel_err, const float *grad_err,
                   double *kappa, double *ebar) {
  for (int c = 0; c < n_classes; ++c) {
    double sxy = 0.0, sxx = 0.0;
    for (int b = 0; b < n_batches; ++b)
      for (int u = 0; u < n_units; ++u) {
        if (unit_class[u] != c) continue;
        const int64_t i = (int64_t)b * n_units + u;
        const double x = (double)exposure[i] * (double)rel_err[i];
        sxy += x * (double)grad_err[i];
        sxx += x * x;
      }
    const double k = sxx > 0.0 ? sxy / sxx : 0.0;
    kappa[c] = k > 0.0 ? k : 0.0;
  }
  for (int u = 0; u < n_units; ++u) {
    double s = 0.0;
    for (int b = 0; b < n_batches; ++b) s += (double)rel_err[(int64_t)b * n_units + u];
    ebar[u] = n_batches > 0 ? s / (double)n_batches : 0.0;
  }
}

/* Calibrated risk of each unit's L action (App. B.1 Eq. app-risk-score):
 *   psi_u = kappa_{c(u)} * E_u * ebar_u,
 * multiplied in that order in fp64.  A unit without a class (outside
 * [0, n_classes)) has no calibration: psi = +inf, which makes L unavailable
 * to the allocator. */
void orc_risk_score(int n_units, const int32_t *unit_class, int n_classes, const double *kappa,
                    const double *ebar, const float *exposure, double *psi) {
  for (int u = 0; u < n_units; ++u) {
    const int c = unit_class[u];
    psi[u] = (c >= 0 && c < n_classes) ? kappa[c] * (double)exposure[u] * ebar[u] : INFINITY;
  }
}

static int cmp_desc(const void *a, const void *b) {
  const double x = *(const double *)a, y = *(const double *)b;
  return x < y ? 1 : (x > y ? -1 : 0);
}

/* Structural sparsity of one batch of update coefficients (the diagnostic
 * replays of App. D.3, Policy-Update Exposure Details): over the n = R*T
 * response slots (padding included), the slots whose policy gradient is zero
 * for each exclusive cause,
 *   counts[0] padding (m = 0),
 *   counts[1] valid slots of a zero-advantage response,
 *   counts[2] valid nonzero-advantage slots on the clipped, flat branch
 *             (flag bit 1 of the coefficient step),
 * and the share of sum |omega| held by the k = max(1, ceil(top_frac * n))
 * largest |omega| (padding counted as 0; 0 when every omega is 0).  The sort
 * puts the largest first, so ties do not change the sum. */
double orc_update_sparsity(const double *coeff, const uint8_t *flags, const float *adv,
                           const uint8_t *mask, int R, int T, double top_frac, int64_t *counts) {
  const int64_t n = (int64_t)R * T;
  counts[0] = counts[1] = counts[2] = 0;
  double *mag = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
  double total = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    const int valid = mask ? mask[i] != 0 : 1;
    if (!valid) counts[0] += 1;
    else if (adv[i / T] == 0.0f) counts[1] += 1;
    else if (flags[i] & 2) counts[2] += 1;
    mag[i] = valid ? fabs(coeff[i]) : 0.0;
    total += mag[i];
  }
  double share = 0.0;
  if (n > 0 && total > 0.0) {
    int64_t k = (int64_t)ceil(top_frac * (double)n);
    if (k < 1) k = 1;
    if (k > n) k = n;
    qsort(mag, (size_t)n, sizeof(double), cmp_desc);
    double top = 0.0;
    for (int64_t i = 0; i < k; ++i) top += mag[i];
    share = top / total;
  }
  free(mag);
  return share;
}

/* ======================================================================= */
/* Backward of the gated MLP activation on a reconstructed unit            */
/* ======================================================================= */

/* The gated MLP of the evaluated models computes h = silu(g) * u from the
 * gate and up projections g, u (silu(g) = g * sigmoid(g)).  When g or u is an L
 * unit, backward uses its reconstruction (App. B.1 Eq. fp8-roundtrip).  Given
 * the gradient dh, in fp64:
 *   du = dh * silu(g)
 *   dg = dh * u * sigmoid(g) * (1 + g * (1 - sigmoid(g)))   (the derivative of silu). */
void orc_swiglu_bwd(const double *g, const double *u, const double *dh, int64_t n, double *dg,
                    double *du) {
  for (int64_t i = 0; i < n; ++i) {
    const double sg = 1.0 / (1.0 + exp(-g[i]));
    du[i] = dh[i] * g[i] * sg;
    dg[i] = dh[i] * u[i] * sg * (1.0 + g[i] * (1.0 - sg));
  }
}
