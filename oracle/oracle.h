/*
 * oracle.h -- plain, slow, single-threaded CPU reference of the HiLoRe hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark load this library.  The GPU product path
 * (libhilore) never includes, links or calls anything in this directory, and
 * this directory never includes anything from the product path.
 *
 * Paper: "HiLoRe: What to Store, Compress, or Recompute for Efficient GRPO
 * Training".  Each function cites the passage it follows.
 *
 * Precision rules:
 *   - values the GPU must reproduce bit for bit (advantages, clip flags,
 *     quantisation codes, block scales, dequantised bf16 values) are computed
 *     in fp32 with the exact operation sequence written out below;
 *   - every value checked against a tolerance (ratios, loss coefficients, row
 *     sums, exposure, risk, relative error, weight gradients) is computed in
 *     fp64 and serves as the "truth".
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math (x86-64 SSE, so
 * every float operation is a single IEEE binary32 operation, rounded to
 * nearest even, with no fused multiply-add).
 */
#ifndef HILORE_ORACLE_H
#define HILORE_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ORC_E4M3FN_CAST is the paper's literal codec: a plain cast, no scales. */
enum { ORC_INT8 = 0, ORC_E4M3FN = 1, ORC_E4M3FN_CAST = 2 };

/* ---- number formats --------------------------------------------------- */
float    orc_bf16_to_f32(uint16_t h);
uint16_t orc_bf16_rne(float v);            /* fp32 -> bf16, nearest-even, by distances */
uint8_t  orc_e4m3fn_rne(float v);          /* fp32 -> OCP E4M3FN, nearest-even, saturating */
uint8_t  orc_e4m3fn_cast(float v);         /* fp32 -> E4M3FN as torch.float8_e4m3fn: nearest-even,
                                              non-saturating (|v| > 464, inf, NaN -> NaN, sign kept) */
uint16_t orc_e4m3fn_cast_to_bf16(uint8_t c); /* exact; NaN codes -> 0x7FC0 */
double   orc_e4m3fn_decode(uint8_t c);     /* exact value of an E4M3FN code (NaN for 0x7f/0xff) */
float    orc_code_value(int code, uint8_t c); /* exact fp32 value of an int8 / E4M3FN code */
/* element-wise array forms of the two roundings, for exhaustive checks */
void     orc_bf16_rne_array(const float *v, int64_t n, uint16_t *out);
void     orc_e4m3fn_rne_array(const float *v, int64_t n, uint8_t *out);
void     orc_e4m3fn_cast_array(const float *v, int64_t n, uint8_t *out);

/* ---- GRPO (Sec. 3.1 Eq. grpo-objective; Sec. 3.2 Eq. update-coefficient) */
void orc_grpo_advantages(const float *rewards, int P, int G, float adv_eps, float *adv);

void orc_grpo_coeffs(const float *rewards, const float *logp_new, const float *logp_old,
                     const float *logp_ref, const uint8_t *mask, int P, int G, int T,
                     float clip_eps, float adv_eps, double beta, double n_norm,
                     float *adv, double *ratio, uint8_t *flags, double *coeff);

double orc_grpo_loss(const float *adv, const double *logp_new, const float *logp_old,
                     const float *logp_ref, const uint8_t *mask, int R, int T,
                     double clip_eps, double beta, double n_norm);

/* ---- blockwise absmax codec (App. B.1 Eq. fp8-roundtrip, scaled reading);
 *      with code ORC_E4M3FN_CAST the literal cast (block and scales unused) */
void orc_quantize(const uint16_t *x, int64_t rows, int64_t cols, int64_t ld, int code,
                  int block, uint8_t *codes, float *scales);
void orc_dequantize(const uint8_t *codes, const float *scales, int64_t rows, int64_t cols,
                    int code, int block, uint16_t *xhat);
void orc_row_stats(const uint16_t *x, int64_t ld, const uint16_t *xhat, int64_t rows,
                   int64_t cols, double *ss_x, double *ss_err);

/* ---- exposure / risk (App. B.1 Eqs. activation-token-weights,
 *      mlp-weighted-exposure, app-calibration-error; Sec. 3.4) */
void orc_unit_exposure_risk(const double *coeff, const uint8_t *mask, int64_t rows,
                            const double *ss_x, const double *ss_err, int64_t d_u,
                            double eps_alpha, double eps_rel,
                            double *exposure, double *risk, double *rel_err);

/* ---- weight gradient on reconstructed activations: dW = deq(X)^T dY ----
 * variant 0: deq = code value * scale in fp64 (unrounded);
 * variant 1: deq = the bf16 value orc_dequantize produces.
 * Computes dW[i][j] for i in [i0,i1), j in [j0,j1) into out[(i-i0)*(j1-j0)+(j-j0)]. */
void orc_wgrad(const uint8_t *codes, const float *scales, int code, int block,
               const uint16_t *dy, int64_t K, int64_t M, int64_t N,
               int64_t i0, int64_t i1, int64_t j0, int64_t j1, int variant, double *out);

/* dW entries at arbitrary (i, j) pairs (for sampled checks at full size). */
void orc_wgrad_entries(const uint8_t *codes, const float *scales, int code, int block,
                       const uint16_t *dy, int64_t K, int64_t M, int64_t N,
                       const int64_t *ii, const int64_t *jj, int64_t n, int variant,
                       double *out);

/* ---- recovery allocation (Sec. 3.4 Eq. joint-allocation; App. B.2 Eqs.
 *      allocation-grid, allocation-integer-costs, allocation-dp; App. B.3 Eq.
 *      available-recovery-actions).  Per unit: q = retained representation and
 *      action ids 0 = R, 1 = H, 2 = L; verified = bit mask of verified actions;
 *      tau_* utilities, dm_* memory costs, psi the risk of L.  m_res and delta_b
 *      are the memory and risk budgets, n_b and n_d the grid intervals (1024 in
 *      the paper).  Returns 0, or -1 on invalid scalars. */
enum { ORC_ACT_R = 0, ORC_ACT_H = 1, ORC_ACT_L = 2 };
int orc_allocate(int U, const uint8_t *q, const uint8_t *verified, const double *tau_h,
                 const double *tau_l, const double *dm_h, const double *dm_l, const double *psi,
                 double m_res, double delta_b, int n_b, int n_d, uint8_t *action,
                 double *totals, int64_t *jk);
/* the same problem by enumerating all 3^U assignments (U <= 16) */
int orc_allocate_brute(int U, const uint8_t *q, const uint8_t *verified, const double *tau_h,
                       const double *tau_l, const double *dm_h, const double *dm_l,
                       const double *psi, double m_res, double delta_b, int n_b, int n_d,
                       uint8_t *action, double *totals, int64_t *jk);

/* ---- calibration scalars (App. B.1 Eqs. app-calibration-error, app-kappa,
 *      app-risk-score; Sec. 3.4 Eqs. calibration-metrics, susceptibility) ---- */
double orc_grad_rel_err(const float *g_l, const float *g_ex, int64_t n, double eps_num);
/* exposure, rel_err, grad_err: fp32 [n_batches][n_units]; kappa f64 [n_classes],
 * ebar f64 [n_units] */
void orc_calibrate(int n_units, int n_batches, int n_classes, const int32_t *unit_class,
                   const float *exposure, const float *rel_err, const float *grad_err,
                   double *kappa, double *ebar);
void orc_risk_score(int n_units, const int32_t *unit_class, int n_classes, const double *kappa,
                    const double *ebar, const float *exposure, double *psi);

/* ---- structural sparsity of the update coefficients (App. D.3, diagnostic
 *      replays).  coeff f64 [R*T], flags u8 [R*T] (bit 1 = clipped), adv f32 [R],
 *      mask u8 [R*T] or NULL.  counts[3] = padding, zero-advantage, clipped slots;
 *      returns the top-k share of sum |omega|. */
double orc_update_sparsity(const double *coeff, const uint8_t *flags, const float *adv,
                           const uint8_t *mask, int R, int T, double top_frac, int64_t *counts);

/* ---- backward of the gated MLP activation h = silu(g) * u (fp64):
 *      du = dh silu(g), dg = dh u silu'(g) */
void orc_swiglu_bwd(const double *g, const double *u, const double *dh, int64_t n, double *dg,
                    double *du);

#ifdef __cplusplus
}
#endif

#endif
