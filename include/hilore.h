/*
 * hilore.h -- C-ABI of the HiLoRe hot path on AMD Instinct MI355X (gfx950).
 *
 * HiLoRe ("HiLoRe: What to Store, Compress, or Recompute for Efficient GRPO
 * Training") decides, for every saved activation unit of a GRPO actor update,
 * whether to keep it in training precision (H), keep a low-precision copy (L)
 * or recompute it (R).  Per microbatch (Algorithm 1) the data-parallel work is:
 *   after forward   encode the L candidates                 -> hilore_compress
 *   Coefficients    per-token GRPO loss coefficients omega  -> hilore_grpo_coeffs
 *   Exposure, psi   per-unit exposure and risk              -> hilore_unit_exposure_risk
 *   Allocate        joint H/L/R choice under memory and risk -> hilore_allocate
 *   in backward     reconstruct L units                     -> hilore_decompress
 *                   and consume them in the weight gradient -> hilore_dequant_wgrad
 *                   or in the LoRA adapter gradient          -> hilore_dequant_lora_grad
 *                   or in the gated-MLP activation backward  -> hilore_dequant_swiglu_bwd
 * Calibration (App. B.1), before training and between refreshes:
 *   single-unit gradient error y                             -> hilore_grad_rel_err
 *   susceptibility kappa_c and mean reconstruction error     -> hilore_calibrate
 *   psi_u = kappa E_u ebar_u, the risk input of Allocate     -> hilore_risk_score
 * Diagnostics (App. D.3): zero-gradient causes, top-k share  -> hilore_update_sparsity
 *
 * Conventions shared by every entry point:
 *   - Every tensor pointer is a DEVICE pointer owned by the caller.  The
 *     library never allocates, frees or retains memory, and keeps no state
 *     between calls (the one exception, hilore_unit_exposure_risk_noalloc,
 *     uses a fixed device array of its own).  hilore_unit_desc arrays are
 *     HOST memory, read during the call only.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     All work is enqueued on it without a host synchronisation; outputs are
 *     valid once the stream reaches them.
 *   - Every argument is validated before anything is launched: on an error
 *     nothing is enqueued and no output is touched.  Validation touches no
 *     device state, so argument errors are reported even without a GPU.
 *   - bf16 tensors are passed as uint16_t* (raw bit patterns).
 *   - Alignment: every tensor pointer must be 16-byte aligned, except the
 *     per-unit outputs of hilore_unit_exposure_risk (4-byte aligned) and the
 *     per-unit arrays of hilore_allocate (8-byte aligned for fp64).
 *   - The functions are re-entrant; calls on different streams may run
 *     concurrently.  No C++ exception crosses this interface.
 *   - Results do not depend on the launch configuration: every reduction is
 *     done in a fixed order, with no floating-point atomics.
 */
#ifndef HILORE_H
#define HILORE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum hilore_status {
  HILORE_OK = 0,
  HILORE_ERR_INVALID_ARG = 1, /* null pointer, negative size, bad enum value      */
  HILORE_ERR_ALIGNMENT = 2,   /* pointer not 16-byte aligned, or bad row stride    */
  HILORE_ERR_UNSUPPORTED = 3, /* valid but unsupported shape (e.g. G > 64)         */
  HILORE_ERR_WORKSPACE = 4,   /* caller-supplied workspace smaller than required   */
  HILORE_ERR_HIP = 5          /* a HIP launch failed (hipGetLastError)             */
} hilore_status;

typedef enum hilore_code {
  HILORE_CODE_INT8 = 0,            /* two's-complement int8, symmetric range [-127, 127],
                                      one fp32 scale per block                          */
  HILORE_CODE_FP8_E4M3FN = 1,      /* OCP E4M3FN (torch.float8_e4m3fn), max 448,
                                      one fp32 scale per block                          */
  HILORE_CODE_FP8_E4M3FN_CAST = 2  /* the paper's literal codec (App. B.1 Eq.
                                      fp8-roundtrip): a plain E4M3FN cast of each bf16
                                      value, no scales (block must be 0, scales unused).
                                      Identical to torch.float8_e4m3fn: nearest-even,
                                      NOT saturating: |x| > 464, +-inf and NaN give the
                                      NaN code 0x7F | sign; (448, 464] gives +-448.  The
                                      cast back is exact; a NaN code gives bf16 0x7FC0. */
} hilore_code;

/* One recovery unit: one saved bf16 activation tensor that receives a single
 * H/L/R action across all its tokens (Sec. 3.4).  Rows are tokens of the
 * microbatch, columns are features; blocks of `block` consecutive columns of
 * one row share one fp32 scale (no scales with HILORE_CODE_FP8_E4M3FN_CAST).
 *   x          bf16 [rows, cols], row stride ld elements (ld >= cols, ld % 8 == 0)
 *   codes      [rows, cols] dense, one byte per element
 *   scales     fp32 [rows, cols / block] dense
 *   xhat       bf16 [rows, cols] dense: output of hilore_decompress
 *   row_ss_x   fp32 [rows] or NULL: per-row sum of x^2
 *   row_ss_err fp32 [rows] or NULL: per-row sum of (xhat - x)^2
 * Each entry point reads only the fields it names. */
typedef struct hilore_unit_desc {
  const uint16_t *x;
  void *codes;
  float *scales;
  uint16_t *xhat;
  float *row_ss_x;
  float *row_ss_err;
  int64_t rows;
  int64_t cols;
  int64_t ld;
} hilore_unit_desc;

/* Human-readable name of a status code (static storage; never NULL). */
const char *hilore_status_string(int status);

/* Library version as 10000 * major + 100 * minor + patch. */
int hilore_version(void);

/*
 * GRPO update quantities for P prompts x G responses x T token slots
 * (Sec. 3.1 Eq. grpo-objective; Sec. 3.2 Eq. update-coefficient; the K3 KL
 * derivative in the proof of Prop. 1; advantages as in App. D.1.1).
 *
 *   rewards  f32 [P*G]          response rewards, prompt-major (group i = rows iG..iG+G-1)
 *   logp_new f32 [P*G*T]        s_t, current-policy log-prob of each slot (response-major)
 *   logp_old f32 [P*G*T]        s_t^old
 *   logp_ref f32 [P*G*T]        s_t^ref; may be NULL only when beta == 0
 *   mask     u8  [P*G*T]        update mask m_t (nonzero = valid); NULL = all valid
 *   clip_eps                    clipping radius eps (> 0, < 1)
 *   adv_eps                     advantage stabiliser (the paper uses 1e-6)
 *   beta                        K3 KL weight (>= 0)
 *   n_norm                      N, the normaliser: > 0 uses this value (all valid tokens of
 *                               the complete rollout batch); <= 0 uses the number of valid
 *                               slots in this call
 * Outputs (device):
 *   adv      f32 [P*G]          A = (R - mean_group) / (population std_group + adv_eps),
 *                               group sums formed as a pairwise tree over a power-of-two
 *                               padding of the group (so the result is reproducible bit
 *                               for bit)
 *   ratio    f32 [P*G*T] or NULL  r_t = exp(s_t - s_t^old)
 *   flags    u8  [P*G*T]        bit0: m_t and chi_t (policy term active);
 *                               bit1: m_t and A != 0 and not chi_t (clipped)
 *   coeff    f32 [P*G*T]        omega_t = (m_t / N) (-chi_t r_t A - beta expm1(s_ref - s_t));
 *                               0 where m_t = 0 or N = 0
 * chi_t is decided in log-ratio space: delta = s_t - s_t^old (fp32), chi = delta <= log1p(eps)
 * when A >= 0, else delta >= log1p(-eps), both thresholds rounded to fp32.
 * workspace: used only to count N (n_norm <= 0 with a mask) over more than 2^16
 * slots: then device memory of at least hilore_grpo_coeffs_workspace_bytes(P, G, T)
 * bytes (4 bytes per 2^16 slots, at most 1 KB), 16-byte aligned, contents on entry
 * irrelevant, and calls sharing it must not overlap; otherwise it may be NULL (the
 * query returns 0 for at most 2^16 slots).
 * Limits: 1 <= G <= 64, P >= 0, T >= 0, P*G*T < 2^31.
 * Errors: bad eps or beta, NaN n_norm, null pointers -> INVALID_ARG; G > 64 or too
 * many slots -> UNSUPPORTED; workspace too small when it is needed -> WORKSPACE.
 */
size_t hilore_grpo_coeffs_workspace_bytes(int P, int G, int T);
hilore_status hilore_grpo_coeffs(const float *rewards, const float *logp_new,
                                 const float *logp_old, const float *logp_ref,
                                 const uint8_t *mask, int P, int G, int T, float clip_eps,
                                 float adv_eps, float beta, double n_norm, float *adv,
                                 float *ratio, uint8_t *flags, float *coeff, void *workspace,
                                 size_t workspace_bytes, void *stream);

/*
 * Blockwise absmax encode of the L candidates after forward (App. B.1 Eq.
 * fp8-roundtrip, in the scaled reading: one fp32 scale per 1 x block run of a
 * row; App. B.3 "post-forward encoding").  For every block, with Q = 127
 * (int8) or 448 (E4M3FN) and amax = max |x| over the block:
 *   amax < 2^-64  -> scale 0 and all codes 0;
 *   otherwise      s = amax / Q and r = Q / amax (IEEE fp32 quotients),
 *                  code = RNE(x * r) (int8: clamped to [-127,127]; E4M3FN: saturating),
 *                  scale = s.
 * With row_ss_x / row_ss_err non-NULL the same pass also writes, per row, the
 * fp32 sums of x^2 (for the token RMS weights of Eq. activation-token-weights)
 * and of (xhat - x)^2 with xhat = bf16(value(code) * s) (the reconstruction
 * error of Eq. app-calibration-error), accumulated in a fixed order.
 *   units[n_units]  host array; uses x, codes, scales, row_ss_x, row_ss_err, rows, cols, ld
 *   block           32, 64, 128 or 256; every unit needs cols % block == 0
 * With code HILORE_CODE_FP8_E4M3FN_CAST (block = 0) each element is cast on its
 * own, scales are neither read nor written, and xhat in the row sums is the
 * cast back (a NaN code makes its row's ss_err NaN).
 * All units of one call are encoded on `stream`; they may differ in shape.
 * Errors: bad code, or block != 0 with the cast code -> INVALID_ARG; other
 * block sizes, or a unit of more than 2^30 rows or 2^30 columns -> UNSUPPORTED.
 */
hilore_status hilore_compress(const hilore_unit_desc *units, int n_units, int code, int block,
                              void *stream);

/*
 * Reconstruction of L units for backward (App. B.1 Eq. fp8-roundtrip, the cast
 * back to bf16): xhat = bf16_RNE(value(code) * scale), elementwise; with
 * HILORE_CODE_FP8_E4M3FN_CAST xhat = value(code) exactly (NaN codes -> 0x7FC0).
 *   units[n_units]  host array; uses codes, scales (not with the cast code), xhat, rows, cols
 * Errors as for hilore_compress.
 */
hilore_status hilore_decompress(const hilore_unit_desc *units, int n_units, int code,
                                int block, void *stream);

/*
 * Per-unit exposure and risk for one microbatch (App. B.1 Eqs.
 * activation-token-weights, mlp-weighted-exposure, app-calibration-error;
 * Sec. 3.4 Eq. token-weighted-risk).  T = rows with a nonzero mask byte.
 *   coeff    f32 [rows]  omega_t aligned to activation rows (zero on prompt/padding rows)
 *   mask     u8  [rows]  valid response tokens T; NULL = all rows
 *   units[n_units]       host array; uses row_ss_x, row_ss_err, rows (== rows), cols
 * For each unit u, with a_t = sqrt(ss_x_t / cols):
 *   exposure[u] = sum_{t in T} |omega_t| (a_t + eps_alpha) / (mean_{s in T} a_s + eps_alpha)
 *   risk[u]     = sum_{t in T} |omega_t| sqrt(ss_err_t)
 *   rel_err[u]  = sqrt(sum_t ss_err_t) / (sqrt(sum_t ss_x_t) + eps_rel)   (all rows)
 * exposure and risk are 0 when T is empty.  Outputs are device f32 [n_units].
 * The sums are fp32: partial sums over chunks of 2048 rows of each unit go to
 * `workspace` and are then added in a fixed order (no floating-point atomics,
 * so repeated calls give identical bits).
 * workspace: device memory of at least hilore_unit_exposure_risk_workspace_bytes(rows,
 * n_units) bytes (32 bytes per unit per 2048 rows; 0, and then NULL is allowed, when
 * rows == 0), 16-byte aligned, contents on entry irrelevant; calls sharing it must
 * not overlap.
 * The calibrated risk of App. B.1 Eq. app-risk-score is kappa * exposure * mean rel_err
 * and the additive distortion of Eq. app-distortion sums it over L units; both are
 * host-side scalar steps.
 * Limits: rows < 2^24 (else UNSUPPORTED).  Errors: negative sizes or eps, null
 * pointers, a unit whose rows differ from `rows` -> INVALID_ARG; workspace too
 * small -> WORKSPACE.
 */
size_t hilore_unit_exposure_risk_workspace_bytes(int64_t rows, int n_units);
hilore_status hilore_unit_exposure_risk(const float *coeff, const uint8_t *mask, int64_t rows,
                                        const hilore_unit_desc *units, int n_units,
                                        float eps_alpha, float eps_rel, float *exposure,
                                        float *risk, float *rel_err, void *workspace,
                                        size_t workspace_bytes, void *stream);

/*
 * hilore_unit_exposure_risk without a workspace, for callers that cannot
 * allocate device memory or pass a buffer for it: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  Same
 * arguments (less the workspace), kernels and results, bit for bit.  The
 * partial sums live in a fixed 1 MiB array in device memory that the library
 * holds on every GPU it runs on until the process ends (its address is looked
 * up once per device, on the first call made with that device current); the
 * call allocates nothing.  One call needs 32 bytes per unit per 2048 rows, so
 * units * ceil(rows / 2048) may be at most 32768 (78 units of 16384 rows use
 * 624), else the call returns WORKSPACE and enqueues nothing.  Every call on
 * one GPU shares that array: calls that overlap on one GPU (other streams,
 * other threads) race and give wrong results; calls in stream order do not.
 * Nothing in the array needs to start at zero.
 */
hilore_status hilore_unit_exposure_risk_noalloc(const float *coeff, const uint8_t *mask,
                                                int64_t rows, const hilore_unit_desc *units,
                                                int n_units, float eps_alpha, float eps_rel,
                                                float *exposure, float *risk, float *rel_err,
                                                void *stream);

/*
 * Weight gradient of a linear layer whose saved input is an L unit, with the
 * reconstruction fused into the GEMM's tile load (the full-parameter setting
 * of App. D "full-parameter" experiments; accumulated over microbatches as in
 * App. D.1.1):
 *   dW[i][j] (+)= sum_t xhat[t][i] * dY[t][j],  xhat = bf16_RNE(value(code[t][i]) * scale[t][i/block])
 *   x_codes  [K, M] one byte per element; x_scales f32 [K, M / block]
 *   dy       bf16 [K, N]; dw f32 [M, N] row-major (the transpose of a [N, M] weight's layout)
 *   accumulate: 0 overwrites dw, 1 adds to it
 * bf16 x bf16 products, fp32 accumulation (MFMA).  xhat is never written to memory.
 * With HILORE_CODE_FP8_E4M3FN_CAST (block = 0, x_scales unused, may be NULL)
 * xhat = value(code) exactly; a NaN code makes its row of dW NaN.
 * Limits: M % block == 0, M % 8 == 0, N % 8 == 0, M and N below 2^22 (else
 * UNSUPPORTED), K >= 0 (K = 0 writes zeros or leaves dw).
 */
hilore_status hilore_dequant_wgrad(const void *x_codes, const float *x_scales, int code,
                                   int block, const uint16_t *dy, float *dw, int64_t K,
                                   int64_t M, int64_t N, int accumulate, void *stream);

/*
 * Gradient of the LoRA down-projection A of a linear layer whose saved input X
 * is an L unit, with the reconstruction fused into the operand load (the
 * paper's default training setting: rank-16 adapters, alpha = 32, on q/k/v/o
 * and gate/up/down, only adapters trainable, App. D.1.1).  With the layer
 * output y = X W^T + scale * (X A^T) B^T and an upstream gradient G, and
 * dh = G B (the gradient of h = X A^T before the scaling):
 *   dA[j][i] (+)= scale * sum_t dh[t][j] * xhat[t][i],
 *   xhat = bf16_RNE(value(code[t][i]) * scale[t][i/block])   (the hilore_decompress value)
 *   x_codes  [K, M] one byte per element; x_scales f32 [K, M / block]
 *   dh       bf16 [K, r] row-major; da f32 [r, M] row-major (the layout of A's gradient)
 *   scale    the adapter scaling alpha / r (applied to the fp32 sum; exact for powers of 2)
 *   accumulate: 0 overwrites da, 1 adds to it
 * bf16 x bf16 products, fp32 accumulation (MFMA), xhat never written to memory;
 * each code is read once per pass of up to 80 adapter rows, so adapters that
 * share one input (q/k/v, gate/up) are best passed side by side in dh (r = 48,
 * 80).  Partial sums over token ranges go to `workspace` and are added in a
 * fixed order (no floating-point atomics).
 * workspace: device memory of at least hilore_lora_grad_workspace_bytes(K, M, r)
 * bytes (below M = 65536 columns: 8 MB per 16 adapter rows of the widest
 * pass, so at most 40 MB), 16-byte aligned, contents on entry irrelevant;
 * calls sharing it must not overlap.
 * With HILORE_CODE_FP8_E4M3FN_CAST (block = 0, x_scales unused) xhat = value(code).
 * Limits: M % block == 0, M % 16 == 0, M < 2^26, K < 2^31, r even, 2 <= r <= 4096.
 * Errors: negative sizes, r < 1, non-finite scale, null pointers -> INVALID_ARG;
 * other shapes (odd r included) -> UNSUPPORTED; workspace too small -> WORKSPACE.
 */
size_t hilore_lora_grad_workspace_bytes(int64_t K, int64_t M, int r);
hilore_status hilore_dequant_lora_grad(const void *x_codes, const float *x_scales, int code,
                                       int block, const uint16_t *dh, float *da, int64_t K,
                                       int64_t M, int r, float scale, int accumulate,
                                       void *workspace, size_t workspace_bytes, void *stream);

/*
 * Joint H/L/R recovery allocation of one microbatch (Sec. 3.4 Eq.
 * joint-allocation, solved exactly on the conservative grid of App. B.2:
 * Eqs. allocation-grid, allocation-integer-costs, allocation-dp, the tie rules
 * and boundary cases that follow them; available actions of App. B.3 Eq.
 * available-recovery-actions).  Actions: 0 = R (recompute; zero utility,
 * memory and risk), 1 = H (keep; tau_h, dm_h, risk 0), 2 = L (low precision;
 * tau_l, dm_l, risk psi).
 *   q[u]         u8: retained representation of unit u under the plan (0/1/2):
 *                H allows {H, L, R}, L allows {L, R}, anything else only R
 *   verified[u]  u8: bit a set when action a is verified for unit u
 *   tau_h, tau_l, dm_h, dm_l, psi   f64 [n_units]: utilities (Delta tau), memory
 *                costs (Delta m) and the L risk (psi_u, e.g. from
 *                hilore_unit_exposure_risk's exposure times the calibration
 *                factor kappa * ebar of App. B.1 Eq. app-risk-score)
 *   m_res        residual memory budget B - M_peak (>= 0), delta_b risk budget (>= 0)
 *   n_b, n_d     grid intervals N_B, N_delta (1024 in the paper), 1 .. 4096
 * A non-R action is available only if verified, allowed by q, with utility
 * > 0 and finite non-negative costs; L also needs delta_b > 0.  Costs round up
 * to integer grid steps (ceil(cost / (budget / n))); a zero budget keeps one
 * state on its axis and admits only zero costs.  Within a state, actions are
 * tried in the order R, H, L and replace the incumbent only when strictly
 * better; the terminal state is the best value, ties to lower risk cost, then
 * lower memory cost; actions come from backtracking.
 * Outputs (device): action u8 [n_units]; totals f64 [3] = (summed utility,
 * memory, risk of the chosen actions, the latter two summed in unit order);
 * jk i64 [2] = terminal integer memory and risk costs.  All arithmetic is
 * fp64 in the order of a sequential implementation, so results are exact.
 * workspace: device memory of at least hilore_allocate_workspace_bytes(n_units,
 * n_b, n_d) bytes, 16-byte aligned, owned by the caller (about 8.9 MB per
 * table plus 279 KB per unit for a 1025 x 1025 grid); its contents on entry
 * do not matter.  Calls that share a workspace must not overlap.
 * Errors: negative or non-finite budgets, n_b or n_d < 1, null pointers ->
 * INVALID_ARG; n_b or n_d > 4096, n_units > 2^20 -> UNSUPPORTED; workspace too
 * small -> WORKSPACE.
 */
size_t hilore_allocate_workspace_bytes(int n_units, int n_b, int n_d);
hilore_status hilore_allocate(int n_units, const uint8_t *q, const uint8_t *verified,
                              const double *tau_h, const double *tau_l, const double *dm_h,
                              const double *dm_l, const double *psi, double m_res,
                              double delta_b, int n_b, int n_d, uint8_t *action, double *totals,
                              int64_t *jk, void *workspace, size_t workspace_bytes,
                              void *stream);

/*
 * Backward of the gated MLP activation h = silu(g) * u (the MLP of the
 * evaluated Qwen/Llama models, whose gate and up activations are complete MLP
 * tensors eligible for L, App. B.1), with an L operand decoded in registers
 * (App. B.1 Eq. fp8-roundtrip; never written to memory):
 *   du = dh * silu(g),   dg = dh * u * sigmoid(g) * (1 + g * (1 - sigmoid(g)))
 *   gate, up   host descriptors of g and u, [rows, cols] each: an L operand gives
 *              codes (+ scales; not with the cast code) and is decoded to exactly
 *              the bf16 value hilore_decompress writes; otherwise x is read as bf16
 *              (row stride ld).  Either or both may be L (then with the same code
 *              and block); rows and cols must agree.
 *   dh         bf16 [rows, cols] dense; dgate, dup bf16 [rows, cols] dense outputs
 * fp32 arithmetic (sigmoid from the hardware exp2 and reciprocal), each output
 * rounded once to bf16.  Limits: cols % 8 == 0, and cols % block == 0 with an L
 * operand.  Errors: null pointers, mismatched shapes -> INVALID_ARG; bad
 * code/block as for hilore_compress; other shapes -> UNSUPPORTED.
 */
hilore_status hilore_dequant_swiglu_bwd(const hilore_unit_desc *gate, const hilore_unit_desc *up,
                                       int code, int block, const uint16_t *dh, uint16_t *dgate,
                                       uint16_t *dup, void *stream);

/*
 * Relative gradient error of one single-unit L intervention, the calibration
 * target y of App. B.1 Eq. app-calibration-error (Sec. 3.4 Eq.
 * calibration-metrics):
 *   y = sqrt( ||g_l - g_ex||^2 / max(||g_ex||^2, eps_num) )    (the paper: eps_num = 1e-30)
 *   g_l, g_ex  f32 [n]: the trainable-parameter gradients with unit u in L and with
 *              exact recovery, e.g. two outputs of hilore_dequant_wgrad (16-byte aligned)
 *   y          f32 [1] (device, 4-byte aligned; may point into the grad_err array of
 *              hilore_calibrate)
 * The sums are fp64 over the fp32 values, in a fixed order (per-workgroup partial
 * sums in `workspace`, then one fixed tree).  workspace: device memory of at least
 * hilore_grad_rel_err_workspace_bytes(n) bytes (at most 16 KB), 16-byte aligned;
 * its contents on entry do not matter; calls sharing it must not overlap.
 * n = 0 gives y = 0.  Errors: n < 0, eps_num not positive and finite, null
 * pointers -> INVALID_ARG; workspace too small -> WORKSPACE.
 */
size_t hilore_grad_rel_err_workspace_bytes(int64_t n);
hilore_status hilore_grad_rel_err(const float *g_l, const float *g_ex, int64_t n, double eps_num,
                                  float *y, void *workspace, size_t workspace_bytes,
                                  void *stream);

/*
 * Calibration of the L risk (App. B.1 Eqs. app-kappa and app-risk-score; Sec.
 * 3.4 Eq. susceptibility), from n_batches calibration microbatches.  Row b of
 * each [n_batches][n_units] f32 array holds, per unit, the exposure E (from
 * hilore_unit_exposure_risk), the reconstruction error e^L (its rel_err output)
 * and the measured gradient error y (hilore_grad_rel_err).  unit_class i32
 * [n_units] gives the class c(u) (saved-state type and layer); units outside
 * [0, n_classes) take no part in any fit.  Outputs (device):
 *   kappa f64 [n_classes]  kappa_c = max(0, sum x y / sum x^2) over the pairs (u, b)
 *                          of class c, x = E e^L: the least-squares fit of y = kappa x
 *                          over kappa >= 0 (0 when sum x^2 = 0)
 *   ebar  f64 [n_units]    mean over b of e^L (0 when n_batches = 0), summed in
 *                          batch order
 * fp64 arithmetic; kappa's sums run in a fixed order.  Errors: negative sizes,
 * null pointers -> INVALID_ARG; n_units * n_batches >= 2^31 -> UNSUPPORTED.
 */
hilore_status hilore_calibrate(int n_units, int n_batches, int n_classes,
                               const int32_t *unit_class, const float *exposure,
                               const float *rel_err, const float *grad_err, double *kappa,
                               double *ebar, void *stream);

/*
 * Calibrated risk of each unit's L action for the current microbatch (App. B.1
 * Eq. app-risk-score, equal to Sec. 3.4 Eq. token-weighted-risk):
 *   psi[u] = kappa[c(u)] * exposure[u] * ebar[u]   (fp64, multiplied in that order)
 * exposure f32 [n_units] from hilore_unit_exposure_risk; kappa, ebar from
 * hilore_calibrate.  A unit whose class is outside [0, n_classes) has psi = +inf,
 * which makes L unavailable in hilore_allocate (psi is its risk input).
 * Errors: negative sizes, null pointers -> INVALID_ARG.
 */
hilore_status hilore_risk_score(int n_units, const int32_t *unit_class, int n_classes,
                                const double *kappa, const double *ebar, const float *exposure,
                                double *psi, void *stream);

/*
 * Structural sparsity of one batch of update coefficients (the diagnostic
 * statistics of App. D.3), over the n = R*T response slots, padding included.
 *   coeff f32 [R*T], flags u8 [R*T], adv f32 [R]: outputs of hilore_grpo_coeffs;
 *   mask u8 [R*T] or NULL (all valid), as passed to it
 * Outputs (device):
 *   counts i64 [3]  slots whose policy gradient is zero, by exclusive cause:
 *                   [0] padding (mask 0), [1] valid slots of a zero-advantage
 *                   response, [2] valid nonzero-advantage slots on the flat clipped
 *                   branch (flag bit 1); divide by n for the fractions
 *   top_share f64 [1]  share of sum |omega| held by the k = max(1, ceil(top_frac * n))
 *                   largest |omega| (padding counts as 0); 0 when every omega is 0
 * The k-th largest |omega| is found exactly (radix select on the fp32 bit patterns)
 * and ties do not change the result; the sums are fp64 in a fixed order.
 * One workgroup (a diagnostic, not a hot-path step).  Errors: negative sizes,
 * top_frac outside (0, 1], null pointers -> INVALID_ARG; R*T >= 2^31 -> UNSUPPORTED.
 */
hilore_status hilore_update_sparsity(const float *coeff, const uint8_t *flags, const float *adv,
                                     const uint8_t *mask, int R, int T, double top_frac,
                                     int64_t *counts, double *top_share, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* HILORE_H */
