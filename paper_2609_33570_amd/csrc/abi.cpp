// C-ABI layer of libhilore: argument validation and dispatch to the gfx950
// kernels.  Every check runs before anything is enqueued and touches no
// device state, so invalid calls fail the same way with or without a GPU.
#include "hilore.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "hilore_internal.hpp"

namespace {

using hilore::CodecBatch;
using hilore::CodecUnit;

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool valid_block(int block) { return block == 32 || block == 64 || block == 128 || block == 256; }

bool valid_code(int code) {
  return code == HILORE_CODE_INT8 || code == HILORE_CODE_FP8_E4M3FN ||
         code == HILORE_CODE_FP8_E4M3FN_CAST;
}

// The blockwise codes need a supported block size; the literal cast has no
// blocks and takes block == 0.
hilore_status check_code_block(int code, int block) {
  if (!valid_code(code)) return HILORE_ERR_INVALID_ARG;
  if (code == HILORE_CODE_FP8_E4M3FN_CAST) return block == 0 ? HILORE_OK : HILORE_ERR_INVALID_ARG;
  return valid_block(block) ? HILORE_OK : HILORE_ERR_UNSUPPORTED;
}

hilore_status hip_status(hipError_t e) { return e == hipSuccess ? HILORE_OK : HILORE_ERR_HIP; }

// Check the fields of one unit that an entry point reads.
enum UnitUse : unsigned {
  kUseX = 1u, kUseCodes = 2u, kUseScales = 4u, kUseXhat = 8u, kUseStats = 16u, kNeedStats = 32u
};

hilore_status check_unit(const hilore_unit_desc &u, int block, unsigned use) {
  if (u.rows < 0 || u.cols < 0) return HILORE_ERR_INVALID_ARG;
  if (block > 0 && u.cols % block != 0) return HILORE_ERR_UNSUPPORTED;
  if (u.rows > hilore::kRowsPerLaunch || u.cols > hilore::kMaxCodecCols)
    return HILORE_ERR_UNSUPPORTED;
  if (u.rows == 0 || u.cols == 0) return HILORE_OK;
  if ((use & kUseX) != 0) {
    if (!u.x) return HILORE_ERR_INVALID_ARG;
    if (u.ld < u.cols) return HILORE_ERR_INVALID_ARG;
    if (u.ld % 8 != 0 || !aligned16(u.x)) return HILORE_ERR_ALIGNMENT;
  }
  if ((use & kUseCodes) != 0) {
    if (!u.codes) return HILORE_ERR_INVALID_ARG;
    if (!aligned16(u.codes)) return HILORE_ERR_ALIGNMENT;
  }
  if ((use & kUseScales) != 0) {
    if (!u.scales) return HILORE_ERR_INVALID_ARG;
    if (!aligned16(u.scales)) return HILORE_ERR_ALIGNMENT;
  }
  if ((use & kUseXhat) != 0) {
    if (!u.xhat) return HILORE_ERR_INVALID_ARG;
    if (!aligned16(u.xhat)) return HILORE_ERR_ALIGNMENT;
  }
  if ((use & (kUseStats | kNeedStats)) != 0) {
    if ((use & kNeedStats) != 0 && (!u.row_ss_x || !u.row_ss_err)) return HILORE_ERR_INVALID_ARG;
    if ((u.row_ss_x && !aligned16(u.row_ss_x)) || (u.row_ss_err && !aligned16(u.row_ss_err)))
      return HILORE_ERR_ALIGNMENT;
  }
  return HILORE_OK;
}

// Validate every unit, then launch in batches of kUnitsPerLaunch.
template <typename Launch>
hilore_status run_codec(const hilore_unit_desc *units, int n_units, int code, int block,
                        unsigned use, bool stats, int lane_steps, Launch launch) {
  if (n_units < 0) return HILORE_ERR_INVALID_ARG;
  if (n_units == 0) return HILORE_OK;
  if (!units) return HILORE_ERR_INVALID_ARG;
  const hilore_status cb = check_code_block(code, block);
  if (cb != HILORE_OK) return cb;
  if (code == HILORE_CODE_FP8_E4M3FN_CAST) use &= ~unsigned(kUseScales);
  for (int i = 0; i < n_units; ++i) {
    const hilore_status st = check_unit(units[i], block, use);
    if (st != HILORE_OK) return st;
  }
  // consecutive units that share a row mapping go to one launch (at most
  // kUnitsPerLaunch units, kRowsPerLaunch rows and, unless one unit alone is
  // larger, kElemsPerLaunch elements per launch)
  CodecBatch b{};
  int64_t rows = 0, elems = 0;
  bool any_stats = false;
  auto flush = [&]() -> hilore_status {
    if (b.n == 0) return HILORE_OK;
    b.row_begin[b.n] = rows;
    b.stats = any_stats ? 1 : 0;
    const hilore_status st = hip_status(launch(b));
    const int wl = b.wpr_log2;
    b = CodecBatch{};
    b.wpr_log2 = wl;
    rows = 0;
    elems = 0;
    any_stats = false;
    return st;
  };
  for (int i = 0; i < n_units; ++i) {
    const hilore_unit_desc &u = units[i];
    if (u.rows == 0 || u.cols == 0) continue;
    const int wl = hilore::codec_wpr_log2(u.cols, lane_steps);
    if (b.n == hilore::kUnitsPerLaunch || (b.n > 0 && wl != b.wpr_log2) ||
        rows + u.rows > hilore::kRowsPerLaunch ||
        (b.n > 0 && elems + u.rows * u.cols > hilore::kElemsPerLaunch)) {
      const hilore_status st = flush();
      if (st != HILORE_OK) return st;
    }
    b.wpr_log2 = wl;
    CodecUnit &c = b.u[b.n];
    c.x = u.x;
    c.codes = static_cast<uint8_t *>(u.codes);
    c.scales = u.scales;
    c.xhat = u.xhat;
    c.ss_x = stats ? u.row_ss_x : nullptr;
    c.ss_err = stats ? u.row_ss_err : nullptr;
    c.rows = u.rows;
    c.cols = u.cols;
    c.ld = u.ld;
    any_stats = any_stats || c.ss_x || c.ss_err;
    b.row_begin[b.n] = rows;
    rows += u.rows;
    elems += u.rows * u.cols;
    ++b.n;
  }
  return flush();
}

// Workspace of hilore_grpo_coeffs: the pre-pass counts, when n slots need one.
size_t grpo_workspace_bytes(int64_t n) {
  return (size_t)hilore::grpo_count_blocks(n) * sizeof(uint32_t);
}

size_t risk_workspace_bytes(int64_t rows, int n_units) {
  return (size_t)n_units * (size_t)hilore::risk_chunks(rows) * hilore::kRiskPartFloats *
         sizeof(float);
}

// Arguments of hilore_unit_exposure_risk other than the workspace.
hilore_status check_exposure_risk(const float *coeff, const uint8_t *mask, int64_t rows,
                                  const hilore_unit_desc *units, int n_units, float eps_alpha,
                                  float eps_rel, const float *exposure, const float *risk,
                                  const float *rel_err) {
  if (rows < 0 || n_units < 0) return HILORE_ERR_INVALID_ARG;
  if (!(eps_alpha >= 0.0f) || !(eps_rel >= 0.0f)) return HILORE_ERR_INVALID_ARG;
  if (n_units == 0) return HILORE_OK;
  if (!units || !exposure || !risk || !rel_err) return HILORE_ERR_INVALID_ARG;
  if (rows >= hilore::kRiskMaxRows) return HILORE_ERR_UNSUPPORTED;
  if (rows > 0 && !coeff) return HILORE_ERR_INVALID_ARG;
  if ((coeff && !aligned16(coeff)) || (mask && !aligned16(mask))) return HILORE_ERR_ALIGNMENT;
  const void *outs[] = {exposure, risk, rel_err};  // written one float at a time
  for (const void *p : outs)
    if ((reinterpret_cast<uintptr_t>(p) & 3u) != 0) return HILORE_ERR_ALIGNMENT;
  for (int i = 0; i < n_units; ++i) {
    const hilore_unit_desc &u = units[i];
    if (u.rows != rows || u.cols <= 0) return HILORE_ERR_INVALID_ARG;
    if (rows > 0) {
      const hilore_status st = check_unit(u, 0, kNeedStats);
      if (st != HILORE_OK) return st;
    }
  }
  return HILORE_OK;
}

// Partial sums of every (row chunk, unit) into part ([unit][chunk] layout),
// then one fold launch over all units.
hilore_status run_exposure_risk(const float *coeff, const uint8_t *mask, int64_t rows,
                                const hilore_unit_desc *units, int n_units, float eps_alpha,
                                float eps_rel, float *exposure, float *risk, float *rel_err,
                                float *part, hipStream_t s) {
  const int64_t n_chunks = hilore::risk_chunks(rows);
  for (int first = 0; first < n_units && n_chunks > 0; first += hilore::kRiskUnitsPerLaunch) {
    hilore::RiskBatch b{};
    b.coeff = coeff;
    b.mask = mask;
    b.rows = rows;
    b.n_chunks = n_chunks;
    b.eps_alpha = eps_alpha;
    b.part = part + (int64_t)first * n_chunks * hilore::kRiskPartFloats;
    for (int i = first; i < n_units && b.n < hilore::kRiskUnitsPerLaunch; ++i) {
      b.ss_x[b.n] = units[i].row_ss_x;
      b.ss_err[b.n] = units[i].row_ss_err;
      b.inv_cols[b.n] = (float)(1.0 / (double)units[i].cols);
      ++b.n;
    }
    const hilore_status st = hip_status(hilore::launch_risk_partial(b, s));
    if (st != HILORE_OK) return st;
  }
  return hip_status(hilore::launch_risk_fold(part, n_units, n_chunks, eps_alpha, eps_rel,
                                             exposure, risk, rel_err, s));
}

}  // namespace

extern "C" {

const char *hilore_status_string(int status) {
  switch (status) {
    case HILORE_OK: return "HILORE_OK";
    case HILORE_ERR_INVALID_ARG: return "HILORE_ERR_INVALID_ARG";
    case HILORE_ERR_ALIGNMENT: return "HILORE_ERR_ALIGNMENT";
    case HILORE_ERR_UNSUPPORTED: return "HILORE_ERR_UNSUPPORTED";
    case HILORE_ERR_WORKSPACE: return "HILORE_ERR_WORKSPACE";
    case HILORE_ERR_HIP: return "HILORE_ERR_HIP";
    default: return "HILORE_ERR_UNKNOWN";
  }
}

int hilore_version(void) { return 10000; }

size_t hilore_grpo_coeffs_workspace_bytes(int P, int G, int T) {
  if (P < 0 || G < 1 || T < 0) return 0;
  return grpo_workspace_bytes((int64_t)P * G * (int64_t)T);
}

hilore_status hilore_grpo_coeffs(const float *rewards, const float *logp_new,
                                 const float *logp_old, const float *logp_ref,
                                 const uint8_t *mask, int P, int G, int T, float clip_eps,
                                 float adv_eps, float beta, double n_norm, float *adv,
                                 float *ratio, uint8_t *flags, float *coeff, void *workspace,
                                 size_t workspace_bytes, void *stream) {
  if (P < 0 || T < 0 || G < 1) return HILORE_ERR_INVALID_ARG;
  if (G > 64) return HILORE_ERR_UNSUPPORTED;
  const int64_t R = (int64_t)P * G;
  const int64_t n = R * (int64_t)T;
  if (n >= (int64_t(1) << 31) || R >= (int64_t(1) << 31)) return HILORE_ERR_UNSUPPORTED;
  if (!(clip_eps > 0.0f && clip_eps < 1.0f) || !(adv_eps >= 0.0f) || !(beta >= 0.0f) ||
      !std::isfinite(beta) || std::isnan(n_norm))
    return HILORE_ERR_INVALID_ARG;
  if (R == 0) return HILORE_OK;
  if (!rewards || !adv) return HILORE_ERR_INVALID_ARG;
  if (!aligned16(rewards) || !aligned16(adv)) return HILORE_ERR_ALIGNMENT;
  if (n > 0) {
    if (!logp_new || !logp_old || !flags || !coeff) return HILORE_ERR_INVALID_ARG;
    if (beta != 0.0f && !logp_ref) return HILORE_ERR_INVALID_ARG;
    const void *ptrs[] = {logp_new, logp_old, logp_ref, mask, ratio, flags, coeff};
    for (const void *p : ptrs)
      if (p && !aligned16(p)) return HILORE_ERR_ALIGNMENT;
  }
  // a pre-pass counts N into the workspace when no N is given for a large masked call
  const bool pre_count = n > 0 && n_norm <= 0.0 && mask && hilore::grpo_count_blocks(n) > 0;
  if (pre_count) {
    if (!workspace) return HILORE_ERR_INVALID_ARG;
    if (!aligned16(workspace)) return HILORE_ERR_ALIGNMENT;
    if (workspace_bytes < grpo_workspace_bytes(n)) return HILORE_ERR_WORKSPACE;
  }
  hilore::GrpoArgs a{};
  a.rewards = rewards;
  a.logp_new = logp_new;
  a.logp_old = logp_old;
  a.logp_ref = beta != 0.0f ? logp_ref : nullptr;
  a.mask = mask;
  a.adv = adv;
  a.ratio = ratio;
  a.coeff = coeff;
  a.flags = flags;
  a.P = P;
  a.G = G;
  a.T = T;
  a.hi = (float)std::log1p((double)clip_eps);
  a.lo = (float)std::log1p(-(double)clip_eps);
  a.adv_eps = adv_eps;
  a.beta = beta;
  a.count_mask = n_norm > 0.0 ? 0 : 1;
  a.inv_n = n_norm > 0.0 ? (float)(1.0 / n_norm) : 0.0f;
  return hip_status(hilore::launch_grpo(a, pre_count ? static_cast<uint32_t *>(workspace) : nullptr,
                                        static_cast<hipStream_t>(stream)));
}

hilore_status hilore_compress(const hilore_unit_desc *units, int n_units, int code, int block,
                              void *stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  return run_codec(units, n_units, code, block, kUseX | kUseCodes | kUseScales | kUseStats, true,
                   hilore::kCompressLaneSteps,
                   [&](const CodecBatch &b) { return hilore::launch_compress(b, code, block, s); });
}

hilore_status hilore_decompress(const hilore_unit_desc *units, int n_units, int code,
                                int block, void *stream) {
  hipStream_t s = static_cast<hipStream_t>(stream);
  return run_codec(units, n_units, code, block, kUseCodes | kUseScales | kUseXhat, false,
                   hilore::kDecompressLaneSteps,
                   [&](const CodecBatch &b) { return hilore::launch_decompress(b, code, block, s); });
}

size_t hilore_unit_exposure_risk_workspace_bytes(int64_t rows, int n_units) {
  if (rows < 0 || n_units < 0 || rows >= hilore::kRiskMaxRows) return 0;
  return risk_workspace_bytes(rows, n_units);
}

hilore_status hilore_unit_exposure_risk(const float *coeff, const uint8_t *mask, int64_t rows,
                                        const hilore_unit_desc *units, int n_units,
                                        float eps_alpha, float eps_rel, float *exposure,
                                        float *risk, float *rel_err, void *workspace,
                                        size_t workspace_bytes, void *stream) {
  const hilore_status st = check_exposure_risk(coeff, mask, rows, units, n_units, eps_alpha,
                                               eps_rel, exposure, risk, rel_err);
  if (st != HILORE_OK || n_units == 0) return st;
  const size_t need = risk_workspace_bytes(rows, n_units);
  if (need > 0 && !workspace) return HILORE_ERR_INVALID_ARG;
  if (workspace && !aligned16(workspace)) return HILORE_ERR_ALIGNMENT;
  if (workspace_bytes < need) return HILORE_ERR_WORKSPACE;
  return run_exposure_risk(coeff, mask, rows, units, n_units, eps_alpha, eps_rel, exposure, risk,
                           rel_err, static_cast<float *>(workspace),
                           static_cast<hipStream_t>(stream));
}

hilore_status hilore_unit_exposure_risk_noalloc(const float *coeff, const uint8_t *mask,
                                                int64_t rows, const hilore_unit_desc *units,
                                                int n_units, float eps_alpha, float eps_rel,
                                                float *exposure, float *risk, float *rel_err,
                                                void *stream) {
  const hilore_status st = check_exposure_risk(coeff, mask, rows, units, n_units, eps_alpha,
                                               eps_rel, exposure, risk, rel_err);
  if (st != HILORE_OK || n_units == 0) return st;
  if (risk_workspace_bytes(rows, n_units) > hilore::kRiskScratchBytes) return HILORE_ERR_WORKSPACE;
  float *part = nullptr;
  if (hilore::risk_scratch(&part) != hipSuccess) return HILORE_ERR_HIP;
  return run_exposure_risk(coeff, mask, rows, units, n_units, eps_alpha, eps_rel, exposure, risk,
                           rel_err, part, static_cast<hipStream_t>(stream));
}

hilore_status hilore_dequant_wgrad(const void *x_codes, const float *x_scales, int code,
                                   int block, const uint16_t *dy, float *dw, int64_t K,
                                   int64_t M, int64_t N, int accumulate, void *stream) {
  if (K < 0 || M < 0 || N < 0) return HILORE_ERR_INVALID_ARG;
  const hilore_status cb = check_code_block(code, block);
  if (cb != HILORE_OK) return cb;
  const bool cast = code == HILORE_CODE_FP8_E4M3FN_CAST;
  if ((!cast && M % block != 0) || M % 8 != 0 || N % 8 != 0) return HILORE_ERR_UNSUPPORTED;
  if (M / 256 + 1 > (1 << 14) || N / 256 + 1 > (1 << 14)) return HILORE_ERR_UNSUPPORTED;
  if (M == 0 || N == 0) return HILORE_OK;
  if (!dw) return HILORE_ERR_INVALID_ARG;
  if (K > 0 && (!x_codes || (!cast && !x_scales) || !dy)) return HILORE_ERR_INVALID_ARG;
  const void *ptrs[] = {x_codes, x_scales, dy, dw};
  for (const void *p : ptrs)
    if (p && !aligned16(p)) return HILORE_ERR_ALIGNMENT;
  hilore::WgradArgs a{};
  a.codes = static_cast<const uint8_t *>(x_codes);
  a.scales = cast ? nullptr : x_scales;
  a.dy = dy;
  a.dw = dw;
  a.K = K;
  a.M = M;
  a.N = N;
  a.accumulate = accumulate ? 1 : 0;
  return hip_status(hilore::launch_wgrad(a, code, block, static_cast<hipStream_t>(stream)));
}

size_t hilore_allocate_workspace_bytes(int n_units, int n_b, int n_d) {
  if (n_units < 0 || n_units > hilore::kAllocMaxUnits || n_b < 1 || n_d < 1 ||
      n_b > hilore::kAllocMaxIntervals || n_d > hilore::kAllocMaxIntervals)
    return 0;
  return hilore::alloc_layout(n_units, n_b + 1, n_d + 1).bytes;
}

hilore_status hilore_allocate(int n_units, const uint8_t *q, const uint8_t *verified,
                              const double *tau_h, const double *tau_l, const double *dm_h,
                              const double *dm_l, const double *psi, double m_res,
                              double delta_b, int n_b, int n_d, uint8_t *action, double *totals,
                              int64_t *jk, void *workspace, size_t workspace_bytes,
                              void *stream) {
  if (n_units < 0 || n_b < 1 || n_d < 1 || !(m_res >= 0.0) || !std::isfinite(m_res) ||
      !(delta_b >= 0.0) || !std::isfinite(delta_b))
    return HILORE_ERR_INVALID_ARG;
  if (n_units > hilore::kAllocMaxUnits || n_b > hilore::kAllocMaxIntervals ||
      n_d > hilore::kAllocMaxIntervals)
    return HILORE_ERR_UNSUPPORTED;
  if (!totals || !jk || !workspace) return HILORE_ERR_INVALID_ARG;
  if (n_units > 0) {
    const void *in[] = {q, verified, tau_h, tau_l, dm_h, dm_l, psi, action};
    for (const void *p : in)
      if (!p) return HILORE_ERR_INVALID_ARG;
    const void *f64[] = {tau_h, tau_l, dm_h, dm_l, psi};
    for (const void *p : f64)
      if ((reinterpret_cast<uintptr_t>(p) & 7u) != 0) return HILORE_ERR_ALIGNMENT;
  }
  if ((reinterpret_cast<uintptr_t>(totals) & 7u) != 0 ||
      (reinterpret_cast<uintptr_t>(jk) & 7u) != 0 || !aligned16(workspace))
    return HILORE_ERR_ALIGNMENT;
  const int KB = m_res > 0.0 ? n_b + 1 : 1;
  const int KD = delta_b > 0.0 ? n_d + 1 : 1;
  if (workspace_bytes < hilore::alloc_layout(n_units, KB, KD).bytes) return HILORE_ERR_WORKSPACE;
  hilore::AllocArgs a{};
  a.q = q;
  a.verified = verified;
  a.tau_h = tau_h;
  a.tau_l = tau_l;
  a.dm_h = dm_h;
  a.dm_l = dm_l;
  a.psi = psi;
  a.m_res = m_res;
  a.delta_b = delta_b;
  a.U = n_units;
  a.n_b = n_b;
  a.n_d = n_d;
  a.action = action;
  a.totals = totals;
  a.jk = jk;
  return hip_status(hilore::launch_allocate(a, KB, KD, workspace, static_cast<hipStream_t>(stream)));
}

size_t hilore_grad_rel_err_workspace_bytes(int64_t n) {
  if (n < 0) return 0;
  return (size_t)hilore::rel_err_partials(n) * 2 * sizeof(double);
}

hilore_status hilore_grad_rel_err(const float *g_l, const float *g_ex, int64_t n, double eps_num,
                                  float *y, void *workspace, size_t workspace_bytes,
                                  void *stream) {
  if (n < 0 || !(eps_num > 0.0) || !std::isfinite(eps_num)) return HILORE_ERR_INVALID_ARG;
  if (!y || !workspace || (n > 0 && (!g_l || !g_ex))) return HILORE_ERR_INVALID_ARG;
  if ((n > 0 && (!aligned16(g_l) || !aligned16(g_ex))) || !aligned16(workspace) ||
      (reinterpret_cast<uintptr_t>(y) & 3u) != 0)
    return HILORE_ERR_ALIGNMENT;
  if (workspace_bytes < hilore_grad_rel_err_workspace_bytes(n)) return HILORE_ERR_WORKSPACE;
  return hip_status(hilore::launch_grad_rel_err(g_l, g_ex, n, eps_num, y,
                                                static_cast<double *>(workspace),
                                                static_cast<hipStream_t>(stream)));
}

hilore_status hilore_calibrate(int n_units, int n_batches, int n_classes,
                               const int32_t *unit_class, const float *exposure,
                               const float *rel_err, const float *grad_err, double *kappa,
                               double *ebar, void *stream) {
  if (n_units < 0 || n_batches < 0 || n_classes < 0) return HILORE_ERR_INVALID_ARG;
  if ((int64_t)n_units * n_batches >= (int64_t(1) << 31)) return HILORE_ERR_UNSUPPORTED;
  if ((n_classes > 0 && !kappa) || (n_units > 0 && (!unit_class || !ebar)) ||
      ((int64_t)n_units * n_batches > 0 && (!exposure || !rel_err || !grad_err)))
    return HILORE_ERR_INVALID_ARG;
  const void *f32[] = {unit_class, exposure, rel_err, grad_err};
  for (const void *p : f32)
    if ((reinterpret_cast<uintptr_t>(p) & 3u) != 0) return HILORE_ERR_ALIGNMENT;
  if ((reinterpret_cast<uintptr_t>(kappa) & 7u) != 0 || (reinterpret_cast<uintptr_t>(ebar) & 7u) != 0)
    return HILORE_ERR_ALIGNMENT;
  hilore::CalibArgs a{};
  a.n_units = n_units;
  a.n_batches = n_batches;
  a.n_classes = n_classes;
  a.unit_class = unit_class;
  a.exposure = exposure;
  a.rel_err = rel_err;
  a.grad_err = grad_err;
  a.kappa = kappa;
  a.ebar = ebar;
  return hip_status(hilore::launch_calibrate(a, static_cast<hipStream_t>(stream)));
}

hilore_status hilore_risk_score(int n_units, const int32_t *unit_class, int n_classes,
                                const double *kappa, const double *ebar, const float *exposure,
                                double *psi, void *stream) {
  if (n_units < 0 || n_classes < 0) return HILORE_ERR_INVALID_ARG;
  if (n_units == 0) return HILORE_OK;
  if (!unit_class || !ebar || !exposure || !psi || (n_classes > 0 && !kappa))
    return HILORE_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(unit_class) & 3u) != 0 ||
      (reinterpret_cast<uintptr_t>(exposure) & 3u) != 0 ||
      (reinterpret_cast<uintptr_t>(kappa) & 7u) != 0 ||
      (reinterpret_cast<uintptr_t>(ebar) & 7u) != 0 || (reinterpret_cast<uintptr_t>(psi) & 7u) != 0)
    return HILORE_ERR_ALIGNMENT;
  return hip_status(hilore::launch_risk_score(n_units, unit_class, n_classes, kappa, ebar,
                                              exposure, psi, static_cast<hipStream_t>(stream)));
}

hilore_status hilore_update_sparsity(const float *coeff, const uint8_t *flags, const float *adv,
                                     const uint8_t *mask, int R, int T, double top_frac,
                                     int64_t *counts, double *top_share, void *stream) {
  if (R < 0 || T < 0 || !(top_frac > 0.0 && top_frac <= 1.0)) return HILORE_ERR_INVALID_ARG;
  const int64_t n = (int64_t)R * T;
  if (n >= (int64_t(1) << 31)) return HILORE_ERR_UNSUPPORTED;
  if (!counts || !top_share || (n > 0 && (!coeff || !flags || !adv))) return HILORE_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(coeff) & 3u) != 0 || (reinterpret_cast<uintptr_t>(adv) & 3u) != 0 ||
      (reinterpret_cast<uintptr_t>(counts) & 7u) != 0 ||
      (reinterpret_cast<uintptr_t>(top_share) & 7u) != 0)
    return HILORE_ERR_ALIGNMENT;
  long long k = (long long)std::ceil(top_frac * (double)n);
  if (k < 1) k = 1;
  if (k > n) k = n;
  hilore::SparsityArgs a{};
  a.coeff = coeff;
  a.flags = flags;
  a.adv = adv;
  a.mask = mask;
  a.R = R;
  a.T = T;
  a.k = k;
  a.counts = counts;
  a.share = top_share;
  return hip_status(hilore::launch_sparsity(a, static_cast<hipStream_t>(stream)));
}

size_t hilore_lora_grad_workspace_bytes(int64_t K, int64_t M, int r) {
  if (K < 0 || M < 0 || r < 1) return 0;
  return hilore::lora_plan(K, M, r).workspace_bytes;
}

hilore_status hilore_dequant_lora_grad(const void *x_codes, const float *x_scales, int code,
                                       int block, const uint16_t *dh, float *da, int64_t K,
                                       int64_t M, int r, float scale, int accumulate,
                                       void *workspace, size_t workspace_bytes, void *stream) {
  if (K < 0 || M < 0 || r < 1 || !std::isfinite(scale)) return HILORE_ERR_INVALID_ARG;
  const hilore_status cb = check_code_block(code, block);
  if (cb != HILORE_OK) return cb;
  const bool cast = code == HILORE_CODE_FP8_E4M3FN_CAST;
  if ((!cast && M % block != 0) || M % 16 != 0 || r % 2 != 0 || r > 4096)
    return HILORE_ERR_UNSUPPORTED;
  if (M >= (int64_t(1) << 26) || K >= (int64_t(1) << 31)) return HILORE_ERR_UNSUPPORTED;
  if (M == 0) return HILORE_OK;
  if (!da || !workspace) return HILORE_ERR_INVALID_ARG;
  if (K > 0 && (!x_codes || (!cast && !x_scales) || !dh)) return HILORE_ERR_INVALID_ARG;
  const void *ptrs[] = {x_codes, x_scales, dh, da, workspace};
  for (const void *p : ptrs)
    if (p && !aligned16(p)) return HILORE_ERR_ALIGNMENT;
  const hilore::LoraPlan plan = hilore::lora_plan(K, M, r);
  if (workspace_bytes < plan.workspace_bytes) return HILORE_ERR_WORKSPACE;
  hilore::LoraArgs a{};
  a.codes = static_cast<const uint8_t *>(x_codes);
  a.scales = cast ? nullptr : x_scales;
  a.dh = dh;
  a.da = da;
  a.part = static_cast<float *>(workspace);
  a.K = K;
  a.M = M;
  a.ldh = r;
  a.scale = scale;
  a.accumulate = accumulate ? 1 : 0;
  a.S = plan.S;
  a.KS = plan.KS;
  a.U = plan.U;
  a.n_wg = plan.n_wg;
  a.xcd_remap = plan.xcd_remap;
  return hip_status(hilore::launch_lora(a, code, block, r, static_cast<hipStream_t>(stream)));
}

hilore_status hilore_dequant_swiglu_bwd(const hilore_unit_desc *gate, const hilore_unit_desc *up,
                                       int code, int block, const uint16_t *dh, uint16_t *dgate,
                                       uint16_t *dup, void *stream) {
  if (!gate || !up) return HILORE_ERR_INVALID_ARG;
  const int64_t rows = gate->rows, cols = gate->cols;
  if (rows < 0 || cols < 0 || up->rows != rows || up->cols != cols) return HILORE_ERR_INVALID_ARG;
  const bool gl = gate->codes != nullptr, ul = up->codes != nullptr;
  if (gl || ul) {
    const hilore_status cb = check_code_block(code, block);
    if (cb != HILORE_OK) return cb;
  }
  if (cols % 8 != 0 || (block > 0 && (gl || ul) && cols % block != 0)) return HILORE_ERR_UNSUPPORTED;
  if (rows == 0 || cols == 0) return HILORE_OK;
  const bool cast = code == HILORE_CODE_FP8_E4M3FN_CAST;
  const hilore_unit_desc *ops[] = {gate, up};
  for (const hilore_unit_desc *o : ops) {
    if (o->codes) {
      if (!cast && !o->scales) return HILORE_ERR_INVALID_ARG;
      if (!aligned16(o->codes) || (!cast && !aligned16(o->scales))) return HILORE_ERR_ALIGNMENT;
    } else {
      if (!o->x || o->ld < cols) return HILORE_ERR_INVALID_ARG;
      if (o->ld % 8 != 0 || !aligned16(o->x)) return HILORE_ERR_ALIGNMENT;
    }
  }
  if (!dh || !dgate || !dup) return HILORE_ERR_INVALID_ARG;
  if (!aligned16(dh) || !aligned16(dgate) || !aligned16(dup)) return HILORE_ERR_ALIGNMENT;
  hilore::SwigluArgs a{};
  a.g_x = gl ? nullptr : gate->x;
  a.u_x = ul ? nullptr : up->x;
  a.g_codes = static_cast<const uint8_t *>(gate->codes);
  a.u_codes = static_cast<const uint8_t *>(up->codes);
  a.g_scales = gl && !cast ? gate->scales : nullptr;
  a.u_scales = ul && !cast ? up->scales : nullptr;
  a.g_ld = gate->ld;
  a.u_ld = up->ld;
  a.dh = dh;
  a.dg = dgate;
  a.du = dup;
  a.rows = rows;
  a.cols = cols;
  return hip_status(hilore::launch_swiglu_bwd(a, code, block, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
