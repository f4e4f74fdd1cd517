// Internal interface between the C-ABI layer (abi.cpp) and the gfx950 kernels.
// Not installed; the public interface is include/hilore.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hilore {

constexpr int kCodeInt8 = 0;
constexpr int kCodeE4M3 = 1;
constexpr int kCodeCast = 2;  // plain E4M3FN cast, no scales

// One unit as the codec kernels see it (a validated copy of hilore_unit_desc).
struct CodecUnit {
  const uint16_t *x;
  uint8_t *codes;
  float *scales;
  uint16_t *xhat;
  float *ss_x;
  float *ss_err;
  int64_t rows;
  int64_t cols;
  int64_t ld;
};

// Units encoded/decoded by one launch travel by value in the kernel
// arguments, so a call needs no device workspace and no host->device copy.
// The units of one launch share the number of waves that sweep a row.
constexpr int kUnitsPerLaunch = 16;
constexpr int64_t kRowsPerLaunch = int64_t(1) << 30;  // bound on a launch's grid
// Elements per launch: units are batched only up to this many (a unit larger
// than it gets a launch of its own).  Launches over a few GB of operands ran
// 3-10% below launches of ~2^28 elements (78 x 16384x3584 int8 and 16 x
// 32768x14336 round trips) while small units gain from sharing a launch.
constexpr int64_t kElemsPerLaunch = int64_t(1) << 28;
// Row lengths the codec kernels support: byte offsets inside a row (2 bytes per
// bf16 element) and the row's buffer range are 32-bit.
constexpr int64_t kMaxCodecCols = int64_t(1) << 30;
struct CodecBatch {
  CodecUnit u[kUnitsPerLaunch];
  int64_t row_begin[kUnitsPerLaunch + 1];  // prefix sum of rows over u[]
  int n;
  int stats;     // compress: write row sums
  int wpr_log2;  // log2 of the waves per row, 0..4
};

// Waves per row (as log2, 0..4) for rows of `cols` columns: the fewest that
// leave each lane at most `lane_steps` steps of 8 columns (measured on
// MI355X over rows of 3584 to 18944 columns: about 5 steps per lane suits
// both directions; fewer waves per row leave the HBM less evenly loaded,
// more waves per row add per-workgroup overhead).
constexpr int kCompressLaneSteps = 5;
constexpr int kDecompressLaneSteps = 5;
inline int codec_wpr_log2(int64_t cols, int lane_steps) {
  const int64_t steps = (cols + 7) / 8;
  int wl = 0;
  while (wl < 4 && (int64_t(64 * lane_steps) << wl) < steps) ++wl;
  return wl;
}

hipError_t launch_compress(const CodecBatch &b, int code, int block, hipStream_t s);
hipError_t launch_decompress(const CodecBatch &b, int code, int block, hipStream_t s);

// Exposure / risk: workgroup (chunk, unit) sums kRiskChunkRows rows of one
// unit into six fp32 partials of kRiskPartFloats floats (padded for 16-byte
// stores), laid out [unit][chunk]; a second launch folds them per unit.
constexpr int kRiskRowsPerThread = 8;
constexpr int64_t kRiskChunkRows = 256 * kRiskRowsPerThread;
constexpr int kRiskPartFloats = 8;
constexpr int64_t kRiskMaxRows = int64_t(1) << 24;  // keeps the valid-row count exact in fp32
constexpr int kRiskUnitsPerLaunch = 96;  // units per partial launch (by value in the arguments)
struct RiskBatch {
  const float *ss_x[kRiskUnitsPerLaunch];
  const float *ss_err[kRiskUnitsPerLaunch];
  float inv_cols[kRiskUnitsPerLaunch];  // 1 / d_u
  float *part;                          // partials of this launch's first unit
  const float *coeff;
  const uint8_t *mask;
  int64_t rows;
  int64_t n_chunks;
  float eps_alpha;
  int n;
};
int64_t risk_chunks(int64_t rows);
hipError_t launch_risk_partial(const RiskBatch &b, hipStream_t s);
hipError_t launch_risk_fold(const float *part, int n_units, int64_t n_chunks, float eps_alpha,
                            float eps_rel, float *exposure, float *risk, float *rel_err,
                            hipStream_t s);
// The allocation-free variant keeps its partials in a fixed device array of
// this many bytes; risk_scratch gives its address on the current device.
constexpr size_t kRiskScratchBytes = size_t(1) << 20;
hipError_t risk_scratch(float **ptr);

struct GrpoArgs {
  const float *rewards, *logp_new, *logp_old, *logp_ref;
  const uint8_t *mask;
  float *adv, *ratio, *coeff;
  uint8_t *flags;
  int P, G, T;
  float hi, lo;       // fp32 log1p(+eps), log1p(-eps)
  float adv_eps, beta;
  float inv_n;        // 1/N when N is given
  int count_mask;     // N = number of valid slots in this call
  const uint32_t *counts;  // set by launch_grpo: pre-pass counts of the mask, or NULL
  int n_counts;
};
// Counting N: up to kGrpoCountInKernelSlots slots every workgroup counts the
// mask itself; beyond, a pre-pass of grpo_count_blocks(slots) workgroups (one
// per kGrpoSlotsPerCount slots, at most kGrpoCounts) writes one uint32 count
// each into the caller's workspace.
constexpr int64_t kGrpoCountInKernelSlots = int64_t(1) << 16;
constexpr int64_t kGrpoSlotsPerCount = int64_t(1) << 16;
constexpr int kGrpoCounts = 256;
int grpo_count_blocks(int64_t slots);
hipError_t launch_grpo(const GrpoArgs &a, uint32_t *counts, hipStream_t s);

struct WgradArgs {
  const uint8_t *codes;
  const float *scales;
  const uint16_t *dy;
  float *dw;
  int64_t K, M, N;
  int accumulate;
};
hipError_t launch_wgrad(const WgradArgs &a, int code, int block, hipStream_t s);

// Joint H/L/R allocation (App. B.2).  Per-unit arrays are device pointers.
struct AllocArgs {
  const uint8_t *q, *verified;
  const double *tau_h, *tau_l, *dm_h, *dm_l, *psi;
  double m_res, delta_b;
  int U, n_b, n_d;
  uint8_t *action;
  double *totals;
  int64_t *jk;
};
struct AllocUnitCost {  // integer costs of one unit on the grid
  int32_t ok_h, ok_l;
  int32_t b_h, b_l, r_l;
  int32_t reach;  // largest memory cost of any state after this unit (cumulative, < KB)
  double tau_h, tau_l;
};
struct AllocLayout {  // the caller's workspace, carved into 256-byte aligned parts
  int S;              // cells per risk row (KB rounded up to 64)
  int64_t cells;      // S * KD
  size_t off_costs, off_f0, off_f1, off_partial, off_pred;
  size_t pred_bytes_per_unit;
  size_t bytes;
};
constexpr int kAllocMaxIntervals = 4096;   // N_B, N_delta at most
constexpr int kAllocMaxUnits = 1 << 20;
AllocLayout alloc_layout(int U, int KB, int KD);
hipError_t launch_allocate(const AllocArgs &a, int KB, int KD, void *workspace, hipStream_t s);

// Calibration scalars (App. B.1 Eqs. app-calibration-error, app-kappa,
// app-risk-score) and the update-sparsity diagnostics (App. D.3).
constexpr int kRelMaxPartials = 1024;  // workgroups of the relative-error reduction (4 per CU)
int rel_err_partials(int64_t n);       // how many of them a reduction over n uses
hipError_t launch_grad_rel_err(const float *g_l, const float *g_ex, int64_t n, double eps_num,
                               float *y, double *part, hipStream_t s);

struct CalibArgs {
  int n_units, n_batches, n_classes;
  const int32_t *unit_class;
  const float *exposure, *rel_err, *grad_err;  // [n_batches][n_units]
  double *kappa, *ebar;
};
hipError_t launch_calibrate(const CalibArgs &a, hipStream_t s);
hipError_t launch_risk_score(int n_units, const int32_t *unit_class, int n_classes,
                             const double *kappa, const double *ebar, const float *exposure,
                             double *psi, hipStream_t s);

struct SparsityArgs {
  const float *coeff;
  const uint8_t *flags;
  const float *adv;
  const uint8_t *mask;
  int R, T;
  long long k;  // ranks in the top share, 1 <= k <= R*T
  int64_t *counts;
  double *share;
};
hipError_t launch_sparsity(const SparsityArgs &a, hipStream_t s);

// LoRA adapter gradient on an L unit (App. D.1.1 adapters; App. B.1 codec).
constexpr int kLoraWorkgroups = 256;  // stream-K grid: one workgroup per CU
struct LoraPlan {
  int64_t S, KS, U;  // strips of 256 columns, k-steps of 32 rows per strip, S * KS
  int64_t n_wg;      // workgroups of the main kernel
  int xcd_remap;     // give each XCD consecutive ranges
  size_t workspace_bytes;
  int passes;        // 16 adapter rows per pass
};
LoraPlan lora_plan(int64_t K, int64_t M, int r);
struct LoraArgs {
  const uint8_t *codes;
  const float *scales;
  const uint16_t *dh;  // bf16 [K, ldh]
  float *da;           // f32 [r, M]
  float *part;         // workspace: 2 partial [16][256] slots per workgroup
  int64_t K, M;
  int ldh, r0, r_pass;
  float scale;
  int accumulate;
  int64_t S, KS, U, n_wg;
  int xcd_remap;
};
hipError_t launch_lora(const LoraArgs &a, int code, int block, int r, hipStream_t s);

// Backward of the gated MLP activation with an L operand decoded in registers.
struct SwigluArgs {
  const uint16_t *g_x, *u_x;       // bf16 operands (row stride g_ld / u_ld), or NULL
  const uint8_t *g_codes, *u_codes;  // L operands: codes [rows, cols] dense, or NULL
  const float *g_scales, *u_scales;
  int64_t g_ld, u_ld;
  const uint16_t *dh;              // bf16 [rows, cols] dense
  uint16_t *dg, *du;               // bf16 [rows, cols] dense
  int64_t rows, cols;
};
hipError_t launch_swiglu_bwd(const SwigluArgs &a, int code, int block, hipStream_t s);

}  // namespace hilore
