// Per-unit policy-update exposure and reconstruction risk on gfx950.
//
// For one microbatch, with T the valid response tokens (App. B.1):
//   a_t      = sqrt(ss_x_t / d_u)                     (Eq. activation-token-weights)
//   alpha_t  = (a_t + eps) / (mean_{s in T} a_s + eps)
//   exposure = sum_{t in T} |omega_t| alpha_t         (Eq. mlp-weighted-exposure)
//   risk     = sum_{t in T} |omega_t| sqrt(ss_err_t)  (token-weighted reconstruction
//                                                      error, Sec. 3.4 / Thm. 1)
//   rel_err  = sqrt(sum ss_err) / (sqrt(sum ss_x) + eps)  (Eq. app-calibration-error)
//
// Since the mean of a_t does not depend on t,
//   exposure = sum_{t in T} |omega_t| (a_t + eps) / (sum_{s in T} a_s / |T| + eps),
// so all six sums are formed in ONE pass over the rows.  One workgroup of 1024
// threads per unit reads the row sums written by the encoder plus omega and
// the mask; thread t takes rows t, t + 1024, ... in that order, issuing the
// loads of kBatch rows before using any, then a butterfly per wave and the 16
// wave totals added in wave order: the result does not depend on anything but
// the inputs.
#include "device_common.hpp"
#include "hilore_internal.hpp"

// Every rounding step is the one written: no implicit fused multiply-add
// (the exact sequences above depend on it; wanted FMAs are explicit fmaf).
#pragma clang fp contract(off)

namespace hilore {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kSums = 6;
constexpr int kBatch = 8;  // rows a thread loads before using them

__global__ __launch_bounds__(kThreads) void exposure_risk_kernel(const RiskBatch b) {
  __shared__ float red[kSums][kWaves];
  const RiskUnit &u = b.u[blockIdx.x];
  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  float s_a = 0.f, s_n = 0.f, s_wa = 0.f, s_r = 0.f, s_x = 0.f, s_e = 0.f;
  for (int64_t t0 = 0; t0 < b.rows; t0 += (int64_t)kThreads * kBatch) {
    float sx[kBatch], se[kBatch], om[kBatch];
    bool in[kBatch], valid[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int64_t t = t0 + (int64_t)j * kThreads + tid;
      in[j] = t < b.rows;
      sx[j] = in[j] ? u.ss_x[t] : 0.f;
      se[j] = in[j] ? u.ss_err[t] : 0.f;
      om[j] = in[j] ? b.coeff[t] : 0.f;
      valid[j] = in[j] && (b.mask ? b.mask[t] != 0 : true);
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (!in[j]) continue;
      s_x += sx[j];
      s_e += se[j];
      if (valid[j]) {
        // per-row square roots by the hardware v_sqrt_f32 (within 1 ulp; the
        // sums are checked to 1e-5 against fp64, not bit for bit)
        const float a = __builtin_amdgcn_sqrtf(sx[j] * u.inv_cols);
        const float w = fabsf(om[j]);
        s_a += a;
        s_n += 1.0f;
        s_wa = fmaf(w, a + b.eps_alpha, s_wa);
        s_r = fmaf(w, __builtin_amdgcn_sqrtf(se[j]), s_r);
      }
    }
  }
  const float v[kSums] = {wave_sum(s_a), wave_sum(s_n), wave_sum(s_wa),
                          wave_sum(s_r), wave_sum(s_x), wave_sum(s_e)};
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < kSums; ++k) red[k][wave] = v[k];
  }
  __syncthreads();
  if (tid == 0) {
    float t[kSums];
#pragma unroll
    for (int k = 0; k < kSums; ++k) {
      t[k] = red[k][0];
      for (int i = 1; i < kWaves; ++i) t[k] += red[k][i];
    }
    const float n = t[1];
    const float expo = n > 0.f ? t[2] / (t[0] / n + b.eps_alpha) : 0.f;
    b.exposure[blockIdx.x] = expo;
    b.risk[blockIdx.x] = t[3];
    b.rel_err[blockIdx.x] = sqrtf(t[5]) / (sqrtf(t[4]) + b.eps_rel);
  }
}

}  // namespace

hipError_t launch_exposure_risk(const RiskBatch &b, hipStream_t s) {
  if (b.n == 0) return hipSuccess;
  hipLaunchKernelGGL(exposure_risk_kernel, dim3(b.n), dim3(kThreads), 0, s, b);
  return hipGetLastError();
}

}  // namespace hilore
