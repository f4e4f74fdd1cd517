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
// so all six sums are formed in ONE pass over the rows.  One workgroup per
// unit reads the row sums written by the encoder plus omega and the mask, each
// thread accumulating a fixed strided subset of rows, followed by a fixed LDS
// tree: the result does not depend on anything but the inputs.
#include "device_common.hpp"
#include "hilore_internal.hpp"

// Every rounding step is the one written: no implicit fused multiply-add
// (the exact sequences above depend on it; wanted FMAs are explicit fmaf).
#pragma clang fp contract(off)

namespace hilore {
namespace {

constexpr int kThreads = 512;
constexpr int kSums = 6;

__global__ __launch_bounds__(kThreads) void exposure_risk_kernel(const RiskBatch b) {
  __shared__ float red[kSums][kThreads];
  const RiskUnit &u = b.u[blockIdx.x];
  const int tid = threadIdx.x;
  float s_a = 0.f, s_n = 0.f, s_wa = 0.f, s_r = 0.f, s_x = 0.f, s_e = 0.f;
  for (int64_t t = tid; t < b.rows; t += kThreads) {
    const float sx = u.ss_x[t];
    const float se = u.ss_err[t];
    s_x += sx;
    s_e += se;
    const bool valid = b.mask ? b.mask[t] != 0 : true;
    if (valid) {
      const float a = sqrtf(sx * u.inv_cols);
      const float w = fabsf(b.coeff[t]);
      s_a += a;
      s_n += 1.0f;
      s_wa = fmaf(w, a + b.eps_alpha, s_wa);
      s_r = fmaf(w, sqrtf(se), s_r);
    }
  }
  red[0][tid] = s_a;
  red[1][tid] = s_n;
  red[2][tid] = s_wa;
  red[3][tid] = s_r;
  red[4][tid] = s_x;
  red[5][tid] = s_e;
  __syncthreads();
  for (int h = kThreads / 2; h > 0; h >>= 1) {
    if (tid < h) {
#pragma unroll
      for (int k = 0; k < kSums; ++k) red[k][tid] += red[k][tid + h];
    }
    __syncthreads();
  }
  if (tid == 0) {
    const float n = red[1][0];
    const float expo = n > 0.f ? red[2][0] / (red[0][0] / n + b.eps_alpha) : 0.f;
    b.exposure[blockIdx.x] = expo;
    b.risk[blockIdx.x] = red[3][0];
    b.rel_err[blockIdx.x] = sqrtf(red[5][0]) / (sqrtf(red[4][0]) + b.eps_rel);
  }
}

}  // namespace

hipError_t launch_exposure_risk(const RiskBatch &b, hipStream_t s) {
  if (b.n == 0) return hipSuccess;
  hipLaunchKernelGGL(exposure_risk_kernel, dim3(b.n), dim3(kThreads), 0, s, b);
  return hipGetLastError();
}

}  // namespace hilore
