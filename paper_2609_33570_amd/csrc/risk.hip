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
// so all six sums (sum a, |T|, sum |omega|(a + eps), sum |omega| sqrt(ss_err),
// sum ss_x, sum ss_err) are formed in ONE pass over the rows.
//
// Two launches.  risk_partial_kernel: workgroup (c, u) sums chunk c (2048
// consecutive rows) of unit u; each of its 256 threads loads its 8 rows as two
// runs of 4 (16-byte loads of the row sums and coefficients, 4 mask bytes)
// before using any, adds them in row order, then a butterfly per wave and the
// 4 wave totals in wave order; the six fp32 partials go to the workspace.  A
// launch covers up to kRiskUnitsPerLaunch units x all chunks, so the chip is
// filled even by a handful of units (2 units of 16384 rows: 16 workgroups of
// one load round trip each; 78 units: 624).  risk_fold_kernel: one wave per
// unit adds its chunk partials (lane l takes chunks l, l + 64, ... in order,
// then a butterfly) and forms the three outputs.  Every order is fixed, so the
// results depend on nothing but the inputs; no floating-point atomics.
#include <mutex>

#include "device_common.hpp"
#include "hilore_internal.hpp"

// Every rounding step is the one written: no implicit fused multiply-add
// (the exact sequences above depend on it; wanted FMAs are explicit fmaf).
#pragma clang fp contract(off)

namespace hilore {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kRun = 4;                          // consecutive rows per 16-byte load
constexpr int kRuns = kRiskRowsPerThread / kRun;  // runs of 4 rows per thread
static_assert(kThreads * kRiskRowsPerThread == kRiskChunkRows, "chunk geometry");
constexpr int kSums = 6;

struct Acc {
  float a = 0.f, n = 0.f, wa = 0.f, r = 0.f, x = 0.f, e = 0.f;
};

__device__ __forceinline__ void add_row(Acc &s, float sx, float se, float om, bool valid,
                                        float inv_cols, float eps_alpha) {
  s.x += sx;
  s.e += se;
  if (valid) {
    // per-row square roots by the hardware v_sqrt_f32 (within 1 ulp; the sums
    // are checked to 1e-5 against fp64, not bit for bit)
    const float a = __builtin_amdgcn_sqrtf(sx * inv_cols);
    const float w = fabsf(om);
    s.a += a;
    s.n += 1.0f;
    s.wa = fmaf(w, a + eps_alpha, s.wa);
    s.r = fmaf(w, __builtin_amdgcn_sqrtf(se), s.r);
  }
}

__global__ __launch_bounds__(kThreads) void risk_partial_kernel(const RiskBatch b) {
  __shared__ float red[kSums][kWaves];
  const int ui = blockIdx.y;
  const float *ss_x = b.ss_x[ui];
  const float *ss_err = b.ss_err[ui];
  const float inv_cols = b.inv_cols[ui];
  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const int64_t r0 = (int64_t)blockIdx.x * kRiskChunkRows;

  // ---- every load of the thread first ----
  float sx[kRuns][kRun], se[kRuns][kRun], om[kRuns][kRun];
  uint32_t mk[kRuns];
#pragma unroll
  for (int g = 0; g < kRuns; ++g) {
    const int64_t t = r0 + (int64_t)g * (kThreads * kRun) + (int64_t)tid * kRun;
    if (t + kRun <= b.rows) {  // rows and all arrays are 16-byte aligned at t
      const float4 x4 = *reinterpret_cast<const float4 *>(ss_x + t);
      const float4 e4 = *reinterpret_cast<const float4 *>(ss_err + t);
      const float4 o4 = *reinterpret_cast<const float4 *>(b.coeff + t);
      sx[g][0] = x4.x; sx[g][1] = x4.y; sx[g][2] = x4.z; sx[g][3] = x4.w;
      se[g][0] = e4.x; se[g][1] = e4.y; se[g][2] = e4.z; se[g][3] = e4.w;
      om[g][0] = o4.x; om[g][1] = o4.y; om[g][2] = o4.z; om[g][3] = o4.w;
      mk[g] = b.mask ? *reinterpret_cast<const uint32_t *>(b.mask + t) : 0x01010101u;
    } else {  // ragged tail: rows past the end contribute nothing
      mk[g] = 0;
#pragma unroll
      for (int k = 0; k < kRun; ++k) {
        const bool in = t + k < b.rows;
        sx[g][k] = in ? ss_x[t + k] : 0.f;
        se[g][k] = in ? ss_err[t + k] : 0.f;
        om[g][k] = in ? b.coeff[t + k] : 0.f;
        const uint32_t m = in ? (b.mask ? (b.mask[t + k] != 0 ? 1u : 0u) : 1u) : 0u;
        mk[g] |= m << (8 * k);
      }
    }
  }

  // ---- the thread's rows in order ----
  Acc s;
#pragma unroll
  for (int g = 0; g < kRuns; ++g) {
#pragma unroll
    for (int k = 0; k < kRun; ++k) {
      const bool valid = ((mk[g] >> (8 * k)) & 0xFFu) != 0;
      add_row(s, sx[g][k], se[g][k], om[g][k], valid, inv_cols, b.eps_alpha);
    }
  }
  const float v[kSums] = {wave_sum(s.a), wave_sum(s.n), wave_sum(s.wa),
                          wave_sum(s.r), wave_sum(s.x), wave_sum(s.e)};
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
#pragma unroll
      for (int i = 1; i < kWaves; ++i) t[k] += red[k][i];
    }
    float4 *dst = reinterpret_cast<float4 *>(
        b.part + ((int64_t)ui * b.n_chunks + blockIdx.x) * kRiskPartFloats);
    dst[0] = make_float4(t[0], t[1], t[2], t[3]);
    dst[1] = make_float4(t[4], t[5], 0.f, 0.f);
  }
}

__global__ __launch_bounds__(kWave) void risk_fold_kernel(const float *part, int64_t n_chunks,
                                                          float eps_alpha, float eps_rel,
                                                          float *exposure, float *risk,
                                                          float *rel_err) {
  const int u = blockIdx.x, lane = threadIdx.x;
  const float *p = part + (int64_t)u * n_chunks * kRiskPartFloats;
  float t[kSums] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int64_t c = lane; c < n_chunks; c += kWave) {
    const float4 a = *reinterpret_cast<const float4 *>(p + c * kRiskPartFloats);
    const float4 q = *reinterpret_cast<const float4 *>(p + c * kRiskPartFloats + 4);
    t[0] += a.x; t[1] += a.y; t[2] += a.z; t[3] += a.w;
    t[4] += q.x; t[5] += q.y;
  }
#pragma unroll
  for (int k = 0; k < kSums; ++k) t[k] = wave_sum(t[k]);
  if (lane == 0) {
    const float n = t[1];
    exposure[u] = n > 0.f ? t[2] / (t[0] / n + eps_alpha) : 0.f;
    risk[u] = t[3];
    rel_err[u] = sqrtf(t[5]) / (sqrtf(t[4]) + eps_rel);
  }
}

// Fixed device scratch of the allocation-free variant: the partials of one
// call.  Every GPU the library runs on holds its own copy until the process
// ends; host code never uses this name as an address, only what
// hipGetSymbolAddress returns for the current device (risk_scratch below).
__device__ __align__(256) float scratch[kRiskScratchBytes / sizeof(float)];

}  // namespace

int64_t risk_chunks(int64_t rows) { return (rows + kRiskChunkRows - 1) / kRiskChunkRows; }

hipError_t launch_risk_partial(const RiskBatch &b, hipStream_t s) {
  if (b.n == 0 || b.n_chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(risk_partial_kernel, dim3((unsigned)b.n_chunks, (unsigned)b.n), dim3(kThreads),
                     0, s, b);
  return hipGetLastError();
}

hipError_t launch_risk_fold(const float *part, int n_units, int64_t n_chunks, float eps_alpha,
                            float eps_rel, float *exposure, float *risk, float *rel_err,
                            hipStream_t s) {
  if (n_units == 0) return hipSuccess;
  hipLaunchKernelGGL(risk_fold_kernel, dim3((unsigned)n_units), dim3(kWave), 0, s, part, n_chunks,
                     eps_alpha, eps_rel, exposure, risk, rel_err);
  return hipGetLastError();
}

hipError_t risk_scratch(float **ptr) {
  constexpr int kMaxDevices = 64;
  static std::once_flag once[kMaxDevices];
  static float *addr[kMaxDevices];
  static hipError_t err[kMaxDevices];
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  // once per device, on the first call made with that device current
  std::call_once(once[dev], [dev]() {
    void *p = nullptr;
    err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    addr[dev] = err[dev] == hipSuccess ? static_cast<float *>(p) : nullptr;
  });
  if (err[dev] != hipSuccess) return err[dev];
  *ptr = addr[dev];
  return hipSuccess;
}

}  // namespace hilore
