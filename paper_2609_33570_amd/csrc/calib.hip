// Calibration scalars and update diagnostics on gfx950.
//
//   relative gradient error  y = sqrt(||g_l - g_ex||^2 / max(||g_ex||^2, eps_num))
//                              (App. B.1 Eq. app-calibration-error; Sec. 3.4 Eq.
//                              calibration-metrics): an HBM-bound dual reduction
//   susceptibility           kappa_c = max(0, sum x y / sum x^2), x = E e^L, over the
//                              calibration pairs (u, b) of class c (Eq. app-kappa)
//   mean reconstruction err  ebar_u = mean_b e^L_{u,b}               (Eq. app-risk-score)
//   calibrated risk          psi_u = kappa_{c(u)} E_u ebar_u           (Eq. app-risk-score)
//   update sparsity          padding / zero-advantage / clipped slot counts and the
//                              top-k share of sum |omega| (App. D.3, diagnostic replays)
//
// Every floating-point sum is fp64 in a fixed order (per-thread strided
// partial sums, then a fixed LDS tree), with no floating-point atomics.
#include "device_common.hpp"
#include "hilore_internal.hpp"

#pragma clang fp contract(off)

namespace hilore {
namespace {

// Fixed-order tree over the kThreads values of `red` (kThreads a power of
// two); every thread returns the total.
template <int kThreads>
__device__ __forceinline__ double block_sum(double v, double *red) {
  const int tid = threadIdx.x;
  red[tid] = v;
  __syncthreads();
#pragma unroll
  for (int h = kThreads / 2; h > 0; h >>= 1) {
    if (tid < h) red[tid] += red[tid + h];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

// ---------------------------------------------------------------- y ------
constexpr int kRelThreads = 256;

// Partial sums of (a - b)^2 and b^2 over a grid-strided range of 16-byte
// groups; the last n % 4 elements go to workgroup 0.  Each thread keeps four
// loads in flight per operand.
__global__ __launch_bounds__(kRelThreads) void rel_err_partial_kernel(const float *a,
                                                                      const float *b, int64_t n,
                                                                      double *part) {
  __shared__ double red[kRelThreads];
  const int64_t n4 = n / 4;
  const float4 *a4 = reinterpret_cast<const float4 *>(a);
  const float4 *b4 = reinterpret_cast<const float4 *>(b);
  const int64_t stride = (int64_t)gridDim.x * kRelThreads;
  double num = 0.0, den = 0.0;
  auto acc = [&](float x, float y) {
    const double d = (double)x - (double)y;
    num = fma(d, d, num);
    den = fma((double)y, (double)y, den);
  };
  int64_t i = (int64_t)blockIdx.x * kRelThreads + threadIdx.x;
  for (; i + 3 * stride < n4; i += 4 * stride) {
    float4 x[4], y[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[k] = a4[i + k * stride];
      y[k] = b4[i + k * stride];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      acc(x[k].x, y[k].x);
      acc(x[k].y, y[k].y);
      acc(x[k].z, y[k].z);
      acc(x[k].w, y[k].w);
    }
  }
  for (; i < n4; i += stride) {
    const float4 x = a4[i], y = b4[i];
    acc(x.x, y.x);
    acc(x.y, y.y);
    acc(x.z, y.z);
    acc(x.w, y.w);
  }
  if (blockIdx.x == 0 && threadIdx.x < n - 4 * n4) acc(a[4 * n4 + threadIdx.x], b[4 * n4 + threadIdx.x]);
  num = block_sum<kRelThreads>(num, red);
  den = block_sum<kRelThreads>(den, red);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = num;
    part[2 * blockIdx.x + 1] = den;
  }
}

__global__ __launch_bounds__(kRelThreads) void rel_err_final_kernel(const double *part, int n_part,
                                                                    double eps_num, float *y) {
  __shared__ double red[kRelThreads];
  double num = 0.0, den = 0.0;
  for (int i = threadIdx.x; i < n_part; i += kRelThreads) {
    num += part[2 * i];
    den += part[2 * i + 1];
  }
  num = block_sum<kRelThreads>(num, red);
  den = block_sum<kRelThreads>(den, red);
  if (threadIdx.x == 0) y[0] = (float)sqrt(num / (den > eps_num ? den : eps_num));
}

// ------------------------------------------------------------ kappa, ebar --
constexpr int kCalThreads = 256;

// One workgroup per class c: sums over every (b, u) with class(u) = c.
__global__ __launch_bounds__(kCalThreads) void kappa_kernel(const CalibArgs a) {
  __shared__ double red[kCalThreads];
  const int c = blockIdx.x;
  const int64_t total = (int64_t)a.n_batches * a.n_units;
  double sxy = 0.0, sxx = 0.0;
  for (int64_t i = threadIdx.x; i < total; i += kCalThreads) {
    const int u = (int)(i % a.n_units);
    if (a.unit_class[u] != c) continue;
    const double x = (double)a.exposure[i] * (double)a.rel_err[i];  // exact
    sxy = fma(x, (double)a.grad_err[i], sxy);
    sxx = fma(x, x, sxx);
  }
  sxy = block_sum<kCalThreads>(sxy, red);
  sxx = block_sum<kCalThreads>(sxx, red);
  if (threadIdx.x == 0) {
    const double k = sxx > 0.0 ? sxy / sxx : 0.0;
    a.kappa[c] = k > 0.0 ? k : 0.0;
  }
}

// One thread per unit, summing its batches in order (so the result is the
// sequential sum, bit for bit).
__global__ __launch_bounds__(kCalThreads) void ebar_kernel(const CalibArgs a) {
  const int u = blockIdx.x * kCalThreads + threadIdx.x;
  if (u >= a.n_units) return;
  double s = 0.0;
  for (int b = 0; b < a.n_batches; ++b) s += (double)a.rel_err[(int64_t)b * a.n_units + u];
  a.ebar[u] = a.n_batches > 0 ? s / (double)a.n_batches : 0.0;
}

__global__ __launch_bounds__(kCalThreads) void risk_score_kernel(int n_units,
                                                                 const int32_t *unit_class,
                                                                 int n_classes,
                                                                 const double *kappa,
                                                                 const double *ebar,
                                                                 const float *exposure,
                                                                 double *psi) {
  const int u = blockIdx.x * kCalThreads + threadIdx.x;
  if (u >= n_units) return;
  const int c = unit_class[u];
  psi[u] = (c >= 0 && c < n_classes) ? kappa[c] * (double)exposure[u] * ebar[u]
                                     : __builtin_inf();
}

// ----------------------------------------------------------- sparsity ------
constexpr int kSpThreads = 1024;
constexpr int kSpWaves = kSpThreads / kWave;

// |omega| of slot (r, t) as its fp32 bit pattern (padding reads 0):
// non-negative fp32 patterns order like their values.
__device__ __forceinline__ uint32_t mag_bits(const SparsityArgs &a, int64_t i) {
  const bool valid = a.mask ? a.mask[i] != 0 : true;
  return valid ? (__float_as_uint(a.coeff[i]) & 0x7FFFFFFFu) : 0u;
}

// One workgroup.  Pass 1 counts the zero-gradient causes and sums |omega|;
// four histogram passes over the digits 30..23, 22..15, 14..7 and 6..0 of the
// magnitude bits find the k-th largest magnitude m_k exactly (radix select);
// a last pass sums the magnitudes above m_k.  The top-k sum is that sum plus
// (k - #{above}) copies of m_k, whichever of the tied slots a sort would pick.
// Waves walk response rows, lanes the token slots of a row.
__global__ __launch_bounds__(kSpThreads) void sparsity_kernel(const SparsityArgs a) {
  __shared__ double red[kSpThreads];
  __shared__ uint32_t hist[256];
  __shared__ unsigned long long cnt[3];
  __shared__ uint32_t s_prefix;
  __shared__ long long s_krem;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  if (tid < 3) cnt[tid] = 0;
  __syncthreads();
  unsigned long long c_pad = 0, c_zero = 0, c_clip = 0;
  double total = 0.0;
  for (int r = wave; r < a.R; r += kSpWaves) {
    const bool zero_adv = a.adv[r] == 0.0f;
    for (int t = lane; t < a.T; t += kWave) {
      const int64_t i = (int64_t)r * a.T + t;
      const bool valid = a.mask ? a.mask[i] != 0 : true;
      if (!valid) ++c_pad;
      else if (zero_adv) ++c_zero;
      else if (a.flags[i] & 2) ++c_clip;
      total += (double)__uint_as_float(mag_bits(a, i));
    }
  }
  atomicAdd(&cnt[0], c_pad);
  atomicAdd(&cnt[1], c_zero);
  atomicAdd(&cnt[2], c_clip);
  total = block_sum<kSpThreads>(total, red);
  if (tid < 3) a.counts[tid] = (int64_t)cnt[tid];
  if (!(total > 0.0)) {
    if (tid == 0) a.share[0] = 0.0;
    return;
  }

  constexpr int kShift[4] = {23, 15, 7, 0};
  constexpr uint32_t kDigit[4] = {0xFFu, 0xFFu, 0xFFu, 0x7Fu};
  uint32_t prefix = 0, known = 0;  // bits of m_k found so far, and their mask
  long long krem = a.k;            // rank of m_k among the slots matching `prefix`
#pragma unroll
  for (int d = 0; d < 4; ++d) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int r = wave; r < a.R; r += kSpWaves)
      for (int t = lane; t < a.T; t += kWave) {
        const uint32_t m = mag_bits(a, (int64_t)r * a.T + t);
        if ((m & known) == prefix) atomicAdd(&hist[(m >> kShift[d]) & kDigit[d]], 1u);
      }
    __syncthreads();
    if (tid == 0) {
      long long above = 0;
      int bin = (int)kDigit[d];
      for (; bin > 0; --bin) {
        if (above + (long long)hist[bin] >= krem) break;
        above += hist[bin];
      }
      s_prefix = prefix | ((uint32_t)bin << kShift[d]);
      s_krem = krem - above;
    }
    __syncthreads();
    prefix = s_prefix;
    krem = s_krem;
    known |= kDigit[d] << kShift[d];
  }
  double top = 0.0;
  for (int r = wave; r < a.R; r += kSpWaves)
    for (int t = lane; t < a.T; t += kWave) {
      const uint32_t m = mag_bits(a, (int64_t)r * a.T + t);
      if (m > prefix) top += (double)__uint_as_float(m);
    }
  top = block_sum<kSpThreads>(top, red);
  if (tid == 0) a.share[0] = (top + (double)krem * (double)__uint_as_float(prefix)) / total;
}

}  // namespace

int rel_err_partials(int64_t n) {
  const int64_t groups = (n / 4 + kRelThreads * 16 - 1) / (kRelThreads * 16);
  return (int)(groups < 1 ? 1 : (groups > kRelMaxPartials ? kRelMaxPartials : groups));
}

hipError_t launch_grad_rel_err(const float *g_l, const float *g_ex, int64_t n, double eps_num,
                               float *y, double *part, hipStream_t s) {
  const int np = rel_err_partials(n);
  hipLaunchKernelGGL(rel_err_partial_kernel, dim3(np), dim3(kRelThreads), 0, s, g_l, g_ex, n,
                     part);
  hipLaunchKernelGGL(rel_err_final_kernel, dim3(1), dim3(kRelThreads), 0, s, part, np, eps_num,
                     y);
  return hipGetLastError();
}

hipError_t launch_calibrate(const CalibArgs &a, hipStream_t s) {
  if (a.n_classes > 0)
    hipLaunchKernelGGL(kappa_kernel, dim3(a.n_classes), dim3(kCalThreads), 0, s, a);
  if (a.n_units > 0)
    hipLaunchKernelGGL(ebar_kernel, dim3((a.n_units + kCalThreads - 1) / kCalThreads),
                       dim3(kCalThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_risk_score(int n_units, const int32_t *unit_class, int n_classes,
                             const double *kappa, const double *ebar, const float *exposure,
                             double *psi, hipStream_t s) {
  if (n_units == 0) return hipSuccess;
  hipLaunchKernelGGL(risk_score_kernel, dim3((n_units + kCalThreads - 1) / kCalThreads),
                     dim3(kCalThreads), 0, s, n_units, unit_class, n_classes, kappa, ebar,
                     exposure, psi);
  return hipGetLastError();
}

hipError_t launch_sparsity(const SparsityArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(sparsity_kernel, dim3(1), dim3(kSpThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace hilore
