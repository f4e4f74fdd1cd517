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
// Every floating-point sum is fp64 in a fixed order (per-thread partial sums
// over a fixed set of elements, then a fixed LDS tree, or a butterfly per wave
// followed by the wave totals in wave order), with no floating-point atomics;
// the histograms of the sparsity diagnostic are integer counts, exact in any
// order.
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
constexpr int kRelGroups = 4;  // 16-byte groups per thread and operand in a chunk
constexpr int64_t kRelChunk = (int64_t)kRelThreads * kRelGroups;  // groups per chunk
constexpr int kRelFinalThreads = 256;
constexpr int kRelFinalBatch = 8;  // partial pairs a thread loads before adding them

// Partial sums of (a - b)^2 and b^2 over chunks of kRelChunk 16-byte groups
// (16 KiB of each operand): workgroup w takes chunks w, w + grid, ...; the
// grid is at most kRelMaxPartials workgroups (four per CU), each streaming
// several chunks on large arrays (four on a 2^24-element pair: 1.15x faster
// than one short-lived workgroup per chunk).  The last n % 4 elements go to
// workgroup 0.  A thread issues all 2 * kRelGroups loads of a chunk before
// using them; inside a chunk thread t takes groups t, t + 256, ...
__global__ __launch_bounds__(kRelThreads) void rel_err_partial_kernel(const float *a,
                                                                      const float *b, int64_t n,
                                                                      double *part) {
  __shared__ double red[kRelThreads];
  const int64_t n4 = n / 4;
  const float4 *a4 = reinterpret_cast<const float4 *>(a);
  const float4 *b4 = reinterpret_cast<const float4 *>(b);
  double num = 0.0, den = 0.0;
  auto acc = [&](float x, float y) {
    const double d = (double)x - (double)y;
    num = fma(d, d, num);
    den = fma((double)y, (double)y, den);
  };
  for (int64_t c0 = (int64_t)blockIdx.x * kRelChunk; c0 < n4; c0 += (int64_t)gridDim.x * kRelChunk) {
    float4 x[kRelGroups], y[kRelGroups];
#pragma unroll
    for (int k = 0; k < kRelGroups; ++k) {
      const int64_t i = c0 + k * kRelThreads + threadIdx.x;
      x[k] = i < n4 ? a4[i] : float4{0.f, 0.f, 0.f, 0.f};
      y[k] = i < n4 ? b4[i] : float4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int k = 0; k < kRelGroups; ++k) {
      acc(x[k].x, y[k].x);
      acc(x[k].y, y[k].y);
      acc(x[k].z, y[k].z);
      acc(x[k].w, y[k].w);
    }
  }
  if (blockIdx.x == 0 && threadIdx.x < n - 4 * n4) acc(a[4 * n4 + threadIdx.x], b[4 * n4 + threadIdx.x]);
  num = block_sum<kRelThreads>(num, red);
  den = block_sum<kRelThreads>(den, red);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = num;
    part[2 * blockIdx.x + 1] = den;
  }
}

// Thread t adds partials t, t + 256, ... in order (loads issued kRelFinalBatch
// at a time), then an xor butterfly per wave and the 4 wave totals in order.
__global__ __launch_bounds__(kRelFinalThreads) void rel_err_final_kernel(const double *part,
                                                                         int n_part, double eps_num,
                                                                         float *y) {
  __shared__ double red[2][kRelFinalThreads / kWave];
  double num = 0.0, den = 0.0;
  for (int i0 = 0; i0 < n_part; i0 += kRelFinalThreads * kRelFinalBatch) {
    double2 v[kRelFinalBatch];
#pragma unroll
    for (int k = 0; k < kRelFinalBatch; ++k) {
      const int i = i0 + k * kRelFinalThreads + (int)threadIdx.x;
      v[k] = i < n_part ? reinterpret_cast<const double2 *>(part)[i] : double2{0.0, 0.0};
    }
#pragma unroll
    for (int k = 0; k < kRelFinalBatch; ++k) {
      num += v[k].x;
      den += v[k].y;
    }
  }
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) {
    num += __shfl_xor(num, off);
    den += __shfl_xor(den, off);
  }
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  if (lane == 0) {
    red[0][w] = num;
    red[1][w] = den;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double n = red[0][0], d = red[1][0];
    for (int k = 1; k < kRelFinalThreads / kWave; ++k) {
      n += red[0][k];
      d += red[1][k];
    }
    y[0] = (float)sqrt(n / (d > eps_num ? d : eps_num));
  }
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
constexpr int kSpBatch = 8;         // slots a thread loads before using them
constexpr int kSpCache = 32768;     // magnitudes kept in LDS when R*T fits (128 KiB)
constexpr int64_t kSpChunk = (int64_t)kSpThreads * kSpBatch;

// |omega| of slot i as its fp32 bit pattern (padding reads 0): non-negative
// fp32 patterns order like their values.
__device__ __forceinline__ uint32_t mag_bits(const SparsityArgs &a, int64_t i) {
  const bool valid = a.mask ? a.mask[i] != 0 : true;
  return valid ? (__float_as_uint(a.coeff[i]) & 0x7FFFFFFFu) : 0u;
}

// Row of flat slot i (< 2^31) of rows of T slots: the fp64 product i * (1/T)
// is within one of the quotient, and one correction step makes it exact.
__device__ __forceinline__ uint32_t row_of(uint32_t i, uint32_t T, double inv_t) {
  uint32_t r = (uint32_t)((double)i * inv_t);
  if (r * T > i) --r;
  else if ((r + 1) * T <= i) ++r;
  return r;
}

// Add into the wave's own histogram: the lanes sharing the first active
// lane's bin are added with one LDS add, the rest one by one.  For the
// exponent digit this covers both shapes of abs(omega): from a GRPO batch a
// few bins hold most lanes (plain atomics would serialise on them), from a
// spread distribution many bins hold a few lanes each (a loop over distinct
// bins would be long).
__device__ __forceinline__ void hist_add_wave(uint32_t *hist, uint32_t bin, bool active) {
  const int lane = threadIdx.x % kWave;
  const uint64_t todo = __ballot(active);
  if (!todo) return;
  const int leader = __ffsll((unsigned long long)todo) - 1;  // wave-uniform
  const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)bin, leader);
  const uint64_t same = __ballot(active && bin == b);
  if (lane == leader) atomicAdd(&hist[b], (uint32_t)__popcll(same));
  if (((todo & ~same) >> lane) & 1u) atomicAdd(&hist[bin], 1u);
}

// Sum of the waves' private histograms for bin threadIdx.x (< 256), in wave
// order, clearing them for the next pass.  One histogram per wave keeps the
// address conflicts of the LDS atomics inside a wave.
__device__ __forceinline__ uint32_t merge_hist(uint32_t (*whist)[256]) {
  uint32_t s = 0;
  for (int w = 0; w < kSpWaves; ++w) {
    s += whist[w][threadIdx.x];
    whist[w][threadIdx.x] = 0;
  }
  return s;
}

// Radix-select step: with `own` the count of bin threadIdx.x (< 256) of the
// current digit among the slots matching the prefix found so far, pick the
// bin holding the krem-th largest of them.  S(b) = #{slots in bins >= b}; the chosen bin is the
// largest b with S(b) >= krem (bin 0 if none).  256 threads scan suffix sums,
// the one thread whose bin satisfies the condition publishes the result.
__device__ __forceinline__ void select_bin(uint32_t own, uint32_t *wtot, int shift,
                                           uint32_t prefix, long long krem, uint32_t *s_prefix,
                                           long long *s_krem) {
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  uint32_t v = 0;
  if (tid < 256) {
    v = own;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {  // suffix scan inside the wave
      const uint32_t o = __shfl_down(v, off);
      if (lane + off < kWave) v += o;
    }
    if (lane == 0) wtot[w] = v;
  }
  __syncthreads();
  if (tid < 256) {
    long long s = v;  // S(tid)
    for (int w2 = w + 1; w2 < 256 / kWave; ++w2) s += wtot[w2];
    const long long above = s - own;  // S(tid + 1)
    if (above < krem && (s >= krem || tid == 0)) {
      *s_prefix = prefix | ((uint32_t)tid << shift);
      *s_krem = krem - above;
    }
  }
  __syncthreads();
}

// Sum over the workgroup in a fixed order: an xor butterfly inside each wave,
// then wave 0 adds the kSpWaves wave totals in index order; every thread gets
// the total.  `red` holds kSpWaves doubles.
__device__ __forceinline__ double sp_block_sum(double v, double *red) {
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
  if (lane == 0) red[w] = v;
  __syncthreads();
  double t = 0.0;
#pragma unroll
  for (int i = 0; i < kSpWaves; ++i) t += red[i];
  __syncthreads();
  return t;
}

// One workgroup.  The first pass over the slots counts the zero-gradient
// causes, sums |omega| in fp64, builds the histogram of the exponent digit
// (bits 30..23 of the magnitude) and, when R*T fits, keeps the magnitudes in
// LDS.  Three more histogram passes over bits 22..15, 14..7 and 6..0 find the
// k-th largest magnitude m_k exactly (radix select), a last pass sums the
// magnitudes above m_k.  The top-k sum is that sum plus (k - #{above}) copies of
// m_k, whichever of the tied slots a sort would pick.  Slots are walked in
// chunks of kSpChunk, thread t taking slots t, t + 1024, ... of a chunk.
__global__ __launch_bounds__(kSpThreads) void sparsity_kernel(const SparsityArgs a) {
  __shared__ uint32_t cache[kSpCache];
  __shared__ double red[kSpWaves];
  __shared__ uint32_t whist[kSpWaves][256];  // one histogram per wave
  __shared__ uint32_t wtot[256 / kWave];
  __shared__ unsigned long long cnt[3];
  __shared__ uint32_t s_prefix;
  __shared__ long long s_krem;
  const int tid = threadIdx.x, lane = tid % kWave;
  const int64_t n = (int64_t)a.R * a.T;
  const bool cached = n <= kSpCache;
  const int wave = tid / kWave;
  const double inv_t = a.T > 0 ? 1.0 / (double)a.T : 0.0;
  if (tid < 3) cnt[tid] = 0;
  for (int e = tid; e < kSpWaves * 256; e += kSpThreads) (&whist[0][0])[e] = 0;
  __syncthreads();

  unsigned long long c_pad = 0, c_zero = 0, c_clip = 0;  // wave totals (uniform)
  double total = 0.0;
  for (int64_t c0 = 0; c0 < n; c0 += kSpChunk) {
    uint32_t m[kSpBatch];
    bool pad[kSpBatch], zero[kSpBatch], clip[kSpBatch];
#pragma unroll
    for (int j = 0; j < kSpBatch; ++j) {
      const int64_t i = c0 + (int64_t)j * kSpThreads + tid;
      const bool in = i < n;
      const bool valid = in && (a.mask ? a.mask[i] != 0 : true);
      const bool zero_adv = in && a.adv[row_of((uint32_t)i, (uint32_t)a.T, inv_t)] == 0.0f;
      const bool clipped = in && (a.flags[i] & 2) != 0;
      m[j] = in ? mag_bits(a, i) : 0u;
      pad[j] = in && !valid;
      zero[j] = valid && zero_adv;
      clip[j] = valid && !zero_adv && clipped;
    }
#pragma unroll
    for (int j = 0; j < kSpBatch; ++j) {
      const int64_t i = c0 + (int64_t)j * kSpThreads + tid;
      c_pad += __popcll(__ballot(pad[j]));
      c_zero += __popcll(__ballot(zero[j]));
      c_clip += __popcll(__ballot(clip[j]));
      total += (double)__uint_as_float(m[j]);
      hist_add_wave(whist[wave], m[j] >> 23, i < n);
      if (cached && i < n) cache[i] = m[j];
    }
  }
  if (lane == 0) {
    atomicAdd(&cnt[0], c_pad);
    atomicAdd(&cnt[1], c_zero);
    atomicAdd(&cnt[2], c_clip);
  }
  total = sp_block_sum(total, red);  // its barriers complete whist and cnt
  if (tid < 3) a.counts[tid] = (int64_t)cnt[tid];
  if (!(total > 0.0)) {
    if (tid == 0) a.share[0] = 0.0;
    return;
  }

  uint32_t prefix = 0;       // bits of m_k found so far
  long long krem = a.k;      // rank of m_k among the slots matching `prefix`
  select_bin(tid < 256 ? merge_hist(whist) : 0u, wtot, 23, prefix, krem, &s_prefix, &s_krem);
  prefix = s_prefix;
  krem = s_krem;
  constexpr int kShift[3] = {15, 7, 0};
  constexpr uint32_t kDigit[3] = {0xFFu, 0xFFu, 0x7Fu};
  // mask of the bits fixed in `prefix` (bit 31 is 0 in every magnitude)
  uint32_t known = 0x80000000u | (0xFFu << 23);
#pragma unroll
  for (int d = 0; d < 3; ++d) {
    for (int64_t c0 = 0; c0 < n; c0 += kSpChunk) {
      uint32_t m[kSpBatch];
#pragma unroll
      for (int j = 0; j < kSpBatch; ++j) {
        const int64_t i = c0 + (int64_t)j * kSpThreads + tid;
        m[j] = i >= n ? 0xFFFFFFFFu : cached ? cache[i] : mag_bits(a, i);
      }
#pragma unroll
      for (int j = 0; j < kSpBatch; ++j)  // the all-ones filler never matches: bit 31
        if ((m[j] & known) == prefix)
          atomicAdd(&whist[wave][(m[j] >> kShift[d]) & kDigit[d]], 1u);
    }
    __syncthreads();
    select_bin(tid < 256 ? merge_hist(whist) : 0u, wtot, kShift[d], prefix, krem, &s_prefix,
               &s_krem);
    prefix = s_prefix;
    krem = s_krem;
    known |= kDigit[d] << kShift[d];
  }
  double top = 0.0;
  for (int64_t c0 = 0; c0 < n; c0 += kSpChunk) {
#pragma unroll
    for (int j = 0; j < kSpBatch; ++j) {
      const int64_t i = c0 + (int64_t)j * kSpThreads + tid;
      if (i < n) {
        const uint32_t m = cached ? cache[i] : mag_bits(a, i);
        if (m > prefix) top += (double)__uint_as_float(m);
      }
    }
  }
  top = sp_block_sum(top, red);
  if (tid == 0) a.share[0] = (top + (double)krem * (double)__uint_as_float(prefix)) / total;
}

}  // namespace

int rel_err_partials(int64_t n) {
  const int64_t chunks = (n / 4 + kRelChunk - 1) / kRelChunk;
  return (int)(chunks < 1 ? 1 : (chunks > kRelMaxPartials ? kRelMaxPartials : chunks));
}

hipError_t launch_grad_rel_err(const float *g_l, const float *g_ex, int64_t n, double eps_num,
                               float *y, double *part, hipStream_t s) {
  const int np = rel_err_partials(n);
  hipLaunchKernelGGL(rel_err_partial_kernel, dim3(np), dim3(kRelThreads), 0, s, g_l, g_ex, n,
                     part);
  hipLaunchKernelGGL(rel_err_final_kernel, dim3(1), dim3(kRelFinalThreads), 0, s, part, np,
                     eps_num, y);
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
