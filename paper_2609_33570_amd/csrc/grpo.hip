// GRPO update quantities on gfx950: group-relative advantages, importance
// ratios, clip flags and the per-token loss coefficients omega_t = dL/ds_t.
//
//   A_j     = (R_j - mean_group) / (population std_group + adv_eps)
//             (Sec. 3.1; App. D.1.1, "GRPO and optimization")
//   r_t     = exp(s_t - s_t^old)                               (Sec. 3.1)
//   chi_t   = [(A >= 0 and r <= 1+eps) or (A < 0 and r >= 1-eps)]
//                                             (Sec. 3.2, Eq. update-coefficient)
//   omega_t = (m_t / N) (-chi_t r_t A - beta expm1(s_ref - s_t))
//             (Eq. update-coefficient with the K3 KL derivative of the proof of
//             Prop. 1)
//
// Each workgroup of grpo_kernel owns a run of 1024 consecutive token slots
// (4 per thread, 128-bit loads).  It first forms, with wave butterflies, the
// advantages of every group its slots touch (a group of G <= 64 rewards sits
// in the lanes of one wave; the group sums are the pairwise tree over the
// next power of two >= G, which the xor butterfly produces exactly) and keeps
// them in LDS; then every thread processes its 4 slots elementwise.
// When N has to be counted (no N given, a mask present), calls of at most
// kGrpoCountInKernelSlots slots let every workgroup count the whole mask
// itself (bytes summed four at a time with a dot product): one launch, no
// scratch, and the mask (at most 64 KB) stays in L2.  Larger calls first run
// count_kernel, whose workgroups each count one contiguous range of the mask
// into the caller's workspace (one 32-bit count each, at most kGrpoCounts),
// and every workgroup of grpo_kernel then adds those counts (exact integer
// sums): the mask is read once more in total instead of once per workgroup.
// Every load a thread makes is issued before the first arithmetic (the mask
// words or counts for N in batches of 8 per thread), so a launch waits on
// memory about once instead of once per phase.
#include "device_common.hpp"
#include "hilore_internal.hpp"

// Every rounding step is the one written: no implicit fused multiply-add
// (the exact sequences above depend on it; wanted FMAs are explicit fmaf).
#pragma clang fp contract(off)

namespace hilore {
namespace {

constexpr int kThreads = 256;
constexpr int kSlotsPerThread = 4;
constexpr int kSlotsPerBlock = kThreads * kSlotsPerThread;
constexpr int kMaxResp = kSlotsPerBlock + 2;  // responses overlapping one run (T >= 1)
constexpr int kMaskBatch = 8;  // 16-byte mask words per thread in flight while counting
static_assert(kGrpoCounts <= kThreads, "one pre-pass count per thread");

// Pairwise-tree sum over the first P2 lanes (P2 a power of two <= 64) by an
// xor butterfly; lanes >= P2 must not be mixed in, so the loop stops at P2/2.
__device__ __forceinline__ float group_sum(float v, int p2) {
  for (int off = 1; off < p2; off <<= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t w) {
  w |= w >> 4;
  w |= w >> 2;
  w |= w >> 1;
  return __builtin_amdgcn_udot4(w & 0x01010101u, 0x01010101u, 0u, false);
}

// Count of the nonzero bytes of mask words [w0, w1) plus, in the last
// workgroup, of the bytes past the last whole word; one 32-bit count per
// workgroup.
__global__ __launch_bounds__(kThreads) void count_kernel(const uint8_t *mask, int64_t n_slots,
                                                         int64_t words_per_wg, uint32_t *counts) {
  __shared__ uint32_t red[kThreads / kWave];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int64_t n_words = n_slots / 16;
  const int64_t w0 = (int64_t)blockIdx.x * words_per_wg;
  const int64_t w1 = w0 + words_per_wg < n_words ? w0 + words_per_wg : n_words;
  const uint4 *m4 = reinterpret_cast<const uint4 *>(mask);
  uint32_t cnt = 0;
  for (int64_t base = w0; base < w1; base += kMaskBatch * kThreads) {
    uint4 mw[kMaskBatch];
#pragma unroll
    for (int u = 0; u < kMaskBatch; ++u) {
      const int64_t i = base + (int64_t)u * kThreads + tid;
      mw[u] = i < w1 ? m4[i] : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < kMaskBatch; ++u)
      cnt += nonzero_bytes(mw[u].x) + nonzero_bytes(mw[u].y) + nonzero_bytes(mw[u].z) +
             nonzero_bytes(mw[u].w);
  }
  if (blockIdx.x == gridDim.x - 1)
    for (int64_t i = n_words * 16 + tid; i < n_slots; i += kThreads) cnt += mask[i] != 0;
  for (int off = 1; off < kWave; off <<= 1) cnt += __shfl_xor(cnt, off, kWave);
  if (lane == 0) red[wave] = cnt;
  __syncthreads();
  if (tid == 0) counts[blockIdx.x] = red[0] + red[1] + red[2] + red[3];
}

__global__ __launch_bounds__(kThreads) void grpo_kernel(const GrpoArgs a, int p2) {
  __shared__ float adv_lds[kMaxResp];
  __shared__ uint32_t red[kThreads / kWave];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int64_t R = (int64_t)a.P * a.G;
  const bool no_tokens = a.T == 0;
  const int64_t T = no_tokens ? 1 : a.T;  // with T == 0 a run covers responses
  const int64_t n_slots = R * T;
  const int64_t c0 = (int64_t)blockIdx.x * kSlotsPerBlock;
  const int64_t c1 = c0 + kSlotsPerBlock < n_slots ? c0 + kSlotsPerBlock : n_slots;
  const int64_t j_lo = c0 / T;
  const int64_t j_hi = (c1 - 1) / T;  // inclusive
  const int64_t g_lo = j_lo / a.G;
  const int64_t g_hi = j_hi / a.G;

  // ---- loads first ----
  // Nothing below changes what a thread reads, so its token slots and the
  // first batch of mask words for the count are requested before any
  // arithmetic: the whole prologue then waits on memory about once.
  const int i0 = (int)c0 + tid * kSlotsPerThread;  // P*G*T < 2^31
  const bool has_slots = !no_tokens && i0 < c1;
  float sn[4] = {0.f, 0.f, 0.f, 0.f}, so[4] = {0.f, 0.f, 0.f, 0.f}, sref[4] = {0.f, 0.f, 0.f, 0.f};
  uint32_t mk = 0x01010101u;
  const bool full = i0 + kSlotsPerThread <= c1;
  if (has_slots) {
    if (full) {
      const float4 n4 = *reinterpret_cast<const float4 *>(a.logp_new + i0);
      const float4 o4 = *reinterpret_cast<const float4 *>(a.logp_old + i0);
      sn[0] = n4.x; sn[1] = n4.y; sn[2] = n4.z; sn[3] = n4.w;
      so[0] = o4.x; so[1] = o4.y; so[2] = o4.z; so[3] = o4.w;
      if (a.beta != 0.0f) {
        const float4 r4 = *reinterpret_cast<const float4 *>(a.logp_ref + i0);
        sref[0] = r4.x; sref[1] = r4.y; sref[2] = r4.z; sref[3] = r4.w;
      }
      if (a.mask) mk = *reinterpret_cast<const uint32_t *>(a.mask + i0);
    } else {
      mk = 0;
      for (int k = 0; k < kSlotsPerThread; ++k) {
        const int i = i0 + k;
        const bool in = i < c1;
        sn[k] = in ? a.logp_new[i] : 0.0f;
        so[k] = in ? a.logp_old[i] : 0.0f;
        if (a.beta != 0.0f) sref[k] = in ? a.logp_ref[i] : 0.0f;
        const uint32_t m = in ? (a.mask ? a.mask[i] : 1u) : 0u;
        mk |= m << (8 * k);
      }
    }
  }
  // counts of a count_kernel pre-pass (one per thread at most), else the mask itself
  uint32_t pre = 0;
  if (!no_tokens && a.count_mask && a.counts && tid < a.n_counts) pre = a.counts[tid];
  const bool count_words = !no_tokens && a.count_mask && a.mask && !a.counts;
  const int64_t n_words = count_words ? n_slots / 16 : 0;
  const uint4 *m4 = reinterpret_cast<const uint4 *>(a.mask);
  uint4 mw[kMaskBatch];
#pragma unroll
  for (int u = 0; u < kMaskBatch; ++u) {
    const int64_t i = (int64_t)u * kThreads + tid;
    mw[u] = i < n_words ? m4[i] : make_uint4(0u, 0u, 0u, 0u);
  }

  // ---- advantages of the groups this run touches ----
  for (int64_t grp = g_lo + wave; grp <= g_hi; grp += kThreads / kWave) {
    const int64_t j = grp * a.G + lane;
    const bool in = lane < a.G;
    const float rew = in ? a.rewards[j] : 0.0f;
    const float mu = group_sum(rew, p2) / (float)a.G;
    const float dv = in ? rew - mu : 0.0f;
    const float sigma = sqrtf(group_sum(dv * dv, p2) / (float)a.G);
    const float adv = dv / (sigma + a.adv_eps);
    if (in) {
      if (j >= j_lo && j <= j_hi) adv_lds[j - j_lo] = adv;
      if (j * T >= c0 && j * T < c1) a.adv[j] = adv;  // owner of the response's first slot
    }
  }

  if (no_tokens) return;  // advantages only

  // ---- normaliser ----
  float inv_n = a.inv_n;
  if (a.count_mask) {
    uint32_t cnt = 0;
    if (a.counts) {
      cnt = pre;
    } else if (a.mask) {
      for (int64_t base = 0; base < n_words; base += kMaskBatch * kThreads) {
        if (base > 0) {  // later batches: all loads of a batch in flight at once
#pragma unroll
          for (int u = 0; u < kMaskBatch; ++u) {
            const int64_t i = base + (int64_t)u * kThreads + tid;
            mw[u] = i < n_words ? m4[i] : make_uint4(0u, 0u, 0u, 0u);
          }
        }
#pragma unroll
        for (int u = 0; u < kMaskBatch; ++u)
          cnt += nonzero_bytes(mw[u].x) + nonzero_bytes(mw[u].y) + nonzero_bytes(mw[u].z) +
                 nonzero_bytes(mw[u].w);
      }
      for (int64_t i = n_words * 16 + tid; i < n_slots; i += kThreads) cnt += a.mask[i] != 0;
    } else {
      cnt = tid == 0 ? (uint32_t)n_slots : 0u;
    }
    for (int off = 1; off < kWave; off <<= 1) cnt += __shfl_xor(cnt, off, kWave);
    if (lane == 0) red[wave] = cnt;
    __syncthreads();
    const uint32_t n = red[0] + red[1] + red[2] + red[3];
    inv_n = n > 0 ? 1.0f / (float)n : 0.0f;
  } else {
    __syncthreads();
  }

  // ---- per-token quantities ----
  if (!has_slots) return;

  float rat[4], om[4];
  uint32_t fl = 0;
#pragma unroll
  for (int k = 0; k < kSlotsPerThread; ++k) {
    const int j = (i0 + k) / (int)T;
    const float A = adv_lds[(j < j_hi ? j : j_hi) - j_lo];
    const bool m = ((mk >> (8 * k)) & 0xFFu) != 0;
    const float delta = sn[k] - so[k];
    const bool chi = A >= 0.0f ? delta <= a.hi : delta >= a.lo;
    const float r = expf(delta);
    const float pol = chi ? r * A : 0.0f;
    const float kl = a.beta != 0.0f ? a.beta * expm1f(sref[k] - sn[k]) : 0.0f;
    rat[k] = r;
    om[k] = m ? (-pol - kl) * inv_n : 0.0f;
    const uint32_t f = (m && chi ? 1u : 0u) | (m && A != 0.0f && !chi ? 2u : 0u);
    fl |= f << (8 * k);
  }
  if (full) {
    *reinterpret_cast<float4 *>(a.coeff + i0) = make_float4(om[0], om[1], om[2], om[3]);
    if (a.ratio) *reinterpret_cast<float4 *>(a.ratio + i0) = make_float4(rat[0], rat[1], rat[2], rat[3]);
    *reinterpret_cast<uint32_t *>(a.flags + i0) = fl;
  } else {
    for (int k = 0; k < kSlotsPerThread; ++k) {
      const int i = i0 + k;
      if (i < c1) {
        a.coeff[i] = om[k];
        if (a.ratio) a.ratio[i] = rat[k];
        a.flags[i] = (uint8_t)(fl >> (8 * k));
      }
    }
  }
}

}  // namespace

int grpo_count_blocks(int64_t slots) {
  if (slots <= kGrpoCountInKernelSlots) return 0;
  const int64_t n = (slots + kGrpoSlotsPerCount - 1) / kGrpoSlotsPerCount;
  return (int)(n < kGrpoCounts ? n : kGrpoCounts);
}

hipError_t launch_grpo(const GrpoArgs &a, uint32_t *counts, hipStream_t s) {
  const int64_t R = (int64_t)a.P * a.G;
  const int64_t slots = a.T == 0 ? R : R * a.T;
  if (slots == 0) return hipSuccess;
  int p2 = 1;
  while (p2 < a.G) p2 <<= 1;
  GrpoArgs b = a;
  b.counts = nullptr;
  b.n_counts = 0;
  if (a.T > 0 && a.count_mask && a.mask && counts) {
    const int nb = grpo_count_blocks(slots);
    if (nb > 0) {  // counted by a pre-pass into the workspace
      const int64_t n_words = slots / 16;
      const int64_t per = (n_words + nb - 1) / nb;
      hipLaunchKernelGGL(count_kernel, dim3((unsigned)nb), dim3(kThreads), 0, s, a.mask, slots,
                         per, counts);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      b.counts = counts;
      b.n_counts = nb;
    }
  }
  const int64_t grid = (slots + kSlotsPerBlock - 1) / kSlotsPerBlock;
  hipLaunchKernelGGL(grpo_kernel, dim3((unsigned)grid), dim3(kThreads), 0, s, b, p2);
  return hipGetLastError();
}

}  // namespace hilore
