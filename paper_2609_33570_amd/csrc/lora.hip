// Adapter gradient of a LoRA linear layer whose saved input is an L unit, with
// the reconstruction fused into the operand load, on gfx950 MFMA:
//   dA[r][i] (+)= scale * sum_t dh[t][r] * xhat[t][i],
//   xhat[t][i] = bf16_RNE(value(code[t][i]) * scale[t][i / BLOCK])
// (or value(code) exactly for the literal cast).  For the layer output
// y = X W^T + scale * (X A^T) B^T and an upstream gradient G, dh = G B; this
// is the paper's default setting (rank-16 adapters on q/k/v/o and gate/up/down,
// alpha = 32, App. D.1.1), where the adapter gradient is the only backward
// consumer of the saved MLP activation that feeds a frozen projection.
//
// The work is a 16-row output contracted over all K tokens: reading the codes
// once (1 + 4/BLOCK bytes per element) bounds it; MFMA serves the 32 FLOP per
// element that a vector unit could not keep up with.
//
// Mapping.  A strip is 256 columns of X; a k-step is 32 token rows of a strip.
// In a k-step, lane (q, h) = (lane % 16, lane / 16) loads rows 8h .. 8h+7 of
// columns 16q .. 16q+15 (one 16-byte load per row: every row of the strip is
// read as 256 contiguous bytes), dequantises them and hands column 16q + c to
// MFMA c (c = 0..15, v_mfma_f32_16x16x32_bf16): its B operand is then 8
// consecutive tokens of one column per lane, as the instruction wants, with
// no transpose.  The A operand is dh^T: lane (q, h) holds dh[8h .. 8h+7][q],
// the same for all 16 MFMAs.  MFMA c accumulates dA[4h + v][16q' + c] in lane
// (q', h), register v.
//
// Balance and locality.  The (strip, k-step) units are numbered strip-major and
// dealt to 256 workgroups in equal contiguous ranges (stream-K), so every CU
// gets the same work whatever the shape; a range meets at most two strips (the
// grid has at least as many workgroups as strips).  Units of fewer than 32
// strips instead split every strip into equal parts, one per workgroup (see
// lora_plan).  With at least 32 strips the
// workgroup index is remapped so that the 32 workgroups on one XCD (dispatch is
// round-robin over the 8 XCDs) take consecutive ranges, i.e. about 1/8 of the
// strips: the scale lines of those strips and the dh rows (read by every strip)
// then stay in that XCD's L2, helped by streaming the codes past it
// (non-temporal loads), instead of being fetched again for every strip.
// Within a strip the 8 waves of a workgroup take every 8th k-step, two of them
// in flight ahead of the one being computed through a ring in LDS (LDS-DMA); at
// the end of its part of a strip a workgroup sums its waves' accumulators
// through LDS in wave order and stores one partial [16][256] to the caller's
// workspace.  A second kernel adds, for each output element, the partials of
// the workgroups that covered its strip in ascending order: no floating-point
// atomics, and the result does not depend on the timing.
#include "device_common.hpp"
#include "hilore_internal.hpp"

// Every rounding step is the one written: no implicit fused multiply-add.
#pragma clang fp contract(off)

namespace hilore {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;
constexpr int kStrip = 256;  // columns per strip, 16 per lane
constexpr int kStep = 32;    // token rows per k-step, 8 per lane
constexpr int kRows = 16;    // adapter rows per pass (the MFMA's M)
constexpr int kPart = kRows * kStrip;
constexpr uint32_t kOob = 0x80000000u;  // a buffer offset past every range: loads 0
constexpr int kNonTemporal = 2;         // cache policy of the streamed codes: NT

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Operands of one k-step for one lane: the codes of rows 8h + j, columns
// 16q .. 16q+15, the block scale of each row and dh[8h + j][r0 + q] (bf16 bits
// in the low half).
struct Raw {
  u32x4 c[8];
  float s[8];
  uint32_t d[8];
};

// Per-lane, loop-invariant parts of the loads.
struct Plan {
  uint32_t vo_c;        // byte offset of row 8h in a k-step (kOob: no data)
  uint32_t st_c;        // byte stride of one token row
  uint32_t vo_d[4];     // dh pair fetched by this lane in each of its dh DMAs
  uint32_t vo_s[4];     // scale fetched by this lane in each of its scale DMAs
  uint32_t rd_s;        // LDS byte offset of its row 8h scale inside the scale area
};

// One ring slot holds a whole k-step for one wave, filled by LDS-DMA:
//   [0, 8192)      codes: row j's 16 bytes of lane l at 1024 j + 16 l
//   [8192, 9216)   dh of the k-step's 32 rows x 16 adapter rows, row-major bf16
//                  (one 4-byte pair per lane and DMA: DMAs of at most 4 bytes
//                  place lane l at 4 l)
//   [9216, 10240)  scales of the k-step's 32 rows x (256 / BLOCK) blocks,
//                  (row, block) at 9216 + 4 (row * nb + block)
// Each lane reads back what it needs; no operand of a k-step in flight lives
// in registers.
constexpr int kSlot = 10240;
constexpr int kDhOff = 8192, kScOff = 9216;
template <int BLOCK>
constexpr int kScaleDmas = (32 * (kStrip / BLOCK) + 63) / 64;

// Rows of k-step kk that exist (0 past K or when the step is not this wave's).
__device__ __forceinline__ int64_t step_rows(const LoraArgs &a, int64_t kk, bool live) {
  const int64_t left = a.K - kk * kStep;
  return !live || left <= 0 ? 0 : (left < kStep ? left : kStep);
}

typedef __attribute__((address_space(3))) void lds_void;

// k-step kk into ring slot `slot`: rows past K and columns past M read as 0.
template <int CODE, int BLOCK>
__device__ __forceinline__ void dma_step(uint8_t *slot, const LoraArgs &a, const Plan &p,
                                         int64_t kk, bool live) {
  const int64_t rows = step_rows(a, kk, live);
  const int64_t t0 = kk * kStep;
  const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(a.codes + t0 * a.M), 0, (int)(rows * a.M), 0x00020000);
#pragma unroll
  for (int j = 0; j < 8; ++j)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (lds_void *)(slot + 1024 * j), 16,
                                             (int)(p.vo_c + j * p.st_c), 0, 0, kNonTemporal);
  const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(a.dh + t0 * a.ldh), 0, (int)(rows * a.ldh * 2), 0x00020000);
#pragma unroll
  for (int i = 0; i < 4; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, (lds_void *)(slot + kDhOff + 256 * i), 4,
                                             (int)p.vo_d[i], 0, 0, 0);
  if constexpr (CODE != kCodeCast) {
    const int64_t sld = a.M / BLOCK;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.scales + t0 * sld), 0, (int)(rows * sld * 4), 0x00020000);
#pragma unroll
    for (int i = 0; i < kScaleDmas<BLOCK>; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)(slot + kScOff + 256 * i), 4,
                                               (int)p.vo_s[i], 0, 0, 0);
  }
}
// VMEM instructions of one k-step
template <int CODE, int BLOCK>
constexpr int kStepLoads = 8 + 4 + (CODE == kCodeCast ? 0 : kScaleDmas<BLOCK>);

// Code bytes C, C+1 (C even) of a 4-byte word -> exact fp32 code values.
template <int CODE, int C>
__device__ __forceinline__ f32x2 decode_pair(uint32_t w) {
  if constexpr (CODE == kCodeInt8) {
    return f32x2{(float)(int)__builtin_amdgcn_sbfe(w, 8 * C, 8),
                 (float)(int)__builtin_amdgcn_sbfe(w, 8 * C + 8, 8)};
  } else {
    return __builtin_amdgcn_cvt_pk_f32_fp8((int)w, C == 2);
  }
}

// Columns 4 D + C and 4 D + C + 1 of the lane's 16 (dword D, byte pair C of
// every row): two B operands of 8 tokens each, xhat rounded to bf16 exactly
// as the decoder rounds it, then the two MFMAs.
template <int CODE, int D, int C>
__device__ __forceinline__ void mma_pair(f32x4 (&acc)[16], const Raw &w, const bf16x8 &A) {
  float lo[8], hi[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t word = D == 0 ? w.c[j].x : D == 1 ? w.c[j].y : D == 2 ? w.c[j].z : w.c[j].w;
    const f32x2 v = decode_pair<CODE, C>(word);
    if constexpr (CODE == kCodeCast) {
      lo[j] = v.x;
      hi[j] = v.y;
    } else {
      lo[j] = v.x * w.s[j];
      hi[j] = v.y * w.s[j];
    }
  }
  u32x4 b0, b1;
  b0.x = pack_bf16(lo[0], lo[1]);
  b0.y = pack_bf16(lo[2], lo[3]);
  b0.z = pack_bf16(lo[4], lo[5]);
  b0.w = pack_bf16(lo[6], lo[7]);
  b1.x = pack_bf16(hi[0], hi[1]);
  b1.y = pack_bf16(hi[2], hi[3]);
  b1.z = pack_bf16(hi[4], hi[5]);
  b1.w = pack_bf16(hi[6], hi[7]);
  constexpr int c0 = 4 * D + C;
  acc[c0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, __builtin_bit_cast(bf16x8, b0), acc[c0],
                                                     0, 0, 0);
  acc[c0 + 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, __builtin_bit_cast(bf16x8, b1),
                                                         acc[c0 + 1], 0, 0, 0);
}

template <int CODE>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[16], const Raw &w) {
  u32x4 a;
  a.x = (w.d[0] & 0xFFFFu) | (w.d[1] << 16);
  a.y = (w.d[2] & 0xFFFFu) | (w.d[3] << 16);
  a.z = (w.d[4] & 0xFFFFu) | (w.d[5] << 16);
  a.w = (w.d[6] & 0xFFFFu) | (w.d[7] << 16);
  const bf16x8 A = __builtin_bit_cast(bf16x8, a);
  // one column pair at a time: its decode stays next to its two MFMAs
  // instead of all 128 values being formed ahead of them
  mma_pair<CODE, 0, 0>(acc, w, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 0, 2>(acc, w, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 1, 0>(acc, w, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 1, 2>(acc, w, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 2, 0>(acc, w, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 2, 2>(acc, w, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 3, 0>(acc, w, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 3, 2>(acc, w, A);
}

// First unit of the range of (remapped) workgroup w.
__device__ __forceinline__ int64_t range_begin(const LoraArgs &a, int64_t w) {
  return a.U * w / a.n_wg;
}

// s_waitcnt with only the vector-memory count limited (expcnt and lgkmcnt
// at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// One k-step of this wave from ring slot `slot`: wait for its DMAs (the next
// k-step's stay in flight), read the operands into registers, refill the
// slot with the k-step after next, and run the MFMAs.
template <int CODE, int BLOCK>
__device__ __forceinline__ void ring_step(f32x4 (&acc)[16], uint8_t *slot, const LoraArgs &a,
                                          const Plan &p, int64_t kk, int64_t k_end, int lane) {
  wait_vmcnt<kStepLoads<CODE, BLOCK>>();
  Raw w;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    w.c[j] = *reinterpret_cast<const u32x4 *>(slot + 1024 * j + 16 * lane);
    w.d[j] = *reinterpret_cast<const uint16_t *>(slot + kDhOff + 2 * (16 * (8 * (lane >> 4) + j) +
                                                                       (lane & 15)));
    if constexpr (CODE != kCodeCast)
      w.s[j] = *reinterpret_cast<const float *>(slot + kScOff + p.rd_s + 4 * j * (kStrip / BLOCK));
  }
  wait_lgkmcnt0();  // the slot is read: refill it
  const int64_t kn = kk + 2 * kWaves;
  dma_step<CODE, BLOCK>(slot, a, p, kn, kn < k_end);
  mma_step<CODE>(acc, w);
}

template <int CODE, int BLOCK>
__global__ __launch_bounds__(kThreads, 1) void lora_kernel(const LoraArgs a) {
  // Two ring slots per wave while streaming (160 KB); at a segment end the
  // first 128 KB hold the 8 waves' accumulators (16 KB each) for the reduction.
  __shared__ __attribute__((aligned(16))) uint8_t ring0[kWaves][kSlot];
  __shared__ __attribute__((aligned(16))) uint8_t ring1[kWaves][kSlot];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;
  const int q = lane & 15, h = lane >> 4;
  // consecutive ranges on one XCD (workgroups are dealt round-robin to the 8 XCDs)
  const int64_t bid = blockIdx.x;
  const int64_t wg = a.xcd_remap ? (bid & 7) * (a.n_wg >> 3) + (bid >> 3) : bid;
  const int64_t u_end = range_begin(a, wg + 1);
  // 16 KB accumulator area of wave w: ring0 holds 5 of them, ring1 the rest
  auto red_of = [&](int w) -> float * {
    return reinterpret_cast<float *>(w < 5 ? &ring0[0][0] + 16384 * w
                                           : &ring1[0][0] + 16384 * (w - 5));
  };
  constexpr int nb = kStrip / BLOCK;  // scale blocks per strip row

  Plan p;
  p.st_c = (uint32_t)a.M;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int e = 64 * i + lane;  // (row, adapter pair) of the k-step's dh
    p.vo_d[i] = 2 * (e % 8) < a.r_pass
                    ? (uint32_t)(e / 8) * (uint32_t)a.ldh * 2u + (uint32_t)(a.r0 + 2 * (e % 8)) * 2u
                    : kOob;
  }
  p.rd_s = (uint32_t)(8 * h * nb + (16 * q) / BLOCK) * 4u;

  int seg = 0;
  // at most two segments per range (the plan keeps n_wg >= S), so two slots
  for (int64_t u = range_begin(a, wg); u < u_end && seg < 2; ++seg) {
    const int64_t s = u / a.KS;
    const int64_t k_end = (u_end - s * a.KS) < a.KS ? (u_end - s * a.KS) : a.KS;
    const int64_t col = s * kStrip + 16 * q;
    p.vo_c = col < a.M ? (uint32_t)(8 * h) * p.st_c + (uint32_t)col : kOob;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int e = 64 * i + lane;  // (row, block) of the k-step's scales
      const int64_t blk = s * nb + e % nb;
      p.vo_s[i] = e < 32 * nb && blk * BLOCK < a.M
                      ? (uint32_t)(e / nb) * (uint32_t)(a.M / BLOCK) * 4u + (uint32_t)blk * 4u
                      : kOob;
    }

    f32x4 acc[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) acc[c] = f32x4{};
    // this wave's k-steps kk, kk + 8, ...; two of them in flight ahead of the
    // one being computed (slot 0 takes the even ones, slot 1 the odd ones)
    int64_t kk = u - s * a.KS + wave;
    dma_step<CODE, BLOCK>(&ring0[wave][0], a, p, kk, kk < k_end);
    dma_step<CODE, BLOCK>(&ring1[wave][0], a, p, kk + kWaves, kk + kWaves < k_end);
    // pairs of k-steps; an odd count ends with a step whose loads are empty
    // (zeros: its MFMAs add nothing)
    const int64_t n_pairs = kk < k_end ? (k_end - kk + 2 * kWaves - 1) / (2 * kWaves) : 0;
    for (int64_t i = 0; i < n_pairs; ++i) {
      ring_step<CODE, BLOCK>(acc, &ring0[wave][0], a, p, kk, k_end, lane);
      ring_step<CODE, BLOCK>(acc, &ring1[wave][0], a, p, kk + kWaves, k_end, lane);
      kk += 2 * kWaves;
    }
    // drain this wave's DMAs (the last ones read nothing but still write the
    // slots) before the ring holds the accumulators
    wait_vmcnt<0>();
    __syncthreads();

    // acc[c][v] = dA[4h + v][16 q + c] of this wave's k-steps
    float *red = red_of(wave);
#pragma unroll
    for (int v = 0; v < 4; ++v)
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4)
        *reinterpret_cast<f32x4 *>(&red[(4 * h + v) * kStrip + 16 * q + 4 * c4]) =
            f32x4{acc[4 * c4][v], acc[4 * c4 + 1][v], acc[4 * c4 + 2][v], acc[4 * c4 + 3][v]};
    __syncthreads();
    float *out = a.part + (2 * wg + seg) * (int64_t)kPart;
#pragma unroll
    for (int e4 = 0; e4 < kPart / 4 / kThreads; ++e4) {
      const int e = 4 * (tid + e4 * kThreads);
      f32x4 sum = *reinterpret_cast<const f32x4 *>(red_of(0) + e);
#pragma unroll
      for (int w = 1; w < kWaves; ++w) sum += *reinterpret_cast<const f32x4 *>(red_of(w) + e);
      *reinterpret_cast<f32x4 *>(out + e) = sum;
    }
    __syncthreads();
    u = (s + 1) * a.KS;
  }
}

// One thread per 4 output elements (strip s, adapter row rr, columns 4c ..
// 4c+3): the partials of the workgroups whose ranges meet strip s, in
// ascending order.  Workgroup w's range begins at floor(U w / n_wg), so the
// first one meeting strip s is floor(((s KS + 1) n_wg - 1) / U) and the last
// floor(((s + 1) KS n_wg - 1) / U); only the first can have begun in an
// earlier strip, and then holds this strip's sums in its second slot.
constexpr int kReduceBatch = 16;

__global__ __launch_bounds__(256) void lora_reduce_kernel(const LoraArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  constexpr int kQuads = kStrip / 4;
  const int64_t per_strip = (int64_t)a.r_pass * kQuads;
  const int64_t s = idx / per_strip;
  const int rr = (int)(idx % per_strip) / kQuads;
  const int c4 = 4 * (int)(idx % kQuads);
  const int64_t col = s * kStrip + c4;
  if (s >= a.S || col >= a.M) return;
  f32x4 sum = {0.f, 0.f, 0.f, 0.f};
  if (a.U > 0) {
    const int64_t first = s * a.KS;
    const int64_t w0 = ((first + 1) * a.n_wg - 1) / a.U;
    const int64_t w1 = ((first + a.KS) * a.n_wg - 1) / a.U;  // inclusive
    const float *base = a.part + rr * kStrip + c4;
    sum = *reinterpret_cast<const f32x4 *>(
        base + (2 * w0 + (range_begin(a, w0) < first ? 1 : 0)) * (int64_t)kPart);
    // up to 16 partials per round trip (a narrow unit's strip has 16 parts);
    // the additions stay in ascending workgroup order
    for (int64_t w = w0 + 1; w <= w1; w += kReduceBatch) {
      f32x4 x[kReduceBatch];
#pragma unroll
      for (int k = 0; k < kReduceBatch; ++k)
        x[k] = w + k <= w1 ? *reinterpret_cast<const f32x4 *>(base + 2 * (w + k) * (int64_t)kPart)
                           : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < kReduceBatch; ++k) sum += x[k];
    }
  }
  float *out = a.da + (int64_t)(a.r0 + rr) * a.M + col;  // M % 16 == 0: 4 in range
  const f32x4 v = sum * a.scale;
  if (a.accumulate) {
    const f32x4 o = {out[0], out[1], out[2], out[3]};
    const f32x4 t = o + v;
    out[0] = t.x; out[1] = t.y; out[2] = t.z; out[3] = t.w;
  } else {
    out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
  }
}

template <int CODE, int BLOCK>
void launch_main(const LoraArgs &a, hipStream_t s) {
  hipLaunchKernelGGL((lora_kernel<CODE, BLOCK>), dim3((unsigned)a.n_wg), dim3(kThreads), 0, s, a);
}

template <int CODE>
void dispatch(const LoraArgs &a, int block, hipStream_t s) {
  switch (block) {
    case 32: return launch_main<CODE, 32>(a, s);
    case 64: return launch_main<CODE, 64>(a, s);
    case 128: return launch_main<CODE, 128>(a, s);
    default: return launch_main<CODE, 256>(a, s);
  }
}

}  // namespace

LoraPlan lora_plan(int64_t K, int64_t M, int r) {
  LoraPlan p{};
  p.S = (M + kStrip - 1) / kStrip;
  p.KS = (K + kStep - 1) / kStep;
  p.U = p.S * p.KS;
  const int64_t want = p.S > kLoraWorkgroups ? p.S : kLoraWorkgroups;
  p.n_wg = p.U < want ? p.U : want;
  // an XCD's share of the strips is at least 1 KB of every row from 32 strips on
  p.xcd_remap = p.n_wg % 8 == 0 && p.S >= 32 ? 1 : 0;
  // Narrow units (fewer than 32 strips, e.g. a hidden-width input): every strip
  // is split into `parts` equal ranges, one per workgroup, so no range crosses a
  // strip (one partial each) and the waves' k-steps come in whole ring pairs.
  // The pairs per wave are the fewest that S * parts <= 256 workgroups allow,
  // and `parts` the smallest count that reaches them.  On 16384 x 3584 (14
  // strips) this gives 224 workgroups of 32 k-steps.
  if (p.S < 32 && p.KS >= 2 * kWaves) {
    const int64_t per = 2 * kWaves;  // k-steps of one ring pair of every wave
    const int64_t pmax = kLoraWorkgroups / p.S;
    const int64_t pairs = (p.KS + per * pmax - 1) / (per * pmax);
    const int64_t parts = (p.KS + per * pairs - 1) / (per * pairs);
    p.n_wg = p.S * parts;
  }
  p.workspace_bytes = (size_t)(p.n_wg > 0 ? p.n_wg : 1) * 2 * kPart * sizeof(float);
  p.passes = (r + kRows - 1) / kRows;
  return p;
}

hipError_t launch_lora(const LoraArgs &base, int code, int block, int r, hipStream_t s) {
  for (int r0 = 0; r0 < r; r0 += kRows) {
    LoraArgs a = base;
    a.r0 = r0;
    a.r_pass = r - r0 < kRows ? r - r0 : kRows;
    if (a.U > 0) {
      if (code == kCodeCast) launch_main<kCodeCast, 256>(a, s);  // no blocks; BLOCK unused
      else if (code == kCodeInt8) dispatch<kCodeInt8>(a, block, s);
      else dispatch<kCodeE4M3>(a, block, s);
    }
    const int64_t threads = a.S * a.r_pass * (kStrip / 4);
    hipLaunchKernelGGL(lora_reduce_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0,
                       s, a);
  }
  return hipGetLastError();
}

}  // namespace hilore
