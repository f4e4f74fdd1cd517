// Adapter gradient of a LoRA linear layer whose saved input is an L unit, with
// the reconstruction fused into the operand load, on gfx950 MFMA:
//   dA[r][i] (+)= scale * sum_t dh[t][r] * xhat[t][i],
//   xhat[t][i] = bf16_RNE(value(code[t][i]) * scale[t][i / BLOCK])
// (or value(code) exactly for the literal cast).  For the layer output
// y = X W^T + scale * (X A^T) B^T and an upstream gradient G, dh = G B; this
// is the paper's default setting (rank-16 adapters on q/k/v/o and gate/up/down,
// alpha = 32, App. D.1.1), where the adapter gradient is the only backward
// consumer of the saved MLP activation that feeds a frozen projection.  The
// q/k/v (and gate/up) adapters share one input, so their dh can be passed side
// by side (r = 48 or 80) and the codes are then read once for all of them.
//
// The work is a (16 R)-row output contracted over all K tokens: reading the
// codes once (1 + 4/BLOCK bytes per element) bounds it; MFMA serves the 32 R
// FLOP per element that a vector unit could not keep up with.
//
// Units and balance (both kernels).  A strip is 256 columns of X; a k-step is
// 32 token rows of a strip.  The (strip, k-step) units are numbered
// strip-major and dealt to the workgroups in equal contiguous ranges
// (stream-K), so every CU gets the same work whatever the shape; a range meets
// at most two strips (the grid has at least as many workgroups as strips).
// Units of fewer than 32 strips instead split every strip into equal parts,
// one per workgroup (see lora_plan).  With at least 32 strips the workgroup
// index is remapped so that the 32 workgroups on one XCD (dispatch is
// round-robin over the 8 XCDs) take consecutive ranges, i.e. about 1/8 of the
// strips: the scale lines of those strips and the dh rows (read by every
// strip) then stay in that XCD's L2, helped by streaming the codes past it
// (non-temporal loads).  At the end of its part of a strip a workgroup stores
// one partial [16 R][256] to the caller's workspace; a second kernel adds, for
// each output element, the partials of the workgroups that covered its strip
// in ascending order: no floating-point atomics, and the result does not
// depend on the timing.
//
// Passes of up to 16 adapter rows: lora_wave_kernel.  The 8 waves of a
// workgroup take every 8th k-step of its range, each on its own: lane
// (q, h) = (lane % 16, lane / 16) loads rows 8h .. 8h+7 of columns 16q .. 16q+15
// (one 16-byte load per row: every row of the strip is read as 256 contiguous
// bytes) straight into registers, two k-steps in flight, dequantises them and
// hands column 16q + c to MFMA c (c = 0..15, v_mfma_f32_16x16x32_bf16): its B
// operand is then 8 consecutive tokens of one column per lane, as the
// instruction wants, with no transpose.  The A operand is dh^T: the k-step's
// [32][16] dh block (one 16-byte load per lane) passes through the wave's own
// 2 KB of LDS and comes back transposed by ds_read_b64_tr_b16, and the
// k-step's (row, block) scale list (one word per lane) through the same area.
// MFMA c accumulates dA[4h + v][16q' + c] in lane (q', h), register v; at a
// segment end the 8 waves' accumulators are summed through LDS in wave order.
//
// Passes of 17 .. 80 adapter rows (R = 2 .. 5 blocks of 16): lora_coop_kernel.
// Per-wave accumulators for 16 R rows x 256 columns would not fit the register
// file, so the workgroup walks its k-steps in order, two per barrier: every
// thread loads 16 code bytes of each (D k-steps in flight in registers) and
// dequantises them once into a double-buffered [64][256] bf16 tile in LDS,
// the dh block goes to LDS next to it, and wave w runs the MFMAs of column
// groups 2w and 2w+1 (16 columns each, B operand by transposing reads of the
// tile) for all R row blocks.  Each wave owns its columns, so a segment ends
// with plain stores of the partial and no cross-wave reduction.
#include "device_common.hpp"
#include "hilore_internal.hpp"

// Every rounding step is the one written: no implicit fused multiply-add.
#pragma clang fp contract(off)

namespace hilore {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * kWave;
constexpr int kStrip = 256;  // columns per strip
constexpr int kStep = 32;    // token rows per k-step
constexpr int kRows = 16;    // adapter rows per row block (the MFMA's M)
constexpr int kMaxR = 5;     // row blocks of one cooperative pass (80 adapter rows)
constexpr int kCoopDepth = 8;  // k-steps in flight per workgroup, cooperative kernel
constexpr uint32_t kOob = 0x80000000u;  // a buffer offset past every range: loads 0
constexpr int kNonTemporal = 2;         // cache policy of the streamed codes: NT

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Adapter rows of a pass, rounded up to whole row blocks.
__host__ __device__ constexpr int pass_blocks(int r_pass) { return (r_pass + kRows - 1) / kRows; }

// Rows of k-step kk that exist (0 past K or when the step is not this one's).
__device__ __forceinline__ int64_t step_rows(const LoraArgs &a, int64_t kk, bool live) {
  const int64_t left = a.K - kk * kStep;
  return !live || left <= 0 ? 0 : (left < kStep ? left : kStep);
}

// First unit of the range of (remapped) workgroup w.
__device__ __forceinline__ int64_t range_begin(const LoraArgs &a, int64_t w) {
  return a.U * w / a.n_wg;
}

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

// dh of one k-step: 32 rows x 16 R adapter rows, read as 16-byte chunks when
// the rank is a multiple of 8 (a chunk is then wholly inside or wholly past the
// pass), else as 4-byte pairs (the rank is even), so that no load straddles
// the end of its range.  Piece t of the block (chunks: 2 R per row, pairs:
// 8 R per row) starts at adapter row `col` of token row `row`; consecutive
// pieces are consecutive in memory and land in the row-major [32][16 R] block
// in LDS at 16 t (chunks) or 4 t (pairs).  Adapter rows past r_pass read 0 or
// the next row's values: their dA rows are never stored.
__device__ __forceinline__ uint32_t dh_offset(const LoraArgs &a, int t, int per_row, int width) {
  const int row = t / per_row, col = width * (t % per_row);
  return col < a.r_pass ? (uint32_t)row * (uint32_t)a.ldh * 2u + (uint32_t)(a.r0 + col) * 2u
                        : kOob;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t dh_rsrc(const LoraArgs &a, int64_t t0,
                                                          int64_t rows) {
  return __builtin_amdgcn_make_buffer_rsrc((void *)(a.dh + t0 * a.ldh), 0,
                                           (int)(rows * a.ldh * 2), 0x00020000);
}

// --------------------------------------------------------- per-wave kernel --

// Scale words each lane loads per k-step (32 rows x 256 / BLOCK blocks).
template <int BLOCK>
constexpr int kScaleWords = (32 * (kStrip / BLOCK) + 63) / 64;

// Operands of one k-step as loaded by one lane: the codes of rows 8h + j,
// columns 16q .. 16q+15; its share of the dh block (chunk `lane`, or pairs
// lane + 64 i); kScaleWords scales of the k-step's (row, block) list.
template <int BLOCK>
struct Raw {
  u32x4 c[8];
  u32x4 d;
  float s[kScaleWords<BLOCK>];
};

// Per-lane, loop-invariant parts of the loads.
template <int BLOCK>
struct Plan {
  uint32_t vo_c;  // byte offset of row 8h of a k-step (kOob: no data)
  uint32_t st_c;  // byte stride of one token row
  uint32_t vo_d[4];
  uint32_t vo_s[kScaleWords<BLOCK>];
};

template <int CODE, int BLOCK, bool WIDE>
__device__ __forceinline__ void load_step(Raw<BLOCK> &w, const LoraArgs &a, const Plan<BLOCK> &p,
                                          int64_t kk, bool live) {
  const int64_t rows = step_rows(a, kk, live);
  const int64_t t0 = kk * kStep;
  const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(a.codes + t0 * a.M), 0, (int)(rows * a.M), 0x00020000);
#pragma unroll
  for (int j = 0; j < 8; ++j)
    w.c[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                           rc, (int)(p.vo_c + j * p.st_c), 0, kNonTemporal));
  const __amdgpu_buffer_rsrc_t rd = dh_rsrc(a, t0, rows);
  if constexpr (WIDE) {
    w.d = __builtin_bit_cast(u32x4,
                             __builtin_amdgcn_raw_buffer_load_b128(rd, (int)p.vo_d[0], 0, 0));
  } else {
    w.d.x = __builtin_amdgcn_raw_buffer_load_b32(rd, (int)p.vo_d[0], 0, 0);
    w.d.y = __builtin_amdgcn_raw_buffer_load_b32(rd, (int)p.vo_d[1], 0, 0);
    w.d.z = __builtin_amdgcn_raw_buffer_load_b32(rd, (int)p.vo_d[2], 0, 0);
    w.d.w = __builtin_amdgcn_raw_buffer_load_b32(rd, (int)p.vo_d[3], 0, 0);
  }
  if constexpr (CODE != kCodeCast) {
    const int64_t sld = a.M / BLOCK;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.scales + t0 * sld), 0, (int)(rows * sld * 4), 0x00020000);
#pragma unroll
    for (int i = 0; i < kScaleWords<BLOCK>; ++i)
      w.s[i] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, (int)p.vo_s[i], 0, 0));
  }
}

// Columns 4 D + C and 4 D + C + 1 of the lane's 16 (dword D, byte pair C of
// every row): two B operands of 8 tokens each, xhat rounded to bf16 exactly
// as the decoder rounds it, then the two MFMAs.
template <int CODE, int D, int C>
__device__ __forceinline__ void mma_pair(f32x4 (&acc)[16], const u32x4 (&cw)[8],
                                         const float (&sc)[8], const bf16x8 &A) {
  float lo[8], hi[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t word = D == 0 ? cw[j].x : D == 1 ? cw[j].y : D == 2 ? cw[j].z : cw[j].w;
    const f32x2 v = decode_pair<CODE, C>(word);
    if constexpr (CODE == kCodeCast) {
      lo[j] = v.x;
      hi[j] = v.y;
    } else {
      lo[j] = v.x * sc[j];
      hi[j] = v.y * sc[j];
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

// A k-step's MFMAs.  The lane's dh share and scale words go through the
// wave's own 2 KB of LDS: dh as the k-step's [32][16] bf16 block, read back
// transposed (ds_read_b64_tr_b16: in each 16-lane group, lane 4a + c gets
// element c of the pieces addressed by lanes a, a+4, a+8, a+12, so pointing
// those at rows 8h + 4i .. +3, adapter rows 4a .. 4a+3 hands lane (q, h)
// dh[8h .. 8h+7][q], the A operand dh^T); scales as the (row, block) list,
// from which lane (q, h) reads row 8h + j's block.
template <int CODE, int BLOCK, bool WIDE>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[16], const Raw<BLOCK> &w, uint8_t *area,
                                         int lane) {
  constexpr int nb = kStrip / BLOCK;
  const int q = lane & 15, h = lane >> 4;
  if constexpr (WIDE) {
    *reinterpret_cast<u32x4 *>(area + 16 * lane) = w.d;
  } else {
    *reinterpret_cast<uint32_t *>(area + 4 * lane) = w.d.x;
    *reinterpret_cast<uint32_t *>(area + 4 * (lane + 64)) = w.d.y;
    *reinterpret_cast<uint32_t *>(area + 4 * (lane + 128)) = w.d.z;
    *reinterpret_cast<uint32_t *>(area + 4 * (lane + 192)) = w.d.w;
  }
  if constexpr (CODE != kCodeCast) {
#pragma unroll
    for (int i = 0; i < kScaleWords<BLOCK>; ++i)
      if (64 * i + lane < 32 * nb)
        *reinterpret_cast<float *>(area + 1024 + 4 * (64 * i + lane)) = w.s[i];
  }
  const uint32_t tr = (uint32_t)(8 * h + ((lane & 15) >> 2)) * 32u + (uint32_t)(lane & 3) * 8u;
  const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(area + tr));
  const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(area + tr + 4 * 32));
  const bf16x8 A =
      __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  float sc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j)
    sc[j] = CODE == kCodeCast ? 1.f
                              : *reinterpret_cast<const float *>(
                                    area + 1024 + 4 * ((8 * h + j) * nb + (16 * q) / BLOCK));
  // one column pair at a time: its decode stays next to its two MFMAs
  // instead of all 128 values being formed ahead of them
  mma_pair<CODE, 0, 0>(acc, w.c, sc, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 0, 2>(acc, w.c, sc, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 1, 0>(acc, w.c, sc, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 1, 2>(acc, w.c, sc, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 2, 0>(acc, w.c, sc, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 2, 2>(acc, w.c, sc, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 3, 0>(acc, w.c, sc, A);
  __builtin_amdgcn_sched_barrier(0);
  mma_pair<CODE, 3, 2>(acc, w.c, sc, A);
}

constexpr int kPart = kRows * kStrip;  // floats of a one-block partial

// WIDE: the rank is a multiple of 8 and dh is read in 16-byte chunks (a
// compile-time choice: a run-time branch between the two load forms inside
// the unrolled loop costs the compiler its load scheduling).
template <int CODE, int BLOCK, bool WIDE>
__global__ __launch_bounds__(kThreads, 1) void lora_wave_kernel(const LoraArgs a) {
  // the 8 waves' accumulators at a segment end (16 KB each); while streaming,
  // 2 KB of each wave's area stage its dh block and scales
  __shared__ __attribute__((aligned(16))) float red[kWaves][kPart];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;
  const int q = lane & 15, h = lane >> 4;
  uint8_t *area = reinterpret_cast<uint8_t *>(&red[wave][0]);
  const int64_t bid = blockIdx.x;
  const int64_t wg = a.xcd_remap ? (bid & 7) * (a.n_wg >> 3) + (bid >> 3) : bid;
  const int64_t u_end = range_begin(a, wg + 1);
  constexpr int nb = kStrip / BLOCK;  // scale blocks per strip row

  Plan<BLOCK> p;
  p.st_c = (uint32_t)a.M;
  if constexpr (WIDE) {
    p.vo_d[0] = dh_offset(a, lane, 2, 8);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) p.vo_d[i] = dh_offset(a, lane + 64 * i, 8, 2);
  }

  int seg = 0;
  // at most two segments per range (the plan keeps n_wg >= S)
  for (int64_t u = range_begin(a, wg); u < u_end && seg < 2; ++seg) {
    const int64_t s = u / a.KS;
    const int64_t k_end = (u_end - s * a.KS) < a.KS ? (u_end - s * a.KS) : a.KS;
    const int64_t col = s * kStrip + 16 * q;
    p.vo_c = col < a.M ? (uint32_t)(8 * h) * p.st_c + (uint32_t)col : kOob;
#pragma unroll
    for (int i = 0; i < kScaleWords<BLOCK>; ++i) {
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
    // one being computed (an odd count ends with a step whose loads are
    // empty: zeros, its MFMAs add nothing)
    int64_t kk = u - s * a.KS + wave;
    Raw<BLOCK> w0, w1;
    load_step<CODE, BLOCK, WIDE>(w0, a, p, kk, kk < k_end);
    load_step<CODE, BLOCK, WIDE>(w1, a, p, kk + kWaves, kk + kWaves < k_end);
    const int64_t n_pairs = kk < k_end ? (k_end - kk + 2 * kWaves - 1) / (2 * kWaves) : 0;
    for (int64_t i = 0; i < n_pairs; ++i) {
      mma_step<CODE, BLOCK, WIDE>(acc, w0, area, lane);
      load_step<CODE, BLOCK, WIDE>(w0, a, p, kk + 2 * kWaves, kk + 2 * kWaves < k_end);
      mma_step<CODE, BLOCK, WIDE>(acc, w1, area, lane);
      load_step<CODE, BLOCK, WIDE>(w1, a, p, kk + 3 * kWaves, kk + 3 * kWaves < k_end);
      kk += 2 * kWaves;
    }

    // acc[c][v] = dA[4h + v][16 q + c] of this wave's k-steps
    float *mine = red[wave];
    __builtin_amdgcn_s_waitcnt(0xC07F);  // this wave's staging reads are done
#pragma unroll
    for (int v = 0; v < 4; ++v)
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4)
        *reinterpret_cast<f32x4 *>(&mine[(4 * h + v) * kStrip + 16 * q + 4 * c4]) =
            f32x4{acc[4 * c4][v], acc[4 * c4 + 1][v], acc[4 * c4 + 2][v], acc[4 * c4 + 3][v]};
    __syncthreads();
    float *out = a.part + (2 * wg + seg) * (int64_t)kPart;
#pragma unroll
    for (int e4 = 0; e4 < kPart / 4 / kThreads; ++e4) {
      const int e = 4 * (tid + e4 * kThreads);
      f32x4 sum = *reinterpret_cast<const f32x4 *>(&red[0][e]);
#pragma unroll
      for (int w = 1; w < kWaves; ++w) sum += *reinterpret_cast<const f32x4 *>(&red[w][e]);
      *reinterpret_cast<f32x4 *>(out + e) = sum;
    }
    __syncthreads();
    u = (s + 1) * a.KS;
  }
}

// ------------------------------------------------------ cooperative kernel --

// One thread's operands of a k-step: codes of row tid / 16, columns
// 16 (tid % 16) .. +15; that row's block scale; its share of the dh block
// (chunk tid when wide, pairs tid + 512 i otherwise).
struct CoopLd {
  u32x4 c;
  float s;
  u32x4 d;
};

template <int CODE, int BLOCK, bool WIDE>
__device__ __forceinline__ void coop_load(CoopLd &l, const LoraArgs &a, uint32_t vo_c,
                                          uint32_t vo_s, const uint32_t (&vo_d)[3], int64_t kk,
                                          bool live) {
  const int64_t rows = step_rows(a, kk, live);
  const int64_t t0 = kk * kStep;
  const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(a.codes + t0 * a.M), 0, (int)(rows * a.M), 0x00020000);
  l.c = __builtin_bit_cast(u32x4,
                           __builtin_amdgcn_raw_buffer_load_b128(rc, (int)vo_c, 0, kNonTemporal));
  if constexpr (CODE != kCodeCast) {
    const int64_t sld = a.M / BLOCK;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(a.scales + t0 * sld), 0, (int)(rows * sld * 4), 0x00020000);
    l.s = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, (int)vo_s, 0, 0));
  }
  // Every thread issues the same loads (threads past the dh block have the
  // out-of-range offset and read 0): a load behind a per-thread condition
  // becomes a branch, and the compiler then drains every load in flight at
  // the loop head instead of keeping D k-steps outstanding.
  const __amdgpu_buffer_rsrc_t rd = dh_rsrc(a, t0, rows);
  if constexpr (WIDE) {
    l.d = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rd, (int)vo_d[0], 0, 0));
  } else {
    l.d.x = __builtin_amdgcn_raw_buffer_load_b32(rd, (int)vo_d[0], 0, 0);
    l.d.y = __builtin_amdgcn_raw_buffer_load_b32(rd, (int)vo_d[1], 0, 0);
    l.d.z = __builtin_amdgcn_raw_buffer_load_b32(rd, (int)vo_d[2], 0, 0);
  }
}

template <int CODE>
__device__ __forceinline__ uint32_t xhat_pair(uint32_t w, float s, int half) {
  const f32x2 v = half ? decode_pair<CODE, 2>(w) : decode_pair<CODE, 0>(w);
  if constexpr (CODE == kCodeCast) return pack_bf16(v.x, v.y);
  return pack_bf16(v.x * s, v.y * s);
}

// 16-byte chunk swizzle of the xhat tile (rows of 512 bytes): the rows t .. t+3
// and t + 8 .. t + 11 of one transposing read land in distinct banks.
__device__ __forceinline__ uint32_t x_swz(uint32_t t) {
  return ((t & 3u) << 1) | (((t >> 3) & 1u) << 3);
}

template <int CODE, int BLOCK, int R, bool WIDE>
__global__ __launch_bounds__(kThreads, 1) void lora_coop_kernel(const LoraArgs a) {
  // two k-steps per barrier, double-buffered: xhat [64][256] bf16 (chunks
  // swizzled) and dh [64][16 R] bf16, row-major blocks of 16 adapter rows
  // side by side
  __shared__ __attribute__((aligned(16))) uint8_t xl[2][2 * kStep * kStrip * 2];
  __shared__ __attribute__((aligned(16))) uint8_t dl[2][2 * kStep * 32 * R];
  constexpr int D = kCoopDepth;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;
  const int q = lane & 15, h = lane >> 4;
  const int64_t bid = blockIdx.x;
  const int64_t wg = a.xcd_remap ? (bid & 7) * (a.n_wg >> 3) + (bid >> 3) : bid;
  const int64_t u_end = range_begin(a, wg + 1);
  constexpr int64_t kSlot = (int64_t)kRows * R * kStrip;
  constexpr int kDhRow = 32 * R;  // bytes of one dh row in LDS

  const int xrow = tid >> 4, xch = tid & 15;  // this thread's row and 16-column chunk
  // this thread's dh pieces: chunk tid (wide) or pairs tid + 512 i
  uint32_t vo_d[3];
  if constexpr (WIDE) {
    vo_d[0] = tid < 64 * R ? dh_offset(a, tid, 2 * R, 8) : kOob;
    vo_d[1] = vo_d[2] = kOob;
  } else {
#pragma unroll
    for (int i = 0; i < 3; ++i)
      vo_d[i] = tid + 512 * i < 256 * R ? dh_offset(a, tid + 512 * i, 8 * R, 2) : kOob;
  }
  // transposing-read addresses (lane 4 e + a of 16-lane group h: row 8 h + e
  // and 8 h + e + 4, columns 4 a .. 4 a + 3 of a 16-column group)
  const uint32_t e4 = (uint32_t)(lane & 15) >> 2, a4 = (uint32_t)lane & 3u;
  const uint32_t trow = 8u * (uint32_t)h + e4;
  uint32_t xo[2][2];  // [column group][read]
#pragma unroll
  for (int gi = 0; gi < 2; ++gi)
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) {
      const uint32_t t = trow + 4u * rd;
      const uint32_t g = 2u * (uint32_t)wave + gi;
      const uint32_t chunk = (2u * g + (a4 >> 1)) ^ x_swz(t);
      xo[gi][rd] = t * 512u + chunk * 16u + 8u * (a4 & 1u);
    }
  const uint32_t dof = trow * kDhRow + a4 * 8u;
  const uint32_t sw = x_swz((uint32_t)xrow);

  int seg = 0;
  for (int64_t u = range_begin(a, wg); u < u_end && seg < 2; ++seg) {
    const int64_t s = u / a.KS;
    const int64_t k0 = u - s * a.KS;
    const int64_t k_end = (u_end - s * a.KS) < a.KS ? (u_end - s * a.KS) : a.KS;
    const int64_t col = s * kStrip + 16 * xch;
    const uint32_t vo_c = col < a.M ? (uint32_t)xrow * (uint32_t)a.M + (uint32_t)col : kOob;
    const uint32_t vo_s =
        col < a.M ? (uint32_t)xrow * (uint32_t)(a.M / BLOCK) * 4u + (uint32_t)(col / BLOCK) * 4u
                  : kOob;

    f32x4 acc[R][2];
#pragma unroll
    for (int b = 0; b < R; ++b) acc[b][0] = acc[b][1] = f32x4{};
    CoopLd L[D];
#pragma unroll
    for (int i = 0; i < D; ++i)
      coop_load<CODE, BLOCK, WIDE>(L[i], a, vo_c, vo_s, vo_d, k0 + i, k0 + i < k_end);

    for (int64_t kb = k0; kb < k_end; kb += D) {
#pragma unroll
      for (int i = 0; i < D; i += 2) {
        const int64_t k = kb + i;
        if (k >= k_end) break;
        const int b = (i / 2) & 1;
        // xhat of this thread's 16 values of k-steps k and k + 1 (past the
        // range: zeros), rounded as the decoder rounds them
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const CoopLd &l = L[i + j];
          u32x4 w0, w1;
          w0.x = xhat_pair<CODE>(l.c.x, l.s, 0);
          w0.y = xhat_pair<CODE>(l.c.x, l.s, 1);
          w0.z = xhat_pair<CODE>(l.c.y, l.s, 0);
          w0.w = xhat_pair<CODE>(l.c.y, l.s, 1);
          w1.x = xhat_pair<CODE>(l.c.z, l.s, 0);
          w1.y = xhat_pair<CODE>(l.c.z, l.s, 1);
          w1.z = xhat_pair<CODE>(l.c.w, l.s, 0);
          w1.w = xhat_pair<CODE>(l.c.w, l.s, 1);
          uint8_t *xb = &xl[b][j * kStep * 512 + xrow * 512];
          *reinterpret_cast<u32x4 *>(xb + ((2u * xch) ^ sw) * 16u) = w0;
          *reinterpret_cast<u32x4 *>(xb + ((2u * xch + 1u) ^ sw) * 16u) = w1;
          uint8_t *db = &dl[b][j * kStep * kDhRow];
          if constexpr (WIDE) {
            if (tid < 64 * R) *reinterpret_cast<u32x4 *>(db + 16 * tid) = l.d;
          } else {
            if (tid < 256 * R) *reinterpret_cast<uint32_t *>(db + 4 * tid) = l.d.x;
            if (tid + 512 < 256 * R) *reinterpret_cast<uint32_t *>(db + 4 * (tid + 512)) = l.d.y;
            if (tid + 1024 < 256 * R) *reinterpret_cast<uint32_t *>(db + 4 * (tid + 1024)) = l.d.z;
          }
        }
        coop_load<CODE, BLOCK, WIDE>(L[i], a, vo_c, vo_s, vo_d, k + D, k + D < k_end);
        coop_load<CODE, BLOCK, WIDE>(L[i + 1], a, vo_c, vo_s, vo_d, k + 1 + D, k + 1 + D < k_end);
        // both tiles written; the reads of this buffer two rounds ago are done
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const uint8_t *xb = &xl[b][j * kStep * 512];
          bf16x8 B[2];
#pragma unroll
          for (int gi = 0; gi < 2; ++gi) {
            const s16x4 lo =
                __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(xb + xo[gi][0]));
            const s16x4 hi =
                __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(xb + xo[gi][1]));
            B[gi] = __builtin_bit_cast(bf16x8,
                                       __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
          }
          const uint8_t *db = &dl[b][j * kStep * kDhRow];
#pragma unroll
          for (int rb = 0; rb < R; ++rb) {
            const s16x4 lo =
                __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(db + dof + 32u * rb));
            const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_s16x4 *)(db + dof + 32u * rb + 4u * kDhRow));
            const bf16x8 A =
                __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
            acc[rb][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B[0], acc[rb][0], 0, 0, 0);
            acc[rb][1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B[1], acc[rb][1], 0, 0, 0);
          }
        }
      }
    }
    // every wave is past its last reads of both buffers before the next
    // segment writes them
    __syncthreads();
    // acc[rb][gi][v] = dA[16 rb + 4 h + v][16 (2 wave + gi) + q]
    float *out = a.part + (2 * wg + seg) * kSlot;
#pragma unroll
    for (int rb = 0; rb < R; ++rb)
#pragma unroll
      for (int gi = 0; gi < 2; ++gi)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          out[(kRows * rb + 4 * h + v) * kStrip + 16 * (2 * wave + gi) + q] = acc[rb][gi][v];
    u = (s + 1) * a.KS;
  }
}

// ---------------------------------------------------------------- reduction --

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
  const int64_t slot = (int64_t)kRows * pass_blocks(a.r_pass) * kStrip;
  f32x4 sum = {0.f, 0.f, 0.f, 0.f};
  if (a.U > 0) {
    const int64_t first = s * a.KS;
    const int64_t w0 = ((first + 1) * a.n_wg - 1) / a.U;
    const int64_t w1 = ((first + a.KS) * a.n_wg - 1) / a.U;  // inclusive
    const float *base = a.part + rr * kStrip + c4;
    sum = *reinterpret_cast<const f32x4 *>(
        base + (2 * w0 + (range_begin(a, w0) < first ? 1 : 0)) * slot);
    // up to 16 partials per round trip (a narrow unit's strip has up to 18
    // parts); the additions stay in ascending workgroup order
    for (int64_t w = w0 + 1; w <= w1; w += kReduceBatch) {
      f32x4 x[kReduceBatch];
#pragma unroll
      for (int k = 0; k < kReduceBatch; ++k)
        x[k] = w + k <= w1 ? *reinterpret_cast<const f32x4 *>(base + 2 * (w + k) * slot)
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

template <int CODE, int BLOCK, bool WIDE>
void launch_main(const LoraArgs &a, hipStream_t s) {
  const dim3 grid((unsigned)a.n_wg), block(kThreads);
  switch (pass_blocks(a.r_pass)) {
    case 1:
      hipLaunchKernelGGL((lora_wave_kernel<CODE, BLOCK, WIDE>), grid, block, 0, s, a);
      return;
    case 2:
      hipLaunchKernelGGL((lora_coop_kernel<CODE, BLOCK, 2, WIDE>), grid, block, 0, s, a);
      return;
    case 3:
      hipLaunchKernelGGL((lora_coop_kernel<CODE, BLOCK, 3, WIDE>), grid, block, 0, s, a);
      return;
    case 4:
      hipLaunchKernelGGL((lora_coop_kernel<CODE, BLOCK, 4, WIDE>), grid, block, 0, s, a);
      return;
    default:
      hipLaunchKernelGGL((lora_coop_kernel<CODE, BLOCK, 5, WIDE>), grid, block, 0, s, a);
      return;
  }
}

template <int CODE, int BLOCK>
void launch_main(const LoraArgs &a, hipStream_t s) {
  if (a.ldh % 8 == 0) launch_main<CODE, BLOCK, true>(a, s);
  else launch_main<CODE, BLOCK, false>(a, s);
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
  // passes of up to 80 adapter rows; the widest sets the partial slot size
  const int widest = pass_blocks(r < kRows * kMaxR ? r : kRows * kMaxR);
  p.workspace_bytes =
      (size_t)(p.n_wg > 0 ? p.n_wg : 1) * 2 * (size_t)(kRows * widest * kStrip) * sizeof(float);
  p.passes = (r + kRows * kMaxR - 1) / (kRows * kMaxR);
  return p;
}

hipError_t launch_lora(const LoraArgs &base, int code, int block, int r, hipStream_t s) {
  for (int r0 = 0; r0 < r; r0 += kRows * kMaxR) {
    LoraArgs a = base;
    a.r0 = r0;
    a.r_pass = r - r0 < kRows * kMaxR ? r - r0 : kRows * kMaxR;
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
