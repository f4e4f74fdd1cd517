// Weight gradient on a reconstructed L unit, dequantisation fused into the
// tile load, on gfx950 MFMA:
//   dW[i][j] (+)= sum_t xhat[t][i] * dY[t][j],
//   xhat[t][i] = bf16_RNE(value(code[t][i]) * scale[t][i / BLOCK]),
// or, for the literal cast code (no scales), xhat[t][i] = value(code[t][i])
// exactly.
// This is the full-parameter weight gradient of a linear layer whose saved
// input is kept in low precision (App. B.1; the full-parameter experiments of
// App. D); gradients accumulate over microbatches (App. D.1.1).
//
// Tiling.  A 256x256 tile of dW per workgroup of 8 waves (2 x 4), each wave a
// 128x64 sub-tile = 4x2 blocks of v_mfma_f32_32x32x16_bf16, i.e. two waves
// per SIMD: while one waits on LDS or memory or runs its dequantisation, the
// other keeps the matrix core busy.  The contraction runs over tokens t in
// stages of 64.  Both operands arrive token-major (t is the slow index of X
// and dY) while MFMA wants 8 consecutive t per lane:
//   - X: every thread loads an 8(t) x 4(column) patch of codes with row loads
//     (a wave covers one full 256-column row of the tile per load),
//     dequantises it and writes 16-byte, t-contiguous bf16 granules to LDS;
//     v_cvt_pk_bf16_f32 packs any two fp32 values, so pairing (t, t+1) in the
//     pack is free.  [256 rows][64 t] bf16, granule index XOR-swizzled by
//     (row ^ row/8): conflict-free both for these writes (8 lanes write rows
//     4 apart) and for the fragment reads (consecutive rows).
//   - dY: copied unchanged from memory to LDS by the buffer unit (16-byte
//     LDS-DMA loads, no registers, no LDS store instructions) as [64 t][256
//     columns] bf16 rows, 16-byte chunk index XOR-swizzled by t.  The B
//     fragments are read back with the transposing ds_read_b64_tr_b16: in
//     each group of 16 lanes, lane 4a + c receives element c of the 8-byte
//     pieces addressed by lanes a, a + 4, a + 8, a + 12, so pointing those
//     lanes at rows t..t+3 of a 4-column slice hands every lane one column
//     with 4 consecutive t; two such reads make a fragment.
// Per stage LDS holds 32 KB of each operand; two stages in flight (128 KB of
// the 160 KB).
//
// Pipeline per stage s (four k-step regions of 8 MFMAs per wave): regions 1
// and 2 dequantise stage s+1's X (already in registers) into the other
// buffer, and region 2 then issues the global loads of stage s+2's X into
// the same registers.  Each thread waits for its own DMA of stage s+1's dY
// and one barrier publishes stage s+1 before the last region, so that
// region 3 finds its fragments in registers: while its MFMAs issue it
// starts the DMA of stage s+2's dY into the buffer just finished and reads
// stage s+1's first fragments, and no wave waits on LDS after the barrier.
// Within a stage every region reads the next k-step's fragments while its
// MFMAs issue; B fragments alternate between two register sets, so the next
// k-step's B is requested right after the first MFMA.
// Work distribution: workgroups are dealt round-robin to the 8 XCDs; the
// launch index is remapped so that each XCD receives a contiguous run of
// tiles, and runs are laid out 8 tile-rows tall, so the 32 CUs of an XCD share
// X and dY panels in their own L2.
#include "device_common.hpp"
#include "hilore_internal.hpp"

// Every rounding step is the one written: no implicit fused multiply-add
// (the exact sequences above depend on it; wanted FMAs are explicit fmaf).
#pragma clang fp contract(off)

namespace hilore {
namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kThreads = 512;
constexpr int kTileBytes = BM * BK * 2;  // one operand stage in LDS (32 KB)
constexpr int kGroupM = 8;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Byte offset of 16-byte granule g (t = 8g..8g+7) of row r in a [256][64] tile.
__device__ __forceinline__ uint32_t lds_off(int r, int g) {
  return (uint32_t)r * 128u + ((uint32_t)((g ^ r ^ (r >> 3)) & 7) << 4);
}

constexpr uint32_t kOob = 0x80000000u;  // a buffer offset past every range: loads 0

// Raw X operand of one stage for one thread: token rows kg..kg+7 (kg = 8 g)
// of columns 4 c .. 4 c + 3 of the tile.
struct Stage {
  uint32_t xc[8];  // codes, 4 bytes per row
  float xs[8];     // the scale of each row's block
};

// dY in LDS: row t of a stage at t * 512 bytes; 16-byte chunk c (columns
// 8c .. 8c+7) stored at chunk position c ^ y_swz(t).  Rows t..t+3 of one
// transposing read then fall in distinct banks, as do the two 16-lane
// groups of a half-wave and the two half-waves.
__device__ __forceinline__ uint32_t y_swz(uint32_t t) {
  return ((t & 3u) << 2) | (((t >> 3) & 1u) << 4);
}

// Per-thread, loop-invariant parts of the stage loads.  Rows past K and
// columns past M (N) fall outside the buffer range of the stage and read as
// 0, so ragged edges need no branches.
struct LoadPlan {
  uint32_t vo_x, vo_s;  // byte offsets of row kg inside a stage
  uint32_t st_x, st_s;  // byte stride of one token row
  uint32_t vo_y[4];     // dY chunk fetched by this lane in each of its 4 DMA loads
};

// Buffer descriptors of one stage of 64 token rows starting at k0.  Past
// the end of K the range is empty and every load returns 0.
struct XRsrc {
  __amdgpu_buffer_rsrc_t x, s;
};

__device__ __forceinline__ int64_t stage_rows(const WgradArgs &a, int64_t k0) {
  const int64_t left = a.K - k0;
  return left <= 0 ? 0 : (left < BK ? left : BK);
}

template <int BLOCK>
__device__ __forceinline__ XRsrc x_rsrc(const WgradArgs &a, int64_t k0) {
  const int64_t rows = stage_rows(a, k0);
  const int64_t sld = a.M / BLOCK;
  XRsrc r;
  r.x = __builtin_amdgcn_make_buffer_rsrc((void *)(a.codes + k0 * a.M), 0, (int)(rows * a.M),
                                          0x00020000);
  r.s = __builtin_amdgcn_make_buffer_rsrc((void *)(a.scales + k0 * sld), 0,
                                          (int)(rows * sld * 4), 0x00020000);
  return r;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t y_rsrc(const WgradArgs &a, int64_t k0) {
  const int64_t rows = stage_rows(a, k0);
  return __builtin_amdgcn_make_buffer_rsrc((void *)(a.dy + k0 * a.N), 0, (int)(rows * a.N * 2),
                                           0x00020000);
}

template <int CODE>
__device__ __forceinline__ void load_stage(Stage &st, const XRsrc &rs, const LoadPlan &lp) {
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    st.xc[r] = __builtin_amdgcn_raw_buffer_load_b32(rs.x, (int)(lp.vo_x + r * lp.st_x), 0, 0);
    if constexpr (CODE != kCodeCast)
      st.xs[r] = __uint_as_float(
          __builtin_amdgcn_raw_buffer_load_b32(rs.s, (int)(lp.vo_s + r * lp.st_s), 0, 0));
  }
}
// VMEM instructions issued by load_stage (the literal cast has no scales)
template <int CODE>
constexpr int kXLoads = CODE == kCodeCast ? 8 : 16;

typedef __attribute__((address_space(3))) void lds_void;

// Stage dY rows 8 w .. 8 w + 7 into b_lds by LDS-DMA: load r of wave w
// writes rows 8 w + 2 r and 8 w + 2 r + 1, lane l to byte 16 l of them.
__device__ __forceinline__ void dma_dy(__amdgpu_buffer_rsrc_t rs, const LoadPlan &lp,
                                       uint8_t *b_lds, int wave) {
#pragma unroll
  for (int r = 0; r < 4; ++r)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)(b_lds + (wave * 8 + 2 * r) * 512),
                                             16, (int)lp.vo_y[r], 0, 0, 0);
}
constexpr int kYLoads = 4;

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

// X columns C, C+1 of the thread's patch: dequantise the 8 token rows and
// write one t-contiguous granule per column (rows (t, t+1) paired per word).
template <int CODE, int C>
__device__ __forceinline__ void fill_x(const Stage &st, uint8_t *a_lds, int lc, int g) {
  float lo[8], hi[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const f32x2 q = decode_pair<CODE, C>(st.xc[r]);
    if constexpr (CODE == kCodeCast) {  // exact bf16 values, no scale
      lo[r] = q.x;
      hi[r] = q.y;
    } else {
      lo[r] = q.x * st.xs[r];
      hi[r] = q.y * st.xs[r];
    }
  }
  u32x4 p;
  p.x = pack_bf16(lo[0], lo[1]);
  p.y = pack_bf16(lo[2], lo[3]);
  p.z = pack_bf16(lo[4], lo[5]);
  p.w = pack_bf16(lo[6], lo[7]);
  *reinterpret_cast<u32x4 *>(a_lds + lds_off(lc * 4 + C, g)) = p;
  p.x = pack_bf16(hi[0], hi[1]);
  p.y = pack_bf16(hi[2], hi[3]);
  p.z = pack_bf16(hi[4], hi[5]);
  p.w = pack_bf16(hi[6], hi[7]);
  *reinterpret_cast<u32x4 *>(a_lds + lds_off(lc * 4 + C + 1, g)) = p;
}

// A fragments of one k-step; B fragments of two (k-steps alternate between
// the two sets, so the next k-step's B can be read while this one's MFMAs
// still use theirs).
struct Frags {
  bf16x8 a[4], b[2][2];
};

typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ s16x4 read_tr16(const uint8_t *p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4 *)p);
}

// Lane-dependent LDS offsets of the fragment reads: A row wm * 128 + lrow,
// and for B block j the transposing-read address at t = 0 (rows 16 KS and
// 16 KS + 4 follow as constant offsets).
struct FragPlan {
  int wm, lrow, lk;
  uint32_t yb[2];
};

// MFMA operands of k-step KS (t = 16 KS .. 16 KS + 15) for this wave.
template <int KS>
__device__ __forceinline__ bf16x8 read_b(const uint8_t *bl, const FragPlan &fp, int j) {
  const s16x4 lo = read_tr16(bl + fp.yb[j] + KS * 16 * 512);
  const s16x4 hi = read_tr16(bl + fp.yb[j] + (KS * 16 + 4) * 512);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

template <int KS>
__device__ __forceinline__ void read_frags(Frags &f, const uint8_t *al, const uint8_t *bl,
                                           const FragPlan &fp) {
#pragma unroll
  for (int j = 0; j < 2; ++j) f.b[KS & 1][j] = read_b<KS>(bl, fp, j);
#pragma unroll
  for (int i = 0; i < 4; ++i)
    f.a[i] = *reinterpret_cast<const bf16x8 *>(
        al + lds_off(fp.wm * 128 + i * 32 + fp.lrow, KS * 2 + fp.lk));
}

// The 8 MFMAs of this k-step (B fragments in set (KS + 3) % 2, i.e. the set
// of k-step KS - 1) with the fragment reads of k-step KS woven in: the B
// fragments of k-step KS go to the other set right after the first MFMA, and
// each A fragment is re-read as soon as its two MFMAs have been issued.
template <int KS>
__device__ __forceinline__ void mma8_read(f32x16 (&acc)[4][2], Frags &f, const uint8_t *al,
                                          const uint8_t *bl, const FragPlan &fp) {
  constexpr int CUR = (KS + 1) & 1, NXT = KS & 1;
#pragma unroll
  for (int j = 0; j < 2; ++j) f.b[NXT][j] = read_b<KS>(bl, fp, j);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc[i][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[CUR][0], acc[i][0], 0, 0, 0);
    acc[i][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[CUR][1], acc[i][1], 0, 0, 0);
    f.a[i] = *reinterpret_cast<const bf16x8 *>(
        al + lds_off(fp.wm * 128 + i * 32 + fp.lrow, KS * 2 + fp.lk));
  }
}

// Instruction order of one k-step region: every MFMA followed by VALU ops
// of the next stage's dequantisation (regions 1 and 2), LDS stores spread
// over the region, global loads after the first MFMAs, and the LDS reads of
// the next k-step's fragments: the four B reads after the first MFMA, one A
// fragment after every second MFMA.
template <bool NEXT, int VALU, int WRITES, int LOADS>
__device__ __forceinline__ void schedule_region() {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // 1 MFMA
    if constexpr (NEXT)
      if (i == 0) __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
    if constexpr (VALU > 0) __builtin_amdgcn_sched_group_barrier(0x002, VALU, 0);
    if constexpr (WRITES > 0)
      if (i % (8 / WRITES) == 8 / WRITES - 1) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
    if constexpr (LOADS > 0)
      if (i < (LOADS + 1) / 2) __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);
    if constexpr (NEXT)
      if (i & 1) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_barrier(0);
}

// One k-step region of a stage s.  Regions 1 and 2 dequantise stage s+1's
// X (already in registers) into the other LDS buffer; region 2 then issues
// the global loads of stage s+2's X into the same registers.  The barrier
// that publishes stage s+1 sits between regions 2 and 3, so region 3 can
// start the DMA of stage s+2's dY into this stage's buffer (no wave reads
// it any more) and read stage s+1's first fragments while its own MFMAs
// issue: no wave waits on LDS after the barrier.
template <int CODE, int KS>
__device__ __forceinline__ void region(f32x16 (&acc)[4][2], Frags &f, const uint8_t *cur_a,
                                       uint8_t *cur_b, uint8_t *nxt_a, uint8_t *nxt_b,
                                       Stage &raw, __amdgpu_buffer_rsrc_t ry, const XRsrc &rx,
                                       const LoadPlan &lp, const FragPlan &fp, int wave, int lc,
                                       int g) {
  if constexpr (KS == 1) fill_x<CODE, 0>(raw, nxt_a, lc, g);
  if constexpr (KS == 2) {
    fill_x<CODE, 2>(raw, nxt_a, lc, g);
    load_stage<CODE>(raw, rx, lp);
  }
  if constexpr (KS == 3) dma_dy(ry, lp, cur_b, wave);
  if constexpr (KS < 3) mma8_read<KS + 1>(acc, f, cur_a, cur_b, fp);
  if constexpr (KS == 3) mma8_read<0>(acc, f, nxt_a, nxt_b, fp);
  if constexpr (KS == 0) schedule_region<true, 0, 0, 0>();
  if constexpr (KS == 1) schedule_region<true, 4, 2, 0>();
  if constexpr (KS == 2) schedule_region<true, 4, 2, kXLoads<CODE>>();
  if constexpr (KS == 3) schedule_region<true, 0, 0, kYLoads>();
}

// s_waitcnt with only the vector-memory count limited (expcnt and lgkmcnt
// at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// A full stage s on `cur` (its first fragments already in f): stage s+1's X
// from `raw` into `nxt`, the loads of stage s+2's X into `raw`, the barrier
// (each thread first waits for its own DMA of stage s+1's dY; the X loads
// issued after it may stay in flight), then the last k-step, the DMA of stage
// s+2's dY into `cur` and the first fragments of stage s+1 from `nxt`.
template <int CODE, int BLOCK>
__device__ __forceinline__ void stage(f32x16 (&acc)[4][2], Frags &f, const uint8_t *cur_a,
                                      uint8_t *cur_b, uint8_t *nxt_a, uint8_t *nxt_b,
                                      Stage &raw, const WgradArgs &a, int64_t k_next2,
                                      const LoadPlan &lp, const FragPlan &fp, int wave, int lc,
                                      int g) {
  const __amdgpu_buffer_rsrc_t ry = y_rsrc(a, k_next2);
  const XRsrc rx = x_rsrc<BLOCK>(a, k_next2);
  region<CODE, 0>(acc, f, cur_a, cur_b, nxt_a, nxt_b, raw, ry, rx, lp, fp, wave, lc, g);
  region<CODE, 1>(acc, f, cur_a, cur_b, nxt_a, nxt_b, raw, ry, rx, lp, fp, wave, lc, g);
  region<CODE, 2>(acc, f, cur_a, cur_b, nxt_a, nxt_b, raw, ry, rx, lp, fp, wave, lc, g);
  wait_vmcnt<kXLoads<CODE>>();
  __syncthreads();
  region<CODE, 3>(acc, f, cur_a, cur_b, nxt_a, nxt_b, raw, ry, rx, lp, fp, wave, lc, g);
}

template <int CODE, int BLOCK>
__global__ __launch_bounds__(kThreads, 1) void wgrad_kernel(const WgradArgs a, int tiles_m,
                                                            int tiles_n) {
  // Two stage buffers, each an A (dequantised X) and a B (dY) tile; separate
  // arrays so that the compiler can tell the DMA targets from the tiles
  // being read.
  __shared__ __attribute__((aligned(16))) uint8_t lds_a0[kTileBytes];
  __shared__ __attribute__((aligned(16))) uint8_t lds_b0[kTileBytes];
  __shared__ __attribute__((aligned(16))) uint8_t lds_a1[kTileBytes];
  __shared__ __attribute__((aligned(16))) uint8_t lds_b1[kTileBytes];

  // XCD-aware tile order.
  const int n_wg = tiles_m * tiles_n;
  int id = blockIdx.x;
  if ((n_wg & 7) == 0) id = (id & 7) * (n_wg >> 3) + (id >> 3);
  const int per_group = kGroupM * tiles_n;
  const int first_m = (id / per_group) * kGroupM;
  const int gm = tiles_m - first_m < kGroupM ? tiles_m - first_m : kGroupM;
  const int tm = first_m + (id % per_group) % gm;
  const int tn = (id % per_group) / gm;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int wn = wave & 3;
  const int lc = tid & 63, g = tid >> 6;  // X loader: 4-column chunk lc, token rows 8 g .. 8 g + 7

  LoadPlan lp;
  {
    const uint32_t kg = (uint32_t)g * 8u;
    const int64_t m = m0 + lc * 4;
    lp.st_x = (uint32_t)a.M;
    lp.st_s = (uint32_t)(a.M / BLOCK) * 4u;
    lp.vo_x = m < a.M ? kg * lp.st_x + (uint32_t)m : kOob;
    lp.vo_s = m < a.M ? kg * lp.st_s + (uint32_t)(m / BLOCK) * 4u : kOob;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint32_t t = (uint32_t)(wave * 8 + 2 * r + (lane >> 5));
      const uint32_t c = (uint32_t)(lane & 31) ^ y_swz(t);
      const int64_t n = n0 + 8 * c;
      lp.vo_y[r] = n < a.N ? t * (uint32_t)a.N * 2u + (uint32_t)n * 2u : kOob;
    }
  }
  FragPlan fp;
  {
    fp.wm = wave >> 2;
    fp.lrow = lane & 31;
    fp.lk = lane >> 5;
    // transposing reads: 16-lane group q = lane / 16, lane 4 a' + c' within
    // it addresses row e = (lane & 15) / 4 of a 4-row slice, columns 4 a
    // .. 4 a + 3 (a = lane & 3) of the group's 16-column half
    const uint32_t q = (uint32_t)lane >> 4, e = ((uint32_t)lane & 15u) >> 2, a4 = lane & 3;
    const uint32_t t = 8u * (q >> 1) + e;                          // t at k-step 0, read 0
    const uint32_t col = 16u * (q & 1u) + 4u * a4;                 // within the 32-column block
    const uint32_t swz = (e << 2) | ((q >> 1) << 4);               // y_swz(t) at every k-step
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const uint32_t chunk = (uint32_t)(wn * 64 + j * 32 + col) >> 3;
      fp.yb[j] = t * 512u + ((chunk ^ swz) << 4) + (col & 7u) * 2u;
    }
  }

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  // Stage s lives in LDS buffer s % 2; the raw X operand of stage s+1 waits
  // in registers.  Loads of stages past K read nothing (empty buffer range)
  // and return 0, so the loop needs no edge branches; the stage count is
  // rounded up to even so that the buffer of every stage is a compile-time
  // constant.
  const int64_t n_stages = ((a.K + BK - 1) / BK + 1) & ~int64_t(1);
  Stage raw;
  Frags f;
  dma_dy(y_rsrc(a, 0), lp, lds_b0, wave);
  load_stage<CODE>(raw, x_rsrc<BLOCK>(a, 0), lp);
  fill_x<CODE, 0>(raw, lds_a0, lc, g);
  fill_x<CODE, 2>(raw, lds_a0, lc, g);
  load_stage<CODE>(raw, x_rsrc<BLOCK>(a, BK), lp);
  dma_dy(y_rsrc(a, BK), lp, lds_b1, wave);
  wait_vmcnt<kXLoads<CODE> + kYLoads>();
  __syncthreads();
  read_frags<0>(f, lds_a0, lds_b0, fp);

  for (int64_t s = 0; s < n_stages; s += 2) {
    stage<CODE, BLOCK>(acc, f, lds_a0, lds_b0, lds_a1, lds_b1, raw, a, (s + 2) * BK, lp, fp,
                       wave, lc, g);
    stage<CODE, BLOCK>(acc, f, lds_a1, lds_b1, lds_a0, lds_b0, raw, a, (s + 3) * BK, lp, fp,
                       wave, lc, g);
  }

  // Epilogue.  32x32 accumulator layout: lane l holds column l % 32 and, for
  // register r, row 8 (r / 4) + 4 (l / 32) + r % 4.
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t col = n0 + wn * 64 + j * 32 + fp.lrow;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + fp.wm * 128 + i * 32 + (r >> 2) * 8 + fp.lk * 4 + (r & 3);
        if (row < a.M && col < a.N) {
          float *p = a.dw + row * a.N + col;
          *p = a.accumulate ? *p + acc[i][j][r] : acc[i][j][r];
        }
      }
    }
  }
}

template <int CODE, int BLOCK>
hipError_t launch_one(const WgradArgs &a, hipStream_t s) {
  const int tiles_m = (int)((a.M + BM - 1) / BM);
  const int tiles_n = (int)((a.N + BN - 1) / BN);
  hipLaunchKernelGGL((wgrad_kernel<CODE, BLOCK>), dim3(tiles_m * tiles_n), dim3(kThreads), 0, s,
                     a, tiles_m, tiles_n);
  return hipGetLastError();
}

template <int CODE>
hipError_t dispatch(const WgradArgs &a, int block, hipStream_t s) {
  switch (block) {
    case 32: return launch_one<CODE, 32>(a, s);
    case 64: return launch_one<CODE, 64>(a, s);
    case 128: return launch_one<CODE, 128>(a, s);
    default: return launch_one<CODE, 256>(a, s);
  }
}

}  // namespace

hipError_t launch_wgrad(const WgradArgs &a, int code, int block, hipStream_t s) {
  if (a.M == 0 || a.N == 0) return hipSuccess;
  if (code == kCodeCast) return launch_one<kCodeCast, 256>(a, s);  // no blocks; BLOCK unused
  return code == kCodeInt8 ? dispatch<kCodeInt8>(a, block, s) : dispatch<kCodeE4M3>(a, block, s);
}

}  // namespace hilore
