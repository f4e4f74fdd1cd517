// Weight gradient on a reconstructed L unit, dequantisation fused into the
// tile load, on gfx950 MFMA:
//   dW[i][j] (+)= sum_t xhat[t][i] * dY[t][j],
//   xhat[t][i] = bf16_RNE(value(code[t][i]) * scale[t][i / BLOCK]).
// This is the full-parameter weight gradient of a linear layer whose saved
// input is kept in low precision (App. B.1; the full-parameter experiments of
// App. D); gradients accumulate over microbatches (App. D.1.1).
//
// Tiling.  A 256x256 tile of dW per workgroup of 8 waves (2 x 4), each wave a
// 128x64 sub-tile = 4x2 blocks of v_mfma_f32_32x32x16_bf16, i.e. two waves
// per SIMD: while one waits on LDS or memory or runs its dequantisation, the
// other keeps the matrix core busy.  The contraction runs over tokens t in
// stages of 64.  Both operands arrive token-major (t is the slow index of X
// and dY) while MFMA wants 8 consecutive t per lane, so every thread loads an
// 8(t) x 4(column) patch with row loads (a wave covers one full 256-column
// row of the tile per load), transposes it in registers and writes 16-byte,
// t-contiguous granules to LDS:
//   - X: the dequantisation produces fp32 values anyway, and
//     v_cvt_pk_bf16_f32 packs any two of them, so pairing (t, t+1) is free;
//   - dY: one v_perm_b32 per output word pairs the bf16 halves of two rows.
// LDS holds [256 rows][64 t] bf16 per operand (32 KB), double buffered
// (128 KB of the 160 KB), with the 16-byte granule index XOR-swizzled by
// (row ^ row/8): conflict-free both for the transposing writes (8 lanes
// write rows 4 apart) and for the MFMA fragment reads (consecutive rows).
//
// Pipeline per stage s (four k-step regions of 8 MFMAs per wave): every
// region reads the next k-step's fragments after its MFMAs; regions 2 and 3
// dequantise / transpose stage s+1 (already in registers) into the other LDS
// buffer, then region 3 issues the global loads of stage s+2 into the same
// registers; one barrier ends the stage.  One register set of raw operands
// keeps the kernel at two waves per SIMD.
//
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

// Raw operands of one stage for one thread: token rows kg..kg+7 (kg = 8 g) of
// columns 4 c .. 4 c + 3 of the tile.
struct Stage {
  uint32_t xc[8];  // X codes, 4 bytes per row
  float xs[8];     // the scale of each row's block
  u32x2 yv[8];     // dY, 4 bf16 per row
};

// Per-thread, loop-invariant parts of the stage loads.  Rows past K and
// columns past M (N) fall outside the buffer range of the stage and read as
// 0, so ragged edges need no branches.
struct LoadPlan {
  uint32_t vo_x, vo_s, vo_y;  // byte offsets of row kg inside a stage
  uint32_t st_x, st_s, st_y;  // byte stride of one token row
};

// Buffer descriptors of one stage of 64 token rows starting at k0.  Past
// the end of K the range is empty and every load returns 0.
struct StageRsrc {
  __amdgpu_buffer_rsrc_t x, s, y;
};

template <int BLOCK>
__device__ __forceinline__ StageRsrc stage_rsrc(const WgradArgs &a, int64_t k0) {
  const int64_t left = a.K - k0;
  const int64_t rows = left <= 0 ? 0 : (left < BK ? left : BK);
  const int64_t sld = a.M / BLOCK;
  StageRsrc r;
  r.x = __builtin_amdgcn_make_buffer_rsrc((void *)(a.codes + k0 * a.M), 0, (int)(rows * a.M),
                                          0x00020000);
  r.s = __builtin_amdgcn_make_buffer_rsrc((void *)(a.scales + k0 * sld), 0,
                                          (int)(rows * sld * 4), 0x00020000);
  r.y = __builtin_amdgcn_make_buffer_rsrc((void *)(a.dy + k0 * a.N), 0, (int)(rows * a.N * 2),
                                          0x00020000);
  return r;
}

__device__ __forceinline__ void load_stage(Stage &st, const StageRsrc &rs, const LoadPlan &lp) {
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    st.xc[r] = __builtin_amdgcn_raw_buffer_load_b32(rs.x, (int)(lp.vo_x + r * lp.st_x), 0, 0);
    st.xs[r] = __uint_as_float(
        __builtin_amdgcn_raw_buffer_load_b32(rs.s, (int)(lp.vo_s + r * lp.st_s), 0, 0));
    st.yv[r] = __builtin_amdgcn_raw_buffer_load_b64(rs.y, (int)(lp.vo_y + r * lp.st_y), 0, 0);
  }
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

// X columns C, C+1 of the thread's patch: dequantise the 8 token rows and
// write one t-contiguous granule per column (rows (t, t+1) paired per word).
template <int CODE, int C>
__device__ __forceinline__ void fill_x(const Stage &st, uint8_t *a_lds, int lc, int g) {
  float lo[8], hi[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const f32x2 q = decode_pair<CODE, C>(st.xc[r]);
    lo[r] = q.x * st.xs[r];
    hi[r] = q.y * st.xs[r];
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

// dY columns C, C+1: pair the bf16 of rows (t, t+1) of each column.
template <int C>
__device__ __forceinline__ void fill_y(const Stage &st, uint8_t *b_lds, int lc, int g) {
#pragma unroll
  for (int c = C; c < C + 2; ++c) {
    const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
    const int w = c >> 1;
    u32x4 p;
    p.x = __builtin_amdgcn_perm(st.yv[1][w], st.yv[0][w], sel);
    p.y = __builtin_amdgcn_perm(st.yv[3][w], st.yv[2][w], sel);
    p.z = __builtin_amdgcn_perm(st.yv[5][w], st.yv[4][w], sel);
    p.w = __builtin_amdgcn_perm(st.yv[7][w], st.yv[6][w], sel);
    *reinterpret_cast<u32x4 *>(b_lds + lds_off(lc * 4 + c, g)) = p;
  }
}

// Quarter Q of a stage's LDS fill (Q = 0..3: X columns 0-1, X 2-3, dY 0-1, dY 2-3).
template <int CODE, int Q>
__device__ __forceinline__ void fill_quarter(const Stage &st, uint8_t *lds_a, int lc, int g) {
  if constexpr (Q == 0) fill_x<CODE, 0>(st, lds_a, lc, g);
  if constexpr (Q == 1) fill_x<CODE, 2>(st, lds_a, lc, g);
  if constexpr (Q == 2) fill_y<0>(st, lds_a + kTileBytes, lc, g);
  if constexpr (Q == 3) fill_y<2>(st, lds_a + kTileBytes, lc, g);
}

struct Frags {
  bf16x8 a[4], b[2];
};

// MFMA operands of k-step KS (t = 16 KS .. 16 KS + 15) for this wave.
template <int KS>
__device__ __forceinline__ void read_frags(Frags &f, const uint8_t *al, int wm, int wn, int lrow,
                                           int lk) {
  const uint8_t *bl = al + kTileBytes;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    f.a[i] = *reinterpret_cast<const bf16x8 *>(al + lds_off(wm * 128 + i * 32 + lrow, KS * 2 + lk));
#pragma unroll
  for (int j = 0; j < 2; ++j)
    f.b[j] = *reinterpret_cast<const bf16x8 *>(bl + lds_off(wn * 64 + j * 32 + lrow, KS * 2 + lk));
}

__device__ __forceinline__ void mma8(f32x16 (&acc)[4][2], const Frags &f) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
}

// Instruction order of one k-step region: every MFMA followed by a few VALU
// ops (the next stage's dequantisation / transposition in the last two
// regions) with that region's LDS stores and global loads spread between,
// then the LDS reads of the next k-step's fragments.
template <bool NEXT, int VALU, int WRITES, int LOADS>
__device__ __forceinline__ void schedule_region() {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // 1 MFMA
    if constexpr (VALU > 0) __builtin_amdgcn_sched_group_barrier(0x002, VALU, 0);
    if constexpr (WRITES > 0)
      if (i % (8 / WRITES) == 8 / WRITES - 1) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
    if constexpr (LOADS > 0) __builtin_amdgcn_sched_group_barrier(0x020, LOADS, 0);
  }
  if constexpr (NEXT) __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);  // 6 LDS reads
  __builtin_amdgcn_sched_barrier(0);
}

// One k-step region of a stage.  Regions 0 and 1 only multiply; region 2
// dequantises the next stage's X patch into the other LDS buffer; region 3
// transposes its dY patch there and then issues the global loads of the
// stage after that into the same registers (so one register set suffices and
// the loads have until region 2 of the next stage to land).  The fragments
// of the next k-step are read into the same registers once this k-step's
// MFMAs have been issued; the other wave on the SIMD covers that latency.
template <int CODE, int KS>
__device__ __forceinline__ void region(f32x16 (&acc)[4][2], Frags &f, const uint8_t *cur,
                                       uint8_t *nxt, Stage &raw, const StageRsrc &rs,
                                       const LoadPlan &lp, int wm, int wn, int lrow, int lk,
                                       int lc, int g) {
  if constexpr (KS == 2) {
    fill_quarter<CODE, 0>(raw, nxt, lc, g);
    fill_quarter<CODE, 1>(raw, nxt, lc, g);
  }
  if constexpr (KS == 3) {
    fill_quarter<CODE, 2>(raw, nxt, lc, g);
    fill_quarter<CODE, 3>(raw, nxt, lc, g);
    load_stage(raw, rs, lp);
  }
  mma8(acc, f);
  if constexpr (KS < 3) read_frags<KS + 1>(f, cur, wm, wn, lrow, lk);
  if constexpr (KS < 2) schedule_region<true, 0, 0, 0>();
  if constexpr (KS == 2) schedule_region<true, 8, 4, 0>();
  if constexpr (KS == 3) schedule_region<false, 2, 4, 3>();
}

// A full stage: MFMAs on `cur`, the LDS fill of the next stage from `raw`
// into `nxt`, then the loads of the stage after that into `raw`.
template <int CODE, int BLOCK>
__device__ __forceinline__ void stage(f32x16 (&acc)[4][2], const uint8_t *cur, uint8_t *nxt,
                                      Stage &raw, const WgradArgs &a, int64_t k_load,
                                      const LoadPlan &lp, int wm, int wn, int lrow, int lk,
                                      int lc, int g) {
  const StageRsrc rs = stage_rsrc<BLOCK>(a, k_load);
  Frags f;
  read_frags<0>(f, cur, wm, wn, lrow, lk);
  region<CODE, 0>(acc, f, cur, nxt, raw, rs, lp, wm, wn, lrow, lk, lc, g);
  region<CODE, 1>(acc, f, cur, nxt, raw, rs, lp, wm, wn, lrow, lk, lc, g);
  region<CODE, 2>(acc, f, cur, nxt, raw, rs, lp, wm, wn, lrow, lk, lc, g);
  region<CODE, 3>(acc, f, cur, nxt, raw, rs, lp, wm, wn, lrow, lk, lc, g);
  __syncthreads();
}

template <int CODE>
__device__ __forceinline__ void fill_stage(const Stage &st, uint8_t *lds_a, int lc, int g) {
  fill_quarter<CODE, 0>(st, lds_a, lc, g);
  fill_quarter<CODE, 1>(st, lds_a, lc, g);
  fill_quarter<CODE, 2>(st, lds_a, lc, g);
  fill_quarter<CODE, 3>(st, lds_a, lc, g);
}

template <int CODE, int BLOCK>
__global__ __launch_bounds__(kThreads, 1) void wgrad_kernel(const WgradArgs a, int tiles_m,
                                                            int tiles_n) {
  // Stage buffer b holds A at lds + 2b * kTileBytes and B right after it.
  __shared__ __attribute__((aligned(16))) uint8_t lds[4 * kTileBytes];

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
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int wm = wave >> 2, wn = wave & 3;
  const int lrow = lane & 31, lk = lane >> 5;
  const int lc = tid & 63, g = tid >> 6;  // loader: 4-column chunk lc, token rows 8 g .. 8 g + 7

  LoadPlan lp;
  {
    const uint32_t kg = (uint32_t)g * 8u;
    const int64_t m = m0 + lc * 4, n = n0 + lc * 4;
    lp.st_x = (uint32_t)a.M;
    lp.st_s = (uint32_t)(a.M / BLOCK) * 4u;
    lp.st_y = (uint32_t)a.N * 2u;
    lp.vo_x = m < a.M ? kg * lp.st_x + (uint32_t)m : kOob;
    lp.vo_s = m < a.M ? kg * lp.st_s + (uint32_t)(m / BLOCK) * 4u : kOob;
    lp.vo_y = n < a.N ? kg * lp.st_y + (uint32_t)n * 2u : kOob;
  }

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  // Stage s lives in LDS buffer s % 2; the raw operands of stage s+1 wait in
  // registers.  Loads of stages past K read nothing (empty buffer range) and
  // return 0, so the loop needs no edge branches; the stage count is rounded
  // up to even so that the buffer of every stage is a compile-time constant.
  const int64_t n_stages = ((a.K + BK - 1) / BK + 1) & ~int64_t(1);
  Stage raw;
  load_stage(raw, stage_rsrc<BLOCK>(a, 0), lp);
  fill_stage<CODE>(raw, lds, lc, g);
  load_stage(raw, stage_rsrc<BLOCK>(a, BK), lp);
  __syncthreads();

  uint8_t *const buf0 = lds;
  uint8_t *const buf1 = lds + 2 * kTileBytes;
  for (int64_t s = 0; s < n_stages; s += 2) {
    stage<CODE, BLOCK>(acc, buf0, buf1, raw, a, (s + 2) * BK, lp, wm, wn, lrow, lk, lc, g);
    stage<CODE, BLOCK>(acc, buf1, buf0, raw, a, (s + 3) * BK, lp, wm, wn, lrow, lk, lc, g);
  }

  // Epilogue.  32x32 accumulator layout: lane l holds column l % 32 and, for
  // register r, row 8 (r / 4) + 4 (l / 32) + r % 4.
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t col = n0 + wn * 64 + j * 32 + lrow;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * 128 + i * 32 + (r >> 2) * 8 + lk * 4 + (r & 3);
        if (row < a.M && col < a.N) {
          float *p = a.dw + row * a.N + col;
          *p = a.accumulate ? *p + acc[i][j][r] : acc[i][j][r];
        }
      }
    }
  }
}

template <int CODE>
hipError_t dispatch(const WgradArgs &a, int block, hipStream_t s) {
  const int tiles_m = (int)((a.M + BM - 1) / BM);
  const int tiles_n = (int)((a.N + BN - 1) / BN);
  const dim3 grid(tiles_m * tiles_n);
  switch (block) {
    case 32: hipLaunchKernelGGL((wgrad_kernel<CODE, 32>), grid, dim3(kThreads), 0, s, a, tiles_m, tiles_n); break;
    case 64: hipLaunchKernelGGL((wgrad_kernel<CODE, 64>), grid, dim3(kThreads), 0, s, a, tiles_m, tiles_n); break;
    case 128: hipLaunchKernelGGL((wgrad_kernel<CODE, 128>), grid, dim3(kThreads), 0, s, a, tiles_m, tiles_n); break;
    default: hipLaunchKernelGGL((wgrad_kernel<CODE, 256>), grid, dim3(kThreads), 0, s, a, tiles_m, tiles_n); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_wgrad(const WgradArgs &a, int code, int block, hipStream_t s) {
  if (a.M == 0 || a.N == 0) return hipSuccess;
  return code == kCodeInt8 ? dispatch<kCodeInt8>(a, block, s) : dispatch<kCodeE4M3>(a, block, s);
}

}  // namespace hilore
