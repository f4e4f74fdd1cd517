// Weight gradient on a reconstructed L unit, dequantisation fused into the
// tile load, on gfx950 MFMA:
//   dW[i][j] (+)= sum_t xhat[t][i] * dY[t][j],
//   xhat[t][i] = bf16_RNE(value(code[t][i]) * scale[t][i / BLOCK]).
// This is the full-parameter weight gradient of a linear layer whose saved
// input is kept in low precision (App. B.1; the full-parameter experiments of
// App. D); gradients accumulate over microbatches (App. D.1.1).
//
// Tiling.  A 256x256 tile of dW per workgroup of 4 waves (2x2), each wave a
// 128x128 sub-tile = 4x4 blocks of v_mfma_f32_32x32x16_bf16.  The contraction
// runs over tokens t in stages of 64.  Both operands arrive token-major (t is
// the slow index of X and dY), while MFMA wants 8 consecutive t per lane, so
// every thread loads an 8(t) x 8(i or j) patch with row loads (X: 8 bytes,
// dY: 16 bytes per row; a wave covers two full 256-column rows per load),
// transposes it in registers and writes 16-byte, t-contiguous granules to LDS:
//   - X: the dequantisation produces fp32 values anyway, and
//     v_cvt_pk_bf16_f32 packs any two of them, so pairing (t, t+1) costs
//     nothing extra;
//   - dY: one v_perm_b32 per output word pairs the bf16 halves of two rows.
// LDS holds [256 rows][64 t] bf16 per operand (32 KB), double buffered
// (128 KB of the 160 KB), with the 16-byte granule index XOR-swizzled by
// (row ^ row/8) so that both the transposing writes (rows 8 apart) and the
// MFMA fragment reads (consecutive rows) spread over the banks.
// The next stage's global loads are issued before the current stage's MFMAs
// and consumed after them, so HBM latency hides under the matrix work.
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
constexpr int kThreads = 256;
constexpr int kTileBytes = BM * BK * 2;  // one operand stage in LDS (32 KB)
constexpr int kGroupM = 8;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Byte offset of 16-byte granule g (t = 8g..8g+7) of row r in a [256][64] tile.
__device__ __forceinline__ uint32_t lds_off(int r, int g) {
  return (uint32_t)r * 128u + ((uint32_t)((g ^ r ^ (r >> 3)) & 7) << 4);
}

// Column c (0..7) of an 8-byte code row -> the exact fp32 code values of
// columns c and c+1 (c even).
template <int CODE, int C>
__device__ __forceinline__ f32x2 decode_pair(u32x2 w) {
  const uint32_t word = C < 4 ? w.x : w.y;
  if constexpr (CODE == kCodeInt8) {
    return f32x2{(float)(int)__builtin_amdgcn_sbfe(word, 8 * (C & 3), 8),
                 (float)(int)__builtin_amdgcn_sbfe(word, 8 * (C & 3) + 8, 8)};
  } else {
    return __builtin_amdgcn_cvt_pk_f32_fp8((int)word, (C & 2) != 0);
  }
}

constexpr uint32_t kOob = 0x80000000u;  // a buffer offset past every range: loads 0

struct Stage {
  u32x2 xc[8];   // X codes: 8 token rows x 8 columns (bytes)
  float xs[8];   // the scale of each of those rows' block
  u32x4 yv[8];   // dY: 8 token rows x 8 columns (bf16)
};

// Per-thread, loop-invariant parts of the stage loads.  Thread t loads token
// rows kg..kg+7 (kg = 8 (t / 32)) of columns 8 (t % 32) .. +7 of the tile.
// Rows past K and columns past M (N) fall outside the buffer range of the
// stage and read as 0, so ragged edges need no branches.
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

// Token rows R0, R0+1 of this thread's 8-row patch (6 loads).
template <int R0>
__device__ __forceinline__ void load_rows(Stage &st, const StageRsrc &rs, const LoadPlan &lp) {
#pragma unroll
  for (int r = R0; r < R0 + 2; ++r) {
    st.xc[r] = __builtin_amdgcn_raw_buffer_load_b64(rs.x, (int)(lp.vo_x + r * lp.st_x), 0, 0);
    st.xs[r] = __uint_as_float(
        __builtin_amdgcn_raw_buffer_load_b32(rs.s, (int)(lp.vo_s + r * lp.st_s), 0, 0));
    st.yv[r] = __builtin_amdgcn_raw_buffer_load_b128(rs.y, (int)(lp.vo_y + r * lp.st_y), 0, 0);
  }
}

template <int BLOCK>
__device__ __forceinline__ void load_stage(Stage &st, const LoadPlan &lp, const WgradArgs &a,
                                           int64_t k0) {
  const StageRsrc rs = stage_rsrc<BLOCK>(a, k0);
  load_rows<0>(st, rs, lp);
  load_rows<2>(st, rs, lp);
  load_rows<4>(st, rs, lp);
  load_rows<6>(st, rs, lp);
}

// Quarter Q of a stage's LDS fill: X columns 2Q, 2Q+1 dequantised and dY
// columns 2Q, 2Q+1, each written as one t-contiguous 16-byte granule per
// column (rows (t, t+1) paired into one word).
template <int CODE, int Q>
__device__ __forceinline__ void store_quarter(const Stage &st, uint8_t *a_lds, uint8_t *b_lds,
                                              int lc, int g) {
  constexpr int C = 2 * Q;
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
  *reinterpret_cast<u32x4 *>(a_lds + lds_off(lc * 8 + C, g)) = p;
  p.x = pack_bf16(hi[0], hi[1]);
  p.y = pack_bf16(hi[2], hi[3]);
  p.z = pack_bf16(hi[4], hi[5]);
  p.w = pack_bf16(hi[6], hi[7]);
  *reinterpret_cast<u32x4 *>(a_lds + lds_off(lc * 8 + C + 1, g)) = p;
#pragma unroll
  for (int c = C; c < C + 2; ++c) {
    const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
    p.x = __builtin_amdgcn_perm(st.yv[1][Q], st.yv[0][Q], sel);
    p.y = __builtin_amdgcn_perm(st.yv[3][Q], st.yv[2][Q], sel);
    p.z = __builtin_amdgcn_perm(st.yv[5][Q], st.yv[4][Q], sel);
    p.w = __builtin_amdgcn_perm(st.yv[7][Q], st.yv[6][Q], sel);
    *reinterpret_cast<u32x4 *>(b_lds + lds_off(lc * 8 + c, g)) = p;
  }
}

template <int CODE>
__device__ __forceinline__ void store_stage(const Stage &st, uint8_t *a_lds, uint8_t *b_lds,
                                            int tid) {
  const int lc = tid & 31, g = tid >> 5;
  store_quarter<CODE, 0>(st, a_lds, b_lds, lc, g);
  store_quarter<CODE, 1>(st, a_lds, b_lds, lc, g);
  store_quarter<CODE, 2>(st, a_lds, b_lds, lc, g);
  store_quarter<CODE, 3>(st, a_lds, b_lds, lc, g);
}

struct Frags {
  bf16x8 a[4], b[4];
};

// MFMA operands of k-step KS (t = 16 KS .. 16 KS + 15) for this wave.
template <int KS>
__device__ __forceinline__ void read_frags(Frags &f, const uint8_t *al, int wm, int wn, int lrow,
                                           int lk) {
  const uint8_t *bl = al + kTileBytes;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f.a[i] = *reinterpret_cast<const bf16x8 *>(al + lds_off(wm * 128 + i * 32 + lrow, KS * 2 + lk));
    f.b[i] = *reinterpret_cast<const bf16x8 *>(bl + lds_off(wn * 128 + i * 32 + lrow, KS * 2 + lk));
  }
}

__device__ __forceinline__ void mma16(f32x16 (&acc)[4][4], const Frags &f) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
}

// Instruction order of one k-step region: the LDS reads of the next
// k-step's fragments first (they have all 16 MFMAs to land), then every MFMA
// followed by three VALU ops of the next stage's dequantisation, with that
// quarter's four LDS stores and six global loads spread between the MFMAs.
template <bool PREFETCH, bool LOADS>
__device__ __forceinline__ void schedule_region() {
  if constexpr (PREFETCH) __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);  // 8 LDS reads
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                  // 1 MFMA
    __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);                  // 3 VALU
    if (i % 4 == 3) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // 1 LDS write
    if (LOADS && i < 8) __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);  // global loads
    if (LOADS && i >= 8) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
  }
  __builtin_amdgcn_sched_barrier(0);
}

// One k-step region of a stage: MFMAs of k-step KS from the current buffer
// and quarter KS of the next stage's LDS fill.  The first region also issues
// every global load of the stage after that: each LDS fill quarter needs all
// eight token rows of its patch, so the loads get a whole stage to land.
template <int CODE, int KS>
__device__ __forceinline__ void region(f32x16 (&acc)[4][4], Frags (&f)[2], const uint8_t *cur,
                                       uint8_t *nxt, const Stage &fill, Stage &load,
                                       const StageRsrc &rs, const LoadPlan &lp, int wm, int wn,
                                       int lrow, int lk, int lc, int g) {
  if constexpr (KS < 3) read_frags<KS + 1>(f[(KS + 1) & 1], cur, wm, wn, lrow, lk);
  if constexpr (KS == 0) {
    load_rows<0>(load, rs, lp);
    load_rows<2>(load, rs, lp);
    load_rows<4>(load, rs, lp);
    load_rows<6>(load, rs, lp);
  }
  store_quarter<CODE, KS>(fill, nxt, nxt + kTileBytes, lc, g);
  mma16(acc, f[KS & 1]);
  schedule_region<(KS < 3), (KS == 0)>();
}

// A full stage: MFMAs on `cur`, the LDS fill of the next stage from `fill`
// into `nxt`, the loads of the stage after that into `load`.
template <int CODE, int BLOCK>
__device__ __forceinline__ void stage(f32x16 (&acc)[4][4], const uint8_t *cur, uint8_t *nxt,
                                      const Stage &fill, Stage &load, const WgradArgs &a,
                                      int64_t k_load, const LoadPlan &lp, int wm, int wn,
                                      int lrow, int lk, int lc, int g) {
  const StageRsrc rs = stage_rsrc<BLOCK>(a, k_load);
  Frags f[2];
  read_frags<0>(f[0], cur, wm, wn, lrow, lk);
  region<CODE, 0>(acc, f, cur, nxt, fill, load, rs, lp, wm, wn, lrow, lk, lc, g);
  region<CODE, 1>(acc, f, cur, nxt, fill, load, rs, lp, wm, wn, lrow, lk, lc, g);
  region<CODE, 2>(acc, f, cur, nxt, fill, load, rs, lp, wm, wn, lrow, lk, lc, g);
  region<CODE, 3>(acc, f, cur, nxt, fill, load, rs, lp, wm, wn, lrow, lk, lc, g);
  __syncthreads();
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
  const int wm = wave >> 1, wn = wave & 1;
  const int lrow = lane & 31, lk = lane >> 5;
  const int lc = tid & 31, g = tid >> 5;

  LoadPlan lp;
  {
    const uint32_t kg = (uint32_t)g * 8u;
    const int64_t m = m0 + lc * 8, n = n0 + lc * 8;
    lp.st_x = (uint32_t)a.M;
    lp.st_s = (uint32_t)(a.M / BLOCK) * 4u;
    lp.st_y = (uint32_t)a.N * 2u;
    lp.vo_x = m < a.M ? kg * lp.st_x + (uint32_t)m : kOob;
    lp.vo_s = m < a.M ? kg * lp.st_s + (uint32_t)(m / BLOCK) * 4u : kOob;
    lp.vo_y = n < a.N ? kg * lp.st_y + (uint32_t)n * 2u : kOob;
  }

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

  // Pipeline.  Stage s of 64 tokens lives in LDS buffer s % 2; the raw
  // (undequantised) operands of stage s+1 wait in registers.  Stage s
  //   - runs its 64 MFMAs from LDS, four k-step regions of 16,
  //   - dequantises and transposes stage s+1 into the other LDS buffer, a
  //     quarter per region, interleaved with the MFMAs,
  //   - issues the global loads of stage s+2 into the register set that
  //     held stage s, a quarter per region,
  //   - ends with one barrier.
  // Loads of stages past K read nothing (empty buffer range) and return 0,
  // so the loop needs no edge branches; the stage count is rounded up to
  // even so that the buffer of every stage is a compile-time constant.
  const int64_t n_stages = ((a.K + BK - 1) / BK + 1) & ~int64_t(1);
  Stage ra, rb;
  load_stage<BLOCK>(ra, lp, a, 0);
  load_stage<BLOCK>(rb, lp, a, BK);
  store_stage<CODE>(ra, lds, lds + kTileBytes, tid);
  __syncthreads();

  uint8_t *const buf0 = lds;
  uint8_t *const buf1 = lds + 2 * kTileBytes;
  for (int64_t s = 0; s < n_stages; s += 2) {
    stage<CODE, BLOCK>(acc, buf0, buf1, rb, ra, a, (s + 2) * BK, lp, wm, wn, lrow, lk, lc, g);
    stage<CODE, BLOCK>(acc, buf1, buf0, ra, rb, a, (s + 3) * BK, lp, wm, wn, lrow, lk, lc, g);
  }

  // Epilogue.  32x32 accumulator layout: lane l holds column l % 32 and, for
  // register r, row 8 (r / 4) + 4 (l / 32) + r % 4.
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t col = n0 + wn * 128 + j * 32 + lrow;
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
