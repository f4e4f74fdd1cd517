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

template <int BLOCK>
__device__ __forceinline__ void load_stage(Stage &st, const LoadPlan &lp, const WgradArgs &a,
                                           int64_t k0) {
  const int64_t left = a.K - k0;
  const int64_t rows = left < BK ? left : BK;
  const int64_t sld = a.M / BLOCK;
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(a.codes + k0 * a.M), 0, (int)(rows * a.M), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(a.scales + k0 * sld), 0, (int)(rows * sld * 4), 0x00020000);
  const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(a.dy + k0 * a.N), 0, (int)(rows * a.N * 2), 0x00020000);
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    st.xc[r] = __builtin_amdgcn_raw_buffer_load_b64(rx, (int)(lp.vo_x + r * lp.st_x), 0, 0);
    st.xs[r] = __uint_as_float(
        __builtin_amdgcn_raw_buffer_load_b32(rs, (int)(lp.vo_s + r * lp.st_s), 0, 0));
    st.yv[r] = __builtin_amdgcn_raw_buffer_load_b128(ry, (int)(lp.vo_y + r * lp.st_y), 0, 0);
  }
}

template <int CODE, int C>
__device__ __forceinline__ void store_x_pair(const Stage &st, uint8_t *a_lds, int lc, int g) {
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
}

template <int CODE>
__device__ __forceinline__ void store_stage(const Stage &st, uint8_t *a_lds, uint8_t *b_lds,
                                            int tid) {
  const int lc = tid & 31;
  const int g = tid >> 5;  // granule = kg / 8
  // X: dequantise two columns of the 8 token rows at a time and pair rows
  // (t, t+1) of each column into one word.
  store_x_pair<CODE, 0>(st, a_lds, lc, g);
  store_x_pair<CODE, 2>(st, a_lds, lc, g);
  store_x_pair<CODE, 4>(st, a_lds, lc, g);
  store_x_pair<CODE, 6>(st, a_lds, lc, g);
  // dY: pair the bf16 of rows (t, t+1) for each column.
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int w = c >> 1;
    const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
    u32x4 p;
    p.x = __builtin_amdgcn_perm(st.yv[1][w], st.yv[0][w], sel);
    p.y = __builtin_amdgcn_perm(st.yv[3][w], st.yv[2][w], sel);
    p.z = __builtin_amdgcn_perm(st.yv[5][w], st.yv[4][w], sel);
    p.w = __builtin_amdgcn_perm(st.yv[7][w], st.yv[6][w], sel);
    *reinterpret_cast<u32x4 *>(b_lds + lds_off(lc * 8 + c, g)) = p;
  }
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

  LoadPlan lp;
  {
    const int lc = tid & 31;
    const uint32_t kg = (uint32_t)(tid >> 5) * 8u;
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

  const int64_t n_stages = (a.K + BK - 1) / BK;
  Stage st;
  if (n_stages > 0) {
    load_stage<BLOCK>(st, lp, a, 0);
    store_stage<CODE>(st, lds, lds + kTileBytes, tid);
  }
  __syncthreads();

  for (int64_t s = 0; s < n_stages; ++s) {
    const int cur = (int)(s & 1);
    const bool more = s + 1 < n_stages;
    if (more) load_stage<BLOCK>(st, lp, a, (s + 1) * BK);
    const uint8_t *al = lds + 2 * cur * kTileBytes;
    const uint8_t *bl = al + kTileBytes;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8 af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const bf16x8 *>(al + lds_off(wm * 128 + i * 32 + lrow, ks * 2 + lk));
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bf[j] = *reinterpret_cast<const bf16x8 *>(bl + lds_off(wn * 128 + j * 32 + lrow, ks * 2 + lk));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      uint8_t *an = lds + 2 * (cur ^ 1) * kTileBytes;
      store_stage<CODE>(st, an, an + kTileBytes, tid);
    }
    __syncthreads();
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
