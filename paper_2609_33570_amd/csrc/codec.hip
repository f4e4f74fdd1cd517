// Blockwise absmax codec for HiLoRe's low-precision (L) action on gfx950.
//
// Encode (App. B.1 Eq. fp8-roundtrip in its scaled reading; App. B.3
// post-forward encoding) and reconstruction for backward.  For every run of
// BLOCK consecutive columns of a row, with Q = 127 (int8) or 448 (E4M3FN):
//   amax < 2^-64 -> scale 0 and codes 0, else
//   s = amax / Q, r = Q / amax (IEEE fp32 quotients), code = RNE(x * r),
//   xhat = bf16_RNE(value(code) * s).
//
// Layout and mapping.  One wave owns one row at a time (rows of all units of
// a launch are numbered consecutively and strided over the waves of the
// grid).  Each lane moves 8 bf16 (one 128-bit load) per step, so a step of a
// wave covers 512 consecutive columns and a block of BLOCK columns is held by
// BLOCK/8 neighbouring lanes; its amax is a DPP/swizzle reduction inside that
// lane group.  Codes leave as one 64-bit store per lane, scales as one 32-bit
// store per block.  The optional per-row sums are kept per lane in a fixed
// order and reduced once per row with a butterfly, so they do not depend on
// the grid size.
//
// The literal codec (code kCodeCast) is the paper's plain cast with no scale:
// code = E4M3FN nearest-even of x where |x| <= 464 (448 for (448, 464]),
// NaN (S.1111.111, sign kept) where |x| > 464 or x is not finite, exactly as
// torch.float8_e4m3fn casts; the cast back is exact, NaN codes giving the
// canonical bf16 NaN 0x7FC0.
//
// Exact quotients without a divide.  amax is the magnitude of one of the
// block's bf16 elements, so amax = m * 2^e with m one of the 128 bf16
// mantissas 1 + k/128.  Because scaling by a power of two commutes with
// rounding in the normal range, RN(amax / Q) = RN(m / Q) * 2^e and
// RN(Q / amax) = RN(Q / m) * 2^-e, and all results stay normal for
// amax >= 2^-64.  The 128 quotients per code are folded at compile time (IEEE
// round-to-nearest) and the exponent is applied by an integer add.
#include "device_common.hpp"
#include "hilore_internal.hpp"

// Every rounding step is the one written: no implicit fused multiply-add
// (the exact sequences above depend on it; wanted FMAs are explicit fmaf).
#pragma clang fp contract(off)

namespace hilore {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;
constexpr int kColsPerStep = kWave * 8;
constexpr int kUnroll = 4;

template <int CODE>
struct QuotientTable {
  uint32_t s[128];  // bits of RN((1 + k/128) / Q)
  uint32_t r[128];  // bits of RN(Q / (1 + k/128))
  constexpr QuotientTable() : s(), r() {
    constexpr float Q = CODE == kCodeInt8 ? 127.0f : 448.0f;
    for (int k = 0; k < 128; ++k) {
      const float m = 1.0f + (float)k / 128.0f;
      s[k] = __builtin_bit_cast(uint32_t, m / Q);
      r[k] = __builtin_bit_cast(uint32_t, Q / m);
    }
  }
};

template <int CODE>
__constant__ constexpr QuotientTable<CODE> kQuot{};

__device__ __forceinline__ int find_unit(const CodecBatch &b, int64_t g) {
  int u = 0;
  while (u + 1 < b.n && g >= b.row_begin[u + 1]) ++u;
  return u;
}

// Scale s and reciprocal r of a block from its amax (see the file comment).
// keep = 0 for a zero block (all codes forced to 0), else ~0.
template <int CODE>
__device__ __forceinline__ void block_quotients(float amax, const uint32_t *tab_s,
                                                const uint32_t *tab_r, float &s, float &r,
                                                uint32_t &keep) {
  const uint32_t ab = __float_as_uint(amax);
  const uint32_t k = (ab >> 16) & 0x7Fu;
  const int e = (int)(ab >> 23) - 127;
  const bool zero = e < -64;  // amax < 2^-64
  const uint32_t sb = tab_s[k] + ((uint32_t)e << 23);
  const uint32_t rb = tab_r[k] - ((uint32_t)e << 23);
  s = zero ? 0.0f : __uint_as_float(sb);
  r = zero ? 0.0f : __uint_as_float(rb);
  keep = zero ? 0u : 0xFFFFFFFFu;
}

// Encode 8 values v[] (already x * r); returns the 8 code bytes and the 8
// code values as fp32 (exact).
template <int CODE>
__device__ __forceinline__ u32x2 encode8(const float v[8], uint32_t keep, float q[8]) {
  u32x2 out;
  if constexpr (CODE == kCodeInt8) {
    // Adding 1.5 * 2^23 rounds to an integer with ties to even and leaves the
    // integer, two's complement, in the low mantissa bits.  |v| <= 127 * (1 +
    // 2^-23) here, so the result is already inside [-127, 127].
    uint32_t b[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float t = v[i] + 12582912.0f;
      b[i] = __float_as_uint(t);
      q[i] = t - 12582912.0f;
    }
    out.x = __builtin_amdgcn_perm(__builtin_amdgcn_perm(b[3], b[2], 0x0c0c0400u),
                                  __builtin_amdgcn_perm(b[1], b[0], 0x0c0c0400u), 0x05040100u);
    out.y = __builtin_amdgcn_perm(__builtin_amdgcn_perm(b[7], b[6], 0x0c0c0400u),
                                  __builtin_amdgcn_perm(b[5], b[4], 0x0c0c0400u), 0x05040100u);
  } else {
    // v_cvt_pk_fp8_f32: round to nearest even onto OCP E4M3FN, sign kept
    // (checked bit for bit against the software rule for every |v| <= 448).
    int lo = __builtin_amdgcn_cvt_pk_fp8_f32(v[0], v[1], 0, false);
    lo = __builtin_amdgcn_cvt_pk_fp8_f32(v[2], v[3], lo, true);
    int hi = __builtin_amdgcn_cvt_pk_fp8_f32(v[4], v[5], 0, false);
    hi = __builtin_amdgcn_cvt_pk_fp8_f32(v[6], v[7], hi, true);
    out.x = (uint32_t)lo & keep;
    out.y = (uint32_t)hi & keep;
    f32x2 d;
    d = __builtin_amdgcn_cvt_pk_f32_fp8((int)out.x, false); q[0] = d.x; q[1] = d.y;
    d = __builtin_amdgcn_cvt_pk_f32_fp8((int)out.x, true);  q[2] = d.x; q[3] = d.y;
    d = __builtin_amdgcn_cvt_pk_f32_fp8((int)out.y, false); q[4] = d.x; q[5] = d.y;
    d = __builtin_amdgcn_cvt_pk_f32_fp8((int)out.y, true);  q[6] = d.x; q[7] = d.y;
  }
  return out;
}

// Code bytes -> exact fp32 values.
template <int CODE>
__device__ __forceinline__ void decode8(u32x2 c, float q[8]) {
  if constexpr (CODE == kCodeInt8) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      q[i] = (float)(int)__builtin_amdgcn_sbfe(c.x, 8 * i, 8);
      q[4 + i] = (float)(int)__builtin_amdgcn_sbfe(c.y, 8 * i, 8);
    }
  } else {
    f32x2 d;
    d = __builtin_amdgcn_cvt_pk_f32_fp8((int)c.x, false); q[0] = d.x; q[1] = d.y;
    d = __builtin_amdgcn_cvt_pk_f32_fp8((int)c.x, true);  q[2] = d.x; q[3] = d.y;
    d = __builtin_amdgcn_cvt_pk_f32_fp8((int)c.y, false); q[4] = d.x; q[5] = d.y;
    d = __builtin_amdgcn_cvt_pk_f32_fp8((int)c.y, true);  q[6] = d.x; q[7] = d.y;
  }
}

// The literal cast of 8 values (see the file comment); q[] receives the
// exact values of the codes (NaN for NaN codes).
__device__ __forceinline__ u32x2 cast8(const float x[8], float q[8]) {
  int lo = __builtin_amdgcn_cvt_pk_fp8_f32(x[0], x[1], 0, false);
  lo = __builtin_amdgcn_cvt_pk_fp8_f32(x[2], x[3], lo, true);
  int hi = __builtin_amdgcn_cvt_pk_fp8_f32(x[4], x[5], 0, false);
  hi = __builtin_amdgcn_cvt_pk_fp8_f32(x[6], x[7], hi, true);
  uint32_t w[2] = {(uint32_t)lo, (uint32_t)hi};
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    // |x| > 464, infinities and NaNs (all of whose magnitude bits exceed those
    // of 464.0f) have no encoding: NaN with the sign of x
    const uint32_t xb = __float_as_uint(x[i]);
    const uint32_t nan = 0x7Fu | ((xb >> 24) & 0x80u);
    const int sh = 8 * (i & 3);
    uint32_t &wd = w[i >> 2];
    wd = (xb & 0x7FFFFFFFu) > 0x43E80000u ? (wd & ~(0xFFu << sh)) | (nan << sh) : wd;
  }
  const u32x2 out = {w[0], w[1]};
  f32x2 d;
  d = __builtin_amdgcn_cvt_pk_f32_fp8((int)out.x, false); q[0] = d.x; q[1] = d.y;
  d = __builtin_amdgcn_cvt_pk_f32_fp8((int)out.x, true);  q[2] = d.x; q[3] = d.y;
  d = __builtin_amdgcn_cvt_pk_f32_fp8((int)out.y, false); q[4] = d.x; q[5] = d.y;
  d = __builtin_amdgcn_cvt_pk_f32_fp8((int)out.y, true);  q[6] = d.x; q[7] = d.y;
  return out;
}

// bf16 of two E4M3FN codes (bytes 2k, 2k+1 of w, k = HI): exact, NaN codes
// -> 0x7FC0.
template <bool HI>
__device__ __forceinline__ uint32_t uncast2(uint32_t w) {
  const f32x2 d = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, HI);
  uint32_t lo = __float_as_uint(d.x) >> 16, hi = __float_as_uint(d.y) >> 16;  // exact
  const uint32_t c0 = (w >> (HI ? 16 : 0)) & 0x7Fu, c1 = (w >> (HI ? 24 : 8)) & 0x7Fu;
  lo = c0 == 0x7Fu ? 0x7FC0u : lo;
  hi = c1 == 0x7Fu ? 0x7FC0u : hi;
  return lo | (hi << 16);
}

// The literal cast, same row-per-wave mapping as compress_kernel.
template <bool STATS>
__global__ __launch_bounds__(kThreads) void cast_kernel(const CodecBatch b) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t n_waves = (int64_t)gridDim.x * kWavesPerBlock;
  const int64_t total = b.row_begin[b.n];
  for (int64_t g = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; g < total;
       g += n_waves) {
    const int u = find_unit(b, g);
    const CodecUnit &d = b.u[u];
    const int64_t row = g - b.row_begin[u];
    const int64_t cols = d.cols;
    const u32x4 *xr = reinterpret_cast<const u32x4 *>(d.x + row * d.ld);
    u32x2 *cr = reinterpret_cast<u32x2 *>(d.codes + row * cols);
    float acc_x = 0.0f, acc_e = 0.0f;
    for (int64_t c0 = 0; c0 < cols; c0 += kColsPerStep * kUnroll) {
      u32x4 w[kUnroll];
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        const int64_t col = c0 + i * kColsPerStep + lane * 8;
        w[i] = col < cols ? __builtin_nontemporal_load(xr + col / 8) : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        const int64_t col = c0 + i * kColsPerStep + lane * 8;
        if (col >= cols) continue;
        float x[8], q[8];
        x[0] = bf16_lo(w[i].x); x[1] = bf16_hi(w[i].x);
        x[2] = bf16_lo(w[i].y); x[3] = bf16_hi(w[i].y);
        x[4] = bf16_lo(w[i].z); x[5] = bf16_hi(w[i].z);
        x[6] = bf16_lo(w[i].w); x[7] = bf16_hi(w[i].w);
        __builtin_nontemporal_store(cast8(x, q), cr + col / 8);
        if constexpr (STATS) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float e = q[j] - x[j];  // exact: both are bf16 values (or NaN)
            acc_e = fmaf(e, e, acc_e);
            acc_x = fmaf(x[j], x[j], acc_x);
          }
        }
      }
    }
    if constexpr (STATS) {
      acc_x = wave_sum(acc_x);
      acc_e = wave_sum(acc_e);
      if (lane == 0) {
        if (d.ss_x) d.ss_x[row] = acc_x;
        if (d.ss_err) d.ss_err[row] = acc_e;
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void uncast_kernel(const CodecBatch b) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t n_waves = (int64_t)gridDim.x * kWavesPerBlock;
  const int64_t total = b.row_begin[b.n];
  for (int64_t g = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; g < total;
       g += n_waves) {
    const int u = find_unit(b, g);
    const CodecUnit &d = b.u[u];
    const int64_t row = g - b.row_begin[u];
    const int64_t cols = d.cols;
    const u32x2 *cr = reinterpret_cast<const u32x2 *>(d.codes + row * cols);
    u32x4 *hr = reinterpret_cast<u32x4 *>(d.xhat + row * cols);
    for (int64_t c0 = 0; c0 < cols; c0 += kColsPerStep * kUnroll) {
      u32x2 c[kUnroll];
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        const int64_t col = c0 + i * kColsPerStep + lane * 8;
        c[i] = col < cols ? __builtin_nontemporal_load(cr + col / 8) : u32x2{0, 0};
      }
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        const int64_t col = c0 + i * kColsPerStep + lane * 8;
        if (col < cols) {
          const u32x4 h = {uncast2<false>(c[i].x), uncast2<true>(c[i].x),
                           uncast2<false>(c[i].y), uncast2<true>(c[i].y)};
          __builtin_nontemporal_store(h, hr + col / 8);
        }
      }
    }
  }
}

template <int CODE, int BLOCK, bool STATS>
__global__ __launch_bounds__(kThreads) void compress_kernel(const CodecBatch b) {
  constexpr int kLanesPerBlock = BLOCK / 8;
  __shared__ uint32_t tab_s[128], tab_r[128];
  if (threadIdx.x < 128) {
    tab_s[threadIdx.x] = kQuot<CODE>.s[threadIdx.x];
    tab_r[threadIdx.x] = kQuot<CODE>.r[threadIdx.x];
  }
  __syncthreads();

  const int lane = threadIdx.x & (kWave - 1);
  const int64_t n_waves = (int64_t)gridDim.x * kWavesPerBlock;
  const int64_t total = b.row_begin[b.n];
  for (int64_t g = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; g < total;
       g += n_waves) {
    const int u = find_unit(b, g);
    const CodecUnit &d = b.u[u];
    const int64_t row = g - b.row_begin[u];
    const int64_t cols = d.cols;
    const u32x4 *xr = reinterpret_cast<const u32x4 *>(d.x + row * d.ld);
    u32x2 *cr = reinterpret_cast<u32x2 *>(d.codes + row * cols);
    float *sr = d.scales + row * (cols / BLOCK);
    float acc_x = 0.0f, acc_e = 0.0f;

    for (int64_t c0 = 0; c0 < cols; c0 += kColsPerStep * kUnroll) {
      u32x4 w[kUnroll];
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        const int64_t col = c0 + i * kColsPerStep + lane * 8;
        w[i] = col < cols ? __builtin_nontemporal_load(xr + col / 8) : u32x4{0, 0, 0, 0};
      }
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        const int64_t col = c0 + i * kColsPerStep + lane * 8;
        if (c0 + i * kColsPerStep >= cols) break;  // wave-uniform
        float x[8];
        x[0] = bf16_lo(w[i].x); x[1] = bf16_hi(w[i].x);
        x[2] = bf16_lo(w[i].y); x[3] = bf16_hi(w[i].y);
        x[4] = bf16_lo(w[i].z); x[5] = bf16_hi(w[i].z);
        x[6] = bf16_lo(w[i].w); x[7] = bf16_hi(w[i].w);
        float am = fmaxf(fmaxf(fmaxf(fabsf(x[0]), fabsf(x[1])), fmaxf(fabsf(x[2]), fabsf(x[3]))),
                         fmaxf(fmaxf(fabsf(x[4]), fabsf(x[5])), fmaxf(fabsf(x[6]), fabsf(x[7]))));
        am = group_max<kLanesPerBlock>(am);
        float s, r;
        uint32_t keep;
        block_quotients<CODE>(am, tab_s, tab_r, s, r, keep);
        float v[8], q[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = x[j] * r;
        const u32x2 code = encode8<CODE>(v, keep, q);
        if (col < cols) {
          __builtin_nontemporal_store(code, cr + col / 8);
          if ((lane & (kLanesPerBlock - 1)) == 0) sr[col / BLOCK] = s;
        }
        if constexpr (STATS) {
#pragma unroll
          for (int j = 0; j < 8; j += 2) {
            const uint32_t h = pack_bf16(q[j] * s, q[j + 1] * s);
            const float e0 = bf16_lo(h) - x[j];
            const float e1 = bf16_hi(h) - x[j + 1];
            acc_e = fmaf(e0, e0, acc_e);
            acc_e = fmaf(e1, e1, acc_e);
            acc_x = fmaf(x[j], x[j], acc_x);
            acc_x = fmaf(x[j + 1], x[j + 1], acc_x);
          }
        }
      }
    }
    if constexpr (STATS) {
      acc_x = wave_sum(acc_x);
      acc_e = wave_sum(acc_e);
      if (lane == 0) {
        if (d.ss_x) d.ss_x[row] = acc_x;
        if (d.ss_err) d.ss_err[row] = acc_e;
      }
    }
  }
}

template <int CODE, int BLOCK>
__global__ __launch_bounds__(kThreads) void decompress_kernel(const CodecBatch b) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t n_waves = (int64_t)gridDim.x * kWavesPerBlock;
  const int64_t total = b.row_begin[b.n];
  for (int64_t g = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; g < total;
       g += n_waves) {
    const int u = find_unit(b, g);
    const CodecUnit &d = b.u[u];
    const int64_t row = g - b.row_begin[u];
    const int64_t cols = d.cols;
    const u32x2 *cr = reinterpret_cast<const u32x2 *>(d.codes + row * cols);
    const float *sr = d.scales + row * (cols / BLOCK);
    u32x4 *hr = reinterpret_cast<u32x4 *>(d.xhat + row * cols);
    for (int64_t c0 = 0; c0 < cols; c0 += kColsPerStep * kUnroll) {
      u32x2 c[kUnroll];
      float s[kUnroll];
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        const int64_t col = c0 + i * kColsPerStep + lane * 8;
        const bool in = col < cols;
        c[i] = in ? __builtin_nontemporal_load(cr + col / 8) : u32x2{0, 0};
        s[i] = in ? sr[col / BLOCK] : 0.0f;
      }
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        const int64_t col = c0 + i * kColsPerStep + lane * 8;
        if (col < cols) {
          float q[8];
          decode8<CODE>(c[i], q);
          u32x4 h;
          h.x = pack_bf16(q[0] * s[i], q[1] * s[i]);
          h.y = pack_bf16(q[2] * s[i], q[3] * s[i]);
          h.z = pack_bf16(q[4] * s[i], q[5] * s[i]);
          h.w = pack_bf16(q[6] * s[i], q[7] * s[i]);
          __builtin_nontemporal_store(h, hr + col / 8);
        }
      }
    }
  }
}

int grid_for(int64_t rows) {
  // Enough 4-wave workgroups to keep every CU of the chip busy (256 CUs,
  // several resident workgroups each); fewer when there are fewer rows.
  const int64_t want = (rows + kWavesPerBlock - 1) / kWavesPerBlock;
  const int64_t cap = 256 * 8;
  return (int)(want < cap ? (want > 0 ? want : 1) : cap);
}

template <int CODE, int BLOCK>
hipError_t compress_dispatch(const CodecBatch &b, hipStream_t s) {
  const int grid = grid_for(b.row_begin[b.n]);
  if (b.stats)
    hipLaunchKernelGGL((compress_kernel<CODE, BLOCK, true>), dim3(grid), dim3(kThreads), 0, s, b);
  else
    hipLaunchKernelGGL((compress_kernel<CODE, BLOCK, false>), dim3(grid), dim3(kThreads), 0, s,
                       b);
  return hipGetLastError();
}

template <int CODE, int BLOCK>
hipError_t decompress_dispatch(const CodecBatch &b, hipStream_t s) {
  const int grid = grid_for(b.row_begin[b.n]);
  hipLaunchKernelGGL((decompress_kernel<CODE, BLOCK>), dim3(grid), dim3(kThreads), 0, s, b);
  return hipGetLastError();
}

template <int CODE>
hipError_t compress_code(const CodecBatch &b, int block, hipStream_t s) {
  switch (block) {
    case 32: return compress_dispatch<CODE, 32>(b, s);
    case 64: return compress_dispatch<CODE, 64>(b, s);
    case 128: return compress_dispatch<CODE, 128>(b, s);
    default: return compress_dispatch<CODE, 256>(b, s);
  }
}

template <int CODE>
hipError_t decompress_code(const CodecBatch &b, int block, hipStream_t s) {
  switch (block) {
    case 32: return decompress_dispatch<CODE, 32>(b, s);
    case 64: return decompress_dispatch<CODE, 64>(b, s);
    case 128: return decompress_dispatch<CODE, 128>(b, s);
    default: return decompress_dispatch<CODE, 256>(b, s);
  }
}

}  // namespace

hipError_t launch_compress(const CodecBatch &b, int code, int block, hipStream_t s) {
  if (code == kCodeCast) {
    const int grid = grid_for(b.row_begin[b.n]);
    if (b.stats)
      hipLaunchKernelGGL((cast_kernel<true>), dim3(grid), dim3(kThreads), 0, s, b);
    else
      hipLaunchKernelGGL((cast_kernel<false>), dim3(grid), dim3(kThreads), 0, s, b);
    return hipGetLastError();
  }
  return code == kCodeInt8 ? compress_code<kCodeInt8>(b, block, s)
                           : compress_code<kCodeE4M3>(b, block, s);
}

hipError_t launch_decompress(const CodecBatch &b, int code, int block, hipStream_t s) {
  if (code == kCodeCast) {
    hipLaunchKernelGGL(uncast_kernel, dim3(grid_for(b.row_begin[b.n])), dim3(kThreads), 0, s, b);
    return hipGetLastError();
  }
  return code == kCodeInt8 ? decompress_code<kCodeInt8>(b, block, s)
                           : decompress_code<kCodeE4M3>(b, block, s);
}

}  // namespace hilore
