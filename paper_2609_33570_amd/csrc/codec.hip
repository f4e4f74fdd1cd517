// Blockwise absmax codec for HiLoRe's low-precision (L) action on gfx950.
//
// Encode (App. B.1 Eq. fp8-roundtrip in its scaled reading; App. B.3
// post-forward encoding) and reconstruction for backward.  For every run of
// BLOCK consecutive columns of a row, with Q = 127 (int8) or 448 (E4M3FN):
//   amax < 2^-64 -> scale 0 and codes 0, else
//   s = amax / Q, r = Q / amax (IEEE fp32 quotients), code = RNE(x * r),
//   xhat = bf16_RNE(value(code) * s).
//
// Layout and mapping.  A row is swept by W = 2^wpr_log2 waves (1 to 16,
// chosen from the row length by the host) and a launch is one pass over its
// rows: a workgroup holds max(W, 4) waves and owns 4/W consecutive rows (W <
// 4) or one row (W >= 4), then exits.  Each lane moves 8 bf16 (one 128-bit
// load) per step, so a step of a wave covers 512 consecutive columns and a
// block of BLOCK columns is held by BLOCK/8 neighbouring lanes; its amax is a
// DPP/swizzle reduction inside that lane group.  Codes leave as one 64-bit
// store per lane, scales as one 32-bit store per block.  Every access goes
// through a buffer range bound to one row of its operand, so lanes past the
// end of a row read zeros and drop their stores without branching, and the
// row's base address stays in scalar registers.  Short-lived
// workgroups that each cover a few KiB to a few tens of KiB of one row keep
// the addresses in flight across the chip inside a narrow moving window,
// which the HBM serves far better than thousands of waves each walking its
// own row.  The optional per-row sums are kept per lane in a fixed order,
// reduced per wave with a butterfly and across the row's waves in wave
// order, so they depend only on the row length.
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

constexpr int kMaxWaves = 16;  // waves per row at most (one workgroup)
constexpr int kMaxThreads = kMaxWaves * kWave;
constexpr int kColsPerStep = kWave * 8;
constexpr int kUnroll = 4;  // loads a lane issues before using the first

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

// The row (numbered over all units of the batch) and the position of this
// wave among the W = 2^wl waves that sweep it (see the file comment).
struct RowSlot {
  int64_t g;  // may be >= the batch's row count for the last workgroup
  int sub;    // 0 .. W-1
};
__device__ __forceinline__ RowSlot row_slot(int wl) {
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x / kWave);  // wave-uniform
  const int rows_per_wg = wl >= 2 ? 1 : 4 >> wl;
  return RowSlot{(int64_t)blockIdx.x * rows_per_wg + (wave >> wl), wave & ((1 << wl) - 1)};
}

// Sum of v over the W = 2^wl waves of each row of the workgroup, in wave
// order, through red[] (one slot per wave); the result is valid in lane 0 of
// the row's first wave.  Every thread of the workgroup must call it (it
// holds a barrier when W > 1).
__device__ __forceinline__ float row_sum(float v, int wl, float *red) {
  v = wave_sum(v);
  if (wl == 0) return v;
  const int wave = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) red[wave] = v;
  __syncthreads();
  if ((wave & ((1 << wl) - 1)) != 0) return v;
  float t = red[wave];
  for (int i = 1; i < (1 << wl); ++i) t += red[wave + i];
  return t;
}

// Buffer range over one row of an operand (bytes [0, bytes) from base).
// Loads past the range return 0 and stores past it are dropped.
struct RowRsrc {
  __amdgpu_buffer_rsrc_t r;
};
__device__ __forceinline__ RowRsrc row_rsrc(const void *base, uint32_t bytes) {
  return RowRsrc{__builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes,
                                                   0x00020000)};
}
constexpr uint32_t kOutOfRange = 0x80000000u;  // an offset past every row range
constexpr int kStream = 2;  // cache policy: nontemporal (data is touched once)
__device__ __forceinline__ u32x4 load_b128(const RowRsrc &r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r.r, (int)off, 0,
                                                                         kStream));
}
__device__ __forceinline__ u32x2 load_b64(const RowRsrc &r, uint32_t off) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r.r, (int)off, 0,
                                                                        kStream));
}
__device__ __forceinline__ uint32_t load_b32(const RowRsrc &r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r.r, (int)off, 0, 0);
}
__device__ __forceinline__ void store_b128(const RowRsrc &r, uint32_t off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r.r, (int)off, 0,
                                         kStream);
}
__device__ __forceinline__ void store_b64(const RowRsrc &r, uint32_t off, u32x2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(v, r.r, (int)off, 0,
                                        kStream);
}
__device__ __forceinline__ void store_b32(const RowRsrc &r, uint32_t off, uint32_t v) {
  __builtin_amdgcn_raw_buffer_store_b32(v, r.r, (int)off, 0, kStream);
}

// acc + lo*lo + hi*hi over the two bf16 halves of w (v_dot2c_f32_bf16).
__device__ __forceinline__ float dot2_bf16(uint32_t w, float acc) {
  const bf16x2 v = __builtin_bit_cast(bf16x2, w);
  return __builtin_amdgcn_fdot2_f32_bf16(v, v, acc, false);
}

// Scale s and reciprocal r of a block from its amax, given as bf16 bits
// (see the file comment).  keep = 0 for a zero block (all codes forced to
// 0), else ~0.
template <int CODE>
__device__ __forceinline__ void block_quotients(uint32_t amax_bits, const uint32_t *tab_s,
                                                const uint32_t *tab_r, float &s, float &r,
                                                uint32_t &keep) {
  const uint32_t k = amax_bits & 0x7Fu;
  const int e = (int)(amax_bits >> 7) - 127;
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
    // the first conversion of each word writes its low half; the high half
    // it keeps (here: whatever keep holds) is overwritten by the second
    int lo = __builtin_amdgcn_cvt_pk_fp8_f32(v[0], v[1], (int)keep, false);
    lo = __builtin_amdgcn_cvt_pk_fp8_f32(v[2], v[3], lo, true);
    int hi = __builtin_amdgcn_cvt_pk_fp8_f32(v[4], v[5], (int)keep, false);
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

// The literal cast, same mapping as compress_kernel.
template <bool STATS>
__global__ __launch_bounds__(kMaxThreads) void cast_kernel(const CodecBatch b) {
  __shared__ float red_x[kMaxWaves], red_e[kMaxWaves];
  const int lane = threadIdx.x & (kWave - 1);
  const int wl = b.wpr_log2;
  const RowSlot rs = row_slot(wl);
  float acc_x = 0.0f, acc_e = 0.0f;
  float *out_x = nullptr, *out_e = nullptr;  // this row's sums (lane 0 of wave 0)
  if (rs.g < b.row_begin[b.n]) {
    const int u = find_unit(b, rs.g);
    const CodecUnit *dp = &b.u[u];
    const int64_t row = rs.g - b.row_begin[u];
    if (rs.sub == 0 && lane == 0) {
      out_x = dp->ss_x ? dp->ss_x + row : nullptr;
      out_e = dp->ss_err ? dp->ss_err + row : nullptr;
    }
    const uint32_t cols = (uint32_t)dp->cols;
    const RowRsrc rx = row_rsrc(dp->x + row * dp->ld, cols * 2);
    const RowRsrc rc = row_rsrc(dp->codes + row * (int64_t)cols, cols);
    const uint32_t step = (uint32_t)kColsPerStep << wl;
    // lanes past the end of the row cast zeros (adding 0 to the sums) and
    // their stores are dropped
    for (uint32_t c0 = (uint32_t)rs.sub * kColsPerStep; c0 < cols; c0 += kUnroll * step) {
      u32x4 w[kUnroll];
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) w[i] = load_b128(rx, (c0 + i * step + lane * 8) * 2);
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        if (c0 + i * step >= cols) break;  // wave-uniform
        float x[8], q[8];
        x[0] = bf16_lo(w[i].x); x[1] = bf16_hi(w[i].x);
        x[2] = bf16_lo(w[i].y); x[3] = bf16_hi(w[i].y);
        x[4] = bf16_lo(w[i].z); x[5] = bf16_hi(w[i].z);
        x[6] = bf16_lo(w[i].w); x[7] = bf16_hi(w[i].w);
        store_b64(rc, c0 + i * step + lane * 8, cast8(x, q));
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
  }
  if constexpr (STATS) {
    acc_x = row_sum(acc_x, wl, red_x);
    acc_e = row_sum(acc_e, wl, red_e);
    if (out_x) *out_x = acc_x;
    if (out_e) *out_e = acc_e;
  }
}

__global__ __launch_bounds__(kMaxThreads) void uncast_kernel(const CodecBatch b) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wl = b.wpr_log2;
  const RowSlot rs = row_slot(wl);
  if (rs.g >= b.row_begin[b.n]) return;
  const int u = find_unit(b, rs.g);
  const CodecUnit &d = b.u[u];
  const int64_t row = rs.g - b.row_begin[u];
  const uint32_t cols = (uint32_t)d.cols;
  const RowRsrc rc = row_rsrc(d.codes + row * (int64_t)cols, cols);
  const RowRsrc rh = row_rsrc(d.xhat + row * (int64_t)cols, cols * 2);
  const uint32_t step = (uint32_t)kColsPerStep << wl;
  for (uint32_t c0 = (uint32_t)rs.sub * kColsPerStep; c0 < cols; c0 += kUnroll * step) {
    u32x2 c[kUnroll];
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) c[i] = load_b64(rc, c0 + i * step + lane * 8);
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
      if (c0 + i * step >= cols) break;  // wave-uniform
      const u32x4 h = {uncast2<false>(c[i].x), uncast2<true>(c[i].x), uncast2<false>(c[i].y),
                       uncast2<true>(c[i].y)};
      store_b128(rh, (c0 + i * step + lane * 8) * 2, h);
    }
  }
}

template <int CODE, int BLOCK, bool STATS>
__global__ __launch_bounds__(kMaxThreads) void compress_kernel(const CodecBatch b) {
  constexpr int kLanesPerBlock = BLOCK / 8;
  __shared__ uint32_t tab_s[128], tab_r[128];
  __shared__ float red_x[kMaxWaves], red_e[kMaxWaves];
  if (threadIdx.x < 128) {
    tab_s[threadIdx.x] = kQuot<CODE>.s[threadIdx.x];
    tab_r[threadIdx.x] = kQuot<CODE>.r[threadIdx.x];
  }
  __syncthreads();

  const int lane = threadIdx.x & (kWave - 1);
  const int wl = b.wpr_log2;
  const RowSlot rs = row_slot(wl);
  float acc_x = 0.0f, acc_e = 0.0f;
  float *out_x = nullptr, *out_e = nullptr;  // this row's sums (lane 0 of wave 0)
  if (rs.g < b.row_begin[b.n]) {
    const int u = find_unit(b, rs.g);
    const CodecUnit *dp = &b.u[u];
    const int64_t row = rs.g - b.row_begin[u];
    if (rs.sub == 0 && lane == 0) {
      out_x = dp->ss_x ? dp->ss_x + row : nullptr;
      out_e = dp->ss_err ? dp->ss_err + row : nullptr;
    }
    // One buffer range per operand row: lanes past the end of the row load
    // zeros (a zero block: scale 0) and their stores fall outside the range
    // and are dropped, so the loop needs no per-lane branches.
    const uint32_t cols = (uint32_t)dp->cols;
    const RowRsrc rx = row_rsrc(dp->x + row * dp->ld, cols * 2);
    const RowRsrc rc = row_rsrc(dp->codes + row * (int64_t)cols, cols);
    const RowRsrc rsc = row_rsrc(dp->scales + row * (int64_t)(cols / BLOCK), cols / BLOCK * 4);
    const bool leader = (lane & (kLanesPerBlock - 1)) == 0;
    const uint32_t step = (uint32_t)kColsPerStep << wl;
    // All of a lane's loads of a round (up to kUnroll steps of the row) are
    // issued before any of them is used; trip counts are wave-uniform.
    for (uint32_t c0 = (uint32_t)rs.sub * kColsPerStep; c0 < cols; c0 += kUnroll * step) {
      u32x4 w[kUnroll];
#pragma unroll
      for (int i = 0; i < kUnroll; ++i)
        w[i] = load_b128(rx, (c0 + i * step + lane * 8) * 2);
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        if (c0 + i * step >= cols) break;  // wave-uniform
        const uint32_t col = c0 + i * step + lane * 8;
        float x[8];
        x[0] = bf16_lo(w[i].x); x[1] = bf16_hi(w[i].x);
        x[2] = bf16_lo(w[i].y); x[3] = bf16_hi(w[i].y);
        x[4] = bf16_lo(w[i].z); x[5] = bf16_hi(w[i].z);
        x[6] = bf16_lo(w[i].w); x[7] = bf16_hi(w[i].w);
        const uint32_t am = group_max_u32<kLanesPerBlock>(absmax_bf16x8(w[i]));
        float s, r;
        uint32_t keep;
        block_quotients<CODE>(am, tab_s, tab_r, s, r, keep);
        float v[8], q[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = x[j] * r;
        const u32x2 code = encode8<CODE>(v, keep, q);
        store_b64(rc, col, code);
        store_b32(rsc, leader ? col / BLOCK * 4 : kOutOfRange, __float_as_uint(s));
        if constexpr (STATS) {
          // sum x^2 straight from the packed bf16 pairs (products are exact)
          acc_x = dot2_bf16(w[i].x, acc_x);
          acc_x = dot2_bf16(w[i].y, acc_x);
          acc_x = dot2_bf16(w[i].z, acc_x);
          acc_x = dot2_bf16(w[i].w, acc_x);
#pragma unroll
          for (int j = 0; j < 8; j += 2) {
            const uint32_t h = pack_bf16(q[j] * s, q[j + 1] * s);
            const float e0 = bf16_lo(h) - x[j];
            const float e1 = bf16_hi(h) - x[j + 1];
            acc_e = fmaf(e0, e0, acc_e);
            acc_e = fmaf(e1, e1, acc_e);
          }
        }
      }
    }
  }
  if constexpr (STATS) {
    acc_x = row_sum(acc_x, wl, red_x);
    acc_e = row_sum(acc_e, wl, red_e);
    if (out_x) *out_x = acc_x;
    if (out_e) *out_e = acc_e;
  }
}

template <int CODE, int BLOCK>
__global__ __launch_bounds__(kMaxThreads) void decompress_kernel(const CodecBatch b) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wl = b.wpr_log2;
  const RowSlot rs = row_slot(wl);
  if (rs.g >= b.row_begin[b.n]) return;
  const int u = find_unit(b, rs.g);
  const CodecUnit &d = b.u[u];
  const int64_t row = rs.g - b.row_begin[u];
  const uint32_t cols = (uint32_t)d.cols;
  const RowRsrc rc = row_rsrc(d.codes + row * (int64_t)cols, cols);
  const RowRsrc rsc = row_rsrc(d.scales + row * (int64_t)(cols / BLOCK), cols / BLOCK * 4);
  const RowRsrc rh = row_rsrc(d.xhat + row * (int64_t)cols, cols * 2);
  const uint32_t step = (uint32_t)kColsPerStep << wl;
  // lanes past the end of the row read zeros and their stores are dropped
  for (uint32_t c0 = (uint32_t)rs.sub * kColsPerStep; c0 < cols; c0 += kUnroll * step) {
    u32x2 c[kUnroll];
    float s[kUnroll];
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
      const uint32_t col = c0 + i * step + lane * 8;
      c[i] = load_b64(rc, col);
      s[i] = __uint_as_float(load_b32(rsc, col / BLOCK * 4));
    }
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
      if (c0 + i * step >= cols) break;  // wave-uniform
      float q[8];
      decode8<CODE>(c[i], q);
      u32x4 h;
      h.x = pack_bf16(q[0] * s[i], q[1] * s[i]);
      h.y = pack_bf16(q[2] * s[i], q[3] * s[i]);
      h.z = pack_bf16(q[4] * s[i], q[5] * s[i]);
      h.w = pack_bf16(q[6] * s[i], q[7] * s[i]);
      store_b128(rh, (c0 + i * step + lane * 8) * 2, h);
    }
  }
}

// One workgroup per row (W >= 4) or per 4/W rows, one pass over the batch.
struct Launch {
  dim3 grid, block;
};
Launch launch_shape(const CodecBatch &b) {
  const int wl = b.wpr_log2;
  const int64_t rows_per_wg = wl >= 2 ? 1 : 4 >> wl;
  const int64_t total = b.row_begin[b.n];
  const int64_t grid = (total + rows_per_wg - 1) / rows_per_wg;
  return Launch{dim3((unsigned)(grid > 0 ? grid : 1)), dim3(kWave << (wl >= 2 ? wl : 2))};
}

template <int CODE, int BLOCK>
hipError_t compress_dispatch(const CodecBatch &b, hipStream_t s) {
  const Launch l = launch_shape(b);
  if (b.stats)
    hipLaunchKernelGGL((compress_kernel<CODE, BLOCK, true>), l.grid, l.block, 0, s, b);
  else
    hipLaunchKernelGGL((compress_kernel<CODE, BLOCK, false>), l.grid, l.block, 0, s, b);
  return hipGetLastError();
}

template <int CODE, int BLOCK>
hipError_t decompress_dispatch(const CodecBatch &b, hipStream_t s) {
  const Launch l = launch_shape(b);
  hipLaunchKernelGGL((decompress_kernel<CODE, BLOCK>), l.grid, l.block, 0, s, b);
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
    const Launch l = launch_shape(b);
    if (b.stats)
      hipLaunchKernelGGL((cast_kernel<true>), l.grid, l.block, 0, s, b);
    else
      hipLaunchKernelGGL((cast_kernel<false>), l.grid, l.block, 0, s, b);
    return hipGetLastError();
  }
  return code == kCodeInt8 ? compress_code<kCodeInt8>(b, block, s)
                           : compress_code<kCodeE4M3>(b, block, s);
}

hipError_t launch_decompress(const CodecBatch &b, int code, int block, hipStream_t s) {
  if (code == kCodeCast) {
    const Launch l = launch_shape(b);
    hipLaunchKernelGGL(uncast_kernel, l.grid, l.block, 0, s, b);
    return hipGetLastError();
  }
  return code == kCodeInt8 ? decompress_code<kCodeInt8>(b, block, s)
                           : decompress_code<kCodeE4M3>(b, block, s);
}

}  // namespace hilore
