// Device helpers shared by the gfx950 kernels (wave64, CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hilore {

constexpr int kWave = 64;

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// bf16 halves of a packed word -> fp32 (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32;
// checked bit for bit against the software rule over every finite fp32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Cross-lane operations inside a wave.  DPP controls (gfx9 encoding).
enum : int {
  kDppQuadXor1 = 0xB1,      // quad_perm [1,0,3,2]
  kDppQuadXor2 = 0x4E,      // quad_perm [2,3,0,1]
  kDppRowHalfMirror = 0x141,
  kDppRowMirror = 0x140,
};

// v and its DPP neighbour combined by an unsigned max: the DPP move folds
// into v_max_u32_dpp (lanes without a source read 0, the identity).
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_max_u32(uint32_t v) {
  return max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true));
}

// Unsigned max over aligned groups of L lanes (L = 4, 8, 16 or 32); every
// lane of the group receives the group maximum.  After the quad steps each
// quad holds its max; the half-row mirror pairs quads 0<->1 and 2<->3, the
// row mirror pairs the two halves of a 16-lane row, and a swizzle pairs the
// two rows of 32.
template <int L>
__device__ __forceinline__ uint32_t group_max_u32(uint32_t v) {
  static_assert(L == 4 || L == 8 || L == 16 || L == 32, "group size");
  v = dpp_max_u32<kDppQuadXor1>(v);
  v = dpp_max_u32<kDppQuadXor2>(v);
  if constexpr (L >= 8) v = dpp_max_u32<kDppRowHalfMirror>(v);
  if constexpr (L >= 16) v = dpp_max_u32<kDppRowMirror>(v);
  if constexpr (L >= 32) v = max(v, (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x401F));
  return v;
}

// Largest magnitude of the 8 bf16 values of w, as bf16 bits in the low half
// (non-negative bf16 patterns order like their values; NaN is out of
// contract).
__device__ __forceinline__ uint32_t absmax_bf16x8(u32x4 w) {
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  const u16x2 a = __builtin_bit_cast(u16x2, w.x & 0x7FFF7FFFu);
  const u16x2 b = __builtin_bit_cast(u16x2, w.y & 0x7FFF7FFFu);
  const u16x2 c = __builtin_bit_cast(u16x2, w.z & 0x7FFF7FFFu);
  const u16x2 d = __builtin_bit_cast(u16x2, w.w & 0x7FFF7FFFu);
  const u16x2 m = __builtin_elementwise_max(__builtin_elementwise_max(a, b),
                                            __builtin_elementwise_max(c, d));
  return max((uint32_t)m.x, (uint32_t)m.y);
}

// Sum over the whole wave as a butterfly (xor 1, 2, 4, ..., 32).  Addition
// is commutative, so every lane ends with the same value: the pairwise tree
// (first half) + (second half), recursively, over the 64 lanes.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

}  // namespace hilore
