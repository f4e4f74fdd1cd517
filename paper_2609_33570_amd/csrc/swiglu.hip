// Backward of the gated MLP activation on gfx950, with an L unit decoded in
// registers.  The evaluated models' MLP computes h = silu(g) * u from the gate
// and up projections g and u (silu(g) = g * sigmoid(g)); when g or u is an L
// unit, backward consumes its reconstruction (App. B.1 Eq. fp8-roundtrip):
//   du = dh * silu(g)
//   dg = dh * u * sigmoid(g) * (1 + g * (1 - sigmoid(g)))
// An L operand is xhat = bf16_RNE(value(code) * scale), bit for bit the value
// hilore_decompress writes, formed in registers and never stored; a bf16
// operand is read as is.  Arithmetic in fp32 (sigmoid from the hardware exp2
// and reciprocal), each output rounded once to bf16 (RNE).
//
// Elementwise and bound by HBM: per element 2 B of dh, 1 + 4/BLOCK B per L
// operand or 2 B per bf16 operand, 4 B of outputs.  A thread takes 8
// consecutive columns of one row (16-byte loads and stores, 8-byte code loads),
// all touched once, so loads and stores are non-temporal.  A workgroup is one
// wave covering 512 columns of a row (4.5 KiB at 9 B per element) and the grid
// is one pass of such short-lived workgroups, columns fastest, rows on the
// grid's second dimension: on 16384 x 18944 this ran ~17% faster than
// 256-thread workgroups over 2048 columns.
#include "device_common.hpp"
#include "hilore_internal.hpp"

// Every rounding step is the one written: no implicit fused multiply-add.
#pragma clang fp contract(off)

namespace hilore {
namespace {

constexpr int kThreads = 64;
constexpr int kColsPerThread = 8;
constexpr int kRowGrid = 65535;

// The raw bits of 8 values of one operand at (row, col .. col+7): a bf16
// operand's 16 bytes, or an L operand's 8 code bytes and its block scale.
struct Raw {
  u32x4 w;
  u32x2 c;
  float s;
};

template <int CODE, int BLOCK, bool L>
__device__ __forceinline__ void load_operand(const uint16_t *x, const uint8_t *codes,
                                             const float *scales, int64_t ld, int64_t cols,
                                             int64_t row, int64_t col, Raw &r) {
  if constexpr (!L) {
    r.w = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(x + row * ld + col));
  } else {
    r.c = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(codes + row * cols + col));
    if constexpr (CODE != kCodeCast) r.s = scales[row * (cols / BLOCK) + col / BLOCK];
  }
}

// The 8 values as fp32: an L operand decoded exactly as decompress does it.
template <int CODE, bool L>
__device__ __forceinline__ void decode_operand(const Raw &r, float v[8]) {
  if constexpr (!L) {
    v[0] = bf16_lo(r.w.x); v[1] = bf16_hi(r.w.x);
    v[2] = bf16_lo(r.w.y); v[3] = bf16_hi(r.w.y);
    v[4] = bf16_lo(r.w.z); v[5] = bf16_hi(r.w.z);
    v[6] = bf16_lo(r.w.w); v[7] = bf16_hi(r.w.w);
  } else {
    float q[8];
    if constexpr (CODE == kCodeInt8) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        q[i] = (float)(int)__builtin_amdgcn_sbfe(r.c.x, 8 * i, 8);
        q[4 + i] = (float)(int)__builtin_amdgcn_sbfe(r.c.y, 8 * i, 8);
      }
    } else {
      f32x2 d;
      d = __builtin_amdgcn_cvt_pk_f32_fp8((int)r.c.x, false); q[0] = d.x; q[1] = d.y;
      d = __builtin_amdgcn_cvt_pk_f32_fp8((int)r.c.x, true);  q[2] = d.x; q[3] = d.y;
      d = __builtin_amdgcn_cvt_pk_f32_fp8((int)r.c.y, false); q[4] = d.x; q[5] = d.y;
      d = __builtin_amdgcn_cvt_pk_f32_fp8((int)r.c.y, true);  q[6] = d.x; q[7] = d.y;
    }
    if constexpr (CODE == kCodeCast) {  // exact bf16 values (NaN codes stay NaN)
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = q[i];
    } else {
#pragma unroll
      for (int i = 0; i < 8; i += 2) {
        const uint32_t h = pack_bf16(q[i] * r.s, q[i + 1] * r.s);  // xhat, as decompress rounds it
        v[i] = bf16_lo(h);
        v[i + 1] = bf16_hi(h);
      }
    }
  }
}

template <int CODE, int BLOCK, bool GL, bool UL>
__global__ __launch_bounds__(kThreads) void swiglu_bwd_kernel(const SwigluArgs a) {
  const int64_t col = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * kColsPerThread;
  if (col >= a.cols) return;
  constexpr float kLog2e = 1.44269504088896340736f;
  for (int64_t row = blockIdx.y; row < a.rows; row += gridDim.y) {
    Raw rg, ru;
    load_operand<CODE, BLOCK, GL>(a.g_x, a.g_codes, a.g_scales, a.g_ld, a.cols, row, col, rg);
    load_operand<CODE, BLOCK, UL>(a.u_x, a.u_codes, a.u_scales, a.u_ld, a.cols, row, col, ru);
    const u32x4 dw =
        __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(a.dh + row * a.cols + col));
    float g[8], u[8], d[8];
    decode_operand<CODE, GL>(rg, g);
    decode_operand<CODE, UL>(ru, u);
    d[0] = bf16_lo(dw.x); d[1] = bf16_hi(dw.x);
    d[2] = bf16_lo(dw.y); d[3] = bf16_hi(dw.y);
    d[4] = bf16_lo(dw.z); d[5] = bf16_hi(dw.z);
    d[6] = bf16_lo(dw.w); d[7] = bf16_hi(dw.w);
    float og[8], ou[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      // sigmoid(g) = 1 / (1 + 2^(-g log2 e)); exp2 overflows to inf for very
      // negative g, giving sigmoid 0 as it should
      const float e = __builtin_amdgcn_exp2f(-g[i] * kLog2e);
      const float sg = __builtin_amdgcn_rcpf(1.0f + e);
      ou[i] = d[i] * (g[i] * sg);
      og[i] = (d[i] * u[i]) * (sg * (1.0f + g[i] * (1.0f - sg)));
    }
    u32x4 pg, pu;
    pg.x = pack_bf16(og[0], og[1]); pg.y = pack_bf16(og[2], og[3]);
    pg.z = pack_bf16(og[4], og[5]); pg.w = pack_bf16(og[6], og[7]);
    pu.x = pack_bf16(ou[0], ou[1]); pu.y = pack_bf16(ou[2], ou[3]);
    pu.z = pack_bf16(ou[4], ou[5]); pu.w = pack_bf16(ou[6], ou[7]);
    __builtin_nontemporal_store(pg, reinterpret_cast<u32x4 *>(a.dg + row * a.cols + col));
    __builtin_nontemporal_store(pu, reinterpret_cast<u32x4 *>(a.du + row * a.cols + col));
  }
}

template <int CODE, int BLOCK, bool GL, bool UL>
void launch_one(const SwigluArgs &a, hipStream_t s) {
  const int64_t chunks = (a.cols / kColsPerThread + kThreads - 1) / kThreads;
  const int64_t rg = a.rows < kRowGrid ? a.rows : kRowGrid;
  hipLaunchKernelGGL((swiglu_bwd_kernel<CODE, BLOCK, GL, UL>), dim3((unsigned)chunks, (unsigned)rg),
                     dim3(kThreads), 0, s, a);
}

template <int CODE, int BLOCK>
void by_operands(const SwigluArgs &a, hipStream_t s) {
  const bool gl = a.g_codes != nullptr, ul = a.u_codes != nullptr;
  if (gl && ul) launch_one<CODE, BLOCK, true, true>(a, s);
  else if (gl) launch_one<CODE, BLOCK, true, false>(a, s);
  else launch_one<CODE, BLOCK, false, true>(a, s);
}

template <int CODE>
void by_block(const SwigluArgs &a, int block, hipStream_t s) {
  switch (block) {
    case 32: return by_operands<CODE, 32>(a, s);
    case 64: return by_operands<CODE, 64>(a, s);
    case 128: return by_operands<CODE, 128>(a, s);
    default: return by_operands<CODE, 256>(a, s);
  }
}

}  // namespace

hipError_t launch_swiglu_bwd(const SwigluArgs &a, int code, int block, hipStream_t s) {
  if (a.rows == 0 || a.cols == 0) return hipSuccess;
  if (a.g_codes == nullptr && a.u_codes == nullptr) launch_one<kCodeInt8, 256, false, false>(a, s);
  else if (code == kCodeCast) by_operands<kCodeCast, 256>(a, s);  // no blocks; BLOCK unused
  else if (code == kCodeInt8) by_block<kCodeInt8>(a, block, s);
  else by_block<kCodeE4M3>(a, block, s);
  return hipGetLastError();
}

}  // namespace hilore
