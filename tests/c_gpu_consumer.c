/* A plain C99 program driving libhilore on the GPU: device memory from the HIP
 * runtime API, no Python or PyTorch anywhere.  Three exact checks:
 *   - codec: bf16 values q * 2^k on the int8 code grid (every block holding
 *     +-127 * 2^k) compress to codes q and scales 2^k and decompress to the
 *     same bits, with a reconstruction error sum of exactly 0;
 *   - coefficients: groups of equal rewards have advantage 0 and, with
 *     beta = 0, coefficient 0 on every slot, and logp_new = logp_old gives
 *     ratio 1 and the policy-term flag on every slot;
 *   - weight gradient: literal E4M3FN codes of small integers times bf16 small
 *     integers, whose sums are exact in fp32, against a host triple loop.
 * Prints one line per check; exit status 0 only if all hold. */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "hilore.h"

#define HIP(x)                                                          \
  do {                                                                  \
    hipError_t e_ = (x);                                                \
    if (e_ != hipSuccess) {                                             \
      printf("HIP error %s in %s\n", hipGetErrorString(e_), #x);        \
      return 2;                                                         \
    }                                                                   \
  } while (0)
#define LIB(x)                                                          \
  do {                                                                  \
    hilore_status s_ = (x);                                             \
    if (s_ != HILORE_OK) {                                              \
      printf("%s -> %s\n", #x, hilore_status_string(s_));               \
      return 3;                                                         \
    }                                                                   \
  } while (0)

/* bf16 bits of a float whose significand fits in 8 bits (exact) */
static uint16_t bf16_exact(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  return (uint16_t)(u >> 16);
}

static int codec_check(void) {
  enum { ROWS = 8, COLS = 256, BLOCK = 32, NB = COLS / BLOCK };
  static uint16_t x[ROWS * COLS], xhat[ROWS * COLS];
  static int8_t q[ROWS * COLS], codes[ROWS * COLS];
  static float s[ROWS * NB], scales[ROWS * NB], ss_err[ROWS];
  for (int r = 0; r < ROWS; ++r)
    for (int b = 0; b < NB; ++b) {
      const int k = (r + b) % 7 - 3;
      s[r * NB + b] = ldexpf(1.0f, k);
      for (int j = 0; j < BLOCK; ++j) {
        const int c = b * BLOCK + j;
        int v = (r * 37 + c * 11) % 255 - 127;
        if (j == 0) v = (b & 1) ? -127 : 127; /* the block's absmax */
        q[r * COLS + c] = (int8_t)v;
        x[r * COLS + c] = bf16_exact(ldexpf((float)v, k));
      }
    }
  void *dx, *dc, *ds, *dh, *dsx, *dse;
  HIP(hipMalloc(&dx, sizeof x));
  HIP(hipMalloc(&dc, sizeof codes));
  HIP(hipMalloc(&ds, sizeof scales));
  HIP(hipMalloc(&dh, sizeof xhat));
  HIP(hipMalloc(&dsx, sizeof ss_err));
  HIP(hipMalloc(&dse, sizeof ss_err));
  HIP(hipMemcpy(dx, x, sizeof x, hipMemcpyHostToDevice));
  hilore_unit_desc u;
  memset(&u, 0, sizeof u);
  u.x = dx;
  u.codes = dc;
  u.scales = ds;
  u.xhat = dh;
  u.row_ss_x = dsx;
  u.row_ss_err = dse;
  u.rows = ROWS;
  u.cols = COLS;
  u.ld = COLS;
  LIB(hilore_compress(&u, 1, HILORE_CODE_INT8, BLOCK, NULL));
  LIB(hilore_decompress(&u, 1, HILORE_CODE_INT8, BLOCK, NULL));
  HIP(hipDeviceSynchronize());
  HIP(hipMemcpy(codes, dc, sizeof codes, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(scales, ds, sizeof scales, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(xhat, dh, sizeof xhat, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(ss_err, dse, sizeof ss_err, hipMemcpyDeviceToHost));
  const int ok_codes = memcmp(codes, q, sizeof q) == 0;
  const int ok_scales = memcmp(scales, s, sizeof s) == 0;
  const int ok_xhat = memcmp(xhat, x, sizeof x) == 0;
  int ok_err = 1;
  for (int r = 0; r < ROWS; ++r) ok_err &= ss_err[r] == 0.0f;
  printf("codec: codes %d scales %d xhat %d zero error %d\n", ok_codes, ok_scales, ok_xhat, ok_err);
  hipFree(dx); hipFree(dc); hipFree(ds); hipFree(dh); hipFree(dsx); hipFree(dse);
  return ok_codes && ok_scales && ok_xhat && ok_err ? 0 : 1;
}

static int grpo_check(void) {
  enum { P = 2, G = 4, T = 8, R = P * G, N = R * T };
  float rewards[R], lp[N], adv[R], ratio[N], coeff[N];
  uint8_t flags[N];
  for (int i = 0; i < R; ++i) rewards[i] = (i / G) ? 0.0f : 1.0f; /* equal within each group */
  for (int i = 0; i < N; ++i) lp[i] = -2.0f - 0.01f * (float)i;
  void *dr, *dl, *da, *dra, *dfl, *dco;
  HIP(hipMalloc(&dr, sizeof rewards));
  HIP(hipMalloc(&dl, sizeof lp));
  HIP(hipMalloc(&da, sizeof adv));
  HIP(hipMalloc(&dra, sizeof ratio));
  HIP(hipMalloc(&dfl, sizeof flags));
  HIP(hipMalloc(&dco, sizeof coeff));
  HIP(hipMemcpy(dr, rewards, sizeof rewards, hipMemcpyHostToDevice));
  HIP(hipMemcpy(dl, lp, sizeof lp, hipMemcpyHostToDevice));
  LIB(hilore_grpo_coeffs(dr, dl, dl, NULL, NULL, P, G, T, 0.2f, 1e-6f, 0.0f, 0.0, da, dra, dfl,
                         dco, NULL, 0, NULL));
  HIP(hipDeviceSynchronize());
  HIP(hipMemcpy(adv, da, sizeof adv, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(ratio, dra, sizeof ratio, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(flags, dfl, sizeof flags, hipMemcpyDeviceToHost));
  HIP(hipMemcpy(coeff, dco, sizeof coeff, hipMemcpyDeviceToHost));
  int ok_adv = 1, ok_ratio = 1, ok_flags = 1, ok_coeff = 1;
  for (int i = 0; i < R; ++i) ok_adv &= adv[i] == 0.0f;
  for (int i = 0; i < N; ++i) {
    ok_ratio &= ratio[i] == 1.0f;
    ok_flags &= flags[i] == 1;
    ok_coeff &= coeff[i] == 0.0f;
  }
  printf("grpo: advantages %d ratios %d flags %d coefficients %d\n", ok_adv, ok_ratio, ok_flags,
         ok_coeff);
  hipFree(dr); hipFree(dl); hipFree(da); hipFree(dra); hipFree(dfl); hipFree(dco);
  return ok_adv && ok_ratio && ok_flags && ok_coeff ? 0 : 1;
}

static int wgrad_check(void) {
  enum { K = 64, M = 256, NN = 256 };
  /* E4M3FN bits of -2, -1, 0, 1, 2 */
  static const uint8_t enc[5] = {0xC0, 0xB8, 0x00, 0x38, 0x40};
  static uint8_t xc[K * M];
  static uint16_t dy[K * NN];
  static float xv[K * M], yv[K * NN], dw[M * NN];
  for (int t = 0; t < K; ++t) {
    for (int i = 0; i < M; ++i) {
      const int v = (t * 7 + i * 3) % 5 - 2;
      xc[t * M + i] = enc[v + 2];
      xv[t * M + i] = (float)v;
    }
    for (int j = 0; j < NN; ++j) {
      const int v = (t * 5 + j * 13) % 7 - 3;
      dy[t * NN + j] = bf16_exact((float)v);
      yv[t * NN + j] = (float)v;
    }
  }
  void *dxc, *ddy, *ddw;
  HIP(hipMalloc(&dxc, sizeof xc));
  HIP(hipMalloc(&ddy, sizeof dy));
  HIP(hipMalloc(&ddw, sizeof dw));
  HIP(hipMemcpy(dxc, xc, sizeof xc, hipMemcpyHostToDevice));
  HIP(hipMemcpy(ddy, dy, sizeof dy, hipMemcpyHostToDevice));
  LIB(hilore_dequant_wgrad(dxc, NULL, HILORE_CODE_FP8_E4M3FN_CAST, 0, ddy, ddw, K, M, NN, 0, NULL));
  HIP(hipDeviceSynchronize());
  HIP(hipMemcpy(dw, ddw, sizeof dw, hipMemcpyDeviceToHost));
  int bad = 0;
  for (int i = 0; i < M; ++i)
    for (int j = 0; j < NN; ++j) {
      float want = 0.0f;
      for (int t = 0; t < K; ++t) want += xv[t * M + i] * yv[t * NN + j];
      bad += dw[i * NN + j] != want;
    }
  printf("wgrad: %d of %d entries differ\n", bad, M * NN);
  hipFree(dxc); hipFree(ddy); hipFree(ddw);
  return bad ? 1 : 0;
}

int main(void) {
  int dev_count = 0;
  HIP(hipGetDeviceCount(&dev_count));
  if (dev_count < 1) {
    printf("no GPU\n");
    return 4;
  }
  HIP(hipSetDevice(0));
  const int fails = codec_check() + grpo_check() + wgrad_check();
  printf("%s\n", fails ? "FAILED" : "OK");
  return fails ? 1 : 0;
}
