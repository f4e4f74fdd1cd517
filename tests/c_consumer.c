/* A plain C caller of libhilore: include/hilore.h compiled as C99 and linked
 * against the library, with no Python in between.  It exercises only calls
 * that return before anything reaches a device (queries and argument
 * validation), so it runs without a GPU; it prints one line per check and
 * exits non-zero on the first mismatch. */
#include <stdio.h>
#include <string.h>

#include "hilore.h"

static int failures = 0;

static void expect(const char *what, long got, long want) {
  printf("%-52s %ld (want %ld)\n", what, got, want);
  if (got != want) ++failures;
}

int main(void) {
  /* any non-null, 16-byte aligned address: no call below dereferences it */
  void *const fake = (void *)(uintptr_t)(1u << 20);
  expect("hilore_version", hilore_version(), 10000);
  expect("status string of UNSUPPORTED",
         strcmp(hilore_status_string(HILORE_ERR_UNSUPPORTED), "HILORE_ERR_UNSUPPORTED"), 0);

  /* workspace queries */
  expect("grad_rel_err workspace, n = 2^24", (long)hilore_grad_rel_err_workspace_bytes(1 << 24),
         1024 * 16);
  expect("allocate workspace, bad grid", (long)hilore_allocate_workspace_bytes(4, 0, 16), 0);
  expect("lora workspace, r = 0", (long)hilore_lora_grad_workspace_bytes(1024, 256, 0), 0);

  /* validation before any launch */
  expect("grpo workspace, 2^18 slots", (long)hilore_grpo_coeffs_workspace_bytes(16, 16, 1024), 16);
  expect("exposure/risk workspace, 78 units", (long)hilore_unit_exposure_risk_workspace_bytes(16384, 78),
         78 * 8 * 32);
  expect("grpo: G = 65", hilore_grpo_coeffs(fake, fake, fake, NULL, NULL, 1, 65, 8, 0.2f, 1e-6f,
                                            0.0f, 0.0, fake, NULL, fake, fake, NULL, 0, NULL),
         HILORE_ERR_UNSUPPORTED);
  hilore_unit_desc u;
  memset(&u, 0, sizeof u);
  u.x = fake;
  u.codes = fake;
  u.scales = fake;
  u.rows = 4;
  u.cols = 200; /* not a multiple of the block */
  u.ld = 200;
  expect("compress: cols % block", hilore_compress(&u, 1, HILORE_CODE_INT8, 128, NULL),
         HILORE_ERR_UNSUPPORTED);
  expect("decompress: bad code", hilore_decompress(&u, 1, 7, 128, NULL), HILORE_ERR_INVALID_ARG);
  expect("wgrad: N % 8", hilore_dequant_wgrad(fake, fake, HILORE_CODE_FP8_E4M3FN, 128, fake, fake,
                                              256, 512, 100, 0, NULL),
         HILORE_ERR_UNSUPPORTED);
  expect("lora: odd rank", hilore_dequant_lora_grad(fake, fake, HILORE_CODE_INT8, 64, fake, fake,
                                                    64, 256, 17, 2.0f, 0, fake, 1 << 20, NULL),
         HILORE_ERR_UNSUPPORTED);
  expect("update_sparsity: top_frac 0", hilore_update_sparsity(fake, fake, fake, NULL, 2, 4, 0.0,
                                                               fake, fake, NULL),
         HILORE_ERR_INVALID_ARG);
  expect("grad_rel_err: workspace too small", hilore_grad_rel_err(fake, fake, 1 << 20, 1e-30, fake,
                                                                 fake, 8, NULL),
         HILORE_ERR_WORKSPACE);
  printf("%s\n", failures ? "FAILED" : "OK");
  return failures ? 1 : 0;
}
