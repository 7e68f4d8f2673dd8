/* A plain C11 consumer of include/gauss_sum.h: compiles the header as C and
 * drives the host-side contract of the library without a GPU (fake device
 * addresses, never dereferenced: every call below is rejected by argument
 * validation before anything is enqueued).
 * Prints one line per check and exits with the number of failed checks. */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "gauss_sum.h"

static int failures = 0;

static void expect(const char* what, int got, int want) {
  printf("%-44s %d%s\n", what, got, got == want ? "" : "   <-- unexpected");
  if (got != want) ++failures;
}

#define A(x) ((const void*)(uintptr_t)(x))
#define F(x) ((float*)(uintptr_t)(x))
#define W(x) ((void*)(uintptr_t)(x))

int main(void) {
  gs_problem p = {1000, 2000, 64, 4, GS_F16, GS_F32};
  const size_t ws = gauss_sum_fwd_workspace_size(&p);
  expect("abi version", gauss_sum_abi_version(), GAUSS_SUM_ABI_VERSION);
  expect("fwd workspace > 0", ws > 0, 1);
  expect("fwd workspace 256-byte multiple", (int)(ws % 256), 0);
  expect("status string of an unknown code", strcmp(gauss_sum_status_string(12345), "unknown status"), 0);
  expect("status string of success", strcmp(gauss_sum_status_string(GS_SUCCESS), "success"), 0);

  const void *q = A(0x100000), *k = A(0x200000), *v = A(0x300000);
  float* out = F(0x400000);
  void* wsp = W(0x1000000);
  expect("NULL problem", gauss_sum_fwd(NULL, q, k, v, 1.0f, out, wsp, ws, 0), GS_ERR_NULL_POINTER);
  expect("NULL output", gauss_sum_fwd(&p, q, k, v, 1.0f, NULL, wsp, ws, 0), GS_ERR_NULL_POINTER);
  expect("tau = 0", gauss_sum_fwd(&p, q, k, v, 0.0f, out, wsp, ws, 0), GS_ERR_BAD_TAU);
  expect("tau = NaN", gauss_sum_fwd(&p, q, k, v, nanf(""), out, wsp, ws, 0), GS_ERR_BAD_TAU);
  expect("workspace too small", gauss_sum_fwd(&p, q, k, v, 1.0f, out, wsp, ws - 256, 0), GS_ERR_WORKSPACE);
  expect("misaligned workspace", gauss_sum_fwd(&p, q, k, v, 1.0f, out, W(0x1000010), ws, 0), GS_ERR_MISALIGNED);
  expect("misaligned fp16 points", gauss_sum_fwd(&p, A(0x100001), k, v, 1.0f, out, wsp, ws, 0), GS_ERR_MISALIGNED);
  expect("output overlaps the values", gauss_sum_fwd(&p, q, k, v, 1.0f, F(0x300000), wsp, ws, 0), GS_ERR_ALIAS);

  gs_problem bad = p;
  bad.D = 257;
  expect("D = 257", gauss_sum_fwd(&bad, q, k, v, 1.0f, out, wsp, ws, 0), GS_ERR_BAD_SHAPE);
  expect("workspace size of a bad shape", (int)gauss_sum_fwd_workspace_size(&bad), 0);
  bad = p;
  bad.qk_dtype = 7; /* not a gs_dtype: an int field, so this is well defined */
  expect("points dtype 7", gauss_sum_fwd(&bad, q, k, v, 1.0f, out, wsp, ws, 0), GS_ERR_UNSUPPORTED);
  bad = p;
  bad.qk_dtype = GS_F32;
  const size_t wsb = gauss_sum_bwd_workspace_size(&bad, 1, 0, 0);
  expect("fp32 points have no gradient (size 0)", (int)wsb, 0);

  printf("%d failed\n", failures);
  return failures;
}
