/* Host-side argument checks of the C ABI, run against a build of libagcn
 * whose host code carries AddressSanitizer and UndefinedBehaviorSanitizer
 * (tests/test_abi_sanitizers.py). No GPU is needed: every call below is
 * refused before the library makes a HIP call, or makes only calls that fail
 * cleanly without a device. Prints "c abi host check ok". */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "agcn.h"

static int g_fail = 0;

static void expect_status(int got, int want, const char* what) {
  if (got != want) {
    printf("FAILED: %s: status %d (%s), expected %d: %s\n", what, got, agcn_status_string(got),
           want, agcn_last_error());
    g_fail = 1;
  }
}

#define P(x) ((void*)(uintptr_t)(x))

static int create(int32_t n_rows, int32_t n_cols, int64_t nnz, uintptr_t rp, uintptr_t ci,
                  uintptr_t v, const agcn_plan_params* prm, agcn_plan_t* h) {
  *h = (agcn_plan_t)P(0xdead);
  return agcn_plan_create(h, n_rows, n_cols, nnz, (const int32_t*)P(rp), (const int32_t*)P(ci),
                          (const float*)P(v), prm, NULL);
}

static agcn_plan_params params(int32_t W, int32_t Z, int32_t H, uint32_t flags) {
  agcn_plan_params p;
  p.max_block_waves = W;
  p.max_wave_nzs = Z;
  p.hub_chunk_nnz = H;
  p.flags = flags;
  return p;
}

int main(void) {
  agcn_plan_params d;
  agcn_default_params(&d);
  if (d.max_block_waves < 1 || d.max_wave_nzs < 1 || d.flags != 0) g_fail = 1;
  agcn_default_params(NULL);
  for (int s = -1; s <= 6; ++s)
    if (agcn_status_string(s) == NULL || strlen(agcn_status_string(s)) == 0) g_fail = 1;

  agcn_plan_t h;
  expect_status(agcn_plan_create(NULL, 4, 4, 4, P(1), P(2), P(3), NULL, NULL),
                AGCN_ERR_INVALID_ARGUMENT, "null out");
  expect_status(create(-1, 4, 4, 0x1000, 0x2000, 0x3000, NULL, &h), AGCN_ERR_INVALID_ARGUMENT,
                "negative n_rows");
  if (h != NULL) g_fail = 1;
  expect_status(create(4, -1, 4, 0x1000, 0x2000, 0x3000, NULL, &h), AGCN_ERR_INVALID_ARGUMENT,
                "negative n_cols");
  expect_status(create(4, 4, -1, 0x1000, 0x2000, 0x3000, NULL, &h), AGCN_ERR_INVALID_ARGUMENT,
                "negative nnz");
  expect_status(create(0, 4, 5, 0x1000, 0x2000, 0x3000, NULL, &h), AGCN_ERR_INVALID_ARGUMENT,
                "nnz without rows");
  expect_status(create(4, 4, (int64_t)1 << 31, 0x1000, 0x2000, 0x3000, NULL, &h),
                AGCN_ERR_UNSUPPORTED, "nnz >= 2^31");
  expect_status(create(4, 4, 4, 0, 0x2000, 0x3000, NULL, &h), AGCN_ERR_INVALID_ARGUMENT,
                "null rowptr");
  expect_status(create(4, 4, 4, 0x1000, 0, 0x3000, NULL, &h), AGCN_ERR_INVALID_ARGUMENT,
                "null colidx");
  const agcn_plan_params bad[] = {params(0, 32, 0, 0),   params(33, 32, 0, 0),
                                  params(16, 0, 0, 0),   params(16, 257, 0, 0),
                                  params(16, 32, -1, 0), params(16, 32, 4097, 0),
                                  params(16, 32, 0, 4),  params(16, 32, 0, 3),
                                  params(32, 128, 0, 0)};
  for (size_t i = 0; i < sizeof bad / sizeof bad[0]; ++i) {
    expect_status(create(4, 4, 4, 0x1000, 0x2000, 0x3000, &bad[i], &h), AGCN_ERR_INVALID_ARGUMENT,
                  "bad parameters");
    if (h != NULL) g_fail = 1;
  }
  const agcn_plan_params h1 = params(16, 32, 1, 0);
  expect_status(create(2147483646, 4, 2147483647LL, 0x1000, 0x2000, 0x3000, &h1, &h),
                AGCN_ERR_UNSUPPORTED, "too many entries");

  size_t n = 0;
  expect_status(agcn_spmm(NULL, 16, (const float*)P(0x1000), 16, (float*)P(0x2000), 16, NULL, NULL),
                AGCN_ERR_INVALID_ARGUMENT, "spmm without plan");
  expect_status(agcn_spmm_ex(NULL, 16, (const float*)P(0x1000), 16, (float*)P(0x2000), 16, NULL,
                             NULL, 1), AGCN_ERR_INVALID_ARGUMENT, "spmm_ex without plan");
  expect_status(agcn_spmm_timed(NULL, 16, (const float*)P(0x1000), 16, (float*)P(0x2000), 16, NULL,
                                NULL, NULL, NULL, NULL), AGCN_ERR_INVALID_ARGUMENT,
                "spmm_timed without plan");
  expect_status(agcn_spmm_workspace_size(NULL, 16, &n), AGCN_ERR_INVALID_ARGUMENT,
                "workspace without plan");
  expect_status(agcn_gcn_workspace_size(NULL, 16, &n), AGCN_ERR_INVALID_ARGUMENT,
                "layer workspace without plan");
  expect_status(agcn_gcn_layer(NULL, 8, 16, (const float*)P(0x1000), 8, (const float*)P(0x2000), 16,
                               (float*)P(0x3000), 16, P(0x4000), NULL, 1),
                AGCN_ERR_INVALID_ARGUMENT, "layer without plan");
  agcn_plan_stats st;
  expect_status(agcn_plan_info(NULL, &st), AGCN_ERR_INVALID_ARGUMENT, "info without plan");
  expect_status(agcn_plan_export(NULL, NULL, NULL, NULL, NULL, NULL), AGCN_ERR_INVALID_ARGUMENT,
                "export without plan");
  agcn_plan_destroy(NULL);
  agcn_release_cached_memory();

  const float* X = (const float*)P(0x1000);
  const float* W = (const float*)P(0x2000);
  float* H = (float*)P(0x3000);
  expect_status(agcn_linear(-1, 4, 4, X, 4, W, 4, H, 4, NULL), AGCN_ERR_INVALID_ARGUMENT, "linear n");
  expect_status(agcn_linear(8, 4, 4, X, 3, W, 4, H, 4, NULL), AGCN_ERR_INVALID_ARGUMENT,
                "linear ldx");
  expect_status(agcn_linear(8, 4, 4, X, 4, W, 4, (float*)P(0x1010), 4, NULL),
                AGCN_ERR_INVALID_ARGUMENT, "linear aliasing");
  expect_status(agcn_linear(8, 4, 4, X, (int64_t)1 << 62, W, 4, H, 4, NULL),
                AGCN_ERR_INVALID_ARGUMENT, "linear extent overflow");
  expect_status(agcn_linear(0, 4, 4, NULL, 4, W, 4, NULL, 4, NULL), AGCN_OK, "empty linear");

  if (strlen(agcn_last_error()) == 0) g_fail = 1;
  if (g_fail) return 1;
  printf("c abi host check ok\n");
  return 0;
}
