/*
 * A plain C caller of libagcn (no Python, no torch): builds a small graph on
 * the host, copies it to the device with the HIP runtime, plans, runs the
 * SpMM with and without the ReLU epilogue and a GCN layer, and compares every
 * element with the CPU oracle (liboracle_agcn, linked for this check only).
 * Exit status 0 when everything matches; prints one line per check.
 *
 * Built and run by tests/test_gpu_c_abi.py.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "agcn.h"
#include "agcn_oracle.h"

#define CHECK_HIP(x)                                                                \
  do {                                                                              \
    hipError_t e_ = (x);                                                            \
    if (e_ != hipSuccess) {                                                         \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x, hipGetErrorString(e_)); \
      return 2;                                                                     \
    }                                                                               \
  } while (0)
#define CHECK_AGCN(x)                                                               \
  do {                                                                              \
    int s_ = (x);                                                                   \
    if (s_ != AGCN_OK) {                                                            \
      fprintf(stderr, "%s:%d %s: %s (%s)\n", __FILE__, __LINE__, #x,                \
              agcn_status_string(s_), agcn_last_error());                           \
      return 3;                                                                     \
    }                                                                               \
  } while (0)

static uint64_t g_state = 0x9e3779b97f4a7c15ull;
static uint32_t next_u32(void) { /* xorshift64* */
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return (uint32_t)((g_state * 0x2545f4914f6cdd1dull) >> 32);
}
static float next_f(void) { return (float)next_u32() / 4294967296.0f * 2.0f - 1.0f; }

/* |got - want| <= 1e-5 * S + 1e-7, elementwise; NaN counts as a mismatch. */
static long count_bad(const float* got, const float* want, const double* S, long m, int relu) {
  long bad = 0;
  for (long i = 0; i < m; ++i) {
    const double w = relu && want[i] < 0.0f ? 0.0 : (double)want[i];
    if (!(fabs((double)got[i] - w) <= 1e-5 * S[i] + 1e-7)) ++bad;
  }
  return bad;
}

int main(void) {
  const int32_t n = 3000, n_cols = 3000, F = 24;
  int32_t* rowptr = (int32_t*)malloc(sizeof(int32_t) * (n + 1));
  rowptr[0] = 0;
  for (int32_t i = 0; i < n; ++i) {
    int32_t d = (int32_t)(next_u32() % 40);
    if (i % 997 == 5) d = 1500 + (int32_t)(next_u32() % 1000); /* hub rows */
    if (i % 13 == 0) d = 0;                                     /* empty rows */
    rowptr[i + 1] = rowptr[i] + d;
  }
  const int64_t nnz = rowptr[n];
  int32_t* colidx = (int32_t*)malloc(sizeof(int32_t) * (size_t)nnz);
  float* vals = (float*)malloc(sizeof(float) * (size_t)nnz);
  for (int64_t e = 0; e < nnz; ++e) {
    colidx[e] = (int32_t)(next_u32() % (uint32_t)n_cols);
    vals[e] = next_f();
  }
  float* X = (float*)malloc(sizeof(float) * (size_t)n_cols * F);
  for (long i = 0; i < (long)n_cols * F; ++i) X[i] = next_f();

  int32_t *d_rowptr, *d_colidx;
  float *d_vals, *d_X, *d_Y;
  CHECK_HIP(hipMalloc((void**)&d_rowptr, sizeof(int32_t) * (n + 1)));
  CHECK_HIP(hipMalloc((void**)&d_colidx, sizeof(int32_t) * (size_t)nnz));
  CHECK_HIP(hipMalloc((void**)&d_vals, sizeof(float) * (size_t)nnz));
  CHECK_HIP(hipMalloc((void**)&d_X, sizeof(float) * (size_t)n_cols * F));
  CHECK_HIP(hipMalloc((void**)&d_Y, sizeof(float) * (size_t)n * F));
  CHECK_HIP(hipMemcpy(d_rowptr, rowptr, sizeof(int32_t) * (n + 1), hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_colidx, colidx, sizeof(int32_t) * (size_t)nnz, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_vals, vals, sizeof(float) * (size_t)nnz, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_X, X, sizeof(float) * (size_t)n_cols * F, hipMemcpyHostToDevice));
  hipStream_t st;
  CHECK_HIP(hipStreamCreate(&st));

  agcn_plan_params prm;
  agcn_default_params(&prm);
  agcn_plan_t plan = NULL;
  CHECK_AGCN(agcn_plan_create(&plan, n, n_cols, nnz, d_rowptr, d_colidx, d_vals, &prm, st));
  agcn_plan_stats stats;
  CHECK_AGCN(agcn_plan_info(plan, &stats));
  printf("plan: n_rows=%d nnz=%lld entries=%lld hub_rows=%d\n", stats.n_rows,
         (long long)stats.nnz, (long long)stats.n_entries, stats.n_hub_rows);

  /* plan metadata against the oracle, bit for bit */
  int32_t* perm = (int32_t*)malloc(sizeof(int32_t) * n);
  int32_t* meta = (int32_t*)malloc(sizeof(int32_t) * 4 * (size_t)stats.n_entries);
  CHECK_AGCN(agcn_plan_export(plan, perm, NULL, NULL, NULL, meta));
  int32_t* operm = (int32_t*)malloc(sizeof(int32_t) * n);
  int32_t* orp = (int32_t*)malloc(sizeof(int32_t) * (n + 1));
  int32_t* oci = (int32_t*)malloc(sizeof(int32_t) * (size_t)nnz);
  float* ova = (float*)malloc(sizeof(float) * (size_t)nnz);
  if (oracle_degree_sort(n, rowptr, operm) != 0 ||
      oracle_relayout(n, rowptr, colidx, vals, operm, orp, oci, ova) != 0)
    return 4;
  const int64_t cap = stats.n_entries + 16;
  int32_t* ometa = (int32_t*)malloc(sizeof(int32_t) * 4 * (size_t)cap);
  const int64_t ne = oracle_partition(n, orp, prm.max_block_waves, prm.max_wave_nzs,
                                      prm.hub_chunk_nnz, ometa, cap);
  const int plan_ok = ne == stats.n_entries && memcmp(perm, operm, sizeof(int32_t) * n) == 0 &&
                      memcmp(meta, ometa, sizeof(int32_t) * 4 * (size_t)ne) == 0;
  printf("plan metadata bit-exact: %s\n", plan_ok ? "yes" : "NO");

  size_t ws_bytes = 0;
  CHECK_AGCN(agcn_spmm_workspace_size(plan, F, &ws_bytes));
  void* d_ws = NULL;
  if (ws_bytes) CHECK_HIP(hipMalloc(&d_ws, ws_bytes));

  float* Y = (float*)malloc(sizeof(float) * (size_t)n * F);
  float* Yo = (float*)malloc(sizeof(float) * (size_t)n * F);
  double* S = (double*)malloc(sizeof(double) * (size_t)n * F);
  if (oracle_spmm(n, n_cols, F, rowptr, colidx, vals, X, F, Yo, F, NULL, S) != 0) return 4;
  long bad_total = 0;
  for (int relu = 0; relu <= 1; ++relu) {
    CHECK_AGCN(agcn_spmm_ex(plan, F, d_X, F, d_Y, F, d_ws, st,
                            relu ? AGCN_EPILOGUE_RELU : AGCN_EPILOGUE_NONE));
    CHECK_HIP(hipStreamSynchronize(st));
    CHECK_HIP(hipMemcpy(Y, d_Y, sizeof(float) * (size_t)n * F, hipMemcpyDeviceToHost));
    const long bad = count_bad(Y, Yo, S, (long)n * F, relu);
    printf("spmm%s: %ld of %ld elements out of tolerance\n", relu ? " + relu" : "", bad,
           (long)n * F);
    bad_total += bad;
  }

  /* one GCN layer: relu(A (X W)), W F x 8 */
  const int32_t fout = 8;
  float* W = (float*)malloc(sizeof(float) * F * fout);
  for (int i = 0; i < F * fout; ++i) W[i] = next_f() * 0.3f;
  float* d_W;
  CHECK_HIP(hipMalloc((void**)&d_W, sizeof(float) * F * fout));
  CHECK_HIP(hipMemcpy(d_W, W, sizeof(float) * F * fout, hipMemcpyHostToDevice));
  size_t lws = 0;
  CHECK_AGCN(agcn_gcn_workspace_size(plan, fout, &lws));
  void* d_lws = NULL;
  CHECK_HIP(hipMalloc(&d_lws, lws));
  CHECK_AGCN(agcn_gcn_layer(plan, F, fout, d_X, F, d_W, fout, d_Y, fout, d_lws, st,
                            AGCN_EPILOGUE_RELU));
  CHECK_HIP(hipStreamSynchronize(st));
  CHECK_HIP(hipMemcpy(Y, d_Y, sizeof(float) * (size_t)n * fout, hipMemcpyDeviceToHost));
  double* S2 = (double*)malloc(sizeof(double) * (size_t)n * fout);
  if (oracle_gcn_layer_rows(n, n_cols, F, fout, rowptr, colidx, vals, X, F, W, fout, 1, NULL, n,
                            Yo, S2) != 0)
    return 4;
  long lbad = 0;
  for (long i = 0; i < (long)n * fout; ++i) {
    const double tol = (1e-5 + (F + 3) * 5.9604644775390625e-08) * S2[i] + 1e-7;
    if (!(fabs((double)Y[i] - (double)Yo[i]) <= tol)) ++lbad;
  }
  printf("gcn layer: %ld of %ld elements out of tolerance\n", lbad, (long)n * fout);
  bad_total += lbad;

  agcn_plan_destroy(plan);
  agcn_release_cached_memory();
  CHECK_HIP(hipStreamDestroy(st));
  const int ok = plan_ok && bad_total == 0;
  printf("C ABI check: %s\n", ok ? "ok" : "FAILED");
  return ok ? 0 : 1;
}
