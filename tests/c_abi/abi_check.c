/*
 * A plain C caller of the library's C ABI (test program, not part of the
 * library).  It allocates device memory with the HIP C runtime API, calls
 * sparselnr_fused_sddmm_spmm and sparselnr_unfused_sddmm_spmm on a seeded
 * 1000-row matrix (row lengths 0..60 plus one 3000-nonzero row, K = L = 64),
 * and checks every row against the CPU oracle (oracle_fused_rows, linked
 * from oracle/liboracle.so) with the parity rule: per row,
 * max |A - Aref| <= 1e-4 * scale.  It also checks that argument errors come
 * back as status codes.  Prints "abi_check: ok" and exits 0 on success.
 */
#define __HIP_PLATFORM_AMD__ 1
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "sparselnr.h"

/* the oracle's C entry point (oracle/oracle.c) */
int64_t oracle_fused_rows(int64_t N, int64_t M, int64_t K, int64_t L, const int32_t *rowptr,
                          const int32_t *colidx, const float *vals, const float *C,
                          const float *D, const float *E, const int64_t *rows, int64_t nrows,
                          double *A_out, double *scale_out, double *Y_out, double *Yscale_out);

/* test-local input generator (64-bit LCG, top 24 bits -> [-1, 1)) */
static uint64_t g_state = 12345;
static uint32_t next_u32(void) {
  g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
  return (uint32_t)(g_state >> 32);
}
static float next_f(void) { return (float)(next_u32() >> 8) * (2.0f / 16777216.0f) - 1.0f; }

#define CHECK_HIP(x)                                                          \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "abi_check: %s failed (%d)\n", #x, (int)e_);            \
      return 2;                                                               \
    }                                                                         \
  } while (0)

static int compare(const char *what, const float *A, const double *ref, const double *scale,
                   int64_t N, int64_t L) {
  double worst = 0.0;
  for (int64_t i = 0; i < N; ++i) {
    double err = 0.0;
    for (int64_t l = 0; l < L; ++l) {
      const double a = A[i * L + l];
      if (!isfinite(a)) {
        fprintf(stderr, "abi_check: %s row %lld not finite\n", what, (long long)i);
        return 1;
      }
      const double d = fabs(a - ref[i * L + l]);
      if (d > err) err = d;
    }
    if (err > 1e-4 * scale[i]) {
      fprintf(stderr, "abi_check: %s row %lld err %.3e scale %.3e\n", what, (long long)i, err,
              scale[i]);
      return 1;
    }
    if (scale[i] > 0 && err / scale[i] > worst) worst = err / scale[i];
  }
  printf("abi_check: %s max err/scale %.3e\n", what, worst);
  return 0;
}

int main(void) {
  const int64_t N = 1000, M = 800, K = 64, L = 64;
  int32_t *rowptr = malloc((N + 1) * sizeof(int32_t));
  rowptr[0] = 0;
  for (int64_t i = 0; i < N; ++i) {
    int32_t n = (int32_t)(next_u32() % 61);
    if (i == 17) n = 3000; /* split over several workers */
    rowptr[i + 1] = rowptr[i] + n;
  }
  const int64_t nnz = rowptr[N];
  int32_t *colidx = malloc(nnz * sizeof(int32_t));
  float *vals = malloc(nnz * sizeof(float));
  for (int64_t p = 0; p < nnz; ++p) {
    colidx[p] = (int32_t)(next_u32() % M);
    vals[p] = next_f();
  }
  float *C = malloc(N * K * sizeof(float)), *D = malloc(M * K * sizeof(float));
  float *E = malloc(M * L * sizeof(float)), *A = malloc(N * L * sizeof(float));
  for (int64_t t = 0; t < N * K; ++t) C[t] = next_f();
  for (int64_t t = 0; t < M * K; ++t) D[t] = next_f();
  for (int64_t t = 0; t < M * L; ++t) E[t] = next_f();

  int dev_count = 0;
  if (hipGetDeviceCount(&dev_count) != hipSuccess || dev_count == 0) {
    fprintf(stderr, "abi_check: no GPU\n");
    return 3;
  }
  int32_t *d_rowptr, *d_colidx;
  float *d_vals, *d_C, *d_D, *d_E, *d_A, *d_Y;
  CHECK_HIP(hipMalloc((void **)&d_rowptr, (N + 1) * sizeof(int32_t)));
  CHECK_HIP(hipMalloc((void **)&d_colidx, nnz * sizeof(int32_t)));
  CHECK_HIP(hipMalloc((void **)&d_vals, nnz * sizeof(float)));
  CHECK_HIP(hipMalloc((void **)&d_C, N * K * sizeof(float)));
  CHECK_HIP(hipMalloc((void **)&d_D, M * K * sizeof(float)));
  CHECK_HIP(hipMalloc((void **)&d_E, M * L * sizeof(float)));
  CHECK_HIP(hipMalloc((void **)&d_A, N * L * sizeof(float)));
  CHECK_HIP(hipMalloc((void **)&d_Y, nnz * sizeof(float)));
  CHECK_HIP(hipMemcpy(d_rowptr, rowptr, (N + 1) * sizeof(int32_t), hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_colidx, colidx, nnz * sizeof(int32_t), hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_vals, vals, nnz * sizeof(float), hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_C, C, N * K * sizeof(float), hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_D, D, M * K * sizeof(float), hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_E, E, M * L * sizeof(float), hipMemcpyHostToDevice));

  /* argument errors are status codes, before any device work */
  if (sparselnr_fused_sddmm_spmm(NULL, d_colidx, d_vals, d_C, d_D, d_E, d_A, N, M, K, L, NULL) !=
      SPARSELNR_ERR_INVALID_ARG) {
    fprintf(stderr, "abi_check: NULL rowptr not rejected\n");
    return 1;
  }
  if (sparselnr_fused_sddmm_spmm(d_rowptr, d_colidx, d_vals, d_C, d_D, d_E, d_A, N, M, -1, L,
                                 NULL) != SPARSELNR_ERR_INVALID_ARG) {
    fprintf(stderr, "abi_check: negative K not rejected\n");
    return 1;
  }

  int64_t *rows = malloc(N * sizeof(int64_t));
  for (int64_t i = 0; i < N; ++i) rows[i] = i;
  double *ref = malloc(N * L * sizeof(double)), *scale = malloc(N * sizeof(double));
  oracle_fused_rows(N, M, K, L, rowptr, colidx, vals, C, D, E, rows, N, ref, scale, NULL, NULL);

  int rc = sparselnr_fused_sddmm_spmm(d_rowptr, d_colidx, d_vals, d_C, d_D, d_E, d_A, N, M, K,
                                      L, NULL);
  if (rc != SPARSELNR_OK) {
    fprintf(stderr, "abi_check: fused call: %s\n", sparselnr_status_string(rc));
    return 1;
  }
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(A, d_A, N * L * sizeof(float), hipMemcpyDeviceToHost));
  if (compare("fused", A, ref, scale, N, L)) return 1;

  CHECK_HIP(hipMemset(d_A, 0xff, N * L * sizeof(float))); /* NaN pattern: every row is written */
  rc = sparselnr_unfused_sddmm_spmm(d_rowptr, d_colidx, d_vals, d_C, d_D, d_E, d_Y, d_A, N, M, K,
                                    L, NULL);
  if (rc != SPARSELNR_OK) {
    fprintf(stderr, "abi_check: unfused call: %s\n", sparselnr_status_string(rc));
    return 1;
  }
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(A, d_A, N * L * sizeof(float), hipMemcpyDeviceToHost));
  if (compare("unfused", A, ref, scale, N, L)) return 1;

  if (sparselnr_release() != SPARSELNR_OK) return 1;
  hipFree(d_rowptr); hipFree(d_colidx); hipFree(d_vals); hipFree(d_C);
  hipFree(d_D); hipFree(d_E); hipFree(d_A); hipFree(d_Y);
  printf("abi_check: ok (N=%lld nnz=%lld K=%lld L=%lld)\n", (long long)N, (long long)nnz,
         (long long)K, (long long)L);
  return 0;
}
