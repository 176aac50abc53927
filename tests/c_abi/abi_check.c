/*
 * A plain C caller of the library's C ABI (test program, not part of the
 * library).  It allocates device memory with the HIP C runtime API, calls
 * sparselnr_fused_sddmm_spmm and sparselnr_unfused_sddmm_spmm on a seeded
 * 1000-row matrix (row lengths 0..60 plus one 3000-nonzero row, K = L = 64),
 * and checks every row against the CPU oracle (oracle_fused_rows) with the
 * parity rule: per row, max |A - Aref| <= 1e-4 * scale.  It also checks that
 * argument errors come back as status codes.  Prints "abi_check: ok" and
 * exits 0 on success.
 *
 * The program reports where it is: stdout is unbuffered, a marker goes to
 * stderr before every phase, and an exit handler prints the last marker, so
 * a crash anywhere (exit-time teardown included) leaves the phase it
 * happened in.
 *
 * With --host-only it runs only the phases that need no GPU (input
 * generation, the oracle, the comparison routine and the argument-error
 * calls, which return before any HIP call) and exits; this is the mode the
 * sanitizer build runs on a host without a GPU.
 */
#define __HIP_PLATFORM_AMD__ 1
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "sparselnr.h"

/* the oracle's C entry point (oracle/oracle.c) */
int64_t oracle_fused_rows(int64_t N, int64_t M, int64_t K, int64_t L, const int32_t *rowptr,
                          const int32_t *colidx, const float *vals, const float *C,
                          const float *D, const float *E, const int64_t *rows, int64_t nrows,
                          double *A_out, double *scale_out, double *Y_out, double *Yscale_out);

static const char *g_phase = "start";

static void phase(const char *name) {
  g_phase = name;
  fprintf(stderr, "abi_check: phase %s\n", name);
}

static void at_exit_marker(void) {
  fprintf(stderr, "abi_check: exit handlers reached (last phase: %s)\n", g_phase);
}

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

int main(int argc, char **argv) {
  setvbuf(stdout, NULL, _IONBF, 0);
  atexit(at_exit_marker);
  const int host_only = argc > 1 && strcmp(argv[1], "--host-only") == 0;
  const int64_t N = 1000, M = 800, K = 64, L = 64;

  phase("inputs");
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

  phase("oracle");
  int64_t *rows = malloc(N * sizeof(int64_t));
  for (int64_t i = 0; i < N; ++i) rows[i] = i;
  double *ref = malloc(N * L * sizeof(double)), *scale = malloc(N * sizeof(double));
  oracle_fused_rows(N, M, K, L, rowptr, colidx, vals, C, D, E, rows, N, ref, scale, NULL, NULL);

  phase("compare routine on the oracle's own rows");
  for (int64_t t = 0; t < N * L; ++t) A[t] = (float)ref[t];
  if (compare("oracle rounded to fp32", A, ref, scale, N, L)) return 1;

  /* argument errors are status codes, returned before any HIP call (the
   * pointers below are never dereferenced) */
  phase("argument errors");
  void *fake = (void *)(uintptr_t)0x1000;
  if (sparselnr_fused_sddmm_spmm(NULL, fake, fake, fake, fake, fake, fake, N, M, K, L, NULL) !=
      SPARSELNR_ERR_INVALID_ARG) {
    fprintf(stderr, "abi_check: NULL rowptr not rejected\n");
    return 1;
  }
  if (sparselnr_fused_sddmm_spmm(fake, fake, fake, fake, fake, fake, fake, N, M, -1, L, NULL) !=
      SPARSELNR_ERR_INVALID_ARG) {
    fprintf(stderr, "abi_check: negative K not rejected\n");
    return 1;
  }
  if (sparselnr_fused_sddmm_spmm_dt(fake, fake, fake, fake, fake, fake, NULL, N, M, K, L, NULL) !=
      SPARSELNR_ERR_INVALID_ARG) {
    fprintf(stderr, "abi_check: NULL A (transposed D) not rejected\n");
    return 1;
  }
  if (sparselnr_unfused_sddmm_spmm(fake, fake, fake, fake, fake, fake, NULL, fake, N, M, K, L,
                                   NULL) != SPARSELNR_ERR_INVALID_ARG) {
    fprintf(stderr, "abi_check: NULL Y not rejected\n");
    return 1;
  }
  if (host_only) {
    phase("done (host only)");
    printf("abi_check: host phases ok (N=%lld nnz=%lld K=%lld L=%lld)\n", (long long)N,
           (long long)nnz, (long long)K, (long long)L);
    free(rowptr); free(colidx); free(vals); free(C); free(D); free(E); free(A);
    free(rows); free(ref); free(scale);
    return 0;
  }

  phase("device setup");
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

  phase("fused call");
  CHECK_HIP(hipMemset(d_A, 0xff, N * L * sizeof(float))); /* NaN pattern: every row is written */
  int rc = sparselnr_fused_sddmm_spmm(d_rowptr, d_colidx, d_vals, d_C, d_D, d_E, d_A, N, M, K,
                                      L, NULL);
  if (rc != SPARSELNR_OK) {
    fprintf(stderr, "abi_check: fused call: %s\n", sparselnr_status_string(rc));
    return 1;
  }
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(A, d_A, N * L * sizeof(float), hipMemcpyDeviceToHost));
  if (compare("fused", A, ref, scale, N, L)) return 1;

  phase("unfused call");
  CHECK_HIP(hipMemset(d_A, 0xff, N * L * sizeof(float)));
  rc = sparselnr_unfused_sddmm_spmm(d_rowptr, d_colidx, d_vals, d_C, d_D, d_E, d_Y, d_A, N, M, K,
                                    L, NULL);
  if (rc != SPARSELNR_OK) {
    fprintf(stderr, "abi_check: unfused call: %s\n", sparselnr_status_string(rc));
    return 1;
  }
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(A, d_A, N * L * sizeof(float), hipMemcpyDeviceToHost));
  if (compare("unfused", A, ref, scale, N, L)) return 1;

  phase("release and free");
  if (sparselnr_release() != SPARSELNR_OK) return 1;
  CHECK_HIP(hipFree(d_rowptr));
  CHECK_HIP(hipFree(d_colidx));
  CHECK_HIP(hipFree(d_vals));
  CHECK_HIP(hipFree(d_C));
  CHECK_HIP(hipFree(d_D));
  CHECK_HIP(hipFree(d_E));
  CHECK_HIP(hipFree(d_A));
  CHECK_HIP(hipFree(d_Y));
  free(rowptr); free(colidx); free(vals); free(C); free(D); free(E); free(A);
  free(rows); free(ref); free(scale);
  phase("return from main");
  printf("abi_check: ok (N=%lld nnz=%lld K=%lld L=%lld)\n", (long long)N, (long long)nnz,
         (long long)K, (long long)L);
  return 0;
}
