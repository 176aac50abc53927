/*
 * Sanitizer driver for the CPU oracle (oracle/oracle.c) and the synthetic
 * input generators (synth/gen.c).  Test program only: tests/test_sanitize.py
 * compiles it together with both sources under
 * -fsanitize=address,undefined and runs it.  It calls every exported
 * function on small inputs, including the edge cases (no rows, no nonzeros,
 * K = 0, L = 0, duplicate and unsorted columns, chosen row subsets), and
 * checks a few properties that tie the functions together, so that an
 * out-of-bounds access, a use of freed memory, a leak or undefined integer
 * arithmetic on any of these paths stops the run.  Prints
 * "sanitize_check: ok" on success.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* synth/gen.c */
uint64_t synth_draw(uint64_t seed, uint64_t id, uint64_t n);
void synth_uniform_f32(uint64_t seed, uint64_t id, double lo, double hi, int64_t n, float *out);
void synth_normal_f32(uint64_t seed, uint64_t id, int64_t n, float *out);
int synth_csr_fixed_degree(uint64_t seed, uint64_t id, int64_t N, int64_t M, int64_t deg,
                           int32_t *rowptr, int32_t *colidx);
int64_t synth_rmat(uint64_t seed, uint64_t id, int levels, int64_t samples, double a, double b,
                   double c, int32_t *rowptr, int32_t *colidx);
int64_t synth_stencil27(int64_t n, int32_t *rowptr, int32_t *colidx);

/* oracle/oracle.c */
int64_t oracle_sddmm(int64_t N, int64_t M, int64_t K, const int32_t *rowptr,
                     const int32_t *colidx, const float *vals, const float *C, const float *D,
                     double *Y, double *Yscale);
int64_t oracle_spmm(int64_t N, int64_t M, int64_t L, const int32_t *rowptr,
                    const int32_t *colidx, const double *Y, const float *E, double *A,
                    const double *Yabs, double *Ascale);
int64_t oracle_fused_rows(int64_t N, int64_t M, int64_t K, int64_t L, const int32_t *rowptr,
                          const int32_t *colidx, const float *vals, const float *C,
                          const float *D, const float *E, const int64_t *rows, int64_t nrows,
                          double *A_out, double *scale_out, double *Y_out, double *Yscale_out);
int64_t oracle_sddmm_spmm_gemm_rows(int64_t K, int64_t L, int64_t Mo, const int32_t *rowptr,
                                    const int32_t *colidx, const float *vals, const float *C,
                                    const float *D, const float *F, const float *Wm,
                                    const int64_t *rows, int64_t nrows, double *out,
                                    double *scale_out);
int64_t oracle_spmm_gemm_rows(int64_t K, int64_t L, const int32_t *rowptr, const int32_t *colidx,
                              const float *vals, const float *C, const float *D,
                              const int64_t *rows, int64_t nrows, double *out, double *scale_out);
int64_t oracle_spmmh_gemm_rows(int64_t J, int64_t L, const int32_t *rowptr,
                               const int32_t *colidx, const float *vals, const float *C,
                               const float *D, const float *E, const int64_t *rows,
                               int64_t nrows, double *out, double *scale_out);
int64_t oracle_fused_rows_dt(int64_t M, int64_t K, int64_t L, const int32_t *rowptr,
                             const int32_t *colidx, const float *vals, const float *C,
                             const float *Dt, const float *E, const int64_t *rows, int64_t nrows,
                             double *out, double *scale_out);

static int g_fail = 0;
#define CHECK(cond, ...)                                   \
  do {                                                     \
    if (!(cond)) {                                         \
      fprintf(stderr, "sanitize_check: " __VA_ARGS__);     \
      fprintf(stderr, "\n");                               \
      g_fail = 1;                                          \
    }                                                      \
  } while (0)

static float *fill(uint64_t id, int64_t n) {
  float *p = malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
  synth_uniform_f32(7, id, -1.0, 1.0, n, p);
  return p;
}

/* Every oracle function on one CSR matrix (N x M), widths K, L, Mo. */
static void oracle_suite(const char *what, int64_t N, int64_t M, const int32_t *rowptr,
                         const int32_t *colidx, int64_t K, int64_t L, int64_t Mo) {
  const int64_t nnz = rowptr[N];
  float *vals = fill(20, nnz), *C = fill(21, N * K), *D = fill(22, M * K), *E = fill(23, M * L);
  float *W = fill(24, L * Mo), *H = fill(25, M * L), *Dk = fill(26, K * L);
  double *Y = malloc(sizeof(double) * (size_t)(nnz + 1));
  double *Ys = malloc(sizeof(double) * (size_t)(nnz + 1));
  double *A = malloc(sizeof(double) * (size_t)(N * L + 1));
  double *As = malloc(sizeof(double) * (size_t)(N + 1));
  double *F = malloc(sizeof(double) * (size_t)(N * L + 1));
  double *Fs = malloc(sizeof(double) * (size_t)(N + 1));
  double *Fy = malloc(sizeof(double) * (size_t)(nnz + 1));
  double *Fys = malloc(sizeof(double) * (size_t)(nnz + 1));
  double *O = malloc(sizeof(double) * (size_t)(N * (Mo > L ? Mo : L) + 1));
  double *Os = malloc(sizeof(double) * (size_t)(N + 1));
  int64_t *rows = malloc(sizeof(int64_t) * (size_t)(N + 1));
  for (int64_t i = 0; i < N; ++i) rows[i] = i;

  /* Figure 2a then 2b against the row-by-row form */
  const int64_t ops_a = oracle_sddmm(N, M, K, rowptr, colidx, vals, C, D, Y, Ys);
  const int64_t ops_b = oracle_spmm(N, M, L, rowptr, colidx, Y, E, A, Ys, As);
  const int64_t ops_f = oracle_fused_rows(N, M, K, L, rowptr, colidx, vals, C, D, E, rows, N, F,
                                          Fs, Fy, Fys);
  CHECK(ops_a == nnz * K && ops_b == nnz * L && ops_f == nnz * (K + L), "%s: op counts", what);
  CHECK(memcmp(Y, Fy, sizeof(double) * (size_t)nnz) == 0, "%s: SDDMM values differ", what);
  CHECK(memcmp(Ys, Fys, sizeof(double) * (size_t)nnz) == 0, "%s: SDDMM scales differ", what);
  CHECK(memcmp(A, F, sizeof(double) * (size_t)(N * L)) == 0, "%s: rows differ", what);
  CHECK(memcmp(As, Fs, sizeof(double) * (size_t)N) == 0, "%s: row scales differ", what);
  /* without the optional outputs */
  oracle_sddmm(N, M, K, rowptr, colidx, vals, C, D, Y, NULL);
  oracle_spmm(N, M, L, rowptr, colidx, Y, E, A, NULL, NULL);
  /* a subset of rows, in another order, with a repeat */
  if (N >= 1) {
    const int64_t sub[4] = {N - 1, 0, N / 2, N / 2};
    int64_t ny = 0;
    for (int t = 0; t < 4; ++t) ny += rowptr[sub[t] + 1] - rowptr[sub[t]];
    double *SA = malloc(sizeof(double) * (size_t)(4 * L + 1));
    double *Ss = malloc(sizeof(double) * 4);
    double *Sy = malloc(sizeof(double) * (size_t)(ny + 1));
    oracle_fused_rows(N, M, K, L, rowptr, colidx, vals, C, D, E, sub, 4, SA, Ss, Sy, NULL);
    CHECK(memcmp(SA, A + (N - 1) * L, sizeof(double) * (size_t)L) == 0, "%s: subset row", what);
    CHECK(Ss[1] == As[0] && Ss[2] == Ss[3], "%s: subset scales", what);
    free(SA); free(Ss); free(Sy);
  }
  /* transposed D gives the plain result */
  float *Dt = malloc(sizeof(float) * (size_t)(M * K + 1));
  for (int64_t j = 0; j < M; ++j)
    for (int64_t k = 0; k < K; ++k) Dt[k * M + j] = D[j * K + k];
  oracle_fused_rows_dt(M, K, L, rowptr, colidx, vals, C, Dt, E, rows, N, O, Os);
  oracle_fused_rows(N, M, K, L, rowptr, colidx, vals, C, D, E, rows, N, F, Fs, NULL, NULL);
  CHECK(memcmp(O, F, sizeof(double) * (size_t)(N * L)) == 0, "%s: transposed D differs", what);
  /* Section 6.2 products */
  oracle_sddmm_spmm_gemm_rows(K, L, Mo, rowptr, colidx, vals, C, D, H, W, rows, N, O, Os);
  oracle_spmm_gemm_rows(K, L, rowptr, colidx, vals, D, Dk, rows, N, O, Os);
  oracle_spmmh_gemm_rows(K, L, rowptr, colidx, vals, D, D, Dk, rows, N, O, Os);
  for (int64_t i = 0; i < N; ++i) CHECK(Os[i] >= 0.0 && isfinite(Os[i]), "%s: scale", what);

  free(vals); free(C); free(D); free(E); free(W); free(H); free(Dk); free(Dt);
  free(Y); free(Ys); free(A); free(As); free(F); free(Fs); free(Fy); free(Fys);
  free(O); free(Os); free(rows);
}

int main(void) {
  setvbuf(stdout, NULL, _IONBF, 0);
  /* counter-based draws and dense fills, odd lengths */
  CHECK(synth_draw(0, 0, 0) == synth_draw(0, 0, 0), "draw not deterministic");
  float *u = malloc(sizeof(float) * 1001);
  synth_uniform_f32(1, 2, -1.0, 1.0, 1001, u);
  for (int t = 0; t < 1001; ++t) CHECK(u[t] >= -1.0f && u[t] < 1.0f, "uniform range");
  synth_normal_f32(1, 3, 1001, u);
  for (int t = 0; t < 1001; ++t) CHECK(isfinite(u[t]), "normal not finite");
  synth_normal_f32(1, 3, 0, u);
  free(u);

  /* fixed degree: rows of distinct sorted columns */
  {
    const int64_t N = 300, M = 40, deg = 12;
    int32_t *rp = malloc(sizeof(int32_t) * (N + 1)), *ci = malloc(sizeof(int32_t) * N * deg);
    CHECK(synth_csr_fixed_degree(5, 1, N, M, deg, rp, ci) == 0, "fixed degree failed");
    for (int64_t i = 0; i < N; ++i)
      for (int64_t p = rp[i] + 1; p < rp[i + 1]; ++p) CHECK(ci[p - 1] < ci[p], "not sorted");
    CHECK(synth_csr_fixed_degree(5, 1, N, M, M + 1, rp, ci) != 0, "deg > M accepted");
    oracle_suite("fixed degree", N, M, rp, ci, 8, 12, 5);
    free(rp); free(ci);
  }
  /* R-MAT: merged duplicates, power-law rows */
  {
    const int levels = 10;
    const int64_t N = (int64_t)1 << levels, samples = 16 * N;
    int32_t *rp = malloc(sizeof(int32_t) * (N + 1)), *ci = malloc(sizeof(int32_t) * samples);
    const int64_t nnz = synth_rmat(3, 1, levels, samples, 0.57, 0.19, 0.19, rp, ci);
    CHECK(nnz > 0 && nnz <= samples && rp[N] == nnz, "rmat nnz");
    for (int64_t i = 0; i < N; ++i)
      for (int64_t p = rp[i] + 1; p < rp[i + 1]; ++p) CHECK(ci[p - 1] < ci[p], "rmat order");
    oracle_suite("rmat", N, N, rp, ci, 16, 4, 3);
    /* unsorted and duplicate columns: reverse every row, repeat a column */
    for (int64_t i = 0; i < N; ++i)
      for (int64_t a = rp[i], b = rp[i + 1] - 1; a < b; ++a, --b) {
        const int32_t t = ci[a]; ci[a] = ci[b]; ci[b] = t;
      }
    for (int64_t i = 0; i < N; ++i)
      if (rp[i + 1] - rp[i] >= 2) ci[rp[i]] = ci[rp[i] + 1];
    oracle_suite("rmat, unsorted with duplicates", N, N, rp, ci, 5, 7, 2);
    CHECK(synth_rmat(3, 1, 31, 10, 0.57, 0.19, 0.19, rp, ci) == -1, "levels > 30 accepted");
    free(rp); free(ci);
  }
  /* stencil: sizes 0, 1 and 6 */
  for (int64_t n = 0; n <= 6; n += (n == 1 ? 5 : 1)) {
    const int64_t N = n * n * n, side = n > 1 ? 3 * n - 2 : n;
    int32_t *rp = malloc(sizeof(int32_t) * (N + 1));
    int32_t *ci = malloc(sizeof(int32_t) * (side * side * side + 1));
    const int64_t nnz = synth_stencil27(n, rp, ci);
    CHECK(nnz == side * side * side, "stencil nnz %lld", (long long)nnz);
    if (N > 0) oracle_suite("stencil", N, N, rp, ci, 4, 9, 4);
    free(rp); free(ci);
  }
  /* degenerate sizes: empty rows only, K = 0, L = 0 */
  {
    int32_t rp[6] = {0, 0, 0, 0, 0, 0}, ci[1] = {0};
    oracle_suite("no nonzeros", 5, 3, rp, ci, 4, 4, 2);
    int32_t rp2[4] = {0, 2, 2, 3}, ci2[3] = {1, 0, 2};
    oracle_suite("K = 0", 3, 3, rp2, ci2, 0, 4, 2);
    oracle_suite("L = 0", 3, 3, rp2, ci2, 4, 0, 0);
  }
  if (g_fail) return 1;
  printf("sanitize_check: ok\n");
  return 0;
}
