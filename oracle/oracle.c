/*
 * CPU ORACLE for A(i,l) = sum_j sum_k B(i,j) * C(i,k) * D(j,k) * E(j,l),
 * B in CSR.  TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the
 * benchmark's CPU-baseline leg call it; the GPU library never links, loads or
 * calls it, and it shares no code with the GPU library.
 *
 * The method (the fused schedule of the paper's Figure 2d) reaches exactly the
 * plain result A = (B .* (C D^T)) E restricted to the nonzeros of B (Section
 * 3.1), only in another loop order.  So the oracle is that definition written
 * out in its two-kernel form: an SDDMM into a value array with the structure
 * of B (Figure 2a; Section 3.1.2 notes the result has exactly B's structure),
 * followed by a row-wise SpMM over that array (Figure 2b).  The paper states
 * that running 2b after 2a gives the same result as the fused forms (caption
 * of Figure 2).
 *
 * Precision: inputs are fp32; every product and sum is taken in fp64 (the
 * paper's listings accumulate in double).  Sums run in index order: k
 * ascending, then nonzeros p ascending.  Operand orientation follows the code
 * of Figure 2 and the text of Section 3.1: C is N x K indexed C[i,k], D is
 * M x K indexed D[j,k], E is M x L indexed E[j,l]; all dense arrays are
 * row-major.  A is overwritten (the listings add into a zero-initialised A).
 *
 * Besides values the oracle returns, per row, the scale used by the parity
 * tolerance:  scale_i = max_l sum_p |b_p| * (sum_k |C_ik| |D_jk|) * |E_jl|,
 * i.e. the same computation on absolute values, and it counts the
 * multiply-adds it performs (Section 3.1.3 gives O(nnz (K + L)) for this
 * schedule).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_abi_version(void) { return 1; }

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Figure 2a: Y[p] = b_p * sum_k C[i,k] * D[j,k] for every nonzero p of row i,
 * j = colidx[p].  If Yscale is not NULL it receives |b_p| sum_k |C_ik||D_jk|.
 * Returns the number of multiply-adds in the k loops (nnz * K). */
int64_t oracle_sddmm(int64_t N, int64_t M, int64_t K, const int32_t *rowptr,
                     const int32_t *colidx, const float *vals, const float *C,
                     const float *D, double *Y, double *Yscale) {
  (void)M;
  int64_t ops = 0;
#pragma omp parallel for schedule(dynamic, 64) reduction(+ : ops)
  for (int64_t i = 0; i < N; ++i) {
    for (int64_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
      const int64_t j = colidx[p];
      double dot = 0.0, adot = 0.0;
      for (int64_t k = 0; k < K; ++k) {
        const double c = (double)C[i * K + k], d = (double)D[j * K + k];
        dot += c * d;
        adot += fabs(c) * fabs(d);
        ++ops;
      }
      Y[p] = (double)vals[p] * dot;
      if (Yscale) Yscale[p] = fabs((double)vals[p]) * adot;
    }
  }
  return ops;
}

/* Figure 2b: A[i,l] = sum_p Y[p] * E[j,l] over the nonzeros p of row i
 * (A overwritten).  If Yabs is not NULL, Ascale receives
 * max_l sum_p Yabs[p] * |E[j,l]| per row.  Returns the multiply-adds (nnz*L). */
int64_t oracle_spmm(int64_t N, int64_t M, int64_t L, const int32_t *rowptr,
                    const int32_t *colidx, const double *Y, const float *E,
                    double *A, const double *Yabs, double *Ascale) {
  (void)M;
  int64_t ops = 0;
#pragma omp parallel reduction(+ : ops)
  {
    double *sacc = (double *)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
#pragma omp for schedule(dynamic, 64)
    for (int64_t i = 0; i < N; ++i) {
      double *a = A + i * L;
      for (int64_t l = 0; l < L; ++l) { a[l] = 0.0; sacc[l] = 0.0; }
      for (int64_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
        const int64_t j = colidx[p];
        for (int64_t l = 0; l < L; ++l) {
          a[l] += Y[p] * (double)E[j * L + l];
          if (Yabs) sacc[l] += Yabs[p] * fabs((double)E[j * L + l]);
          ++ops;
        }
      }
      if (Ascale) {
        double m = 0.0;
        for (int64_t l = 0; l < L; ++l) m = sacc[l] > m ? sacc[l] : m;
        Ascale[i] = m;
      }
    }
    free(sacc);
  }
  return ops;
}

/* The result on a list of rows, computed row by row as the two kernels above
 * do it: SDDMM of the row into a row-local value array, then the row's SpMM.
 * rows[r] selects the row; A_out is nrows x L (fp64), scale_out is nrows.
 * If Y_out is not NULL it receives the row's SDDMM values, rows concatenated
 * in list order (Yscale_out likewise, may be NULL).
 * Returns the multiply-adds performed (sum of row lengths times K + L). */
int64_t oracle_fused_rows(int64_t N, int64_t M, int64_t K, int64_t L,
                          const int32_t *rowptr, const int32_t *colidx,
                          const float *vals, const float *C, const float *D,
                          const float *E, const int64_t *rows, int64_t nrows,
                          double *A_out, double *scale_out, double *Y_out,
                          double *Yscale_out) {
  (void)N; (void)M;
  int64_t *yoff = NULL;
  if (Y_out || Yscale_out) {
    yoff = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nrows + 1));
    yoff[0] = 0;
    for (int64_t r = 0; r < nrows; ++r)
      yoff[r + 1] = yoff[r] + (rowptr[rows[r] + 1] - rowptr[rows[r]]);
  }
  int64_t ops = 0;
#pragma omp parallel reduction(+ : ops)
  {
    int64_t cap = 0;
    double *y = NULL, *yabs = NULL;
    double *sacc = (double *)malloc(sizeof(double) * (size_t)(L > 0 ? L : 1));
#pragma omp for schedule(dynamic, 64)
    for (int64_t r = 0; r < nrows; ++r) {
      const int64_t i = rows[r];
      const int64_t p0 = rowptr[i], p1 = rowptr[i + 1], n = p1 - p0;
      if (n > cap) {
        cap = n;
        y = (double *)realloc(y, sizeof(double) * (size_t)cap);
        yabs = (double *)realloc(yabs, sizeof(double) * (size_t)cap);
      }
      /* producer: the row's SDDMM values */
      for (int64_t p = p0; p < p1; ++p) {
        const int64_t j = colidx[p];
        double dot = 0.0, adot = 0.0;
        for (int64_t k = 0; k < K; ++k) {
          const double c = (double)C[i * K + k], d = (double)D[j * K + k];
          dot += c * d;
          adot += fabs(c) * fabs(d);
          ++ops;
        }
        y[p - p0] = (double)vals[p] * dot;
        yabs[p - p0] = fabs((double)vals[p]) * adot;
      }
      /* consumer: the row's SpMM */
      double *a = A_out + r * L;
      for (int64_t l = 0; l < L; ++l) { a[l] = 0.0; sacc[l] = 0.0; }
      for (int64_t p = p0; p < p1; ++p) {
        const int64_t j = colidx[p];
        for (int64_t l = 0; l < L; ++l) {
          const double e = (double)E[j * L + l];
          a[l] += y[p - p0] * e;
          sacc[l] += yabs[p - p0] * fabs(e);
          ++ops;
        }
      }
      double m = 0.0;
      for (int64_t l = 0; l < L; ++l) m = sacc[l] > m ? sacc[l] : m;
      scale_out[r] = m;
      if (Y_out)
        for (int64_t q = 0; q < n; ++q) Y_out[yoff[r] + q] = y[q];
      if (Yscale_out)
        for (int64_t q = 0; q < n; ++q) Yscale_out[yoff[r] + q] = yabs[q];
    }
    free(y);
    free(yabs);
    free(sacc);
  }
  free(yoff);
  return ops;
}

/* ------------------------------------------------------------------------
 * Further computations of the paper's Section 6.2 benchmarks, each written
 * in its fused loop order on the chosen rows, fp64, with the abs-value scale
 * of the result (the same loops on |.|).  out is nrows x (output width).
 */

/* Scratch of one thread: two vectors of length n. */
static int ensure(double **a, double **b, int64_t *cap, int64_t n) {
  if (n <= *cap) return 0;
  *a = (double *)realloc(*a, sizeof(double) * (size_t)n);
  *b = (double *)realloc(*b, sizeof(double) * (size_t)n);
  *cap = n;
  return (*a && *b) ? 0 : 1;
}

/* <SDDMM, SpMM, GEMM>: A(i,m) = sum_{j,k,l} B(i,j) C(i,k) D(j,k) F(j,l) W(l,m).
 * Per row: t_l = sum_p b_p (sum_k C_ik D_jk) F_jl (the <SDDMM, SpMM> row),
 * then A_im = sum_l t_l W_lm.  C: N x K, D: M x K, F: M x L, W: L x Mo. */
int64_t oracle_sddmm_spmm_gemm_rows(int64_t K, int64_t L, int64_t Mo, const int32_t *rowptr,
                                    const int32_t *colidx, const float *vals, const float *C,
                                    const float *D, const float *F, const float *Wm,
                                    const int64_t *rows, int64_t nrows, double *out,
                                    double *scale_out) {
  int64_t ops = 0;
#pragma omp parallel reduction(+ : ops)
  {
    double *t = NULL, *ta = NULL;
    int64_t cap = 0;
    ensure(&t, &ta, &cap, L > 0 ? L : 1);
#pragma omp for schedule(dynamic, 64)
    for (int64_t r = 0; r < nrows; ++r) {
      const int64_t i = rows[r];
      for (int64_t l = 0; l < L; ++l) { t[l] = 0.0; ta[l] = 0.0; }
      for (int64_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
        const int64_t j = colidx[p];
        double dot = 0.0, adot = 0.0;
        for (int64_t k = 0; k < K; ++k) {
          const double c = (double)C[i * K + k], d = (double)D[j * K + k];
          dot += c * d;
          adot += fabs(c) * fabs(d);
          ++ops;
        }
        const double y = (double)vals[p] * dot, ya = fabs((double)vals[p]) * adot;
        for (int64_t l = 0; l < L; ++l) {
          t[l] += y * (double)F[j * L + l];
          ta[l] += ya * fabs((double)F[j * L + l]);
          ++ops;
        }
      }
      double m_scale = 0.0;
      for (int64_t m = 0; m < Mo; ++m) {
        double s = 0.0, sa = 0.0;
        for (int64_t l = 0; l < L; ++l) {
          s += t[l] * (double)Wm[l * Mo + m];
          sa += ta[l] * fabs((double)Wm[l * Mo + m]);
          ++ops;
        }
        out[r * Mo + m] = s;
        m_scale = sa > m_scale ? sa : m_scale;
      }
      scale_out[r] = m_scale;
    }
    free(t);
    free(ta);
  }
  return ops;
}

/* <SpMM, GEMM>: A(i,l) = sum_{j,k} B(i,j) C(j,k) D(k,l).  Per row: the SpMM
 * row t_k = sum_p b_p C_jk, then A_il = sum_k t_k D_kl.  C: M x K, D: K x L. */
int64_t oracle_spmm_gemm_rows(int64_t K, int64_t L, const int32_t *rowptr,
                              const int32_t *colidx, const float *vals, const float *C,
                              const float *D, const int64_t *rows, int64_t nrows, double *out,
                              double *scale_out) {
  int64_t ops = 0;
#pragma omp parallel reduction(+ : ops)
  {
    double *t = NULL, *ta = NULL;
    int64_t cap = 0;
    ensure(&t, &ta, &cap, K > 0 ? K : 1);
#pragma omp for schedule(dynamic, 64)
    for (int64_t r = 0; r < nrows; ++r) {
      const int64_t i = rows[r];
      for (int64_t k = 0; k < K; ++k) { t[k] = 0.0; ta[k] = 0.0; }
      for (int64_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
        const int64_t j = colidx[p];
        const double b = (double)vals[p];
        for (int64_t k = 0; k < K; ++k) {
          t[k] += b * (double)C[j * K + k];
          ta[k] += fabs(b) * fabs((double)C[j * K + k]);
          ++ops;
        }
      }
      double m_scale = 0.0;
      for (int64_t l = 0; l < L; ++l) {
        double s = 0.0, sa = 0.0;
        for (int64_t k = 0; k < K; ++k) {
          s += t[k] * (double)D[k * L + l];
          sa += ta[k] * fabs((double)D[k * L + l]);
          ++ops;
        }
        out[r * L + l] = s;
        m_scale = sa > m_scale ? sa : m_scale;
      }
      scale_out[r] = m_scale;
    }
    free(t);
    free(ta);
  }
  return ops;
}

/* <SpMMH, GEMM>: A(i,l) = sum_{k,j} B(i,k) C(k,j) D(k,j) E(j,l).  Per row: the
 * Hadamard SpMM row t_j = sum_p b_p C_kj D_kj (k = colidx[p]), then
 * A_il = sum_j t_j E_jl.  C, D: M x J, E: J x L. */
int64_t oracle_spmmh_gemm_rows(int64_t J, int64_t L, const int32_t *rowptr,
                               const int32_t *colidx, const float *vals, const float *C,
                               const float *D, const float *E, const int64_t *rows,
                               int64_t nrows, double *out, double *scale_out) {
  int64_t ops = 0;
#pragma omp parallel reduction(+ : ops)
  {
    double *t = NULL, *ta = NULL;
    int64_t cap = 0;
    ensure(&t, &ta, &cap, J > 0 ? J : 1);
#pragma omp for schedule(dynamic, 64)
    for (int64_t r = 0; r < nrows; ++r) {
      const int64_t i = rows[r];
      for (int64_t jj = 0; jj < J; ++jj) { t[jj] = 0.0; ta[jj] = 0.0; }
      for (int64_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
        const int64_t k = colidx[p];
        const double b = (double)vals[p];
        for (int64_t jj = 0; jj < J; ++jj) {
          const double c = (double)C[k * J + jj], d = (double)D[k * J + jj];
          t[jj] += b * c * d;
          ta[jj] += fabs(b) * fabs(c) * fabs(d);
          ++ops;
        }
      }
      double m_scale = 0.0;
      for (int64_t l = 0; l < L; ++l) {
        double s = 0.0, sa = 0.0;
        for (int64_t jj = 0; jj < J; ++jj) {
          s += t[jj] * (double)E[jj * L + l];
          sa += ta[jj] * fabs((double)E[jj * L + l]);
          ++ops;
        }
        out[r * L + l] = s;
        m_scale = sa > m_scale ? sa : m_scale;
      }
      scale_out[r] = m_scale;
    }
    free(t);
    free(ta);
  }
  return ops;
}

/* <SDDMM, SpMM> with D stored transposed (Section 4.3.1): Dt is K x M and
 * D(j,k) is read as Dt[k*M + j].  Otherwise as oracle_fused_rows. */
int64_t oracle_fused_rows_dt(int64_t M, int64_t K, int64_t L, const int32_t *rowptr,
                             const int32_t *colidx, const float *vals, const float *C,
                             const float *Dt, const float *E, const int64_t *rows,
                             int64_t nrows, double *out, double *scale_out) {
  int64_t ops = 0;
#pragma omp parallel reduction(+ : ops)
  {
    double *t = NULL, *ta = NULL;
    int64_t cap = 0;
    ensure(&t, &ta, &cap, L > 0 ? L : 1);
#pragma omp for schedule(dynamic, 64)
    for (int64_t r = 0; r < nrows; ++r) {
      const int64_t i = rows[r];
      for (int64_t l = 0; l < L; ++l) { t[l] = 0.0; ta[l] = 0.0; }
      for (int64_t p = rowptr[i]; p < rowptr[i + 1]; ++p) {
        const int64_t j = colidx[p];
        double dot = 0.0, adot = 0.0;
        for (int64_t k = 0; k < K; ++k) {
          const double c = (double)C[i * K + k], d = (double)Dt[k * M + j];
          dot += c * d;
          adot += fabs(c) * fabs(d);
          ++ops;
        }
        const double y = (double)vals[p] * dot, ya = fabs((double)vals[p]) * adot;
        for (int64_t l = 0; l < L; ++l) {
          t[l] += y * (double)E[j * L + l];
          ta[l] += ya * fabs((double)E[j * L + l]);
          ++ops;
        }
      }
      double m_scale = 0.0;
      for (int64_t l = 0; l < L; ++l) {
        out[r * L + l] = t[l];
        m_scale = ta[l] > m_scale ? ta[l] : m_scale;
      }
      scale_out[r] = m_scale;
    }
    free(t);
    free(ta);
  }
  return ops;
}
