/*
 * sparselnr.h -- C ABI of the MI355X (gfx950) fused SDDMM->SpMM library.
 *
 * Computes, for a sparse matrix B in CSR form and dense C, D, E,
 *
 *     A(i,l) = sum_{j,k} B(i,j) * C(i,k) * D(j,k) * E(j,l)
 *
 * the <SDDMM, SpMM> computation of Dias et al., "SparseLNR: Accelerating
 * Sparse Tensor Computations Using Loop Nest Restructuring" (ICS 2022),
 * Section 3.1 and Figure 2.  The fused entry point runs the paper's
 * loop-fused, kernel-distributed schedule (Figure 2d; Section 3.1.3): one
 * pass over the rows of B in which, for every nonzero, a scalar SDDMM value
 * is produced and immediately consumed by the SpMM update of the row, so no
 * nnz-sized intermediate exists (Section 4.2: the temporary of this
 * expression is a scalar because no index below the nest boundary is shared
 * by producer and consumer).  The unfused entry points are the paper's
 * separate-kernel schedule (Figures 2a and 2b, Section 3.1.2), kept as the
 * in-library comparison.
 *
 * Layouts (all row-major, densely packed, fp32 values, int32 indices):
 *   rowptr  int32[N+1]   CSR row offsets; rowptr[0] = 0, non-decreasing
 *   colidx  int32[nnz]   column of every nonzero, 0 <= colidx[p] < M
 *   vals    float[nnz]   value of every nonzero
 *   C       float[N*K]   C(i,k) at C[i*K + k]
 *   D       float[M*K]   D(j,k) at D[j*K + k]
 *   E       float[M*L]   E(j,l) at E[j*L + l]
 *   A       float[N*L]   A(i,l) at A[i*L + l]   (output, overwritten)
 *   Y       float[nnz]   SDDMM values with the structure of B (unfused only)
 * where nnz = rowptr[N] (read on the device; never passed in).
 *
 * Conventions shared by every compute entry point:
 *   - All array pointers are DEVICE pointers owned by the caller; the library
 *     never frees or retains them.  The base pointers must be 4-byte aligned;
 *     16-byte alignment with K and L multiples of 4 enables the fast paths.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL is the null
 *     stream).  No call synchronises with the host.
 *   - Columns within a row may be unsorted and may repeat (repeats add).
 *     Preconditions on the CSR arrays are not checked on the device; use
 *     sparselnr_validate_csr in tests.  nnz and N + nnz must be < 2^31.
 *   - N = 0 or L = 0 is a no-op.  K = 0 makes every SDDMM value zero.  Rows
 *     without nonzeros produce zero rows of A.
 *   - rowptr must be non-NULL when N > 0.  colidx and vals (Y for SpMM) must
 *     be non-NULL when N > 0; pass any valid device address when nnz = 0.
 *     C must be non-NULL when N > 0 and K > 0; D when N, M, K > 0; E when
 *     N, M, L > 0; A when N > 0 and L > 0; Y (unfused/SDDMM) when N > 0.
 *   - Argument errors are reported BEFORE any HIP call, with no side effect.
 *   - The fused, unfused and SpMM calls use a workspace per (device, stream)
 *     for rows whose nonzeros are split between workers (2 partial rows per
 *     worker: tens of MB for matrices of millions of rows); it is allocated
 *     on first use, grown when a call needs more, reused, and freed by
 *     sparselnr_release().
 *     Calls on different streams use different workspaces; calls on one
 *     stream are ordered by the stream.
 *   - HIP graph capture: once a stream's workspace is large enough (after
 *     one uncaptured call of the same size, width and grid factor on that
 *     stream), a call launches kernels only, with no allocation,
 *     synchronisation or memset, and can be captured on that stream.  The
 *     graph records the workspace address: while it may still be replayed,
 *     do not call sparselnr_release() and make no call on that stream that
 *     needs a larger workspace (more rows, a wider L, a larger grid factor),
 *     since either frees the workspace.
 *   - Results are deterministic: the same inputs give bit-identical outputs
 *     on the same device model (no floating-point atomics).
 *   - No C++ exception crosses this interface.
 */
#ifndef SPARSELNR_H
#define SPARSELNR_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__)
#define SPARSELNR_API __attribute__((visibility("default")))
#else
#define SPARSELNR_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every int-valued entry point. */
enum sparselnr_status_code {
  SPARSELNR_OK = 0,
  SPARSELNR_ERR_INVALID_ARG = 1, /* NULL pointer, negative size, misuse      */
  SPARSELNR_ERR_UNSUPPORTED = 2, /* K or L above SPARSELNR_MAX_WIDTH, or
                                    sizes beyond the int32 index range        */
  SPARSELNR_ERR_HIP = 3,         /* a HIP call failed; see last_hip_error      */
  SPARSELNR_ERR_NO_MEMORY = 4,   /* workspace allocation failed               */
  SPARSELNR_ERR_INVALID_CSR = 5  /* sparselnr_validate_csr found a violation  */
};

/* Largest accepted K and L. */
#define SPARSELNR_MAX_WIDTH 65536

/* Version of this interface (incremented on incompatible change). */
SPARSELNR_API int sparselnr_abi_version(void);

/*
 * Fused SDDMM->SpMM (Figure 2d; Section 3.1.3):
 *   A(i,:) = sum_{p in row i} vals[p] * dot(C(i,:), D(colidx[p],:)) * E(colidx[p],:)
 * A is overwritten.  Arithmetic is fp32 (fused multiply-add), with the
 * k-reduction done as a lane-parallel tree and the l-update accumulated in
 * nonzero order.  Needs the per-(device, stream) workspace.
 */
SPARSELNR_API int sparselnr_fused_sddmm_spmm(const int32_t *rowptr, const int32_t *colidx,
                                             const float *vals, const float *C,
                                             const float *D, const float *E, float *A,
                                             int64_t N, int64_t M, int64_t K, int64_t L,
                                             void *stream);

/* Size in bytes of the device array of sparselnr_fused_sddmm_spmm_noalloc. */
#define SPARSELNR_NOALLOC_SCRATCH_BYTES (64u * 1024u * 1024u)

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same
 * computation, arguments, layouts and argument errors as
 * sparselnr_fused_sddmm_spmm, with no allocation of any kind (no hipMalloc,
 * hipFree or allocating library routine).  The partial rows of rows split
 * between workers go to a fixed device array of
 * SPARSELNR_NOALLOC_SCRATCH_BYTES (64 MiB) inside the library, one per GPU,
 * held from the first call on that GPU until the process ends.  The call
 * runs at the grid factor the fused entry point would use, halved until the
 * partial rows fit the array (so results may differ from the fused entry
 * point's in rounding order, within its accuracy; they are bit-identical
 * when the same factor fits, as it does at the automatic factor for the
 * workloads of this library).  It returns SPARSELNR_ERR_UNSUPPORTED if they
 * do not fit even at one resident grid (not reached for K, L <= 512).
 * All calls on one GPU share that GPU's array and it keeps the last call's
 * contents: calls that overlap in time on one GPU (different streams, or
 * different host threads) RACE and corrupt each other's results; order them
 * on one stream.  Nothing in the array needs clearing between calls.
 */
SPARSELNR_API int sparselnr_fused_sddmm_spmm_noalloc(const int32_t *rowptr,
                                                     const int32_t *colidx, const float *vals,
                                                     const float *C, const float *D,
                                                     const float *E, float *A, int64_t N,
                                                     int64_t M, int64_t K, int64_t L,
                                                     void *stream);

/*
 * Unfused comparison (Figure 2a then Figure 2b, Section 3.1.2): the SDDMM
 * writes Y (nnz floats, structure of B, same order as colidx), then the SpMM
 * reads it.  Same result as the fused call up to rounding order.
 */
SPARSELNR_API int sparselnr_unfused_sddmm_spmm(const int32_t *rowptr, const int32_t *colidx,
                                               const float *vals, const float *C,
                                               const float *D, const float *E, float *Y,
                                               float *A, int64_t N, int64_t M, int64_t K,
                                               int64_t L, void *stream);

/* SDDMM alone (Figure 2a): Y[p] = vals[p] * dot(C(i,:), D(colidx[p],:)). */
SPARSELNR_API int sparselnr_sddmm(const int32_t *rowptr, const int32_t *colidx,
                                  const float *vals, const float *C, const float *D,
                                  float *Y, int64_t N, int64_t M, int64_t K, void *stream);

/* SpMM alone (Figure 2b): A(i,:) = sum_{p in row i} Y[p] * E(colidx[p],:).
 * A is overwritten.  Needs the per-(device, stream) workspace. */
SPARSELNR_API int sparselnr_spmm(const int32_t *rowptr, const int32_t *colidx,
                                 const float *Y, const float *E, float *A, int64_t N,
                                 int64_t M, int64_t L, void *stream);

/*
 * <SDDMM, SpMM, GEMM> (Section 6.2; the recursive application of the fusion
 * in Section 4.2):
 *   A(i,m) = sum_{j,k,l} B(i,j) C(i,k) D(j,k) F(j,l) W(l,m)
 * computed as the fused <SDDMM, SpMM> row t_i (Figure 2d) followed, in the
 * same pass, by the per-row product A_i = t_i W, so neither the nnz-sized
 * SDDMM values nor the N x L matrix t is ever stored.  The row products
 * run on the matrix cores over tiles of finished rows.
 *   C: N x K, D: M x K, F: M x L, W: L x Mo, A: N x Mo (overwritten).
 * Supported: K == L in {16, 32, 64, 128, 256, 512}, any Mo; C, D and F
 * 16-byte aligned.  Other shapes return SPARSELNR_ERR_UNSUPPORTED.
 */
SPARSELNR_API int sparselnr_fused_sddmm_spmm_gemm(const int32_t *rowptr, const int32_t *colidx,
                                                  const float *vals, const float *C,
                                                  const float *D, const float *F,
                                                  const float *W, float *A, int64_t N,
                                                  int64_t M, int64_t K, int64_t L, int64_t Mo,
                                                  void *stream);

/*
 * <SpMM, GEMM> (Section 6.2; the GNN hidden-state update):
 *   A(i,l) = sum_{j,k} B(i,j) C(j,k) D(k,l)
 * computed per row as the SpMM row t_i = sum_j B(i,j) C(j,:) (a vector
 * temporary of length K, Section 6.3) followed by A_i = t_i D.
 *   C: M x K, D: K x L, A: N x L (overwritten).
 * Supported: K in {16, 32, 64, 128, 256, 512}, any L; C 16-byte aligned.
 */
SPARSELNR_API int sparselnr_spmm_gemm(const int32_t *rowptr, const int32_t *colidx,
                                      const float *vals, const float *C, const float *D,
                                      float *A, int64_t N, int64_t M, int64_t K, int64_t L,
                                      void *stream);

/*
 * <SpMMH, GEMM> (Section 6.2):
 *   A(i,l) = sum_{k,j} B(i,k) C(k,j) D(k,j) E(j,l)
 * computed per row as t_i = sum_k B(i,k) (C(k,:) .* D(k,:)) (length J)
 * followed by A_i = t_i E.  B is N x M; C, D: M x J; E: J x L; A: N x L.
 * Supported: J in {16, 32, 64, 128, 256, 512}, any L; C and D 16-byte
 * aligned.
 * C .* D does not depend on the row i.  When nnz >= 3 M (decided on the
 * device, which alone knows nnz) it is formed once into a per-(device,
 * stream) workspace of M x J floats and gathered as one row per nonzero;
 * otherwise each nonzero multiplies its two gathered rows.  Both schedules
 * round the same products in the same order, so A is bit-identical either
 * way.  The workspace is allocated on the first call of a shape (failure:
 * SPARSELNR_ERR_NO_MEMORY) and freed by sparselnr_release().
 */
SPARSELNR_API int sparselnr_spmmh_gemm(const int32_t *rowptr, const int32_t *colidx,
                                       const float *vals, const float *C, const float *D,
                                       const float *E, float *A, int64_t N, int64_t M,
                                       int64_t J, int64_t L, void *stream);

/*
 * <SDDMM, SpMM> with D stored transposed (Section 4.3.1: the layout whose
 * temporary becomes a vector over j unless the loops are reordered):
 *   A(i,l) = sum_{j,k} B(i,j) C(i,k) Dt(k,j) E(j,l),   Dt: K x M.
 * On the GPU the reorder is done on the data: Dt is transposed once into a
 * per-(device, stream) workspace of M x K floats (coalesced tile transpose),
 * then the fused kernel runs.  Same result, shapes and errors as
 * sparselnr_fused_sddmm_spmm; the workspace is freed by sparselnr_release().
 */
SPARSELNR_API int sparselnr_fused_sddmm_spmm_dt(const int32_t *rowptr, const int32_t *colidx,
                                                const float *vals, const float *C,
                                                const float *Dt, const float *E, float *A,
                                                int64_t N, int64_t M, int64_t K, int64_t L,
                                                void *stream);

/*
 * Checks the CSR preconditions on the device: rowptr[0] == 0, rowptr
 * non-decreasing, 0 <= rowptr[N] <= colidx_len, N + rowptr[N] < 2^31, every
 * colidx in [0, M).  colidx_len is the number of int32 entries the caller
 * allocated for colidx; at most that many are read.  SYNCHRONOUS (waits for
 * `stream`); meant for tests and debugging, not the hot path.  Writes
 * nnz = rowptr[N] to *nnz_out (host pointer, may be NULL).
 * Returns SPARSELNR_OK or SPARSELNR_ERR_INVALID_CSR (or an error code).
 */
SPARSELNR_API int sparselnr_validate_csr(const int32_t *rowptr, const int32_t *colidx,
                                         int64_t N, int64_t M, int64_t colidx_len,
                                         int64_t *nnz_out, void *stream);

/* Static text for a status code (never NULL). */
SPARSELNR_API const char *sparselnr_status_string(int status);

/* hipError_t of the last failing HIP call made by this library on the
 * calling thread (0 if none). */
SPARSELNR_API int sparselnr_last_hip_error(void);

/*
 * Launch tuning (no counterpart in the paper, which fixes no GPU launch).
 * Every walk launch runs `factor` resident grids of workers, each worker
 * taking one merge-path slice of rows + nonzeros, so a larger factor gives
 * more, shorter slices: the workers resident at one moment then cover a
 * narrower band of rows, which changes how D and E rows are shared in the
 * caches.  factor 0 restores the automatic choice (8 when the matrix has at
 * least 8 rows per resident worker, else 1); 1..64 fixes the factor for every
 * later call in the process, on every device and stream (the environment
 * variable SPARSELNR_GRID_FACTOR gives the first value).  Results are
 * deterministic for a fixed factor; another factor splits rows between slices
 * elsewhere and so changes the fp32 summation order (within the accuracy
 * stated for each entry point).  The carry workspace grows with the number
 * of workers: 2 * L floats per worker.  Launches already made are not
 * affected.  Returns SPARSELNR_OK, or SPARSELNR_ERR_INVALID_ARG for a factor
 * outside 0..64.
 */
SPARSELNR_API int sparselnr_set_grid_factor(int factor);

/* The factor fixed by sparselnr_set_grid_factor or SPARSELNR_GRID_FACTOR,
 * or 0 when it is chosen per call. */
SPARSELNR_API int sparselnr_get_grid_factor(void);

/* Waits for the device(s) and frees every workspace the library allocated.
 * Safe to call at any time; later calls allocate again. */
SPARSELNR_API int sparselnr_release(void);

#ifdef __cplusplus
} /* extern "C" */
#endif

#endif /* SPARSELNR_H */
