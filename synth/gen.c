/*
 * Seeded synthetic inputs for the fused SDDMM->SpMM workloads.
 *
 * This file holds no arithmetic of the method itself: it only draws sparse
 * structures (CSR rowptr/colidx) and dense fp32 arrays.  Both the CPU oracle
 * and the GPU library are fed from the arrays it writes; neither links it.
 *
 * Random numbers come from one counter-based generator: element n of stream
 * (seed, id) is splitmix64_mix(key(seed, id) + (n + 1) * GOLDEN), where
 * splitmix64_mix is the 64-bit finaliser of SplitMix64 (Steele, Lea and Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA 2014; the
 * constants are the "Mix13" variant published with Java's SplittableRandom).
 * Because every element has its own counter, the output does not depend on
 * how many OpenMP threads run.
 *
 * The paper draws its dense operands at random without naming a distribution
 * (Section 6.1, datasets paragraph); the sparse matrices here stand in for its
 * Table 1 inputs by shape and structure class.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t id) {
  return mix64(mix64(seed + GOLDEN) ^ (id * 0xD1B54A32D192ED03ULL));
}

static inline uint64_t draw(uint64_t key, uint64_t n) {
  return mix64(key + (n + 1) * GOLDEN);
}

/* 53-bit uniform double in [0, 1). */
static inline double u53(uint64_t r) { return (double)(r >> 11) * 0x1.0p-53; }

/* Uniform integer in [0, bound) by Lemire's multiply-shift. */
static inline uint64_t below(uint64_t r, uint64_t bound) {
  return (uint64_t)(((__uint128_t)r * bound) >> 64);
}

int synth_abi_version(void) { return 1; }

int synth_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

uint64_t synth_draw(uint64_t seed, uint64_t id, uint64_t n) {
  return draw(stream_key(seed, id), n);
}

/* out[n] = lo + (hi - lo) * u, u = 24-bit uniform in [0, 1).  For the ranges
 * used here ([-1, 1) and [0, 1)) every value is exactly representable. */
void synth_uniform_f32(uint64_t seed, uint64_t id, double lo, double hi,
                       int64_t n, float *out) {
  const uint64_t key = stream_key(seed, id);
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < n; ++t) {
    const double u = (double)(draw(key, (uint64_t)t) >> 40) * 0x1.0p-24;
    out[t] = (float)(lo + (hi - lo) * u);
  }
}

/* Standard normal by the Box-Muller transform: elements 2m and 2m+1 share the
 * uniform pair (draw 2m, draw 2m+1) and take the cosine and sine branch. */
void synth_normal_f32(uint64_t seed, uint64_t id, int64_t n, float *out) {
  const uint64_t key = stream_key(seed, id);
  const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
  for (int64_t m = 0; m < (n + 1) / 2; ++m) {
    const double u1 = 1.0 - u53(draw(key, 2 * (uint64_t)m)); /* (0, 1] */
    const double u2 = u53(draw(key, 2 * (uint64_t)m + 1));
    const double rad = sqrt(-2.0 * log(u1));
    out[2 * m] = (float)(rad * cos(two_pi * u2));
    if (2 * m + 1 < n) out[2 * m + 1] = (float)(rad * sin(two_pi * u2));
  }
}

static int cmp_i32(const void *a, const void *b) {
  const int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return (x > y) - (x < y);
}

static void sort_small(int32_t *v, int64_t n) {
  if (n > 32) {
    qsort(v, (size_t)n, sizeof(int32_t), cmp_i32);
    return;
  }
  for (int64_t a = 1; a < n; ++a) {
    const int32_t x = v[a];
    int64_t b = a - 1;
    while (b >= 0 && v[b] > x) { v[b + 1] = v[b]; --b; }
    v[b + 1] = x;
  }
}

/* Every row holds exactly `deg` distinct columns drawn uniformly from [0, M)
 * by Floyd's sampling, sorted ascending.  rowptr: N+1, colidx: N*deg. */
int synth_csr_fixed_degree(uint64_t seed, uint64_t id, int64_t N, int64_t M,
                           int64_t deg, int32_t *rowptr, int32_t *colidx) {
  if (N < 0 || M < 0 || deg < 0 || deg > M || N * deg > INT32_MAX) return 1;
  const uint64_t key = stream_key(seed, id);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < N; ++i) {
    int32_t *row = colidx + i * deg;
    for (int64_t t = 0; t < deg; ++t) {
      const int64_t top = M - deg + t; /* candidate range [0, top] */
      const int64_t pick = (int64_t)below(draw(key, (uint64_t)(i * deg + t)),
                                          (uint64_t)(top + 1));
      int taken = 0;
      for (int64_t q = 0; q < t; ++q)
        if (row[q] == (int32_t)pick) { taken = 1; break; }
      row[t] = (int32_t)(taken ? top : pick);
    }
    sort_small(row, deg);
  }
  for (int64_t i = 0; i <= N; ++i) rowptr[i] = (int32_t)(i * deg);
  return 0;
}

/* R-MAT (Chakrabarti, Zhan and Faloutsos, SDM 2004): each of `samples` edges
 * descends `levels` times into one of four quadrants with probabilities
 * (a, b, c, 1-a-b-c), most significant bit first; no noise, no vertex
 * permutation, self loops kept.  Duplicate (row, col) pairs are merged.
 * colidx must hold `samples` entries; returns nnz (>= 0) or -1 on error. */
int64_t synth_rmat(uint64_t seed, uint64_t id, int levels, int64_t samples,
                   double a, double b, double c, int32_t *rowptr,
                   int32_t *colidx) {
  if (levels < 0 || levels > 30 || samples < 0 || samples > INT32_MAX) return -1;
  const int64_t N = (int64_t)1 << levels;
  const uint64_t key = stream_key(seed, id);
  const double ta = a, tb = a + b, tc = a + b + c;
  int32_t *rows = (int32_t *)malloc(sizeof(int32_t) * (size_t)(samples ? samples : 1));
  int32_t *cols = (int32_t *)malloc(sizeof(int32_t) * (size_t)(samples ? samples : 1));
  int64_t *start = (int64_t *)calloc((size_t)N + 1, sizeof(int64_t));
  int64_t *fill = (int64_t *)calloc((size_t)N + 1, sizeof(int64_t));
  int32_t *ucount = (int32_t *)calloc((size_t)N + 1, sizeof(int32_t));
  if (!rows || !cols || !start || !fill || !ucount) {
    free(rows); free(cols); free(start); free(fill); free(ucount);
    return -1;
  }
#pragma omp parallel for schedule(static)
  for (int64_t s = 0; s < samples; ++s) {
    uint32_t r = 0, q = 0;
    for (int t = 0; t < levels; ++t) {
      const double u = u53(draw(key, (uint64_t)s * (uint64_t)levels + (uint64_t)t));
      const uint32_t bit = 1u << (levels - 1 - t);
      if (u < ta) {
      } else if (u < tb) {
        q |= bit;
      } else if (u < tc) {
        r |= bit;
      } else {
        r |= bit;
        q |= bit;
      }
    }
    rows[s] = (int32_t)r;
    cols[s] = (int32_t)q;
  }
  /* bucket the samples by row */
#pragma omp parallel for schedule(static)
  for (int64_t s = 0; s < samples; ++s)
    __atomic_fetch_add(&start[rows[s] + 1], 1, __ATOMIC_RELAXED);
  for (int64_t i = 0; i < N; ++i) start[i + 1] += start[i];
  int32_t *tmp = (int32_t *)malloc(sizeof(int32_t) * (size_t)(samples ? samples : 1));
  if (!tmp) {
    free(rows); free(cols); free(start); free(fill); free(ucount);
    return -1;
  }
#pragma omp parallel for schedule(static)
  for (int64_t s = 0; s < samples; ++s) {
    const int32_t r = rows[s];
    const int64_t pos = start[r] + __atomic_fetch_add(&fill[r], 1, __ATOMIC_RELAXED);
    tmp[pos] = cols[s];
  }
  /* sort and merge duplicates inside every row */
#pragma omp parallel for schedule(dynamic, 256)
  for (int64_t i = 0; i < N; ++i) {
    int32_t *v = tmp + start[i];
    const int64_t n = start[i + 1] - start[i];
    sort_small(v, n);
    int64_t u = 0;
    for (int64_t t = 0; t < n; ++t)
      if (u == 0 || v[u - 1] != v[t]) v[u++] = v[t];
    ucount[i] = (int32_t)u;
  }
  rowptr[0] = 0;
  for (int64_t i = 0; i < N; ++i) rowptr[i + 1] = rowptr[i] + ucount[i];
#pragma omp parallel for schedule(dynamic, 256)
  for (int64_t i = 0; i < N; ++i)
    memcpy(colidx + rowptr[i], tmp + start[i], sizeof(int32_t) * (size_t)ucount[i]);
  const int64_t nnz = rowptr[N];
  free(rows); free(cols); free(start); free(fill); free(ucount); free(tmp);
  return nnz;
}

/* 27-point stencil on an n*n*n grid: row r = x + n*y + n*n*z couples to every
 * grid point (x+dx, y+dy, z+dz), dx,dy,dz in {-1,0,1}, that lies inside the
 * grid (itself included).  Columns come out sorted ascending.
 * rowptr: n^3 + 1 entries; colidx: (3n-2)^3 entries. */
int64_t synth_stencil27(int64_t n, int32_t *rowptr, int32_t *colidx) {
  if (n < 0 || n > 1290) return -1;
  const int64_t N = n * n * n;
  /* row lengths are products of per-axis neighbour counts */
  rowptr[0] = 0;
  for (int64_t r = 0; r < N; ++r) {
    const int64_t x = r % n, y = (r / n) % n, z = r / (n * n);
    const int64_t cx = 3 - (x == 0) - (x == n - 1);
    const int64_t cy = 3 - (y == 0) - (y == n - 1);
    const int64_t cz = 3 - (z == 0) - (z == n - 1);
    rowptr[r + 1] = (int32_t)(rowptr[r] + cx * cy * cz);
  }
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < N; ++r) {
    const int64_t x = r % n, y = (r / n) % n, z = r / (n * n);
    int64_t p = rowptr[r];
    for (int dz = -1; dz <= 1; ++dz)
      for (int dy = -1; dy <= 1; ++dy)
        for (int dx = -1; dx <= 1; ++dx) {
          const int64_t X = x + dx, Y = y + dy, Z = z + dz;
          if (X < 0 || Y < 0 || Z < 0 || X >= n || Y >= n || Z >= n) continue;
          colidx[p++] = (int32_t)(X + n * Y + n * n * Z);
        }
  }
  return rowptr[N];
}
