// Device code of the fused SDDMM->SpMM library for gfx950 (CDNA4, wave64).
//
// Work decomposition (all kernels): merge-path partitioning of the CSR rows.
// The row ends of B (rowptr[1..N]) and its nonzeros 0..nnz-1 form one merged
// sequence of N + nnz items; every worker (a group of W lanes inside a wave)
// takes an equal slice of it.  A worker therefore owns a contiguous run of
// nonzeros plus the rows ending inside it, so power-law rows (tens of
// thousands of nonzeros) are split over many workers and empty rows still get
// their zero store, while no worker waits on another.  A row whose nonzeros
// straddle workers leaves partial rows in a workspace ("carry"); a second
// small kernel adds them in worker order, so results are deterministic.
//
// Per row, the loop body is the fused schedule of the paper's Figure 2d: for
// each nonzero the producer (SDDMM inner k-loop) forms the scalar
//     y = b * dot(C_i, D_j)
// with C_i held in registers and the dot reduced across lanes with DPP /
// swizzle, then the consumer (SpMM inner l-loop) adds y * E_j into the row
// accumulators, also in registers.  The scalar temporary is the one the
// paper's Algorithm 1 derives for this expression (Section 4.2: no index
// below the nest boundary is shared, so the temporary is a scalar).  The
// producer and consumer may use different lane mappings inside one row, the
// GPU reading of the branched iteration graph (Section 4.1): with K = 16 and
// L = 256, 4-lane groups compute 16 scalars at once and the whole wave then
// streams each 1 KB row of E.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace slnr {

enum Mode : int { kFused = 0, kSddmm = 1, kSpmm = 2 };

struct WalkArgs {
  const int32_t *rowptr;
  const int32_t *colidx;
  const float *vals;  // B values (fused, SDDMM) or Y values (SpMM)
  const float *C;     // N x K
  const float *D;     // M x K
  const float *E;     // M x L (row stride L)
  float *out;         // A (fused, SpMM; row stride L) or Y (SDDMM)
  float *carry;       // [workers][2][Lw] partial rows: slot 0 head, slot 1 tail
  int32_t *meta;      // [workers][2]: tail row (or -1), head row (or -1)
  int64_t N;
  int32_t K;
  int32_t L;          // row stride of E and A
  int32_t l0;         // first column of the l-tile handled by this launch
  int32_t Lw;         // width of that tile
  int32_t workers;    // workers in the grid
  int32_t min_chunk;  // smallest merge-path slice per worker
  int32_t xcd_span;   // blocks per XCD for the XCD-contiguous remap (0: off)
  int32_t xcds;       // XCDs the hardware deals blocks across
};

// ---------------------------------------------------------------- lane ops

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                         0xF, 0xF, false));
}

__device__ __forceinline__ int bperm_i(int src_lane, int v) {
  return __builtin_amdgcn_ds_bpermute(src_lane << 2, v);
}

__device__ __forceinline__ float bperm_f(int src_lane, float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_ds_bpermute(src_lane << 2, __builtin_bit_cast(int, v)));
}

// Sum over aligned groups of G lanes; every lane of the group receives the
// same bits (each step adds a value and its partner's, and fp addition is
// commutative).
template <int G>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(G == 1 || G == 2 || G == 4 || G == 8 || G == 16 || G == 32 || G == 64,
                "group size");
  if constexpr (G >= 2) v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]: lane ^ 1
  if constexpr (G >= 4) v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]: lane ^ 2
  if constexpr (G >= 8) v += dpp<0x141>(v);  // row_half_mirror: other quad of 8
  if constexpr (G >= 16) v += dpp<0x140>(v); // row_mirror: other half of 16
  if constexpr (G >= 32)                     // swizzle bit mode, xor 16
    v += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
  if constexpr (G >= 64) v += bperm_f((int)(threadIdx.x & 63) ^ 32, v);
  return v;
}

template <int V>
__device__ __forceinline__ void ldv(float (&r)[V], const float *p) {
  if constexpr (V % 4 == 0) {
#pragma unroll
    for (int t = 0; t < V / 4; ++t) {
      const float4 x = reinterpret_cast<const float4 *>(p)[t];
      r[4 * t] = x.x; r[4 * t + 1] = x.y; r[4 * t + 2] = x.z; r[4 * t + 3] = x.w;
    }
  } else if constexpr (V % 2 == 0) {
#pragma unroll
    for (int t = 0; t < V / 2; ++t) {
      const float2 x = reinterpret_cast<const float2 *>(p)[t];
      r[2 * t] = x.x; r[2 * t + 1] = x.y;
    }
  } else {
#pragma unroll
    for (int t = 0; t < V; ++t) r[t] = p[t];
  }
}

template <int V>
__device__ __forceinline__ void stv(float *p, const float (&r)[V]) {
  if constexpr (V % 4 == 0) {
#pragma unroll
    for (int t = 0; t < V / 4; ++t)
      reinterpret_cast<float4 *>(p)[t] = make_float4(r[4 * t], r[4 * t + 1], r[4 * t + 2], r[4 * t + 3]);
  } else if constexpr (V % 2 == 0) {
#pragma unroll
    for (int t = 0; t < V / 2; ++t)
      reinterpret_cast<float2 *>(p)[t] = make_float2(r[2 * t], r[2 * t + 1]);
  } else {
#pragma unroll
    for (int t = 0; t < V; ++t) p[t] = r[t];
  }
}

// ------------------------------------------------------------ merge path

// Largest row i in [max(0, d - nnz), min(d, N)] with rowptr[i] + i <= d: the
// merge-path coordinate (i row ends, d - i nonzeros consumed) of diagonal d.
// rowptr[i] + i is strictly increasing, so this is a plain bisection.
__device__ __forceinline__ int64_t mp_search(const int32_t *rowptr, int64_t N,
                                             int64_t nnz, int64_t d) {
  int64_t lo = d > nnz ? d - nnz : 0;
  int64_t hi = d < N ? d : N;
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) >> 1;
    if ((int64_t)rowptr[mid] + mid <= d) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

struct Slice {
  int64_t i0, p0, i1, p1;  // start and end coordinates
  bool head;               // row i0 began in an earlier slice and ends here
  bool active;
};

__device__ __forceinline__ int64_t logical_block(const WalkArgs &a) {
  // Blocks are dealt round-robin over the XCDs; remap so that each XCD works
  // through one contiguous range of slices (neighbouring rows share L2).
  if (a.xcd_span > 0)
    return (int64_t)(blockIdx.x % a.xcds) * a.xcd_span + blockIdx.x / a.xcds;
  return blockIdx.x;
}

__device__ __forceinline__ Slice make_slice(const WalkArgs &a, int64_t worker) {
  Slice s;
  const int64_t N = a.N;
  const int64_t nnz = a.rowptr[N];
  const int64_t items = N + nnz;
  int64_t S = (items + a.workers - 1) / a.workers;
  if (S < a.min_chunk) S = a.min_chunk;
  const int64_t d0 = worker * S;
  s.active = d0 < items;
  if (!s.active) {
    s.i0 = s.p0 = s.i1 = s.p1 = 0;
    s.head = false;
    return s;
  }
  const int64_t d1 = d0 + S < items ? d0 + S : items;
  s.i0 = mp_search(a.rowptr, N, nnz, d0);
  s.p0 = d0 - s.i0;
  s.i1 = mp_search(a.rowptr, N, nnz, d1);
  s.p1 = d1 - s.i1;
  s.head = (s.i0 < s.i1) && (s.p0 > (int64_t)a.rowptr[s.i0]);
  return s;
}

// ------------------------------------------------------ fast-path kernel
//
// W   lanes per worker (4..64); the consumer spreads E_j / A_i over them.
// NB  nonzeros per producer pass; PS = W / NB lanes form one dot product.
// KV  floats of C_i / D_j per producer lane (K = PS * KV).
// LV  floats of E_j / A_i per lane (L = W * LV).
// U   nonzeros per loop step (their gathers are all in flight together).
template <int MODE, int W, int NB, int KV, int LV, int U>
__global__ __launch_bounds__(256) void walk_fast(WalkArgs a) {
  constexpr int PS = W / NB;
  static_assert(W >= 4 && W <= 64 && (W & (W - 1)) == 0, "W");
  static_assert(NB >= 1 && W % NB == 0, "NB");
  static_assert(NB == 1 || U == NB, "a producer pass handles one step");
  static_assert(U <= W, "the index window must cover a step");
  const int lane = threadIdx.x & 63;
  const int glane = lane & (W - 1);
  const int gbase = lane - glane;
  const int q = glane % PS;   // k-slice of this lane in its dot product
  const int sub = glane / PS; // which nonzero of a producer pass (NB > 1)
  const int64_t worker =
      (logical_block(a) * (blockDim.x >> 6) + (threadIdx.x >> 6)) * (64 / W) + lane / W;
  if (worker >= a.workers) return;
  int32_t *meta = a.meta + 2 * worker;
  const Slice s = make_slice(a, worker);
  if (!s.active) {
    if (MODE != kSddmm && glane == 0) { meta[0] = -1; meta[1] = -1; }
    return;
  }
  const int32_t *__restrict__ rowptr = a.rowptr;
  const int32_t *__restrict__ colidx = a.colidx;
  const float *__restrict__ vals = a.vals;
  const float *__restrict__ Cm = a.C;
  const float *__restrict__ Dm = a.D;
  const float *__restrict__ Em = a.E;
  float *__restrict__ out = a.out;
  const int64_t K = a.K, L = a.L, N = a.N;

  int64_t i = s.i0, p = s.p0;
  int64_t wb = -(int64_t)(1 << 30);  // base of the index window
  int wj = 0;                        // colidx[wb + glane]
  float wv = 0.f;                    // vals[wb + glane]
  while (true) {
    const bool has_end = i < s.i1;
    if (!has_end && i >= N) break;
    const int64_t r_end = has_end ? (int64_t)rowptr[i + 1] : s.p1;
    float acc[LV];
#pragma unroll
    for (int v = 0; v < LV; ++v) acc[v] = 0.f;
    float c[KV];
#pragma unroll
    for (int v = 0; v < KV; ++v) c[v] = 0.f;
    if (MODE != kSpmm && p < r_end) ldv<KV>(c, Cm + i * K + q * KV);
    while (p < r_end) {
      const int n = (int)(r_end - p < U ? r_end - p : U);
      if (p + n > wb + W) {  // refill the index window
        wb = p;
        const int64_t pw = wb + glane;
        if (pw < s.p1) { wj = colidx[pw]; wv = vals[pw]; }
      }
      const int off = (int)(p - wb);
      if constexpr (NB == 1) {
        float dr[U][KV];
        float er[U][LV];
        float bb[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (u < n) {
            const int64_t j = bperm_i(gbase + off + u, wj);
            bb[u] = bperm_f(gbase + off + u, wv);
            if (MODE != kSpmm) ldv<KV>(dr[u], Dm + j * K + q * KV);
            if (MODE != kSddmm) ldv<LV>(er[u], Em + j * L + glane * LV);
          }
        }
        float ysel = 0.f;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          if (u < n) {
            float y;
            if (MODE == kSpmm) {
              y = bb[u];
            } else {
              float t = 0.f;
#pragma unroll
              for (int v = 0; v < KV; ++v) t = fmaf(c[v], dr[u][v], t);
              t = group_sum<W>(t);
              y = bb[u] * t;
            }
            if (MODE == kSddmm) {
              if (glane == u) ysel = y;
            } else {
#pragma unroll
              for (int v = 0; v < LV; ++v) acc[v] = fmaf(y, er[u][v], acc[v]);
            }
          }
        }
        if (MODE == kSddmm && glane < n) out[p + glane] = ysel;
      } else {
        // one producer pass: sub-group `sub` forms the scalar of nonzero p+sub
        const bool act = sub < n;
        float y = 0.f;
        if (MODE != kSpmm) {
          // (lanes with sub >= n read a stale window entry and discard it)
          const int src = (gbase + off + sub) & 63;
          const int64_t js = bperm_i(src, wj);
          const float bs = bperm_f(src, wv);
          float dr[KV];
          float t = 0.f;
          if (act) {
            ldv<KV>(dr, Dm + js * K + q * KV);
#pragma unroll
            for (int v = 0; v < KV; ++v) t = fmaf(c[v], dr[v], t);
          }
          t = group_sum<PS>(t);
          y = bs * t;
          if (MODE == kSddmm && act && q == 0) out[p + sub] = y;
        }
        if (MODE != kSddmm) {
          float er[U][LV];
          float yy[U];
#pragma unroll
          for (int u = 0; u < U; ++u) {
            if (u < n) {
              const int64_t j = bperm_i(gbase + off + u, wj);
              yy[u] = (MODE == kSpmm) ? bperm_f(gbase + off + u, wv) : bperm_f(gbase + u * PS, y);
              ldv<LV>(er[u], Em + j * L + glane * LV);
            }
          }
#pragma unroll
          for (int u = 0; u < U; ++u) {
            if (u < n) {
#pragma unroll
              for (int v = 0; v < LV; ++v) acc[v] = fmaf(yy[u], er[u][v], acc[v]);
            }
          }
        }
      }
      p += n;
    }
    if (MODE != kSddmm) {
      float *dst;
      if (!has_end) dst = a.carry + (worker * 2 + 1) * (int64_t)a.Lw;
      else if (i == s.i0 && s.head) dst = a.carry + (worker * 2) * (int64_t)a.Lw;
      else dst = out + i * L;
      stv<LV>(dst + glane * LV, acc);
    }
    if (!has_end) break;
    ++i;
  }
  if (MODE != kSddmm && glane == 0) {
    meta[0] = s.i1 < N ? (int32_t)s.i1 : -1;
    meta[1] = s.head ? (int32_t)s.i0 : -1;
  }
}

// -------------------------------------------------------- generic kernel
//
// Any K and any l-tile of up to 64 * LT columns: one wave per worker, one
// nonzero at a time, scalar loads.  Used when K or L has no fast variant or
// the operands are not 16-byte aligned.
template <int MODE, int LT>
__global__ __launch_bounds__(256) void walk_generic(WalkArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t worker = logical_block(a) * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (worker >= a.workers) return;
  int32_t *meta = a.meta + 2 * worker;
  const Slice s = make_slice(a, worker);
  if (!s.active) {
    if (MODE != kSddmm && lane == 0) { meta[0] = -1; meta[1] = -1; }
    return;
  }
  const int32_t *__restrict__ rowptr = a.rowptr;
  const int64_t K = a.K, L = a.L, N = a.N, Lw = a.Lw, l0 = a.l0;
  int64_t i = s.i0, p = s.p0;
  while (true) {
    const bool has_end = i < s.i1;
    if (!has_end && i >= N) break;
    const int64_t r_end = has_end ? (int64_t)rowptr[i + 1] : s.p1;
    float acc[LT];
#pragma unroll
    for (int t = 0; t < LT; ++t) acc[t] = 0.f;
    for (; p < r_end; ++p) {
      const int64_t j = a.colidx[p];
      float y;
      if (MODE == kSpmm) {
        y = a.vals[p];
      } else {
        float t = 0.f;
        for (int64_t k = lane; k < K; k += 64) t = fmaf(a.C[i * K + k], a.D[j * K + k], t);
        t = group_sum<64>(t);
        y = a.vals[p] * t;
      }
      if (MODE == kSddmm) {
        if (lane == 0) a.out[p] = y;
      } else {
#pragma unroll
        for (int t = 0; t < LT; ++t) {
          const int64_t l = lane + 64 * t;
          if (l < Lw) acc[t] = fmaf(y, a.E[j * L + l0 + l], acc[t]);
        }
      }
    }
    if (MODE != kSddmm) {
      float *dst;
      int64_t stride_base;
      if (!has_end) { dst = a.carry; stride_base = (worker * 2 + 1) * Lw; }
      else if (i == s.i0 && s.head) { dst = a.carry; stride_base = (worker * 2) * Lw; }
      else { dst = a.out; stride_base = i * L + l0; }
#pragma unroll
      for (int t = 0; t < LT; ++t) {
        const int64_t l = lane + 64 * t;
        if (l < Lw) dst[stride_base + l] = acc[t];
      }
    }
    if (!has_end) break;
    ++i;
  }
  if (MODE != kSddmm && lane == 0) {
    meta[0] = s.i1 < N ? (int32_t)s.i1 : -1;
    meta[1] = s.head ? (int32_t)s.i0 : -1;
  }
}

// ------------------------------------------------------------ carry fixup
//
// One wave per worker slice.  A slice whose first row is a head row (begun
// by earlier slices) adds, in slice order, the tail partials of the earlier
// slices that end inside that row, then its own head partial, and writes
// the row of A.
__global__ __launch_bounds__(256) void carry_fixup(const float *__restrict__ carry,
                                                   const int32_t *__restrict__ meta,
                                                   float *__restrict__ A, int32_t workers,
                                                   int32_t Lw, int32_t L, int32_t l0) {
  const int lane = threadIdx.x & 63;
  const int64_t c = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (c >= workers) return;
  const int32_t r = meta[2 * c + 1];
  if (r < 0) return;
  int64_t first = c;
  while (true) {  // slices with tail row r are contiguous and end at c - 1
    const int64_t idx = first - 1 - lane;
    const bool same = idx >= 0 && meta[2 * idx] == r;
    const uint64_t m = __ballot(same);
    const int run = (~m == 0) ? 64 : __builtin_ctzll(~m);
    first -= run;
    if (run < 64) break;
  }
  for (int64_t l = lane; l < Lw; l += 64) {
    float sum = 0.f;
    for (int64_t cc = first; cc < c; ++cc) sum += carry[(cc * 2 + 1) * Lw + l];
    sum += carry[(c * 2) * Lw + l];
    A[(int64_t)r * L + l0 + l] = sum;
  }
}

// ------------------------------------------------------------ validation
//
// flags[0] |= 1: rowptr[0] != 0; 2: rowptr decreasing; 4: colidx out of
// range; 8: nnz negative, too large, or beyond the colidx length given.
// Reads at most colidx_len entries of colidx.
__global__ void validate_csr_kernel(const int32_t *rowptr, const int32_t *colidx, int64_t N,
                                    int64_t M, int64_t colidx_len, int32_t *flags) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t nnz = rowptr[N];
  if (tid == 0) {
    if (rowptr[0] != 0) atomicOr(flags, 1);
    if (nnz < 0 || nnz + N >= ((int64_t)1 << 31) || nnz > colidx_len) atomicOr(flags, 8);
  }
  for (int64_t i = tid; i < N; i += stride)
    if (rowptr[i + 1] < rowptr[i]) atomicOr(flags, 2);
  const int64_t n = nnz < colidx_len ? nnz : colidx_len;
  for (int64_t p = tid; p < n; p += stride) {
    const int32_t j = colidx[p];
    if (j < 0 || j >= M) atomicOr(flags, 4);
  }
}

}  // namespace slnr
