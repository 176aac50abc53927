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

#include <type_traits>

namespace slnr {

// Streams read or written once per call carry the nontemporal hint (C, the
// CSR arrays, A).  Measured on MI355X against plain loads and stores: the
// fused walk is 0.5-1.5% faster with the hint, the unfused passes 0.4-2%.
constexpr bool kNT = true;

enum Mode : int { kFused = 0, kSddmm = 1, kSpmm = 2 };

// Gather schedules of a step of nonzeros:
//  kPipelined  a depth-2 software pipeline (nonzero u's rows in flight while
//              u-1 is reduced and applied); few registers, high occupancy.
//  kPaced      all index broadcasts of the step first, then the gathers one
//              nonzero at a time, each issued once the previous nonzero's D
//              row has arrived, then all arithmetic.  Fewer requests in
//              flight per worker keeps workers of an XCD in step, which keeps
//              rows shared by neighbouring rows (banded matrices) in L2.
//  kBurst      all index broadcasts of the step, then all of its gathers at
//              once, then all arithmetic: one memory latency per step.  For
//              inputs too small to fill the GPU, whose time is the chain of
//              dependent loads of one worker, not the traffic.
enum Sched : int { kPipelined = 0, kPaced = 1, kBurst = 2 };

// s_waitcnt immediate (gfx9 encoding) waiting for vmcnt <= V only.
template <int V>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(V >= 0 && V < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((V & 15) | ((V >> 4) << 14) | (7 << 4) | (15 << 8));
}

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
  // consumer row width and the optional parts of the Section 6.2 benchmarks
  int32_t Lin;        // width of the gathered consumer rows (E, G2); == L without epilogue
  const float *G2;    // second gathered row source, multiplied elementwise (M x Lin)
  const float *Wep;   // per-row epilogue matrix (Lin x L): A_i = t_i * Wep
  // Gate of a launch whose schedule depends on nnz, which only the device
  // knows: kGateNone runs always, kGateDense only if nnz >= gate_nnz,
  // kGateSparse only if nnz < gate_nnz.  A closed launch exits at once.
  int64_t gate_nnz;
  int32_t gate;
};

enum Gate : int { kGateNone = 0, kGateDense = 1, kGateSparse = 2 };

// True when the gate of this launch is closed (uniform over the grid).
__device__ __forceinline__ bool gate_closed(int gate, const int32_t *rowptr, int64_t N,
                                            int64_t gate_nnz) {
  if (gate == kGateNone) return false;
  const bool dense = (int64_t)rowptr[N] >= gate_nnz;
  return gate == kGateDense ? !dense : dense;
}

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

__device__ __forceinline__ float readlane(float v, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

// Sum over aligned groups of G lanes; every lane of the group receives the
// same bits (each step adds a value and its partner's, and fp addition is
// commutative).  Inside rows of 16 lanes the steps are DPP moves; the rows
// of a 32- or 64-lane group are then combined from their first lanes read
// into scalar registers, (R0 + R1) + (R2 + R3), the same sums as an
// exchange of halves would form, without a trip through the LDS unit.  The
// callers keep each group's lanes active together, so the lanes read hold
// the group's own row sums.
template <int G>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(G == 1 || G == 2 || G == 4 || G == 8 || G == 16 || G == 32 || G == 64,
                "group size");
  if constexpr (G >= 2) v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]: lane ^ 1
  if constexpr (G >= 4) v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]: lane ^ 2
  if constexpr (G >= 8) v += dpp<0x141>(v);  // row_half_mirror: other quad of 8
  if constexpr (G >= 16) v += dpp<0x140>(v); // row_mirror: other half of 16
  if constexpr (G == 32) {
    const float lo = readlane(v, 0) + readlane(v, 16);
    const float hi = readlane(v, 32) + readlane(v, 48);
    return (threadIdx.x & 32) ? hi : lo;
  }
  if constexpr (G == 64)
    return (readlane(v, 0) + readlane(v, 16)) + (readlane(v, 32) + readlane(v, 48));
  return v;
}

typedef float f4_t __attribute__((ext_vector_type(4)));
typedef float f2_t __attribute__((ext_vector_type(2)));

// Loads V consecutive floats.  NT marks a stream read once per call
// (nontemporal hint: the line is not kept in L2 ahead of the D/E rows that
// are gathered again and again).
template <int V, bool NT = false>
__device__ __forceinline__ void ldv(float (&r)[V], const float *p) {
  if constexpr (V % 4 == 0) {
#pragma unroll
    for (int t = 0; t < V / 4; ++t) {
      const f4_t *q = reinterpret_cast<const f4_t *>(p) + t;
      const f4_t x = NT ? __builtin_nontemporal_load(q) : *q;
      r[4 * t] = x[0]; r[4 * t + 1] = x[1]; r[4 * t + 2] = x[2]; r[4 * t + 3] = x[3];
    }
  } else if constexpr (V % 2 == 0) {
#pragma unroll
    for (int t = 0; t < V / 2; ++t) {
      const f2_t *q = reinterpret_cast<const f2_t *>(p) + t;
      const f2_t x = NT ? __builtin_nontemporal_load(q) : *q;
      r[2 * t] = x[0]; r[2 * t + 1] = x[1];
    }
  } else {
#pragma unroll
    for (int t = 0; t < V; ++t) r[t] = NT ? __builtin_nontemporal_load(p + t) : p[t];
  }
}

template <int V, bool NT = false>
__device__ __forceinline__ void stv(float *p, const float (&r)[V]) {
  if constexpr (V % 4 == 0) {
#pragma unroll
    for (int t = 0; t < V / 4; ++t) {
      f4_t x;
      x[0] = r[4 * t]; x[1] = r[4 * t + 1]; x[2] = r[4 * t + 2]; x[3] = r[4 * t + 3];
      f4_t *q = reinterpret_cast<f4_t *>(p) + t;
      if constexpr (NT) __builtin_nontemporal_store(x, q);
      else *q = x;
    }
  } else if constexpr (V % 2 == 0) {
#pragma unroll
    for (int t = 0; t < V / 2; ++t) {
      f2_t x;
      x[0] = r[2 * t]; x[1] = r[2 * t + 1];
      f2_t *q = reinterpret_cast<f2_t *>(p) + t;
      if constexpr (NT) __builtin_nontemporal_store(x, q);
      else *q = x;
    }
  } else {
#pragma unroll
    for (int t = 0; t < V; ++t) {
      if constexpr (NT) __builtin_nontemporal_store(r[t], p + t);
      else p[t] = r[t];
    }
  }
}

// Loads V floats at byte offset `off` from `base`.  The offset is 32-bit
// (the host only selects the fast kernels when every gathered array is
// below 4 GiB), so the address is formed from the kernel-argument base in
// SGPRs plus one VGPR.
template <int V>
__device__ __forceinline__ void ldv_off(float (&r)[V], const float *__restrict__ base,
                                        uint32_t off) {
  ldv<V>(r, reinterpret_cast<const float *>(reinterpret_cast<const char *>(base) + off));
}

template <typename T>
__device__ __forceinline__ T ld_stream(const T *p) {
  return __builtin_nontemporal_load(p);
}

// ------------------------------------------------------------ merge path

// Largest row i in [max(0, d - nnz), min(d, N)] with rowptr[i] + i <= d: the
// merge-path coordinate (i row ends, d - i nonzeros consumed) of diagonal d,
// for the two diagonals da and db at once.  rowptr[i] + i is strictly
// increasing in i.  The G lanes of a worker probe G points of each current
// interval at once and keep the sub-interval the ballot points to, so a
// search takes log_G(N) steps instead of log_2(N) dependent loads, and the
// two searches share their steps (both probes of a step are loaded before
// either ballot).  All lanes of the group return the same values.
template <int G>
__device__ __forceinline__ void mp_search2(const int32_t *rowptr, int64_t N, int64_t nnz,
                                           int64_t da, int64_t db, int64_t *ia, int64_t *ib) {
  const int lane = threadIdx.x & 63;
  const int glane = lane & (G - 1);
  const int gbase = lane - glane;
  const int64_t d[2] = {da, db};
  int64_t lo[2], hi[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    lo[t] = d[t] > nnz ? d[t] - nnz : 0;  // rowptr[lo] + lo <= d always holds
    hi[t] = d[t] < N ? d[t] : N;
  }
  while (lo[0] < hi[0] || lo[1] < hi[1]) {
    int64_t step[2], x[2];
    int32_t r[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {  // a finished search probes its own end, which is in range
      step[t] = (hi[t] - lo[t] + G - 1) / G;
      x[t] = lo[t] + (int64_t)(glane + 1) * step[t];
      if (x[t] > hi[t]) x[t] = hi[t];
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) r[t] = rowptr[x[t]];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (lo[t] < hi[t]) {  // uniform in the group
        const uint64_t ball = __ballot((int64_t)r[t] + x[t] <= d[t]);
        const uint64_t bits = G == 64 ? ball : (ball >> gbase) & ((1ull << (G & 63)) - 1);
        const int m = (~bits == 0) ? 64 : __builtin_ctzll(~bits);  // probes 0..m-1 hold
        const int64_t xm1 = lo[t] + (int64_t)m * step[t];           // probe m-1 (if m > 0)
        const int64_t xm = lo[t] + (int64_t)(m + 1) * step[t];      // probe m (if m < G)
        if (m > 0) lo[t] = xm1 < hi[t] ? xm1 : hi[t];
        if (m < G) hi[t] = (xm < hi[t] ? xm : hi[t]) - 1;
      }
    }
  }
  *ia = lo[0];
  *ib = lo[1];
}

struct Slice {
  int64_t id;              // slice index in merge order
  int64_t i0, p0, i1, p1;  // start and end coordinates
  bool head;               // row i0 began in an earlier slice and ends here
  bool active;
};

// Slice length of inputs too small to fill the GPU, and the row length that
// slices shorter than 64 items still keep whole.
constexpr int64_t kShortSlice = 16;
constexpr int64_t kSnapRow = 16;

// Slices are S = ceil(items / workers) items long, raised to min_chunk (or
// to kShortSlice, below), so small inputs use only the first
// ns = ceil(items / S) of them.  An input with
// fewer than kShortSlice items per worker cannot fill the GPU however it is
// cut: its time is one worker's chain of dependent loads.  If its rows
// average at most kSnapRow nonzeros, its slices are kShortSlice items (about
// one short row and its end), so it spreads over as many workers as it has
// rows.  Measured on MI355X, 2048 rows of 10 nonzeros at K = L = 32: fused
// 22.6 -> 13.2 us per call, unfused 32.8 -> 19.2 us, results bit-identical
// (no row is split either way).  Inputs with longer rows on average keep
// 64-item slices: a hub row there would split into 4x more partial rows,
// which one wave of the fixup sums (1000 rows with one of 10^5 nonzeros:
// 172 us against 90 at K = L = 32).  Inputs with 16 to 64 items per worker
// also keep 64-item slices (65536 rows of 16 nonzeros: the unfused passes
// 1.7% slower with 34-item slices).  With the XCD
// remap, XCD x (blocks are dealt round-robin over the XCDs) takes the
// contiguous run of slices [x * ns / xcds, (x + 1) * ns / xcds), so that the
// workers sharing an L2 walk neighbouring rows and every XCD gets an equal
// share however small the input.
__device__ __forceinline__ void slice_count(const WalkArgs &a, int64_t *S_out, int64_t *ns_out,
                                            int64_t *items_out, int64_t *nnz_out) {
  const int64_t nnz = a.rowptr[a.N];
  const int64_t items = a.N + nnz;
  int64_t S = (items + a.workers - 1) / a.workers;
  if (S < kShortSlice && nnz <= kSnapRow * a.N) S = kShortSlice;
  else if (S < a.min_chunk) S = a.min_chunk;
  *S_out = S;
  *ns_out = (items + S - 1) / S;
  *items_out = items;
  *nnz_out = nnz;
}

template <int W>
__device__ __forceinline__ Slice make_slice(const WalkArgs &a) {
  Slice s;
  int64_t S, ns, items, nnz;
  slice_count(a, &S, &ns, &items, &nnz);
  constexpr int kWorkersPerWave = 64 / W;
  const int64_t wpb = (int64_t)(blockDim.x >> 6) * kWorkersPerWave;
  const int64_t local = (threadIdx.x >> 6) * kWorkersPerWave + (threadIdx.x & 63) / W;
  if (a.xcd_span > 0) {
    const int64_t xcd = blockIdx.x % a.xcds;
    const int64_t in_xcd = (int64_t)(blockIdx.x / a.xcds) * wpb + local;
    const int64_t per_xcd = (ns + a.xcds - 1) / a.xcds;
    s.id = xcd * per_xcd + in_xcd;
    s.active = in_xcd < per_xcd && s.id < ns;
  } else {
    s.id = (int64_t)blockIdx.x * wpb + local;
    s.active = s.id < ns;
  }
  s.i0 = s.p0 = s.i1 = s.p1 = 0;
  s.head = false;
  if (!s.active) return s;
  const int64_t d0 = s.id * S;
  const int64_t d1 = d0 + S < items ? d0 + S : items;
  mp_search2<W>(a.rowptr, a.N, nnz, d0, d1, &s.i0, &s.i1);
  s.p0 = d0 - s.i0;
  s.p1 = d1 - s.i1;
  // A boundary inside a short row moves back to the row's start, so only
  // long rows are ever split between slices.  Short means at most S/4
  // nonzeros for slices of 64 items or more; the shorter slices of small
  // inputs keep rows of up to min(S, 16) nonzeros whole, so that such inputs
  // leave no partial rows to the fixup.  Both slices sharing the boundary
  // apply the same rule, and the rule is monotone, so slices stay contiguous
  // and ordered; snap never exceeds S, so no slice is left empty by it.
  const int64_t snap_short = S < kSnapRow ? S : kSnapRow;
  const int64_t snap = S / 4 > snap_short ? S / 4 : snap_short;
  auto snap_back = [&](int64_t i, int64_t &p) {
    if (i < a.N) {
      const int64_t r0 = a.rowptr[i];
      if (p > r0 && (int64_t)a.rowptr[i + 1] - r0 <= snap) p = r0;
    }
  };
  snap_back(s.i0, s.p0);
  snap_back(s.i1, s.p1);
  s.head = (s.i0 < s.i1) && (s.p0 > (int64_t)a.rowptr[s.i0]);
  return s;
}

// Registers holding one nonzero's gathered rows.
template <int MODE, int KV, int LV, int HAD>
struct Gather {
  float d[MODE == kSpmm ? 1 : KV];
  float e[MODE == kSddmm ? 1 : LV];
  float h[HAD ? LV : 1];
  float b;
};

// ------------------------------------------------------------ row walk
//
// The nonzero loop of one row inside one slice, shared by the walk kernels.
// W   lanes per worker (4..64); the consumer spreads E_j / A_i over them.
// NB  nonzeros per producer pass; PS = W / NB lanes form one dot product.
// KV  floats of C_i / D_j per producer lane (K = PS * KV).
// LV  floats of E_j / A_i per lane (L = W * LV).
// SCHED, U  gather schedule and, for kPaced and kBurst, the nonzeros per step.
// HAD  the consumer row is E_j .* G2_j (Hadamard product of two gathers).
//
// The state is group-uniform (all W lanes agree on p, n), so lane-group
// divergence inside a wave only masks whole groups.  The colidx / vals window
// (one entry per lane) keeps the dependent loads off the critical path; the
// gathered D_j and E_j rows are plain loads so the hot columns stay in L2.
// A paced step issues a nonzero's gathers once every load of the previous
// nonzero but the newest has arrived (vmcnt <= 1).  Letting two stay in
// flight measured 9-10% slower on MI355X for the 64-lane worker with one
// float of each row per lane (R-MAT 2^22, K = L = 64, three boxes, builds
// compared in one process), and slower for the wider rows of rmat1m and
// the stencil.

template <int MODE, int W, int NB, int KV, int LV, int SCHED, int U, int HAD = 0>
struct RowWalk {
  static constexpr int PS = W / NB;
  static_assert(W >= 4 && W <= 64 && (W & (W - 1)) == 0, "W");
  static_assert(NB >= 1 && W % NB == 0, "NB");
  static_assert(SCHED == kPipelined || (U >= 1 && U <= W && (NB == 1 || U == NB)), "U");
  static_assert(SCHED != kBurst || NB == 1, "burst steps are built for one dot per pass");
  static constexpr bool kStep = SCHED == kPaced || SCHED == kBurst;
  static_assert(!HAD || (NB == 1 && MODE == kSpmm), "Hadamard rows come with the one-dot SpMM");

  const int32_t *__restrict__ colidx;
  const float *__restrict__ vals;
  const float *__restrict__ Dm;
  const float *__restrict__ Em;
  const float *__restrict__ Gm;
  float *__restrict__ out;  // SDDMM values (kSddmm)
  int64_t p1;               // end of the slice's nonzeros
  uint32_t strideD, strideE, offD, offE;  // row strides and this lane's offset, in bytes
  int glane, gbase, q, sub;
  int64_t wb;  // nonzero window: wj = colidx[wb + glane], wv = vals[wb + glane]
  int wj;
  float wv;
  // multi-dot SDDMM passes: this lane's slice of the D row of the next
  // pass's nonzero, gathered one pass ahead.  (In the fused walk the same
  // prefetch gains nothing at its best grid factor on the 27-point stencil,
  // and its 8 extra registers cost a wave per SIMD, so the fused passes
  // gather their own D rows.)
  float dnext[KV];
  int64_t pnext;  // first nonzero of the pass dnext belongs to (never a p otherwise)

  __device__ __forceinline__ RowWalk(const WalkArgs &a, int64_t p1_, uint32_t strideE_)
      : colidx(a.colidx), vals(a.vals), Dm(a.D), Em(a.E), Gm(a.G2), out(a.out), p1(p1_),
        strideD((uint32_t)a.K * 4u), strideE(strideE_), wb(-((int64_t)1 << 40)), wj(0),
        wv(0.f), pnext(-((int64_t)1 << 40)) {
    const int lane = threadIdx.x & 63;
    glane = lane & (W - 1);
    gbase = lane - glane;
    q = glane % PS;    // k-slice of this lane in its dot product
    sub = glane / PS;  // which nonzero of a producer pass (NB > 1)
    offD = (uint32_t)(q * KV) * 4u;
    offE = (uint32_t)(glane * LV) * 4u;
  }

  // Nonzeros p .. r_end-1 of the current row: their products with C_i (held
  // in c) are formed and applied to acc (or written out for the SDDMM).
  __device__ __forceinline__ void row(int64_t &p, int64_t r_end, const float (&c)[KV],
                                      float (&acc)[LV]) {
      while (p < r_end) {
        if (p >= wb + W) {  // refill the nonzero window
          wb = p;
          const int64_t pw = wb + glane;
          if (pw < p1) {
            wj = kNT ? ld_stream(colidx + pw) : colidx[pw];
            wv = kNT ? ld_stream(vals + pw) : vals[pw];
          }
        }
        // this step: the row's nonzeros inside the window (at most NB for a
        // producer pass of the multi-dot variant)
        int n = (int)(r_end - p < wb + W - p ? r_end - p : wb + W - p);
        if (NB > 1 && n > NB) n = NB;
        if (kStep && n > U) n = U;
        const int off = (int)(p - wb);
        if constexpr (NB == 1 && kStep) {
          uint32_t jj[U];
          float bb[U];
  #pragma unroll
          for (int u = 0; u < U; ++u) {  // lanes past n read stale entries, unused
            const int src = (gbase + off + u) & 63;
            jj[u] = (uint32_t)bperm_i(src, wj);
            bb[u] = bperm_f(src, wv);
          }
          float dr[U][KV];
          float er[U][LV];
          float hr[HAD ? U : 1][HAD ? LV : 1];
  #pragma unroll
          for (int u = 0; u < U; ++u) {
            if (u < n) {
              if (SCHED == kPaced && u > 0) wait_vmcnt<1>();
              if constexpr (MODE != kSpmm) ldv_off<KV>(dr[u], Dm, jj[u] * strideD + offD);
              if constexpr (MODE != kSddmm) ldv_off<LV>(er[u], Em, jj[u] * strideE + offE);
              if constexpr (HAD) ldv_off<LV>(hr[u], Gm, jj[u] * strideE + offE);
            }
          }
          float ysel = 0.f;
  #pragma unroll
          for (int u = 0; u < U; ++u) {
            if (u < n) {
              float y;
              if constexpr (MODE == kSpmm) {
                y = bb[u];
              } else {
                float t = 0.f;
  #pragma unroll
                for (int v = 0; v < KV; ++v) t = fmaf(c[v], dr[u][v], t);
                t = group_sum<W>(t);
                y = bb[u] * t;
              }
              if constexpr (MODE == kSddmm) {
                if (glane == u) ysel = y;
              } else if constexpr (HAD) {
  #pragma unroll
                for (int v = 0; v < LV; ++v) acc[v] = fmaf(y, er[u][v] * hr[u][v], acc[v]);
              } else {
  #pragma unroll
                for (int v = 0; v < LV; ++v) acc[v] = fmaf(y, er[u][v], acc[v]);
              }
            }
          }
          if (MODE == kSddmm && glane < n) out[p + glane] = ysel;
        } else if constexpr (NB == 1) {
          // Depth-2 software pipeline: the gathers of nonzero u are in flight
          // while nonzero u-1 is reduced and applied.  The loop body is
          // straight-line, so the wait before each consume covers exactly the
          // older pair of loads.
          Gather<MODE, KV, LV, HAD> ga, gb;
          float ysel = 0.f;
          auto issue = [&](Gather<MODE, KV, LV, HAD> &g, int u) {
            const int src = gbase + off + u;
            const uint32_t j = (uint32_t)bperm_i(src, wj);
            g.b = bperm_f(src, wv);
            if constexpr (MODE != kSpmm) ldv_off<KV>(g.d, Dm, j * strideD + offD);
            if constexpr (MODE != kSddmm) ldv_off<LV>(g.e, Em, j * strideE + offE);
            if constexpr (HAD) ldv_off<LV>(g.h, Gm, j * strideE + offE);
          };
          auto consume = [&](const Gather<MODE, KV, LV, HAD> &g, int u) {
            float y;
            if constexpr (MODE == kSpmm) {
              y = g.b;
            } else {
              float t = 0.f;
  #pragma unroll
              for (int v = 0; v < KV; ++v) t = fmaf(c[v], g.d[v], t);
              t = group_sum<W>(t);
              y = g.b * t;
            }
            if constexpr (MODE == kSddmm) {
              if (glane == u) ysel = y;
            } else if constexpr (HAD) {
  #pragma unroll
              for (int v = 0; v < LV; ++v) acc[v] = fmaf(y, g.e[v] * g.h[v], acc[v]);
            } else {
  #pragma unroll
              for (int v = 0; v < LV; ++v) acc[v] = fmaf(y, g.e[v], acc[v]);
            }
          };
          issue(ga, 0);
          int u = 1;
          for (; u + 1 < n; u += 2) {
            issue(gb, u);
            consume(ga, u - 1);
            issue(ga, u + 1);
            consume(gb, u);
          }
          if (u < n) {
            issue(gb, u);
            consume(ga, u - 1);
            consume(gb, u);
          } else {
            consume(ga, u - 1);
          }
          if (MODE == kSddmm && glane < n) out[p + glane] = ysel;
        } else {
          // one producer pass: sub-group `sub` forms the scalar of nonzero p+sub
          const bool act = sub < n;
          float y = 0.f;
          if (MODE != kSpmm) {
            // (lanes with sub >= n read a stale window entry and discard it)
            const int src = (gbase + off + sub) & 63;
            const uint32_t js = (uint32_t)bperm_i(src, wj);
            const float bs = bperm_f(src, wv);
            if constexpr (MODE == kSddmm) {
              // the D rows of this pass, unless the previous pass gathered them
              if (p != pnext && act) ldv_off<KV>(dnext, Dm, js * strideD + offD);
              float t = 0.f;
              if (act) {
  #pragma unroll
                for (int v = 0; v < KV; ++v) t = fmaf(c[v], dnext[v], t);
              }
              t = group_sum<PS>(t);
              y = bs * t;
              if (act && q == 0) out[p + sub] = y;
              // Gather the next pass's D rows before this pass's loop
              // overhead and store.  The next pass starts at p + n and takes
              // at most NB nonzeros, none past the window or the slice (it
              // may belong to the next row: its dot waits for that row's C_i,
              // not for D).  If the window ends here, the next pass refills
              // it and gathers its own rows.
              const int64_t pn = p + n;
              const int offn = (int)(pn - wb) + sub;
              const uint32_t jn = (uint32_t)bperm_i((gbase + offn) & 63, wj);
              if (pn - wb < W) {
                pnext = pn;
                if (offn < W && pn + sub < p1) ldv_off<KV>(dnext, Dm, jn * strideD + offD);
              } else {
                pnext = -((int64_t)1 << 40);
              }
            } else {
              float dr[KV];
              float t = 0.f;
              if (act) {
                ldv_off<KV>(dr, Dm, js * strideD + offD);
  #pragma unroll
                for (int v = 0; v < KV; ++v) t = fmaf(c[v], dr[v], t);
              }
              t = group_sum<PS>(t);
              y = bs * t;
            }
          }
          if (MODE != kSddmm && SCHED == kPaced) {
            // consumer: the whole worker streams each E row, one row issued
            // after the previous one has arrived
            uint32_t jj[NB];
            float yy[NB];
  #pragma unroll
            for (int u = 0; u < NB; ++u) {
              const int src = (gbase + off + u) & 63;
              jj[u] = (uint32_t)bperm_i(src, wj);
              yy[u] = (MODE == kSpmm) ? bperm_f(src, wv) : bperm_f((gbase + u * PS) & 63, y);
            }
            float er[NB][LV];
  #pragma unroll
            for (int u = 0; u < NB; ++u) {
              if (u < n) {
                if (u > 0) wait_vmcnt<1>();
                ldv_off<LV>(er[u], Em, jj[u] * strideE + offE);
              }
            }
  #pragma unroll
            for (int u = 0; u < NB; ++u) {
              if (u < n) {
  #pragma unroll
                for (int v = 0; v < LV; ++v) acc[v] = fmaf(yy[u], er[u][v], acc[v]);
              }
            }
          } else if (MODE != kSddmm) {
            // consumer: the whole worker streams each E row, depth-2 pipeline
            float ea[LV], eb[LV];
            float ya = 0.f, yb = 0.f;
            auto issue = [&](float (&e)[LV], float &yv, int u) {
              const int src = gbase + off + u;
              const uint32_t j = (uint32_t)bperm_i(src, wj);
              yv = (MODE == kSpmm) ? bperm_f(src, wv) : bperm_f(gbase + u * PS, y);
              ldv_off<LV>(e, Em, j * strideE + offE);
            };
            auto consume = [&](const float (&e)[LV], float yv) {
  #pragma unroll
              for (int v = 0; v < LV; ++v) acc[v] = fmaf(yv, e[v], acc[v]);
            };
            issue(ea, ya, 0);
            int u = 1;
            for (; u + 1 < n; u += 2) {
              issue(eb, yb, u);
              consume(ea, ya);
              issue(ea, ya, u + 1);
              consume(eb, yb);
            }
            if (u < n) {
              issue(eb, yb, u);
              consume(ea, ya);
              consume(eb, yb);
            } else {
              consume(ea, ya);
            }
          }
        }
        p += n;
      }
  }
};

// ------------------------------------------------------ fast-path kernel
//
// One worker (W lanes) per merge-path slice; per row of the slice, C_i is
// loaded once, RowWalk applies the row's nonzeros, and the row (or its
// partial) is stored.  Besides the nonzero window of RowWalk, a rowptr
// window (one row end per lane) keeps the row ends off the critical path.
// C_i, the CSR arrays and A are streamed once per call and carry the
// nontemporal hint.
template <int MODE, int W, int NB, int KV, int LV, int SCHED, int U>
__global__ __launch_bounds__(256) void walk_fast(WalkArgs a) {
  const Slice s = make_slice<W>(a);
  if (!s.active) return;
  RowWalk<MODE, W, NB, KV, LV, SCHED, U> rw(a, s.p1, (uint32_t)a.L * 4u);
  const int glane = rw.glane, gbase = rw.gbase;
  const int64_t worker = s.id;  // carry slots and metadata are per slice
  int32_t *meta = a.meta + 2 * worker;
  const int32_t *__restrict__ rowptr = a.rowptr;
  const float *__restrict__ Cm = a.C;
  float *__restrict__ out = a.out;
  const int64_t K = a.K, L = a.L, N = a.N;
  constexpr int64_t kFar = -((int64_t)1 << 40);

  int64_t i = s.i0, p = s.p0;
  int64_t rb = kFar;  // rowptr window: wr = rowptr[rb + glane]
  int wr = 0;
  while (true) {
    const bool has_end = i < s.i1;
    if (!has_end && i >= N) break;
    int64_t r_end = s.p1;
    if (has_end) {
      if (i + 1 >= rb + W) {
        rb = i + 1;
        if (rb + glane <= N) wr = kNT ? ld_stream(rowptr + rb + glane) : rowptr[rb + glane];
      }
      r_end = bperm_i(gbase + (int)(i + 1 - rb), wr);
    }
    float acc[LV];
#pragma unroll
    for (int v = 0; v < LV; ++v) acc[v] = 0.f;
    float c[KV];
#pragma unroll
    for (int v = 0; v < KV; ++v) c[v] = 0.f;
    if (MODE != kSpmm && p < r_end) ldv<KV, kNT>(c, Cm + i * K + rw.q * KV);
    rw.row(p, r_end, c, acc);
    if constexpr (MODE != kSddmm) {
      if (!has_end) stv<LV>(a.carry + (worker * 2 + 1) * (int64_t)a.Lw + glane * LV, acc);
      else if (i == s.i0 && s.head) stv<LV>(a.carry + (worker * 2) * (int64_t)a.Lw + glane * LV, acc);
      else stv<LV, kNT>(out + i * L + glane * LV, acc);
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
  const Slice s = make_slice<64>(a);
  if (!s.active) return;
  const int64_t worker = s.id;  // carry slots and metadata are per slice
  int32_t *meta = a.meta + 2 * worker;
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
// A slice whose first row is a head row (begun by earlier slices) owns that
// row's fixup: it adds, in slice order, the tail partials of the earlier
// slices that end inside the row, then its own head partial, and writes the
// row of A.  Each wave takes groups of G consecutive slices (G a power of
// two up to 64, grid-stride): lanes 0..G-1 read the group's head entries at
// once and the wave then fixes the group's head rows one after another.  The
// host picks G so that the grid holds at most 32 waves per CU: a call on a
// small matrix does not pay for one wave per possible slice, and a power-law
// matrix, where a large share of the slices start inside a long row, still
// spreads its head rows over many waves.

// The run of slices [first, c) whose tail row is r (they are contiguous and
// end at c - 1), found with one ballot per 64 slices.  Uniform in the wave.
__device__ __forceinline__ int64_t tail_run_start(const int32_t *__restrict__ meta, int64_t c,
                                                  int32_t r) {
  const int lane = threadIdx.x & 63;
  int64_t first = c;
  while (true) {
    const int64_t idx = first - 1 - lane;
    const bool same = idx >= 0 && meta[2 * idx] == r;
    const uint64_t m = __ballot(same);
    const int run = (~m == 0) ? 64 : __builtin_ctzll(~m);
    first -= run;
    if (run < 64) break;
  }
  return first;
}

// Partials first .. c-1 (tail slots) and c (head slot) of one row summed in
// slice order, V consecutive columns per lane (V = 4: one 16-byte load per
// partial, so a row of Lw columns takes Lw / 256 passes instead of Lw / 64;
// each column's sum is taken in the same order either way, so the results
// are bit-identical).  The loads of a batch are issued together, so a row
// split over hundreds of slices (a power-law hub row) costs a few memory
// latencies rather than one per slice.
template <int V>
__device__ __forceinline__ void fix_cols(const float *__restrict__ carry, float *__restrict__ arow,
                                         int64_t Lw, int64_t first, int64_t c) {
  typedef typename std::conditional<V == 4, f4_t, float>::type vec;
  constexpr int kBatch = V == 4 ? 4 : 16;
  const int lane = threadIdx.x & 63;
  auto at = [&](int64_t slot, int64_t l) {
    return *reinterpret_cast<const vec *>(carry + slot * Lw + l);
  };
  for (int64_t l = (int64_t)V * lane; l < Lw; l += 64 * V) {
    vec sum = vec{};
    int64_t cc = first;
    for (; cc + kBatch <= c; cc += kBatch) {
      vec v[kBatch];
#pragma unroll
      for (int t = 0; t < kBatch; ++t) v[t] = at((cc + t) * 2 + 1, l);
#pragma unroll
      for (int t = 0; t < kBatch; ++t) sum += v[t];
    }
    if (cc < c) {
      vec v[kBatch];
#pragma unroll
      for (int t = 0; t < kBatch; ++t)
        if (cc + t < c) v[t] = at((cc + t) * 2 + 1, l);
#pragma unroll
      for (int t = 0; t < kBatch; ++t)
        if (cc + t < c) sum += v[t];
    }
    sum += at(c * 2, l);
    *reinterpret_cast<vec *>(arow + l) = sum;
  }
}

// Row r of A from its partials: 16-byte pieces when the widths and the
// addresses allow them (uniform over the grid), single floats otherwise.
__device__ __forceinline__ void fix_row(const WalkArgs &a, int64_t c, int32_t r) {
  const int64_t Lw = a.Lw;
  const int64_t first = tail_run_start(a.meta, c, r);
  float *const arow = a.out + (int64_t)r * a.L + a.l0;
  const bool v4 = (Lw & 3) == 0 && (a.L & 3) == 0 && (a.l0 & 3) == 0 &&
                  (reinterpret_cast<uintptr_t>(a.out) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(a.carry) & 15) == 0;
  if (v4) fix_cols<4>(a.carry, arow, Lw, first, c);
  else fix_cols<1>(a.carry, arow, Lw, first, c);
}

__global__ __launch_bounds__(256) void carry_fixup(WalkArgs a, int G) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t waves = (int64_t)gridDim.x * (blockDim.x >> 6);
  int64_t S, ns, items, nnz;
  slice_count(a, &S, &ns, &items, &nnz);
  // meta entries past ns belong to no slice of this call and are never read
  for (int64_t g0 = wave * G; g0 < ns; g0 += waves * G) {
    const int64_t cl = g0 + lane;
    const int32_t rl = (lane < G && cl < ns) ? a.meta[2 * cl + 1] : -1;
    uint64_t heads = __ballot(rl >= 0);
    while (heads) {  // wave-uniform
      const int b = __builtin_ctzll(heads);
      heads &= heads - 1;
      fix_row(a, g0 + b, bperm_i(b, rl));
    }
  }
}

// ------------------------------------------------------------ Hadamard
//
// H = C .* D elementwise over n4 float4 elements (16-byte aligned arrays),
// grid-stride.  C and D are streamed once (nontemporal); H is stored plainly
// because the walk that follows gathers it.  Gated like the walks: the
// launch does nothing unless its gate is open.
__global__ __launch_bounds__(256) void hadamard4_kernel(const float *__restrict__ C,
                                                        const float *__restrict__ D,
                                                        float *__restrict__ H, int64_t n4,
                                                        const int32_t *rowptr, int64_t N,
                                                        int64_t gate_nnz, int gate) {
  if (gate_closed(gate, rowptr, N, gate_nnz)) return;
  const f4_t *c4 = reinterpret_cast<const f4_t *>(C);
  const f4_t *d4 = reinterpret_cast<const f4_t *>(D);
  f4_t *h4 = reinterpret_cast<f4_t *>(H);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n4; t += stride) {
    const f4_t x = __builtin_nontemporal_load(c4 + t);
    const f4_t y = __builtin_nontemporal_load(d4 + t);
    h4[t] = x * y;
  }
}

// ------------------------------------------------------------ transpose
//
// dst (cols x rows) = src (rows x cols) transposed, through a 32 x 32 tile in
// LDS so that both the reads and the writes are coalesced.  Block 32 x 8.
__global__ __launch_bounds__(256) void transpose_kernel(const float *__restrict__ src,
                                                        float *__restrict__ dst, int64_t rows,
                                                        int64_t cols, int64_t tiles_c) {
  __shared__ float tile[32][33];
  const int64_t tr = blockIdx.x / tiles_c, tc = blockIdx.x % tiles_c;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  const int64_t r0 = tr * 32, c0 = tc * 32;
#pragma unroll
  for (int k = 0; k < 32; k += 8) {
    const int64_t r = r0 + ty + k, c = c0 + tx;
    if (r < rows && c < cols) tile[ty + k][tx] = src[r * cols + c];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 32; k += 8) {
    const int64_t c = c0 + ty + k, r = r0 + tx;
    if (r < rows && c < cols) dst[c * rows + r] = tile[tx][ty + k];
  }
}

// The same for rows and cols multiples of 4 and 16-byte aligned arrays: a
// 64 x 64 tile per block of 256 threads, read and written as float4 (16 lanes
// cover 256 contiguous bytes of a row on both sides).  The LDS pitch of 65
// makes the column reads of the write phase conflict-free.
__global__ __launch_bounds__(256) void transpose4_kernel(const float *__restrict__ src,
                                                         float *__restrict__ dst, int64_t rows,
                                                         int64_t cols, int64_t tiles_c) {
  __shared__ float tile[64][65];
  const int64_t tr = blockIdx.x / tiles_c, tc = blockIdx.x % tiles_c;
  const int64_t r0 = tr * 64, c0 = tc * 64;
  const int q = threadIdx.x & 15, g = threadIdx.x >> 4;  // float4 column, row group
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int lr = g + 16 * it;
    const int64_t r = r0 + lr, c = c0 + 4 * q;
    if (r < rows && c < cols) {  // cols % 4 == 0: the float4 lies inside the row
      const f4_t x = __builtin_nontemporal_load(reinterpret_cast<const f4_t *>(src + r * cols + c));
      tile[lr][4 * q] = x[0];
      tile[lr][4 * q + 1] = x[1];
      tile[lr][4 * q + 2] = x[2];
      tile[lr][4 * q + 3] = x[3];
    }
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int lc = g + 16 * it;
    const int64_t c = c0 + lc, r = r0 + 4 * q;
    if (c < cols && r < rows) {  // rows % 4 == 0
      f4_t x;
      x[0] = tile[4 * q][lc];
      x[1] = tile[4 * q + 1][lc];
      x[2] = tile[4 * q + 2][lc];
      x[3] = tile[4 * q + 3][lc];
      *reinterpret_cast<f4_t *>(dst + c * rows + r) = x;
    }
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
