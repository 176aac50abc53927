// Device code of the per-row epilogue kernel of the fused SDDMM->SpMM
// library for gfx950: the <SDDMM, SpMM, GEMM>, <SpMM, GEMM> and
// <SpMMH, GEMM> computations of the paper's Section 6.2, built on the
// merge-path walk of walker.hpp.
#pragma once

#include "walker.hpp"

namespace slnr {

// ------------------------------------------------------- epilogue kernel
//
// <SDDMM, SpMM, GEMM>, <SpMM, GEMM> and <SpMMH, GEMM> of the paper's Section
// 6.2: the row t_i of the sparse product (fused SDDMM->SpMM, or an SpMM whose
// gathered row is E_j, or E_j .* G2_j for the Hadamard form) is multiplied by
// the dense Wep (Lin x Lout) before it is stored, A_i = t_i Wep.  The product
// is linear, so the partial rows of a row split between slices take it too
// and the carry fixup adds them.
//
// The walk is RowWalk (W lanes per worker, LV floats of the row per lane;
// the schedule is a template choice), run as a loop that is uniform across
// the wave: a worker whose slice is done idles.  A worker that finishes a row with
// nonzeros in its slice writes t_i to its wave's tile in LDS (TR rows, filled
// in order across the wave's workers) and the row's destination (an A row or
// a carry slot) beside it.  Once the next round of rows might not fit, the
// wave multiplies the tile on the matrix cores: v_mfma_f32_4x4x1f32 over
// quads of rows, one input k per step, lane l supplying t[4q + (l & 3)][k]
// and Wep[k][l] and receiving column l of the four rows, so each row is
// stored by 64 lanes in one coalesced pass per 64 columns.  Wep is read
// through the caches (it is small and every wave reads it), which leaves LDS
// to the tiles.
//
// With WL = 1 the block first copies the whole Wep into LDS (one copy shared
// by the block's waves, which are then many: the host launches up to 16
// waves per block) and the tile products read it from there; otherwise they
// read it through the caches.  LDS layout: [Wep, Lin x Lout floats rounded
// up to a multiple of 4] [tiles, TR rows of TS floats per wave]
// [destinations, TR per wave].
template <int MODE, int W, int LV, int HAD, int TR, int SCHED, int U, int WL = 0>
__global__ __launch_bounds__(WL ? 1024 : 256) void walk_epi(WalkArgs a) {
  constexpr int KV = LV;  // fused form: K = Lin
  constexpr int LIN = W * LV;
  constexpr int WPW = 64 / W;  // workers per wave
  constexpr int TS = LIN + 4;  // tile row stride in floats (16-byte rows, staggered banks)
  static_assert(MODE == kFused || MODE == kSpmm, "mode");
  static_assert(TR % 4 == 0 && TR >= WPW && TR <= 16, "tile rows");
  static_assert(!(HAD && MODE == kFused), "Hadamard rows come with the SpMM form");
  extern __shared__ float smem[];
  const int lane = threadIdx.x & 63;
  const int glane = lane & (W - 1);
  const int gbase = lane - glane;
  const int wave = threadIdx.x >> 6;
  const int wsize = WL ? ((LIN * a.L + 3) & ~3) : 0;  // floats of the staged Wep
  float *wlds = smem;
  float *tile = smem + wsize + wave * (TR * TS);
  uint64_t *tdst =
      reinterpret_cast<uint64_t *>(smem + wsize + (blockDim.x >> 6) * (TR * TS)) + wave * TR;

  if (gate_closed(a.gate, a.rowptr, a.N, a.gate_nnz)) return;
  if constexpr (WL) {  // the whole block takes part (the gate is uniform over the grid)
    const int n = LIN * a.L;
    for (int t = threadIdx.x; t < n; t += blockDim.x) wlds[t] = a.Wep[t];
    __syncthreads();
  }
  const Slice s = make_slice<W>(a);
  const int64_t worker = s.id;
  RowWalk<MODE, W, 1, KV, LV, SCHED, U, HAD> rw(a, s.p1, (uint32_t)LIN * 4u);
  const int32_t *__restrict__ rowptr = a.rowptr;
  const float *__restrict__ Cm = a.C;
  const float *__restrict__ Wm = a.Wep;
  float *__restrict__ out = a.out;
  const int64_t K = a.K, L = a.L, N = a.N;
  const int lout = a.L;
  constexpr int64_t kFar = -((int64_t)1 << 40);

  // Tile product and stores of rows 0..cnt-1.  All lanes of the wave take
  // part (the caller is in uniform control flow).  Inputs go in blocks of
  // kBk steps of 4, and the Wep values of the next block are loaded while
  // the current block is multiplied: two steps for the SpMM forms, one for
  // the fused form, whose walk needs the registers (measured on MI355X).
  constexpr int kBk = MODE == kFused ? 1 : 2;
  static_assert(LIN % (4 * kBk) == 0, "input blocks");
  auto flush = [&](int cnt) {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    const int nq = (cnt + 3) >> 2;
    const float *arow = tile + (lane & 3) * TS;
    for (int c0 = 0; c0 < lout; c0 += 64) {
      const int col = c0 + lane;
      const int wc = col < lout ? col : c0;  // lanes past Lout read a valid column
      const float *wcol = WL ? wlds + wc : Wm + wc;
      f4_t o[TR / 4];
#pragma unroll
      for (int q = 0; q < TR / 4; ++q) o[q] = f4_t{0.f, 0.f, 0.f, 0.f};
      float bn[4 * kBk];
#pragma unroll
      for (int t = 0; t < 4 * kBk; ++t) bn[t] = wcol[t * lout];
#pragma unroll 1
      for (int k0 = 0; k0 < LIN; k0 += 4 * kBk) {
        float b[4 * kBk];
#pragma unroll
        for (int t = 0; t < 4 * kBk; ++t) b[t] = bn[t];
        if (k0 + 4 * kBk < LIN) {
#pragma unroll
          for (int t = 0; t < 4 * kBk; ++t) bn[t] = wcol[(int64_t)(k0 + 4 * kBk + t) * lout];
        }
#pragma unroll
        for (int u = 0; u < kBk; ++u) {
#pragma unroll
          for (int q = 0; q < TR / 4; ++q) {
            if (q < nq) {
              const f4_t av = *reinterpret_cast<const f4_t *>(arow + q * 4 * TS + k0 + 4 * u);
#pragma unroll
              for (int kk = 0; kk < 4; ++kk)
                o[q] = __builtin_amdgcn_mfma_f32_4x4x1f32(av[kk], b[4 * u + kk], o[q], 0, 0, 0);
            }
          }
        }
      }
      if (col < lout) {
#pragma unroll
        for (int q = 0; q < TR / 4; ++q) {
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int r = 4 * q + v;
            if (r < cnt) {
              // destination: element offset << 1, low bit set for a carry slot
              const uint64_t dd = tdst[r];
              const int64_t off = (int64_t)(dd >> 1) + col;
              if (dd & 1) a.carry[off] = o[q][v];
              else __builtin_nontemporal_store(o[q][v], out + off);
            }
          }
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  };

  int64_t i = s.i0, p = s.p0;
  int64_t rb = kFar;  // rowptr window: wr = rowptr[rb + glane]
  int wr = 0;
  int cnt = 0;  // rows waiting in the tile (the same in every lane)
  bool live = s.active;
  while (__ballot(live) != 0) {
    float acc[LV];
#pragma unroll
    for (int v = 0; v < LV; ++v) acc[v] = 0.f;
    bool fin = false;
    uint64_t dd = 0;
    if (live) {
      const bool has_end = i < s.i1;
      if (!has_end && i >= N) {
        live = false;
      } else {
        int64_t r_end = s.p1;
        if (has_end) {
          if (i + 1 >= rb + W) {
            rb = i + 1;
            if (rb + glane <= N) wr = ld_stream(rowptr + rb + glane);
          }
          r_end = bperm_i(gbase + (int)(i + 1 - rb), wr);
        }
        const int64_t row_start = p;
        float c[KV];
#pragma unroll
        for (int v = 0; v < KV; ++v) c[v] = 0.f;
        if (MODE == kFused && p < r_end) ldv<KV, kNT>(c, Cm + i * K + glane * KV);
        rw.row(p, r_end, c, acc);
        // destination: a row of A, or a carry slot of a row split between slices
        int64_t off = i * L;
        bool carry = false;
        if (!has_end) {
          off = (worker * 2 + 1) * (int64_t)a.Lw;
          carry = true;
        } else if (i == s.i0 && s.head) {
          off = (worker * 2) * (int64_t)a.Lw;
          carry = true;
        }
        if (p == row_start) {  // no nonzero of the row in this slice: a zero product
          for (int l = glane; l < lout; l += W) {
            if (carry) a.carry[off + l] = 0.f;
            else __builtin_nontemporal_store(0.f, out + off + l);
          }
        } else {
          fin = true;
          dd = ((uint64_t)off << 1) | (carry ? 1u : 0u);
        }
        if (!has_end) live = false;
        else ++i;
      }
    }
    // uniform point: finished rows take the next tile rows, in worker order
    const uint64_t fm = __ballot(fin && glane == 0);
    if (fm != 0) {
      if (fin) {
        const int r = cnt + __builtin_popcountll(fm & ((1ull << gbase) - 1));
        stv<LV>(tile + r * TS + glane * LV, acc);
        if (glane == 0) tdst[r] = dd;
      }
      cnt += __builtin_popcountll(fm);
      if (cnt > TR - WPW) {
        flush(cnt);
        cnt = 0;
      }
    }
  }
  if (cnt > 0) flush(cnt);
  if (s.active && glane == 0) {
    int32_t *meta = a.meta + 2 * worker;
    meta[0] = s.i1 < N ? (int32_t)s.i1 : -1;
    meta[1] = s.head ? (int32_t)s.i0 : -1;
  }
}

}  // namespace slnr
