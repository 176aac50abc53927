// Host side of the fused SDDMM->SpMM library: argument checks, variant
// choice, workspace management and launches.  The C ABI is declared in
// include/sparselnr.h.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <cstdlib>
#include <map>
#include <mutex>
#include <utility>

#include "sparselnr.h"
#include "walker.hpp"
#include "epilogue.hpp"

namespace {

using slnr::WalkArgs;

thread_local int g_last_hip_error = 0;

constexpr int kBlock = 256;       // threads per block (4 waves)
// The plain walks (walk_fast) launch one wave per block.  Measured on
// MI355X against 4-wave blocks: fused 1.2-2.9% and unfused 0.7-3.6% faster
// on R-MAT 2^20 / 2^22, the 27-point stencil and 2048 rows of 10 nonzeros
// (uniform 65536 x 16: fused +1.5%, unfused -1.4%).  Smaller blocks leave the
// dispatcher a finer-grained tail and spread each XCD's share more evenly.
constexpr int kWalkBlock = 64;
constexpr int kMinChunk = 64;     // smallest merge-path slice per worker (see slice_count)
constexpr int kXcds = 8;          // MI355X deals blocks over 8 XCDs
constexpr int kGridFactor = 8;    // resident grids per walk launch for large inputs
constexpr int kGenericLT = 4;     // generic path: 4 x 64 = 256 columns per tile
// <SpMMH, GEMM>: C .* D is formed once when nnz >= kHoistRatio * M (12 M J
// bytes for the product against 4 J bytes per nonzero for a second gather).
constexpr int64_t kHoistRatio = 3;

int hip_fail(hipError_t e) {
  g_last_hip_error = (int)e;
  return SPARSELNR_ERR_HIP;
}

struct Workspace {
  void *ptr = nullptr;
  size_t bytes = 0;
};

std::mutex g_mu;
std::map<int, int> g_cus;                                    // device -> CUs
std::map<std::pair<int, std::pair<uintptr_t, size_t>>, int> g_occupancy;  // (device, (kernel, LDS)) -> blocks/CU
// Resident grids per walk launch: 0 not read yet (SPARSELNR_GRID_FACTOR gives
// the first value), -1 chosen per call by size, 1..kMaxGridFactor fixed
// (sparselnr_set_grid_factor).
constexpr int kMaxGridFactor = 64;
std::atomic<int> g_grid_factor{0};
// workspaces per (device, stream, slot): slot 0 carry partials, slot 1 the
// transposed D of the transposed-D entry point
struct WsKey {
  int dev;
  uintptr_t stream;
  int slot;
  bool operator<(const WsKey &o) const {
    if (dev != o.dev) return dev < o.dev;
    if (stream != o.stream) return stream < o.stream;
    return slot < o.slot;
  }
};
std::map<WsKey, Workspace> g_workspace;

int current_device(int *dev) {
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return hip_fail(e);
  return SPARSELNR_OK;
}

std::map<int, size_t> g_max_lds;  // device -> largest LDS of one block

int device_max_lds(int dev, size_t *out) {
  std::lock_guard<std::mutex> lock(g_mu);
  auto it = g_max_lds.find(dev);
  if (it != g_max_lds.end()) {
    *out = it->second;
    return SPARSELNR_OK;
  }
  int n = 0;
  hipError_t e = hipDeviceGetAttribute(&n, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return hip_fail(e);
  g_max_lds[dev] = n > 0 ? (size_t)n : 0;
  *out = g_max_lds[dev];
  return SPARSELNR_OK;
}

int device_cus(int dev, int *cus) {
  std::lock_guard<std::mutex> lock(g_mu);
  auto it = g_cus.find(dev);
  if (it != g_cus.end()) {
    *cus = it->second;
    return SPARSELNR_OK;
  }
  int n = 0;
  hipError_t e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_fail(e);
  if (n <= 0) n = 1;
  g_cus[dev] = n;
  *cus = n;
  return SPARSELNR_OK;
}

// Workspace of at least `bytes` for (device, stream); grows by reallocation
// after the stream has drained (only on the first calls of a new shape).
int get_workspace(int dev, hipStream_t stream, size_t bytes, void **out, int slot = 0) {
  std::lock_guard<std::mutex> lock(g_mu);
  Workspace &w = g_workspace[WsKey{dev, (uintptr_t)stream, slot}];
  if (w.bytes < bytes) {
    if (w.ptr) {
      hipError_t e = hipStreamSynchronize(stream);
      if (e != hipSuccess) return hip_fail(e);
      e = hipFree(w.ptr);
      w.ptr = nullptr;
      w.bytes = 0;
      if (e != hipSuccess) return hip_fail(e);
    }
    void *p = nullptr;
    hipError_t e = hipMalloc(&p, bytes);
    if (e != hipSuccess) {
      g_last_hip_error = (int)e;
      (void)hipGetLastError();
      return SPARSELNR_ERR_NO_MEMORY;
    }
    w.ptr = p;
    w.bytes = bytes;
  }
  *out = w.ptr;
  return SPARSELNR_OK;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// The fast kernels address gathered rows with 32-bit byte offsets.
bool offsets32(int64_t rows, int64_t width) { return rows * width * 4 < ((int64_t)1 << 32); }

// ----------------------------------------------------------- variants

enum Mode { kFused = slnr::kFused, kSddmm = slnr::kSddmm, kSpmm = slnr::kSpmm };

using KernelFn = void (*)(WalkArgs);

struct Variant {
  KernelFn fn = nullptr;
  int W = 64;          // lanes per worker
  bool generic = true; // generic kernel (l-tiles of 256 columns)
  size_t lds = 0;      // dynamic LDS bytes per block (the epilogue matrix)
  int block = kBlock;  // threads per block
  KernelFn fn_small = nullptr;  // same mapping, for inputs that fit one resident grid
  KernelFn fn_wide = nullptr;   // wider workers, for inputs that need several resident grids
  int W_wide = 64;
  KernelFn fn_fine = nullptr;   // same mapping, for grids of at least fine_factor resident grids
  int fine_factor = 0;
};

template <int MODE, int W, int NB, int KV, int LV, int SCHED = slnr::kPipelined, int U = 1>
Variant fast() {
  Variant v;
  v.fn = slnr::walk_fast<MODE, W, NB, KV, LV, SCHED, U>;
  v.W = W;
  v.generic = false;
  v.block = kWalkBlock;
  return v;
}

// Epilogue kernel: W-lane workers, Lin = W * LV, tiles of TR rows per wave,
// pipelined walk.  (The paced walk of the plain fused kernel needs 20 more
// VGPRs here and measured 27-30% slower for the fused form on MI355X.)
template <int MODE, int W, int LV, int HAD, int TR>
Variant epi() {
  Variant v;
  v.fn = slnr::walk_epi<MODE, W, LV, HAD, TR, slnr::kPipelined, 1>;
  v.W = W;
  v.generic = false;
  constexpr int TS = W * LV + 4;
  v.lds = (size_t)(kBlock / 64) * TR * (TS * sizeof(float) + sizeof(uint64_t));
  return v;
}

// The same with the dense matrix staged in LDS once per block of `block`
// threads (Lin x Lout floats, Lout known per call).
template <int MODE, int W, int LV, int HAD, int TR>
Variant epi_wl(int64_t Lout, int block) {
  Variant v;
  v.fn = slnr::walk_epi<MODE, W, LV, HAD, TR, slnr::kPipelined, 1, 1>;
  v.W = W;
  v.generic = false;
  v.block = block;
  constexpr int LIN = W * LV;
  constexpr int TS = LIN + 4;
  const size_t wfloats = ((size_t)LIN * Lout + 3) & ~(size_t)3;
  v.lds = wfloats * sizeof(float) + (size_t)(block / 64) * TR * (TS * sizeof(float) +
                                                                   sizeof(uint64_t));
  return v;
}

template <int MODE>
Variant generic() {
  Variant v;
  v.fn = slnr::walk_generic<MODE, kGenericLT>;
  v.W = 64;
  v.generic = true;
  return v;
}

// Gather schedule of the fused kernels and of the unfused (SDDMM, SpMM)
// kernels, each set to what measured fastest for it on MI355X: the fused
// kernels pace their gathers (the K = 16, L = 256 one only for coarse slices,
// see with_fine), the unfused ones pipeline them.  Nonzeros per
// step of the paced schedule: 8 for the 128-wide rows, 4 otherwise (the
// 64-lane kernels of large inputs take their own, below).
constexpr int kFS = slnr::kPaced;
constexpr int kUS = slnr::kPipelined;
constexpr int kPU = 4;
constexpr int kPU128 = 8;

// Inputs that fit one resident grid (few rows per worker) run with more
// nonzeros per paced step at K = L = 32 and 64 (measured on MI355X: 8 per step
// is 8% faster on 65536 rows of 16 nonzeros, 4 is 1% faster on R-MAT 2^22).
constexpr int kPUs = 8;
// Gather schedule of the small-input fused kernel at K = L = 32: all gathers
// of a step at once.  Measured on MI355X, 2048 rows of 10 nonzeros (16-item
// slices): 12.3 us per call against 13.2 paced.  At K = L = 64 the burst
// walk is 5% slower on 65536 rows of 16 nonzeros, which keep 64-item slices
// and the paced walk.
constexpr int kSmall32 = slnr::kBurst;

// The 64-lane fused kernel of large inputs at K = L = 128 takes 10 nonzeros
// per paced step (measured on MI355X, R-MAT 2^20: 1.5-2.3% faster than 8 on
// two boxes; 6 and 16 slower, as are 2 or 3 loads in flight per issue).
constexpr int kPU128W = 10;

Variant with_small(Variant v, KernelFn small) {
  v.fn_small = small;
  return v;
}

// Large inputs (several resident grids) walk with one 64-lane worker per
// wave instead of several narrower ones.  Measured on MI355X, the fused
// kernel and both unfused passes at K = L = 64 and 128 on R-MAT graphs with
// 2^20 and 2^22 vertices: 1-8% faster (fewer nonzeros in flight per CU keep
// the gathered rows of an XCD's workers closer together in L2).  Inputs
// that fit one resident grid keep the narrow workers: on 65536 rows of 16
// nonzeros the 64-lane walk is 35-55% slower (4x fewer workers).
template <int MODE, int KV, int LV, int SCHED, int U>
Variant with_wide(Variant v) {
  v.fn_wide = slnr::walk_fast<MODE, 64, 1, KV, LV, SCHED, U>;
  v.W_wide = 64;
  return v;
}

// Fine slices (many resident grids per launch) take the pipelined schedule.
// Measured on MI355X, the fused kernel at K = 16, L = 256 on the 27-point
// stencil of a 128^3 grid (2^21 rows), ms per call by resident grids:
//             8     12     24     48     64
//   paced   5.85  5.77   5.79   5.80   6.02
//   piped   6.61  6.10   5.61   5.04   5.09
// With fine slices the rows walked at one moment on an XCD lie close
// together and their E rows come back from the caches; the pipelined walk
// holds 56 fewer registers of gathered rows than the 16-nonzero paced step,
// so more waves share the CU and more gathers are in flight.  With coarse
// slices the gathers go further out and the paced walk, which keeps fewer
// in flight per wave, is faster.
template <int MODE, int W, int NB, int KV, int LV, int U>
Variant with_fine(Variant v, int from) {
  v.fn_fine = slnr::walk_fast<MODE, W, NB, KV, LV, slnr::kPipelined, U>;
  v.fine_factor = from;
  return v;
}

// Lane mapping of a fused fast variant for K, L in {16, ..., 512}: the
// consumer spreads E_j / A_i over W lanes of LV floats (L = W * LV); the
// producer forms NB dot products per pass, each over PS = W / NB lanes of KV
// floats (K = PS * KV).  LV is 4 (8 at L = 512) unless K is so wide against
// L that a dot over all W lanes would need more than 16 floats per lane;
// then the consumer takes 2 or 1 floats per lane on more lanes.  KV is 4
// where it fits, larger when K is wide against L (one dot per pass over the
// whole worker, at most 32 floats), 2 when 4 would need more than 64
// registers of gathered E rows per pass.  U: nonzeros per paced step (NB for
// the multi-dot passes, else as many as 64 registers of gathered rows allow,
// at most 4).  W == 0: no fast variant.
struct FusedMap {
  int W, LV, KV, NB, U;
};

constexpr FusedMap fused_map(int K, int L) {
  int LV = L == 512 ? 8 : 4;
  while (LV > 1 && K / (L / LV) > 16) LV /= 2;
  const int W = L / LV;
  if (W > 64) return FusedMap{0, 0, 0, 0, 0};
  int KV = 4;
  while (KV <= 32 && K / KV > W) KV *= 2;
  if (KV > 32) return FusedMap{0, 0, 0, 0, 0};
  int PS = K / KV;
  int NB = W / PS;
  if (NB * LV > 64) {
    KV = 2;
    PS = K / KV;
    NB = W / PS;
  }
  if (PS < 1 || PS > W || NB * PS != W || NB * LV > 64) return FusedMap{0, 0, 0, 0, 0};
  const int fit = 64 / (KV + LV);
  const int U = NB > 1 ? NB : (fit < 1 ? 1 : (fit < 4 ? fit : 4));
  return FusedMap{W, LV, KV, NB, U};
}

template <int K, int L>
Variant fused_fast() {
  constexpr FusedMap m = fused_map(K, L);
  if constexpr (m.W == 0) {
    return generic<kFused>();
  } else {
    return fast<kFused, m.W, m.NB, m.KV, m.LV, kFS, m.U>();
  }
}

template <int K>
Variant fused_fast_l(int64_t L) {
  switch (L) {
    case 16: return fused_fast<K, 16>();
    case 32: return fused_fast<K, 32>();
    case 64: return fused_fast<K, 64>();
    case 128: return fused_fast<K, 128>();
    case 256: return fused_fast<K, 256>();
    case 512: return fused_fast<K, 512>();
    default: return generic<kFused>();
  }
}

// Fast variants exist for every K, L in {16, 32, 64, 128, 256, 512}, with
// 16-byte aligned operands.  The widths of the benchmark workloads (K = L = 32, 64,
// 128, 256 and K = 16, L = 256) keep their measured schedules; other
// widths take the mapping of fused_map.
Variant pick_fused(int64_t K, int64_t L, bool al) {
  if (al) {
    if (K == 32 && L == 32) return with_small(fast<kFused, 8, 1, 4, 4, kFS, kPU>(),
                                              slnr::walk_fast<kFused, 8, 1, 4, 4, kSmall32, kPUs>);
    if (K == 64 && L == 64)
      return with_wide<kFused, 1, 1, kFS, kPU>(with_small(
          fast<kFused, 16, 1, 4, 4, kFS, kPU>(), slnr::walk_fast<kFused, 16, 1, 4, 4, kFS, kPUs>));
    if (K == 128 && L == 128)
      return with_wide<kFused, 2, 2, kFS, kPU128W>(fast<kFused, 32, 1, 4, 4, kFS, kPU128>());
    if (K == 256 && L == 256) return fast<kFused, 64, 1, 4, 4, kFS, kPU>();
    if (K == 16 && L == 256)
      return with_fine<kFused, 64, 16, 4, 4, 16>(fast<kFused, 64, 16, 4, 4, kFS, 16>(), 24);
    switch (K) {
      case 16: return fused_fast_l<16>(L);
      case 32: return fused_fast_l<32>(L);
      case 64: return fused_fast_l<64>(L);
      case 128: return fused_fast_l<128>(L);
      case 256: return fused_fast_l<256>(L);
      case 512: return fused_fast_l<512>(L);
      default: break;
    }
  }
  return generic<kFused>();
}

Variant pick_sddmm(int64_t K, bool al) {
  if (al) {
    if (K == 16) return fast<kSddmm, 64, 16, 4, 4, kUS, 16>();
    if (K == 32) return fast<kSddmm, 8, 1, 4, 4, kUS, kPU>();
    if (K == 64) return with_wide<kSddmm, 1, 1, kUS, kPU>(fast<kSddmm, 16, 1, 4, 4, kUS, kPU>());
    if (K == 128)
      return with_wide<kSddmm, 2, 2, kUS, kPU128>(fast<kSddmm, 32, 1, 4, 4, kUS, kPU128>());
    if (K == 256) return fast<kSddmm, 64, 1, 4, 4, kUS, kPU>();
    if (K == 512) return fast<kSddmm, 64, 1, 8, 4, kUS, kPU>();
  }
  return generic<kSddmm>();
}

Variant pick_spmm(int64_t L, bool al) {
  if (al) {
    if (L == 16) return fast<kSpmm, 4, 1, 4, 4, kUS, kPU>();
    if (L == 32) return fast<kSpmm, 8, 1, 4, 4, kUS, kPU>();
    if (L == 64) return with_wide<kSpmm, 1, 1, kUS, kPU>(fast<kSpmm, 16, 1, 4, 4, kUS, kPU>());
    if (L == 128)
      return with_wide<kSpmm, 2, 2, kUS, kPU128>(fast<kSpmm, 32, 1, 4, 4, kUS, kPU128>());
    if (L == 256) return fast<kSpmm, 64, 1, 4, 4, kUS, kPU>();
    if (L == 512) return fast<kSpmm, 64, 1, 4, 8, kUS, kPU>();
  }
  return generic<kSpmm>();
}

// Section 6.2 benchmarks with a per-row epilogue.  Lin (the width of the
// gathered rows and of t_i) in {16, 32, 64, 128, 256, 512}; any Lout.
// Workers of Lin / 4 lanes (4 floats per lane) from Lin = 64 on, of 16 lanes
// below: 4- and 8-lane workers put 16 and 8 workers in a wave, so a 16-row
// tile fills every round or two and is multiplied nearly empty, and the
// shorter slices of the extra workers split more rows, whose partial rows
// are Lout wide (measured on MI355X, R-MAT 2^20, <SpMM, GEMM>: 16 x 512
// 2.03 against 2.79 ms, 16 x 256 1.38 against 1.71, 32 x 512 2.25 against
// 2.52, 32 x 128 1.06 against 1.09; within 1% at Lout <= 64).  Tiles of 16
// rows per wave up to Lin = 64, 12 at 128 and 4 above, so that LDS does not
// limit occupancy (measured on MI355X, R-MAT 2^20 rows).
//
// For the fused form (<SDDMM, SpMM, GEMM>) at Lin <= 64, the dense matrix is
// staged in LDS once per block (epi_wl) when it takes at most 64 KB, with
// TRW rows per tile, and the block size is the one of 256, 512 or 1024
// threads that gives the most waves per CU within the LDS of a CU (at most
// 24, the register limit of these kernels; ties go to the larger block,
// which copies the matrix fewer times).  Measured on MI355X, R-MAT 2^20 rows
// at the paper's sizes: 2-3% faster for <SDDMM, SpMM, GEMM> (64 x 64, 512
// threads, 24 waves per CU); 1.2-1.4x slower for the SpMM forms at Lin = 128
// (64 KB or 32 KB staged leave 16 waves per CU) and 1.2x slower for
// <SpMM, GEMM> at 64 x 64, so those read the matrix through the caches.
constexpr size_t kLdsPerCu = 160 * 1024;
constexpr int kEpiWavesCap = 24;

template <int MODE, int W, int LV, int HAD, int TR, int TRW>
Variant epi_best(int64_t Lout, size_t max_lds_block) {
  constexpr int LIN = W * LV;
  if constexpr (MODE == kFused && LIN <= 64) {
    if ((int64_t)LIN * Lout * 4 > 65536) return epi<MODE, W, LV, HAD, TR>();
    Variant best{};
    int best_waves = 0;
    for (int block : {1024, 512, 256}) {
      Variant v = epi_wl<MODE, W, LV, HAD, TRW>(Lout, block);
      if (v.lds > max_lds_block || v.lds > kLdsPerCu) continue;
      int waves = (int)(kLdsPerCu / v.lds) * (block / 64);
      if (waves > kEpiWavesCap) waves = kEpiWavesCap;
      if (waves > best_waves) {
        best = v;
        best_waves = waves;
      }
    }
    if (best.fn) return best;
  }
  return epi<MODE, W, LV, HAD, TR>();
}

bool epi_width(int64_t Lin) {
  return Lin == 16 || Lin == 32 || Lin == 64 || Lin == 128 || Lin == 256 || Lin == 512;
}

template <int MODE, int HAD>
Variant pick_epi(int64_t Lin, int64_t Lout, size_t max_lds_block) {
  switch (Lin) {
    case 16: return epi_best<MODE, 16, 1, HAD, 16, 16>(Lout, max_lds_block);
    case 32: return epi_best<MODE, 16, 2, HAD, 16, 16>(Lout, max_lds_block);
    case 64: return epi_best<MODE, 16, 4, HAD, 16, 16>(Lout, max_lds_block);
    case 128: return epi_best<MODE, 32, 4, HAD, 12, 8>(Lout, max_lds_block);
    case 256: return epi_best<MODE, 64, 4, HAD, 4, 4>(Lout, max_lds_block);
    case 512: return epi_best<MODE, 64, 8, HAD, 4, 4>(Lout, max_lds_block);
    default: return Variant{};
  }
}

struct Grid {
  int blocks;
  int workers;
  int xcd_span;
  int factor;
};

// Resident blocks per CU for `fn` (occupancy query, cached per device).
int blocks_per_cu(int dev, KernelFn fn, int block, size_t lds, int *out) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_grid_factor.load() == 0) {
    const char *env = getenv("SPARSELNR_GRID_FACTOR");
    const int f = env ? atoi(env) : -1;
    int unset = 0;
    g_grid_factor.compare_exchange_strong(unset, f >= 1 && f <= kMaxGridFactor ? f : -1);
  }
  auto key = std::make_pair(dev, std::make_pair((uintptr_t)fn, lds));
  auto it = g_occupancy.find(key);
  if (it != g_occupancy.end()) {
    *out = it->second;
    return SPARSELNR_OK;
  }
  int nb = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, (const void *)fn, block, lds);
  if (e != hipSuccess) return hip_fail(e);
  if (nb <= 0) nb = 1;
  g_occupancy[key] = nb;
  *out = nb;
  return SPARSELNR_OK;
}

// The grid is `factor` resident grids.  Large matrices use kGridFactor:
// many more slices than resident workers, so the blocks resident on an XCD
// at any moment walk a compact window of rows (neighbouring rows of banded
// matrices share their D/E rows in L2) and the dispatcher balances the tail.
// Small matrices (fewer than 8 rows per resident worker) use one resident
// grid, because extra blocks would only find empty slices.  A factor > 0
// fixes the number of grids (the wide-worker kernels keep the factor chosen
// for the narrow ones).
Grid make_grid(int cus, int per_cu, int block, int W, int64_t N, int factor = 0) {
  Grid g;
  const int64_t resident_blocks = (int64_t)cus * per_cu;
  const int64_t resident_workers = resident_blocks * (block / 64) * (64 / W);
  if (factor < 1) factor = g_grid_factor.load();
  if (factor < 1) factor = N >= 8 * resident_workers ? kGridFactor : 1;
  int blocks = (int)(resident_blocks * factor);
  blocks = ((blocks + kXcds - 1) / kXcds) * kXcds;
  g.blocks = blocks;
  g.workers = blocks * (block / 64) * (64 / W);
  g.xcd_span = blocks / kXcds;  // XCD-contiguous slice numbering
  g.factor = factor;
  return g;
}

// Launch shape of the carry fixup: each wave takes groups of G slices, G
// the smallest power of two from 8 to 64 that covers all `workers` slices
// with at most 32 waves per CU.
struct FixupShape {
  int blocks;
  int G;
};

FixupShape fixup_shape(int cus, int64_t workers) {
  const int64_t max_waves = (int64_t)cus * 32;
  int G = 8;
  while (G < 64 && (workers + G - 1) / G > max_waves) G *= 2;
  const int64_t waves = (workers + G - 1) / G;
  int64_t blocks = (waves + (kBlock / 64) - 1) / (kBlock / 64);
  if (blocks > max_waves / (kBlock / 64)) blocks = max_waves / (kBlock / 64);
  return FixupShape{(int)(blocks > 0 ? blocks : 1), G};
}

// Kernel and grid of a walk launch at a requested grid factor (0: the
// automatic or process-wide choice): one resident grid takes the
// small-input kernel, several the wide-worker kernel, fine slices the
// fine-slice kernel, where the variant has them.
int choose_launch(int dev, int cus, const Variant *vs, int nv, int64_t N, int factor,
                  Variant *v_out, Grid *g_out) {
  int rc;
  Variant v = vs[0];
  int per_cu = 1;
  if ((rc = blocks_per_cu(dev, v.fn, v.block, v.lds, &per_cu)) != SPARSELNR_OK) return rc;
  for (int t = 1; t < nv; ++t) {
    if (vs[t].W != v.W || vs[t].block != v.block || vs[t].generic != v.generic)
      return SPARSELNR_ERR_UNSUPPORTED;  // alternatives must split the matrix alike
    int pc = 1;
    if ((rc = blocks_per_cu(dev, vs[t].fn, vs[t].block, vs[t].lds, &pc)) != SPARSELNR_OK)
      return rc;
    if (pc < per_cu) per_cu = pc;
  }
  Grid g = make_grid(cus, per_cu, v.block, v.W, N, factor);
  if (nv == 1 && g.factor == 1 && v.fn_small) {  // one resident grid: the small-input schedule
    v.fn = v.fn_small;
    if ((rc = blocks_per_cu(dev, v.fn, v.block, v.lds, &per_cu)) != SPARSELNR_OK) return rc;
    g = make_grid(cus, per_cu, v.block, v.W, N, factor);
  } else if (nv == 1 && g.factor > 1 && v.fn_wide) {  // several grids: the wide workers
    v.fn = v.fn_wide;
    v.W = v.W_wide;
    if ((rc = blocks_per_cu(dev, v.fn, v.block, v.lds, &per_cu)) != SPARSELNR_OK) return rc;
    g = make_grid(cus, per_cu, v.block, v.W, N, g.factor);
  } else if (nv == 1 && v.fn_fine && g.factor >= v.fine_factor) {  // fine slices
    v.fn = v.fn_fine;
    if ((rc = blocks_per_cu(dev, v.fn, v.block, v.lds, &per_cu)) != SPARSELNR_OK) return rc;
    g = make_grid(cus, per_cu, v.block, v.W, N, g.factor);
  }
  *v_out = v;
  *g_out = g;
  return SPARSELNR_OK;
}

// Carry workspace of a walk launch: two partial rows of the l-tile width
// plus two int32 of metadata per worker.
struct CarrySize {
  size_t carry, meta;
  size_t total() const { return carry + meta; }
};

CarrySize carry_size(const Grid &g, int64_t tile_w) {
  return CarrySize{(size_t)g.workers * 2 * (size_t)tile_w * sizeof(float),
                   (size_t)g.workers * 2 * sizeof(int32_t)};
}

// A buffer the caller provides instead of the per-(device, stream)
// workspace (the no-allocation entry point): its device address and size.
struct FixedBuffer {
  void *ptr;
  size_t bytes;
};

// Runs one merge-path walk (+ carry fixup unless SDDMM) over the whole matrix.
// With nv > 1, the variants are gated alternatives, each with its own
// arguments as[k] (only the one whose gate opens on the device does any
// work): they share one grid, workspace and slice split, so the one carry
// fixup serves whichever ran.  With `fixed`, the partial rows go to that
// buffer instead of the workspace, and the grid factor is halved until they
// fit (ERR_UNSUPPORTED if they do not fit at one resident grid); the walk
// then allocates nothing.
int run_walk(Mode mode, const Variant *vs, const WalkArgs *as, int nv, hipStream_t stream,
             const FixedBuffer *fixed = nullptr) {
  WalkArgs a = as[0];
  int dev = 0, cus = 0, rc;
  if ((rc = current_device(&dev)) != SPARSELNR_OK) return rc;
  if ((rc = device_cus(dev, &cus)) != SPARSELNR_OK) return rc;
  Variant v;
  Grid g;
  if ((rc = choose_launch(dev, cus, vs, nv, a.N, 0, &v, &g)) != SPARSELNR_OK) return rc;
  const int64_t tiles = vs[0].generic ? (a.L + 64 * kGenericLT - 1) / (64 * kGenericLT) : 1;
  const int64_t tile_w = vs[0].generic ? 64 * kGenericLT : a.L;
  if (fixed && mode != kSddmm) {
    while (carry_size(g, tile_w).total() > fixed->bytes && g.factor > 1)
      if ((rc = choose_launch(dev, cus, vs, nv, a.N, g.factor / 2, &v, &g)) != SPARSELNR_OK)
        return rc;
    if (carry_size(g, tile_w).total() > fixed->bytes) return SPARSELNR_ERR_UNSUPPORTED;
  }
  a.workers = g.workers;
  a.min_chunk = kMinChunk;
  a.xcd_span = g.xcd_span;
  a.xcds = kXcds;
  if (mode != kSddmm) {
    const CarrySize cs = carry_size(g, tile_w);
    void *ws = nullptr;
    if (fixed) {
      ws = fixed->ptr;
    } else if ((rc = get_workspace(dev, stream, cs.total(), &ws)) != SPARSELNR_OK) {
      return rc;
    }
    a.carry = (float *)ws;
    a.meta = (int32_t *)((char *)ws + cs.carry);
  } else {
    a.carry = nullptr;
    a.meta = nullptr;
  }
  for (int64_t t = 0; t < (mode == kSddmm ? 1 : tiles); ++t) {
    a.l0 = (int32_t)(t * tile_w);
    a.Lw = (int32_t)((a.L - a.l0) < tile_w ? (a.L - a.l0) : tile_w);
    for (int k = 0; k < nv; ++k) {
      WalkArgs ak = as[k];  // the shared fields come from a
      ak.workers = a.workers;
      ak.min_chunk = a.min_chunk;
      ak.xcd_span = a.xcd_span;
      ak.xcds = a.xcds;
      ak.carry = a.carry;
      ak.meta = a.meta;
      ak.l0 = a.l0;
      ak.Lw = a.Lw;
      const Variant &vk = k == 0 ? v : vs[k];  // v: the kernel chosen for this input
      hipLaunchKernelGGL(vk.fn, dim3(g.blocks), dim3(vk.block), vk.lds, stream, ak);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return hip_fail(e);
    }
    if (mode != kSddmm) {
      const FixupShape fs = fixup_shape(cus, g.workers);
      hipLaunchKernelGGL(slnr::carry_fixup, dim3(fs.blocks), dim3(kBlock), 0, stream, a, fs.G);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return hip_fail(e);
    }
  }
  return SPARSELNR_OK;
}

int run_walk(Mode mode, const Variant &v, WalkArgs a, hipStream_t stream,
             const FixedBuffer *fixed = nullptr) {
  return run_walk(mode, &v, &a, 1, stream, fixed);
}

bool bad_size(int64_t N, int64_t M, int64_t K, int64_t L) {
  return N < 0 || M < 0 || K < 0 || L < 0;
}

int check_range(int64_t N, int64_t M, int64_t K, int64_t L) {
  if (K > SPARSELNR_MAX_WIDTH || L > SPARSELNR_MAX_WIDTH) return SPARSELNR_ERR_UNSUPPORTED;
  if (N >= ((int64_t)1 << 31) - 1 || M >= ((int64_t)1 << 31)) return SPARSELNR_ERR_UNSUPPORTED;
  return SPARSELNR_OK;
}

// Argument checks of the fused <SDDMM, SpMM> entry points (plain and
// transposed D): pointers, signs and ranges, all before any HIP call.
int check_fused_args(const int32_t *rowptr, const int32_t *colidx, const float *vals,
                     const float *C, const float *D, const float *E, const float *A, int64_t N,
                     int64_t M, int64_t K, int64_t L) {
  if (bad_size(N, M, K, L)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && (!rowptr || !colidx || !vals)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && K > 0 && !C) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && M > 0 && K > 0 && !D) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && M > 0 && L > 0 && !E) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && L > 0 && !A) return SPARSELNR_ERR_INVALID_ARG;
  return check_range(N, M, K, L);
}

// Device array of the no-allocation fused entry point: the partial rows of
// split rows and their metadata.  Each GPU the library runs on holds one copy
// for the life of the process.  Host code never uses the name `scratch` as
// an address: the device address of each GPU's copy comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kScratchBytes = SPARSELNR_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "scratch size");
constexpr int kMaxDevices = 64;
void *g_scratch_ptr[kMaxDevices] = {};

}  // namespace

static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

namespace {

int scratch_address(int dev, void **out) {
  if (dev < 0 || dev >= kMaxDevices) return SPARSELNR_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e);
    if (!p) return hip_fail(hipErrorInvalidSymbol);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SPARSELNR_OK;
}

WalkArgs base_args(const int32_t *rowptr, const int32_t *colidx, const float *vals,
                   int64_t N, int64_t K, int64_t L) {
  WalkArgs a{};
  a.rowptr = rowptr;
  a.colidx = colidx;
  a.vals = vals;
  a.N = N;
  a.K = (int32_t)K;
  a.L = (int32_t)L;
  a.l0 = 0;
  a.Lw = (int32_t)L;
  a.Lin = (int32_t)L;
  a.G2 = nullptr;
  a.Wep = nullptr;
  a.gate_nnz = 0;
  a.gate = slnr::kGateNone;
  return a;
}

// Shared driver of the epilogue entry points.
int run_epilogue(Mode mode, bool had, const int32_t *rowptr, const int32_t *colidx,
                 const float *vals, const float *C, const float *D, const float *E,
                 const float *G2, const float *Wm, float *A, int64_t N, int64_t Kdot,
                 int64_t Lin, int64_t Lout, void *stream) {
  if (!epi_width(Lin)) return SPARSELNR_ERR_UNSUPPORTED;  // before any HIP call
  int dev = 0, rc;
  size_t max_lds = 0;
  if ((rc = current_device(&dev)) != SPARSELNR_OK) return rc;
  if ((rc = device_max_lds(dev, &max_lds)) != SPARSELNR_OK) return rc;
  Variant v = mode == kFused ? pick_epi<kFused, 0>(Lin, Lout, max_lds)
                             : (had ? pick_epi<kSpmm, 1>(Lin, Lout, max_lds)
                                    : pick_epi<kSpmm, 0>(Lin, Lout, max_lds));
  if (!v.fn) return SPARSELNR_ERR_UNSUPPORTED;
  WalkArgs a = base_args(rowptr, colidx, vals, N, Kdot, Lout);
  a.C = C;
  a.D = D;
  a.E = E;
  a.G2 = G2;
  a.Wep = Wm;
  a.Lin = (int32_t)Lin;
  a.out = A;
  return run_walk(mode, v, a, (hipStream_t)stream);
}

}  // namespace

extern "C" {

int sparselnr_abi_version(void) { return 1; }

const char *sparselnr_status_string(int status) {
  switch (status) {
    case SPARSELNR_OK: return "ok";
    case SPARSELNR_ERR_INVALID_ARG: return "invalid argument";
    case SPARSELNR_ERR_UNSUPPORTED: return "unsupported size";
    case SPARSELNR_ERR_HIP: return "HIP call failed";
    case SPARSELNR_ERR_NO_MEMORY: return "workspace allocation failed";
    case SPARSELNR_ERR_INVALID_CSR: return "CSR preconditions violated";
    default: return "unknown status";
  }
}

int sparselnr_last_hip_error(void) { return g_last_hip_error; }

int sparselnr_set_grid_factor(int factor) {
  if (factor < 0 || factor > kMaxGridFactor) return SPARSELNR_ERR_INVALID_ARG;
  g_grid_factor.store(factor == 0 ? -1 : factor);
  return SPARSELNR_OK;
}

int sparselnr_get_grid_factor(void) {
  const int f = g_grid_factor.load();
  if (f != 0) return f > 0 ? f : 0;
  const char *env = getenv("SPARSELNR_GRID_FACTOR");
  const int e = env ? atoi(env) : 0;
  return e >= 1 && e <= kMaxGridFactor ? e : 0;
}

int sparselnr_fused_sddmm_spmm(const int32_t *rowptr, const int32_t *colidx,
                               const float *vals, const float *C, const float *D,
                               const float *E, float *A, int64_t N, int64_t M, int64_t K,
                               int64_t L, void *stream) {
  int rc = check_fused_args(rowptr, colidx, vals, C, D, E, A, N, M, K, L);
  if (rc != SPARSELNR_OK) return rc;
  if (N == 0 || L == 0) return SPARSELNR_OK;
  const bool al = aligned16(C) && aligned16(D) && aligned16(E) && aligned16(A) &&
                  offsets32(M, K) && offsets32(M, L);
  WalkArgs a = base_args(rowptr, colidx, vals, N, K, L);
  a.C = C;
  a.D = D;
  a.E = E;
  a.out = A;
  return run_walk(kFused, pick_fused(K, L, al), a, (hipStream_t)stream);
}

int sparselnr_fused_sddmm_spmm_noalloc(const int32_t *rowptr, const int32_t *colidx,
                                       const float *vals, const float *C, const float *D,
                                       const float *E, float *A, int64_t N, int64_t M,
                                       int64_t K, int64_t L, void *stream) {
  int rc = check_fused_args(rowptr, colidx, vals, C, D, E, A, N, M, K, L);
  if (rc != SPARSELNR_OK) return rc;
  if (N == 0 || L == 0) return SPARSELNR_OK;
  const bool al = aligned16(C) && aligned16(D) && aligned16(E) && aligned16(A) &&
                  offsets32(M, K) && offsets32(M, L);
  int dev = 0;
  if ((rc = current_device(&dev)) != SPARSELNR_OK) return rc;
  FixedBuffer fb{nullptr, kScratchBytes};
  if ((rc = scratch_address(dev, &fb.ptr)) != SPARSELNR_OK) return rc;
  WalkArgs a = base_args(rowptr, colidx, vals, N, K, L);
  a.C = C;
  a.D = D;
  a.E = E;
  a.out = A;
  return run_walk(kFused, pick_fused(K, L, al), a, (hipStream_t)stream, &fb);
}

int sparselnr_sddmm(const int32_t *rowptr, const int32_t *colidx, const float *vals,
                    const float *C, const float *D, float *Y, int64_t N, int64_t M, int64_t K,
                    void *stream) {
  if (bad_size(N, M, K, 0)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && (!rowptr || !colidx || !vals || !Y)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && K > 0 && !C) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && M > 0 && K > 0 && !D) return SPARSELNR_ERR_INVALID_ARG;
  int rc = check_range(N, M, K, 0);
  if (rc != SPARSELNR_OK) return rc;
  if (N == 0) return SPARSELNR_OK;
  const bool al = aligned16(C) && aligned16(D) && offsets32(M, K);
  WalkArgs a = base_args(rowptr, colidx, vals, N, K, 0);
  a.C = C;
  a.D = D;
  a.out = Y;
  return run_walk(kSddmm, pick_sddmm(K, al), a, (hipStream_t)stream);
}

int sparselnr_spmm(const int32_t *rowptr, const int32_t *colidx, const float *Y,
                   const float *E, float *A, int64_t N, int64_t M, int64_t L, void *stream) {
  if (bad_size(N, M, 0, L)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && (!rowptr || !colidx || !Y)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && M > 0 && L > 0 && !E) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && L > 0 && !A) return SPARSELNR_ERR_INVALID_ARG;
  int rc = check_range(N, M, 0, L);
  if (rc != SPARSELNR_OK) return rc;
  if (N == 0 || L == 0) return SPARSELNR_OK;
  const bool al = aligned16(E) && aligned16(A) && offsets32(M, L);
  WalkArgs a = base_args(rowptr, colidx, Y, N, 0, L);
  a.E = E;
  a.out = A;
  return run_walk(kSpmm, pick_spmm(L, al), a, (hipStream_t)stream);
}

int sparselnr_unfused_sddmm_spmm(const int32_t *rowptr, const int32_t *colidx,
                                 const float *vals, const float *C, const float *D,
                                 const float *E, float *Y, float *A, int64_t N, int64_t M,
                                 int64_t K, int64_t L, void *stream) {
  if (bad_size(N, M, K, L)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && (!rowptr || !colidx || !vals || !Y)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && K > 0 && !C) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && M > 0 && K > 0 && !D) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && M > 0 && L > 0 && !E) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && L > 0 && !A) return SPARSELNR_ERR_INVALID_ARG;
  int rc = check_range(N, M, K, L);
  if (rc != SPARSELNR_OK) return rc;
  if (N == 0) return SPARSELNR_OK;
  rc = sparselnr_sddmm(rowptr, colidx, vals, C, D, Y, N, M, K, stream);
  if (rc != SPARSELNR_OK) return rc;
  return sparselnr_spmm(rowptr, colidx, Y, E, A, N, M, L, stream);
}

int sparselnr_fused_sddmm_spmm_gemm(const int32_t *rowptr, const int32_t *colidx,
                                    const float *vals, const float *C, const float *D,
                                    const float *F, const float *Wm, float *A, int64_t N,
                                    int64_t M, int64_t K, int64_t L, int64_t Mo, void *stream) {
  if (bad_size(N, M, K, L) || Mo < 0) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && (!rowptr || !colidx || !vals)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && (!C || !Wm || !A || (M > 0 && (!D || !F)))) return SPARSELNR_ERR_INVALID_ARG;
  int rc = check_range(N, M, K, L > Mo ? L : Mo);
  if (rc != SPARSELNR_OK) return rc;
  if (N == 0 || Mo == 0) return SPARSELNR_OK;
  if (K != L || !(aligned16(C) && aligned16(D) && aligned16(F) && offsets32(M, K) &&
                  offsets32(M, L)))
    return SPARSELNR_ERR_UNSUPPORTED;
  return run_epilogue(kFused, false, rowptr, colidx, vals, C, D, F, nullptr, Wm, A, N, K, L, Mo,
                      stream);
}

int sparselnr_spmm_gemm(const int32_t *rowptr, const int32_t *colidx, const float *vals,
                        const float *C, const float *D, float *A, int64_t N, int64_t M,
                        int64_t K, int64_t L, void *stream) {
  if (bad_size(N, M, K, L)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && (!rowptr || !colidx || !vals)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && L > 0 && (!A || (K > 0 && !D) || (M > 0 && K > 0 && !C)))
    return SPARSELNR_ERR_INVALID_ARG;
  int rc = check_range(N, M, K, L);
  if (rc != SPARSELNR_OK) return rc;
  if (N == 0 || L == 0) return SPARSELNR_OK;
  if (!(aligned16(C) && offsets32(M, K))) return SPARSELNR_ERR_UNSUPPORTED;
  return run_epilogue(kSpmm, false, rowptr, colidx, vals, nullptr, nullptr, C, nullptr, D, A, N,
                      0, K, L, stream);
}

int sparselnr_spmmh_gemm(const int32_t *rowptr, const int32_t *colidx, const float *vals,
                         const float *C, const float *D, const float *E, float *A, int64_t N,
                         int64_t M, int64_t J, int64_t L, void *stream) {
  if (bad_size(N, M, J, L)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && (!rowptr || !colidx || !vals)) return SPARSELNR_ERR_INVALID_ARG;
  if (N > 0 && L > 0 && (!A || (J > 0 && !E) || (M > 0 && J > 0 && (!C || !D))))
    return SPARSELNR_ERR_INVALID_ARG;
  int rc = check_range(N, M, J, L);
  if (rc != SPARSELNR_OK) return rc;
  if (N == 0 || L == 0) return SPARSELNR_OK;
  if (!(aligned16(C) && aligned16(D) && offsets32(M, J))) return SPARSELNR_ERR_UNSUPPORTED;
  if (!epi_width(J)) return SPARSELNR_ERR_UNSUPPORTED;
  if (M == 0 || J == 0)  // no rows to gather: the per-nonzero form alone
    return run_epilogue(kSpmm, true, rowptr, colidx, vals, nullptr, nullptr, C, D, E, A, N, 0, J,
                        L, stream);
  // C .* D does not depend on the row, so it can be formed once (M x J,
  // 12 M J bytes) and gathered as one row per nonzero, or formed per nonzero
  // from two gathered rows (4 J more bytes per nonzero).  The first moves
  // fewer bytes when nnz >= 3 M.  nnz is known on the device only, so both
  // schedules are launched, gated on it, and exactly one of them runs.
  int dev = 0;
  size_t max_lds = 0;
  if ((rc = current_device(&dev)) != SPARSELNR_OK) return rc;
  if ((rc = device_max_lds(dev, &max_lds)) != SPARSELNR_OK) return rc;
  Variant vs[2] = {pick_epi<kSpmm, 0>(J, L, max_lds), pick_epi<kSpmm, 1>(J, L, max_lds)};
  if (!vs[0].fn || !vs[1].fn) return SPARSELNR_ERR_UNSUPPORTED;
  hipStream_t s = (hipStream_t)stream;
  void *ws = nullptr;
  if ((rc = get_workspace(dev, s, (size_t)M * J * sizeof(float), &ws, 2)) != SPARSELNR_OK)
    return rc;
  float *H = (float *)ws;
  const int64_t gate_nnz = kHoistRatio * M;
  int cus = 0;
  if ((rc = device_cus(dev, &cus)) != SPARSELNR_OK) return rc;
  const int64_t n4 = M * J / 4;  // J is a multiple of 4 (supported widths)
  int64_t hb = (n4 + kBlock - 1) / kBlock;
  if (hb > (int64_t)cus * 8) hb = (int64_t)cus * 8;
  hipLaunchKernelGGL(slnr::hadamard4_kernel, dim3((unsigned)hb), dim3(kBlock), 0, s, C, D, H, n4,
                     rowptr, N, gate_nnz, (int)slnr::kGateDense);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e);
  WalkArgs as[2];
  as[0] = base_args(rowptr, colidx, vals, N, 0, L);
  as[0].Wep = E;
  as[0].Lin = (int32_t)J;
  as[0].out = A;
  as[0].gate_nnz = gate_nnz;
  as[1] = as[0];
  as[0].E = H;  // hoisted: one gathered row of H = C .* D per nonzero
  as[0].gate = slnr::kGateDense;
  as[1].E = C;  // per nonzero: C_k .* D_k from two gathered rows
  as[1].G2 = D;
  as[1].gate = slnr::kGateSparse;
  return run_walk(kSpmm, vs, as, 2, s);
}

int sparselnr_fused_sddmm_spmm_dt(const int32_t *rowptr, const int32_t *colidx,
                                  const float *vals, const float *C, const float *Dt,
                                  const float *E, float *A, int64_t N, int64_t M, int64_t K,
                                  int64_t L, void *stream) {
  // every argument is checked before the transpose touches the device
  int rc = check_fused_args(rowptr, colidx, vals, C, Dt, E, A, N, M, K, L);
  if (rc != SPARSELNR_OK) return rc;
  if (N == 0 || L == 0) return SPARSELNR_OK;
  if (M == 0 || K == 0)  // D is empty: nothing to transpose
    return sparselnr_fused_sddmm_spmm(rowptr, colidx, vals, C, Dt, E, A, N, M, K, L, stream);
  int dev = 0;
  if ((rc = current_device(&dev)) != SPARSELNR_OK) return rc;
  hipStream_t s = (hipStream_t)stream;
  void *ws = nullptr;
  if ((rc = get_workspace(dev, s, (size_t)M * K * sizeof(float), &ws, 1)) != SPARSELNR_OK)
    return rc;
  float *D = (float *)ws;
  if (M % 4 == 0 && K % 4 == 0 && aligned16(Dt)) {
    const int64_t tiles_c = (M + 63) / 64, tiles_r = (K + 63) / 64;
    hipLaunchKernelGGL(slnr::transpose4_kernel, dim3((unsigned)(tiles_r * tiles_c)), dim3(256), 0,
                       s, Dt, D, K, M, tiles_c);
  } else {
    const int64_t tiles_c = (M + 31) / 32, tiles_r = (K + 31) / 32;
    hipLaunchKernelGGL(slnr::transpose_kernel, dim3((unsigned)(tiles_r * tiles_c)), dim3(256), 0,
                       s, Dt, D, K, M, tiles_c);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e);
  return sparselnr_fused_sddmm_spmm(rowptr, colidx, vals, C, D, E, A, N, M, K, L, stream);
}

int sparselnr_validate_csr(const int32_t *rowptr, const int32_t *colidx, int64_t N, int64_t M,
                           int64_t colidx_len, int64_t *nnz_out, void *stream) {
  if (N < 0 || M < 0 || colidx_len < 0 || !rowptr) return SPARSELNR_ERR_INVALID_ARG;
  if (colidx_len > 0 && !colidx) return SPARSELNR_ERR_INVALID_ARG;
  if (N >= ((int64_t)1 << 31) - 1) return SPARSELNR_ERR_UNSUPPORTED;
  hipStream_t s = (hipStream_t)stream;
  int32_t *flags = nullptr;
  hipError_t e = hipMalloc(&flags, 2 * sizeof(int32_t));
  if (e != hipSuccess) return hip_fail(e);
  int32_t host[2] = {0, 0};
  int rc = SPARSELNR_OK;
  e = hipMemsetAsync(flags, 0, 2 * sizeof(int32_t), s);
  if (e == hipSuccess) {
    hipLaunchKernelGGL(slnr::validate_csr_kernel, dim3(1024), dim3(256), 0, s, rowptr, colidx,
                       N, M, colidx_len, flags);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipMemcpyAsync(&host[0], flags, sizeof(int32_t),
                                          hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipMemcpyAsync(&host[1], rowptr + N, sizeof(int32_t),
                                          hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) rc = hip_fail(e);
  hipError_t ef = hipFree(flags);
  if (rc == SPARSELNR_OK && ef != hipSuccess) rc = hip_fail(ef);
  if (rc != SPARSELNR_OK) return rc;
  if (nnz_out) *nnz_out = host[1];
  return host[0] == 0 ? SPARSELNR_OK : SPARSELNR_ERR_INVALID_CSR;
}

int sparselnr_release(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  int rc = SPARSELNR_OK;
  int saved = 0;
  (void)hipGetDevice(&saved);
  for (auto &kv : g_workspace) {
    if (!kv.second.ptr) continue;
    hipError_t e = hipSetDevice(kv.first.dev);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipFree(kv.second.ptr);
    if (e != hipSuccess) rc = hip_fail(e);
  }
  g_workspace.clear();
  (void)hipSetDevice(saved);
  return rc;
}

}  // extern "C"
