// Choice of the two-plane groups and the plane-1 CSR of a linear (gfx950).
//
// Paper: section 4.2 (E2M-ATQ) gives a second ternary plane to a minority
// of blocks; section 3 chooses them with salience masks fitted on
// calibration activations, which are not available here, so groups are
// ranked by their one-plane residual energy (written by tq_ternarize).  The
// rule: the nnz groups with the largest energy, ties to the lower flat index
// (row-major (r, g)); a NaN energy ranks below every number, -0 and +0 tie.
// Records are numbered in flat order, which is CSR order by row.
//
// Steps, all on the caller's stream, with scratch in the caller's workspace:
// 1. Radix select of the nnz-th largest 64-bit key, eight passes of 8-bit
//    digits from the most significant: per pass one histogram launch over
//    the keys that match the digits found so far, then a one-block launch
//    that picks the digit holding the wanted rank and clears the histogram.
//    The result is the threshold key T and the number `need` of groups with
//    key T to take (the first `need` of them in flat order).
// 2. Per tile of kTile groups: how many keys are above T and equal to T.
// 3. One block: each tile's offset among the equal keys and among the
//    selected groups (a tile takes its equal keys while the running count
//    of equal keys is below `need`).
// 4. Per tile: block-local scans give each selected group its record
//    index, written to rec_index and gidx1, and the row pointers of the
//    rows whose first group lies in the tile.
// Counts are integers, so the result is deterministic and unique.

#include <mutex>

#include "tq_internal.h"

namespace tq {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;                  // groups per thread per tile
constexpr int kTile = kThreads * kItems;    // 4096 groups per tile
constexpr int kOffsetThreads = 1024;

// Workspace layout: histogram, state, then four uint32 arrays over tiles.
constexpr size_t kHistBytes = 256 * sizeof(uint32_t);
struct SelState {
  uint64_t prefix;   // digits found so far (the threshold key T at the end)
  uint64_t mask;     // which bits of prefix are set
  uint64_t rank;     // wanted rank among keys matching prefix (1-based, from the top)
  uint64_t pad;
};
constexpr size_t kStateOff = kHistBytes;
constexpr size_t kTilesOff = kStateOff + sizeof(SelState);

__host__ __device__ constexpr int64_t num_tiles(int64_t n) { return (n + kTile - 1) / kTile; }

constexpr size_t workspace_bytes_for(int64_t n) {
  return (kTilesOff + 4 * sizeof(uint32_t) * (size_t)num_tiles(n) + 255) & ~(size_t)255;
}

// Scratch of the allocation-free entry point: one copy per GPU, held until
// the process ends.  Host code never passes this name to a kernel; it uses
// the device address obtained for it below.
constexpr size_t kScratchBytes = workspace_bytes_for(TQ_SELECT_NOALLOC_MAX_GROUPS);
static __device__ __attribute__((aligned(256))) unsigned char scratch[kScratchBytes];

// Orderable key of an energy: larger energy, larger key; NaN is 0, below
// every number (-inf maps to 0x000FFFFFFFFFFFFF); both zeros map to the key
// of +0.
__device__ inline uint64_t energy_key(double e) {
  uint64_t b = __builtin_bit_cast(uint64_t, e);
  if ((b & 0x7FFFFFFFFFFFFFFFull) > 0x7FF0000000000000ull) return 0;   // NaN
  if ((b & 0x7FFFFFFFFFFFFFFFull) == 0) b = 0;                          // -0 -> +0
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ inline uint32_t wave_inclusive_scan(uint32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t u = __shfl_up(v, d, 64);
    if (lane >= d) v += u;
  }
  return v;
}

// Exclusive scan of v over the block (blockDim.x a multiple of 64, at most
// 1024 threads); *total receives the block's sum.  Every thread must call.
__device__ inline uint32_t block_exclusive_scan(uint32_t v, uint32_t* total) {
  __shared__ uint32_t wsum[16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const uint32_t inc = wave_inclusive_scan(v);
  if (lane == 63) wsum[wave] = inc;
  __syncthreads();
  uint32_t before = 0, tot = 0;
  for (int w = 0; w < nw; ++w) {
    const uint32_t s = wsum[w];
    before += w < wave ? s : 0u;
    tot += s;
  }
  __syncthreads();   // wsum is reused by the next call
  *total = tot;
  return before + inc - v;
}

// One block of 256 threads: clear the histogram and set the state.  With
// nothing to select the threshold is the all-ones key, which no energy maps
// to, and no equal key is taken.
__global__ void __launch_bounds__(256) sel_init(uint32_t* hist, SelState* st, uint64_t rank) {
  hist[threadIdx.x] = 0u;
  if (threadIdx.x == 0) {
    st->prefix = rank == 0 ? ~0ull : 0ull;
    st->mask = 0;
    st->rank = rank;
    st->pad = 0;
  }
}

// Histogram of the digit at `shift` over keys that match the digits found
// so far (LDS counts per block, then one global add per bin).
__global__ void __launch_bounds__(kThreads) sel_hist(const double* __restrict__ energy, int64_t n,
                                                     const SelState* st, uint32_t* hist, int shift) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0u;
  __syncthreads();
  const uint64_t prefix = st->prefix, mask = st->mask;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
    const uint64_t k = energy_key(energy[i]);
    if ((k & mask) == prefix) atomicAdd(&h[(k >> shift) & 255u], 1u);
  }
  __syncthreads();
  const uint32_t c = h[threadIdx.x];
  if (c) atomicAdd(&hist[threadIdx.x], c);
}

// One block of 256 threads: the digit holding the wanted rank (counting
// from the largest digit), then the histogram is cleared for the next pass.
__global__ void __launch_bounds__(256) sel_pick(SelState* st, uint32_t* hist, int shift) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = hist[threadIdx.x];
  __syncthreads();
  hist[threadIdx.x] = 0u;
  if (threadIdx.x == 0) {
    const uint64_t rank = st->rank;
    uint64_t above = 0;
    int d = 255;
    for (; d > 0; --d) {
      if (above + h[d] >= rank) break;
      above += h[d];
    }
    st->rank = rank - above;
    st->prefix |= (uint64_t)d << shift;
    st->mask |= 255ull << shift;
  }
}

// Per tile: keys above and equal to the threshold.
__global__ void __launch_bounds__(kThreads) sel_count(const double* __restrict__ energy, int64_t n,
                                                      const SelState* st, uint32_t* gt, uint32_t* eq) {
  const uint64_t T = st->prefix;
  const int64_t base = (int64_t)blockIdx.x * kTile;
  uint32_t cg = 0, ce = 0;
#pragma unroll 4
  for (int j = 0; j < kItems; ++j) {
    const int64_t i = base + (int64_t)j * kThreads + threadIdx.x;
    if (i < n) {
      const uint64_t k = energy_key(energy[i]);
      cg += k > T ? 1u : 0u;
      ce += k == T ? 1u : 0u;
    }
  }
  uint32_t tg, te;
  block_exclusive_scan(cg, &tg);
  block_exclusive_scan(ce, &te);
  if (threadIdx.x == 0) {
    gt[blockIdx.x] = tg;
    eq[blockIdx.x] = te;
  }
}

// One block: each tile's offsets among the equal keys and among the
// selected groups, in chunks of blockDim.x tiles with running carries.
__global__ void __launch_bounds__(kOffsetThreads) sel_offsets(const SelState* st, const uint32_t* gt,
                                                              const uint32_t* eq, uint32_t* eq_off,
                                                              uint32_t* sel_off, int64_t ntiles) {
  const uint64_t need = st->rank;
  uint64_t carry_eq = 0, carry_sel = 0;
  for (int64_t c0 = 0; c0 < ntiles; c0 += blockDim.x) {
    const int64_t b = c0 + threadIdx.x;
    const uint32_t e = b < ntiles ? eq[b] : 0u, g = b < ntiles ? gt[b] : 0u;
    uint32_t te, ts;
    const uint64_t eoff = carry_eq + block_exclusive_scan(e, &te);
    const uint64_t left = need > eoff ? need - eoff : 0;
    const uint32_t take = (uint32_t)(left < e ? left : e);
    const uint64_t soff = carry_sel + block_exclusive_scan(g + take, &ts);
    if (b < ntiles) {
      eq_off[b] = (uint32_t)eoff;
      sel_off[b] = (uint32_t)soff;
    }
    carry_eq += te;
    carry_sel += ts;
  }
}

// Per tile: thread t takes the kItems consecutive groups base + kItems t ..,
// so block-local scans follow flat order.
__global__ void __launch_bounds__(kThreads) sel_write(const double* __restrict__ energy, int64_t n, int32_t G,
                                                      int64_t n_out, int64_t nnz, const SelState* st,
                                                      const uint32_t* eq_off, const uint32_t* sel_off,
                                                      int32_t* rec_index, int32_t* rowptr1, uint16_t* gidx1) {
  const uint64_t T = st->prefix, need = st->rank;
  const int64_t base = (int64_t)blockIdx.x * kTile + (int64_t)threadIdx.x * kItems;
  uint32_t gtm = 0, eqm = 0;
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const int64_t i = base + j;
    if (i < n) {
      const uint64_t k = energy_key(energy[i]);
      gtm |= (k > T ? 1u : 0u) << j;
      eqm |= (k == T ? 1u : 0u) << j;
    }
  }
  uint32_t total;
  uint64_t r = (uint64_t)eq_off[blockIdx.x] + block_exclusive_scan((uint32_t)__builtin_popcount(eqm), &total);
  uint32_t selm = gtm;
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    if ((eqm >> j) & 1u) {
      if (r < need) selm |= 1u << j;
      ++r;
    }
  }
  uint32_t rec = sel_off[blockIdx.x] + block_exclusive_scan((uint32_t)__builtin_popcount(selm), &total);
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const int64_t i = base + j;
    if (i < n) {
      const bool s = (selm >> j) & 1u;
      const int64_t row = i / G, g = i - row * G;
      rec_index[i] = s ? (int32_t)rec : -1;
      if (s && rec < (uint64_t)nnz) gidx1[rec] = (uint16_t)g;
      if (g == 0) rowptr1[row] = (int32_t)rec;   // records before the row's first group
      rec += s ? 1u : 0u;
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) rowptr1[n_out] = (int32_t)nnz;
}

}  // namespace

size_t select_workspace_bytes(int64_t n) { return workspace_bytes_for(n); }

hipError_t launch_select(const double* energy, int64_t n_out, int32_t G, int64_t nnz, int32_t* rec_index,
                         int32_t* rowptr1, uint16_t* gidx1, void* workspace, hipStream_t s) {
  const int64_t n = n_out * G;
  const int64_t nt = num_tiles(n);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  uint32_t* hist = reinterpret_cast<uint32_t*>(ws);
  SelState* st = reinterpret_cast<SelState*>(ws + kStateOff);
  uint32_t* gt = reinterpret_cast<uint32_t*>(ws + kTilesOff);
  uint32_t* eq = gt + nt;
  uint32_t* eq_off = eq + nt;
  uint32_t* sel_off = eq_off + nt;
  // A writable stand-in for gidx1 when nothing is selected (never written).
  uint16_t* gidx = nnz > 0 ? gidx1 : reinterpret_cast<uint16_t*>(hist);

  hipLaunchKernelGGL(sel_init, dim3(1), dim3(256), 0, s, hist, st, (uint64_t)nnz);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (nnz > 0) {
    const unsigned hb = (unsigned)(nt < 1024 ? nt : 1024);
    for (int shift = 56; shift >= 0; shift -= 8) {
      hipLaunchKernelGGL(sel_hist, dim3(hb), dim3(kThreads), 0, s, energy, n, st, hist, shift);
      hipLaunchKernelGGL(sel_pick, dim3(1), dim3(256), 0, s, st, hist, shift);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  hipLaunchKernelGGL(sel_count, dim3((unsigned)nt), dim3(kThreads), 0, s, energy, n, st, gt, eq);
  hipLaunchKernelGGL(sel_offsets, dim3(1), dim3(kOffsetThreads), 0, s, st, gt, eq, eq_off, sel_off, nt);
  hipLaunchKernelGGL(sel_write, dim3((unsigned)nt), dim3(kThreads), 0, s, energy, n, G, n_out, nnz, st, eq_off,
                     sel_off, rec_index, rowptr1, gidx);
  return hipGetLastError();
}

// Device address of `scratch` on the current GPU, looked up once per device
// (each GPU holds its own copy of the array at its own address).
static hipError_t scratch_address(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

hipError_t launch_select_noalloc(const double* energy, int64_t n_out, int32_t G, int64_t nnz, int32_t* rec_index,
                                 int32_t* rowptr1, uint16_t* gidx1, hipStream_t s) {
  if (n_out * G > TQ_SELECT_NOALLOC_MAX_GROUPS) return hipErrorInvalidValue;
  void* ws = nullptr;
  const hipError_t e = scratch_address(&ws);
  if (e != hipSuccess) return e;
  return launch_select(energy, n_out, G, nnz, rec_index, rowptr1, gidx1, ws, s);
}

}  // namespace tq
