// A chain of dependent grouped GEMVs in one launch: the decode step's
// projections, stage after stage (gfx950).
//
// Paper: section 13 runs the packed model's whole decode step; within a
// decoder layer q, k and v read one input, o reads the attention output,
// gate and up read the normalised residual, and down reads the activated
// MLP state, so at batch 1 the step is a chain of dependent GEMVs (the
// operation of each stage is that of tq_gemv_grouped, eq. 3).
//
// Design for CDNA4:
// * One workgroup of 1024 threads per CU, all resident at once (cooperative
//   launch), each with the 16-copy LDS table built once for the whole chain
//   instead of once per launch.
// * Every stage is split over the workgroups by rows (a plan built on the
//   host: one 128-byte work record per workgroup and stage); inside a
//   workgroup the lanes own half-groups and decode exactly as the batch-1
//   GEMV does (gemv_decode.h), so every output equals tq_gemv's bit for bit.
// * Stage s+1 reads its x only after every workgroup has finished stage s.
//   A workgroup writes its outputs with device-coherent stores (sc1), waits
//   for them to complete, then publishes its own flag (one per workgroup,
//   64 bytes apart, so no two workgroups write one cache line).  The first
//   wave of every workgroup polls all flags with four independent coherent
//   loads per lane and round, and x is then read with coherent loads too:
//   every access that crosses workgroups bypasses the non-coherent caches,
//   so no cache-wide write-back or invalidate is needed (measured on
//   MI355X: 1.8 us per stage transition this way, 6.8 us with agent-scope
//   fences).
// * A workgroup issues the loads of its next stage's first two passes,
//   first records and row bounds before it waits, so they stream in while
//   the flags propagate; later passes go out after x, each once the pass
//   two before it is computed (a wave's loads return in order, so every
//   load issued before x delays x).
// * Flags carry an epoch, generation * stages + stage + 1, compared modulo
//   2^32; the last workgroup to finish a call advances the generation, so
//   no flag is ever reset.  Every wait is bounded: past its limit a
//   workgroup sets the sync block's sticky error word and carries on, so
//   the launch always ends.

#include <mutex>

#include "tq_internal.h"

#pragma clang fp contract(off)

namespace tq {
namespace {

#include "gemv_decode.h"

constexpr int kChainThreads = 1024;
constexpr int kChainMaxPasses = 6;
constexpr int kSpinLimit = 1 << 17;     // poll rounds (~0.1 s) before a wait gives up
constexpr int kSyncHeadBytes = 256;
constexpr int kFlagStrideDw = 16;       // 64 bytes between workgroup flags

struct ChainSyncHead {
  uint32_t generation;   // calls completed
  uint32_t exit_count;   // workgroups that finished the current call
  uint32_t error;        // sticky: a wait hit its limit
  uint32_t pad[61];
};
static_assert(sizeof(ChainSyncHead) == kSyncHeadBytes, "sync head size");

__device__ inline uint32_t ld_dev(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void st_dev(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline bool epoch_reached(uint32_t f, uint32_t e) { return (int32_t)(f - e) >= 0; }

constexpr int kCoherent = 16;   // sc1: device scope, bypassing the per-XCD caches

// Wave 0 waits until every workgroup has published epoch e; then the whole
// workgroup proceeds.  Bounded: past kSpinLimit rounds, or once another
// workgroup has given up, the error word is set and the wait ends.
__device__ void wait_all(const uint32_t* flags, ChainSyncHead* head, int nwg, uint32_t e) {
  if (threadIdx.x < 64) {
    const int l = threadIdx.x;
    for (int b = 0; b < nwg; b += 256) {
      const int w0 = min(b + l, nwg - 1), w1 = min(b + l + 64, nwg - 1);
      const int w2 = min(b + l + 128, nwg - 1), w3 = min(b + l + 192, nwg - 1);
      int spins = 0;
      while (true) {
        const uint32_t f0 = ld_dev(flags + kFlagStrideDw * w0), f1 = ld_dev(flags + kFlagStrideDw * w1);
        const uint32_t f2 = ld_dev(flags + kFlagStrideDw * w2), f3 = ld_dev(flags + kFlagStrideDw * w3);
        const bool ok = epoch_reached(f0, e) && epoch_reached(f1, e) && epoch_reached(f2, e) && epoch_reached(f3, e);
        if (__ballot(!ok) == 0) break;
        ++spins;
        if (spins > kSpinLimit || ((spins & 15) == 0 && ld_dev(&head->error) != 0)) {
          if (l == 0) st_dev(&head->error, 1u);
          break;
        }
      }
    }
  }
  __syncthreads();
  asm volatile("" ::: "memory");
}

// x of a stage, 16 bytes per load, coherent with stores made earlier in the
// same launch by other workgroups.
__device__ inline uint4 load_x16(__amdgpu_buffer_rsrc_t xr, int i) {
  typedef uint32_t u4v __attribute__((ext_vector_type(4)));
  const u4v v = __builtin_amdgcn_raw_buffer_load_b128(xr, 16 * i, 0, kCoherent);
  return uint4{v.x, v.y, v.z, v.w};
}

__device__ inline void store_y_dev(__amdgpu_buffer_rsrc_t yr, int i, float v, bool f32) {
  if (f32)
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), yr, 4 * i, 0, kCoherent);
  else
    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, (_Float16)v), yr, 2 * i, 0, kCoherent);
}

// One plane-0 pass of a lane: its 12 body bytes in one load.
struct __attribute__((aligned(4))) Body3 {
  uint32_t a, b, c;
};
__device__ inline void load_pass_c(Pass& p, const uint8_t* body0, const uint8_t* tail0, const uint16_t* scale0,
                                   const uint16_t* offset0, uint32_t f) {
  const Body3 b = *reinterpret_cast<const Body3*>(body0 + (size_t)(kMainBytes * f));
  p.w[0] = b.a;
  p.w[1] = b.b;
  p.w[2] = b.c;
  p.w[3] = __builtin_nontemporal_load(tail0 + (size_t)(2 * f));
  p.sc = __builtin_nontemporal_load(scale0 + (size_t)f);
  p.mu = __builtin_nontemporal_load(offset0 + (size_t)f);
}

// Plane-0 passes whose loads are issued before the wait; the rest go out
// after x, each once the pass two before it is computed (a wave's loads
// return in order, so loads issued before x delay x).
constexpr int kChainAhead = 2;

// One stage for one workgroup: issue its loads, wait for the previous
// stage (wait_e != 0), stage x, decode, write the outputs, publish my_e.
// The arithmetic is the batch-1 GEMV's, in the same order.
template <int kPasses>
__device__ __attribute__((always_inline)) inline void run_stage(const ChainWork& W, const unsigned char* lut,
                                                                unsigned char* smem, int lds_dyn, uint32_t* flags,
                                                                ChainSyncHead* head, int nwg, uint32_t wait_e,
                                                                uint32_t my_e) {
  constexpr int T = kChainThreads;
  const int tid = threadIdx.x;
  const int G = W.G;
  const int S = 2 * G;
  const int SP = padded_slots(S);
  const int segs = SP > 64 ? SP >> 6 : 1;
  const int ri = T / SP;
  const int K = G * kGroup;
  const int row_begin = W.row_begin;
  const int nrb = W.row_end - W.row_begin;
  const bool out_f32 = (W.flags & 1) != 0;

  uint32_t* xsw = reinterpret_cast<uint32_t*>(smem);
  float* rowsum = reinterpret_cast<float*>(smem + 4 * kXStrideDw * G);
  float* recval = rowsum + ((nrb * segs + 1) & ~1);
  const int rec_cap = (int)((lds_dyn - (reinterpret_cast<unsigned char*>(recval) - smem)) / 8);

  const bool in_rows = tid < ri * SP;
  const int sl = in_rows ? tid % SP : 0;
  const bool active = in_rows && sl < S;
  const int g = active ? sl >> 1 : 0;
  const int h = sl & 1;
  const int rl = in_rows ? tid / SP : 0;
  const uint32_t slot = (uint32_t)(tid & (kRep - 1)) << 4;
  const bool has_rec = W.nnz1 > 0;

  // ---- 1. Loads of this stage (before waiting for the previous one).
  // Record range: from the plan, or the device row pointers.
  // Without records x stands in as a readable address (at least 256 bytes).
  const int* rpb = has_rec ? W.rowptr1 + row_begin : reinterpret_cast<const int*>(W.x);
  int k0 = W.rec_begin, k1 = W.rec_end;
  const bool dev_range = has_rec && k0 < 0;
  if (dev_range) {
    k0 = rpb[0];
    k1 = rpb[nrb];
  }
  if (!has_rec) k0 = k1 = 0;
  const int hh = tid & 1;
  const int kr = k0 + (tid >> 1);
  constexpr int per_sweep = T >> 1;
  RecSrc MR;
  MR.codes1 = has_rec ? W.codes1 : W.codes0;
  MR.nnz1 = has_rec ? (uint32_t)W.nnz1 : 0u;
  MR.gidx1 = has_rec ? W.gidx1 : W.scale0;
  MR.offset1 = has_rec ? W.offset1 : W.scale0;
  MR.scale1 = has_rec ? W.scale1 : W.scale0;
  const int kmax = has_rec ? W.nnz1 - 1 : 0;
  auto rec_index = [&](int k) -> uint32_t { return (uint32_t)max(min(k, min(max(k1 - 1, k0), kmax)), 0); };
  RecHalf rec;
  load_rec_half(rec, MR, rec_index(kr), has_rec ? hh : 0);

  const uint32_t ngroups = (uint32_t)W.n_out * (uint32_t)G;
  const uint8_t* body0 = W.codes0 + kHalfBytes * h;
  const uint8_t* tail0 = W.codes0 + (size_t)(kMainBytes * ngroups) + h;
  const bool has_off = W.offset0 != nullptr;
  const uint16_t* off0 = has_off ? W.offset0 : W.scale0;
  Pass buf[kPasses];
  auto issue_pass = [&](int d) {
    const int r = min(row_begin + rl + d * ri, W.row_end - 1);
    uint32_t rg = (uint32_t)r * (uint32_t)G;
    asm volatile("" : "+v"(rg));
    load_pass_c(buf[d], body0, tail0, W.scale0, off0, rg + (uint32_t)g);
  };
  constexpr int kAhead = kPasses < kChainAhead ? kPasses : kChainAhead;
#pragma unroll
  for (int d = 0; d < kAhead; ++d) issue_pass(d);
  const int tr = has_rec ? min(tid, nrb - 1) : 0;
  const int rpa = rpb[tr];
  const int rpz = rpb[has_rec ? tr + 1 : 0];

  // ---- 2. The previous stage must be complete before x is read.
  if (wait_e != 0) wait_all(flags, head, nwg, wait_e);

  // ---- 3. x, coherent loads, into the 68-dword group slots.
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc((void*)W.x, 0, 2 * K, 0x00020000);
  for (int i = tid; i < K / 8; i += T) {
    typedef uint32_t u2v __attribute__((ext_vector_type(2)));
    const uint4 v = load_x16(xr, i);
    const int c = i & 15;
    uint32_t* xg = xsw + kXStrideDw * (i >> 4);
    *reinterpret_cast<u2v*>(xg + x_slot_dw(8 * c)) = u2v{v.x, v.y};
    *reinterpret_cast<u2v*>(xg + x_slot_dw(8 * c + 4)) = u2v{v.z, v.w};
  }
  __syncthreads();

  uint32_t xr_[kXrRegs];
  load_xr(xr_, xsw, g, h);
  float xsum = 0.f;
  if (has_off) {
    typedef _Float16 h2v __attribute__((ext_vector_type(2)));
    const h2v ones = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
    for (int i = 0; i < kXrRegs; ++i) xsum = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2v, xr_[i]), ones, xsum, false);
  }

  // ---- 4. Plane 0, one row per pass.
  const int seg = SP < 64 ? SP : 64;
#pragma unroll
  for (int d = 0; d < kPasses; ++d) {
    const int row = rl + d * ri;
    pass_priority<kPasses>(d);
    float v = code_dot(lut, slot, buf[d].w, xr_) * h2f(buf[d].sc);
    v = v + (has_off ? h2f(buf[d].mu) : 0.f) * xsum;
    asm volatile("" : "+v"(v));
    if (d + kAhead < kPasses) issue_pass(d + kAhead);
    v = (active && row < nrb) ? v : 0.f;
    const float sum = segment_sum(v, seg);
    if (in_rows && row < nrb && (sl & (seg - 1)) == seg - 1) rowsum[row * segs + (sl >> 6)] = sum;
    __builtin_amdgcn_sched_barrier(0);
  }
  __builtin_amdgcn_s_setprio(0);

  // ---- 5. Plane 1: two threads per record, sweeps of T / 2 records.
  if (has_rec) {
    for (int k = kr, first = 1; k < k1; k += per_sweep, first = 0) {
      if (!first) load_rec_half(rec, MR, rec_index(k), hh);
      if (k >= 0 && k - k0 < rec_cap) recval[2 * (k - k0) + hh] = record_half_value(lut, slot, xsw, rec, hh, G);
    }
  }
  __syncthreads();

  // ---- 6. Row totals in a fixed order (the GEMV's), coherent stores.
  if (tid < nrb) {
    float a = rowsum[tid * segs];
    for (int c = 1; c < segs; ++c) a += rowsum[tid * segs + c];
    if (has_rec) {
      typedef float f2v __attribute__((ext_vector_type(2)));
      const int kb = max(rpa, k0), ke = min(min(rpz, k1), k0 + rec_cap);
      for (int k = kb; k < ke; k += 8) {
        f2v v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = *reinterpret_cast<const f2v*>(recval + 2 * (min(k + u, ke - 1) - k0));
#pragma unroll
        for (int u = 0; u < 8; ++u) a += k + u < ke ? v[u].x + v[u].y : 0.f;
      }
    }
    const __amdgpu_buffer_rsrc_t yr =
        __builtin_amdgcn_make_buffer_rsrc(W.y, 0, W.n_out * (out_f32 ? 4 : 2), 0x00020000);
    store_y_dev(yr, row_begin + tid, a, out_f32);
  }

  // ---- 7. Publish: every output store of the workgroup has completed.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0) st_dev(flags + kFlagStrideDw * blockIdx.x, my_e);
}

// A workgroup with no rows in a stage still keeps the chain's order.
__device__ inline void idle_stage(uint32_t* flags, ChainSyncHead* head, int nwg, uint32_t wait_e, uint32_t my_e) {
  if (wait_e != 0) wait_all(flags, head, nwg, wait_e);
  if (threadIdx.x == 0) st_dev(flags + kFlagStrideDw * blockIdx.x, my_e);
}

__global__ void __launch_bounds__(kChainThreads) __attribute__((amdgpu_waves_per_eu(4)))
chain_kernel(const ChainWork* __restrict__ plan, int32_t n_stages, unsigned char* sync, int32_t nwg,
             int32_t lds_dyn) {
  __shared__ __attribute__((aligned(16))) unsigned char lut[kLutBytes];
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  ChainSyncHead* head = reinterpret_cast<ChainSyncHead*>(sync);
  uint32_t* flags = reinterpret_cast<uint32_t*>(sync + kSyncHeadBytes);
  const uint32_t gen = __builtin_amdgcn_readfirstlane(ld_dev(&head->generation));
  const uint32_t e0 = gen * (uint32_t)n_stages;

  for (int c = threadIdx.x; c < 256; c += kChainThreads) {
    const uint4 e = lut_entry(c);
#pragma unroll
    for (int q = 0; q < kRep; ++q) reinterpret_cast<uint4*>(lut)[c * kRep + ((q + c) & (kRep - 1))] = e;
  }
  // The table is complete before the first stage reads it (the first
  // stage's x barrier also orders it; this keeps idle first stages simple).
  __syncthreads();

  for (int s = 0; s < n_stages; ++s) {
    const ChainWork W = plan[(int64_t)s * nwg + blockIdx.x];
    const uint32_t wait_e = s == 0 ? 0u : e0 + (uint32_t)s;   // epoch of stage s - 1
    const uint32_t my_e = e0 + (uint32_t)s + 1u;
    const int passes = (W.flags >> 8) & 255;
    if (W.row_end <= W.row_begin) {
      idle_stage(flags, head, nwg, wait_e, my_e);
      continue;
    }
    switch (passes) {
      case 1: run_stage<1>(W, lut, smem, lds_dyn, flags, head, nwg, wait_e, my_e); break;
      case 2: run_stage<2>(W, lut, smem, lds_dyn, flags, head, nwg, wait_e, my_e); break;
      case 3: run_stage<3>(W, lut, smem, lds_dyn, flags, head, nwg, wait_e, my_e); break;
      case 4: run_stage<4>(W, lut, smem, lds_dyn, flags, head, nwg, wait_e, my_e); break;
      case 5: run_stage<5>(W, lut, smem, lds_dyn, flags, head, nwg, wait_e, my_e); break;
      default: run_stage<6>(W, lut, smem, lds_dyn, flags, head, nwg, wait_e, my_e); break;
    }
  }

  // The last workgroup to finish advances the generation for the next call.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t done = __hip_atomic_fetch_add(&head->exit_count, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (done == (uint32_t)nwg - 1) {
      st_dev(&head->exit_count, 0u);
      st_dev(&head->generation, gen + 1u);
    }
  }
}

__global__ void __launch_bounds__(256) sync_clear(uint32_t* sync, int64_t ndw) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < ndw; i += (int64_t)gridDim.x * 256) sync[i] = 0u;
}

// LDS bytes beyond the table for one stage's work: x slots, wave sums of
// every row, two values per record.
size_t stage_lds(int G, int rows, int64_t records) {
  const int SP = padded_slots(2 * G);
  const int segs = SP > 64 ? SP / 64 : 1;
  return 4 * (size_t)kXStrideDw * G + 4 * (size_t)((rows * segs + 1) & ~1) + 8 * (size_t)records;
}

struct ChainDevice {
  int cus = 0;
  bool attr_set = false;
};

hipError_t chain_device(ChainDevice** out) {
  static std::mutex mu;
  static ChainDevice devs[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  ChainDevice& d = devs[dev];
  if (d.cus == 0) {
    e = hipDeviceGetAttribute(&d.cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
  }
  *out = &d;
  return hipSuccess;
}

}  // namespace

int chain_lds_limit() { return 160 * 1024 - kLutBytes; }
int chain_sync_head_bytes() { return kSyncHeadBytes; }
int chain_flag_stride_bytes() { return 4 * kFlagStrideDw; }

hipError_t chain_workgroups(int* nwg) {
  ChainDevice* d = nullptr;
  const hipError_t e = chain_device(&d);
  if (e == hipSuccess) *nwg = d->cus;
  return e;
}

// Plan of one stage: rows per workgroup and passes, or false where the
// stage does not fit one round of nwg workgroups of 1024 threads.
bool plan_stage(const MatDev* ms, int n, int nwg, int* rows_per_wg, int* passes, int* used) {
  const int G = ms[0].n_groups;
  const int SP = padded_slots(2 * G);
  if (SP > kChainThreads) return false;
  const int ri = kChainThreads / SP;
  int64_t total = 0;
  for (int i = 0; i < n; ++i) total += ms[i].n_out;
  int64_t rpw = (total + nwg - 1) / nwg;
  if (rpw < 1) rpw = 1;
  for (;; ++rpw) {
    int64_t wgs = 0;
    for (int i = 0; i < n; ++i) wgs += (ms[i].n_out + rpw - 1) / rpw;
    if (wgs <= nwg) {
      *used = (int)wgs;
      break;
    }
  }
  const int64_t p = (rpw + ri - 1) / ri;
  if (p > kChainMaxPasses || rpw > kChainThreads) return false;
  *rows_per_wg = (int)rpw;
  *passes = (int)p;
  return true;
}

hipError_t chain_plan_fill(const ChainStageDev* st, int n_stages, int nwg, ChainWork* plan, int64_t* max_lds) {
  int64_t lds = 0;
  for (int s = 0; s < n_stages; ++s) {
    const ChainStageDev& S = st[s];
    int rpw = 0, passes = 0, used = 0;
    if (!plan_stage(S.m, S.n, nwg, &rpw, &passes, &used)) return hipErrorInvalidValue;
    ChainWork* row = plan + (int64_t)s * nwg;
    int w = 0;
    for (int i = 0; i < S.n; ++i) {
      const MatDev& m = S.m[i];
      for (int64_t r0 = 0; r0 < m.n_out; r0 += rpw, ++w) {
        ChainWork& W = row[w];
        W = ChainWork{};
        W.codes0 = m.codes0;
        W.scale0 = m.scale0;
        W.rowptr1 = m.rowptr1;
        W.gidx1 = m.gidx1;
        W.codes1 = m.codes1;
        W.offset1 = m.offset1;
        W.scale1 = m.scale1;
        W.offset0 = m.offset0;
        W.x = S.x;
        W.y = S.ys[i];
        W.n_out = m.n_out;
        W.nnz1 = (int32_t)m.nnz1;
        W.row_begin = (int32_t)r0;
        W.row_end = (int32_t)(r0 + rpw < m.n_out ? r0 + rpw : m.n_out);
        W.G = m.n_groups;
        W.flags = (S.out_f32 ? 1 : 0) | (passes << 8);
        int64_t recs = (int64_t)W.row_end - W.row_begin;   // bound without host pointers: all groups
        recs *= m.n_groups;
        if (m.nnz1 > 0 && m.rowptr1_host != nullptr) {
          int64_t a = m.rowptr1_host[W.row_begin], b = m.rowptr1_host[W.row_end];
          a = a < 0 ? 0 : (a > m.nnz1 ? m.nnz1 : a);   // in bounds whatever the host copy holds
          b = b < 0 ? 0 : (b > m.nnz1 ? m.nnz1 : b);
          W.rec_begin = (int32_t)a;
          W.rec_end = (int32_t)b;
          recs = b > a ? b - a : 0;
        } else if (m.nnz1 > 0) {
          W.rec_begin = -1;
          W.rec_end = -1;
          if (recs > m.nnz1) recs = m.nnz1;
        } else {
          recs = 0;
        }
        const int64_t need = (int64_t)stage_lds(W.G, W.row_end - W.row_begin, recs);
        if (need > lds) lds = need;
      }
    }
    for (; w < nwg; ++w) {   // idle in this stage
      row[w] = ChainWork{};
      row[w].G = S.m[0].n_groups;
    }
  }
  *max_lds = lds;
  return hipSuccess;
}

hipError_t launch_chain_clear(void* sync, int64_t bytes, hipStream_t s) {
  const int64_t ndw = bytes / 4;
  const int64_t b = (ndw + 255) / 256;
  hipLaunchKernelGGL(sync_clear, dim3((unsigned)(b < 1 ? 1 : (b > 4096 ? 4096 : b))), dim3(256), 0, s,
                     static_cast<uint32_t*>(sync), ndw);
  return hipGetLastError();
}

hipError_t launch_chain(const ChainWork* plan, int n_stages, int nwg, int lds_dyn, void* sync, hipStream_t s) {
  ChainDevice* d = nullptr;
  hipError_t e = chain_device(&d);
  if (e != hipSuccess) return e;
  if (!d->attr_set) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(chain_kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                            chain_lds_limit());
    if (e != hipSuccess) return e;
    d->attr_set = true;
  }
  unsigned char* sp = static_cast<unsigned char*>(sync);
  void* args[] = {(void*)&plan, (void*)&n_stages, (void*)&sp, (void*)&nwg, (void*)&lds_dyn};
  return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(chain_kernel), dim3(nwg), dim3(kChainThreads), args,
                                    (unsigned)lds_dyn, s);
}

}  // namespace tq
