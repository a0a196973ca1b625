// Packed ternary GEMV y = W^ x for gfx950 (batch 1), and its grouped form.
//
// Paper: section 3, eq. 3 (W^ = (mu + a0 T0 + a1 T1) (.) M, T_i in
// {-1, 0, +1}; per-group offsets/scales on a salience-selected subset), A16
// activations (section 3), packed supports (section 12).  The paper's own
// kernel (section 13) is a prototype for another GPU and gives no design;
// this one is built for CDNA4:
//
// * Lane ownership.  A row of G groups is split into S = 2G half-groups: half
//   h of group g holds code bytes 12h .. 12h+11 (inputs 60h .. 60h+59) plus
//   tail byte 24+h (inputs 120+5h ..).  Rows are laid on SP lanes, SP = S
//   rounded up to a divisor or a multiple of 64, so that no row straddles a
//   wave boundary; a workgroup of T threads covers RI = T / SP rows per pass
//   and thread t always owns half-group t % SP, so its activations stay in 33
//   VGPRs for the whole launch: per pair of code bytes (j, j+1) the fp16
//   pairs (x0, x1), (x2, x3) of each byte and (x4 of j, x4 of j+1); for the
//   tail byte (x0, x1), (x2, x3), (x4, 0).
// * Decode.  A 256-entry table maps a code to four dwords of fp16 patterns
//   (+1 = 0x3C00, -1 = 0xBC00, 0 = 0): (t0, t1), (t2, t3), (t4, 0), (0, t4).
//   A pair of bytes takes two 16-byte table reads and five v_dot2_f32_f16
//   (the fifth on (t4 of j) | (t4 of j+1)), accumulating in fp32.  The table is
//   replicated kRep = 16 times in LDS (copy q of code c at byte 16 (16 c + q),
//   64 KiB); a lane reads copy lane % 16 (12 bytes), so lanes read together
//   sit on different banks whatever codes they hold (four copies cost two to
//   three times as many LDS cycles in bank conflicts).
// * Loads.  Per pass a lane loads 12 body bytes (three dwords, 4-aligned in
//   the split layout), its tail byte and its group's scale; lanes of a row
//   read consecutive bytes, so every wave load is contiguous.  Every wave
//   issues its x loads before any wave issues weight loads (a barrier
//   between), then the records' and the first two passes' loads; each later
//   pass is issued after the pass two before it is computed (issuing every
//   pass up front stalls the waves at issue, and the set-up with them).
//   Loads go out in the order their data is needed and every one is
//   unconditional (clamped addresses), so each wait is an exact vmcnt.
//   x is staged in LDS with each half-group's 60 inputs 16-byte aligned, so
//   a lane fetches its activations with ten reads.  The matrix record is read
//   from the kernel-argument
//   segment with one scalar round trip; the leading arguments that select it
//   are preloaded into SGPRs.
// * Per-group offsets (optional, on every group): a lane sums its own
//   activations once and adds mu0 * sum(x) to each pass's value; the
//   offsets are loaded with the scales.
// * Plane 1.  Each record is handled by two threads (one per half).  A
//   record half computes s1 * sum(t1 x) + mu * sum(x) over its half-group and
//   stores it in its own LDS slot (records of a workgroup are contiguous in
//   CSR order, so the slot is the record's index in that range).  When the
//   host passes each workgroup's record range, their loads go out with the
//   first batch, and if extra waves (within 1024 threads) can take every
//   record of a workgroup in one sweep, they do so while the other waves
//   run plane 0.  Otherwise the plane-0 waves take the records after plane
//   0 (without host ranges the range also needs the row pointers first, one
//   more memory round trip).
// * Reduction.  After each pass the lanes of a row add their plane-0 values
//   with DPP (quad permutes, mirrors and row broadcasts folded into the
//   adds); the last lane of each 64-lane segment writes the segment sum to
//   LDS.  After one barrier, one thread per row adds the row's segment sums
//   and then its records' two halves, always in the same order.  No atomics:
//   results are bit-identical run to run.

#include "tq_internal.h"

// Products and sums are rounded as written (no fused multiply-add), so the
// result does not depend on which of the kernel variants runs.
#pragma clang fp contract(off)

namespace tq {
namespace {

#include "gemv_decode.h"

#include "gemv_args.h"

// Plane-0 passes whose loads are issued before the set-up.
constexpr int kPrefetch = 2;
// Most record sweeps a record wave may take (more sweeps measured slower:
// the record waves then compete with plane 0 for the LDS).
constexpr int kMaxRecSweeps = 1;

// kPasses: plane-0 passes per lane (the first kPrefetch loaded before the
// set-up).  kXLoads: 16-byte
// loads of x per thread (ceil(K / 8 / T)).  kHostRanges: the host passes
// each workgroup's record range.
template <int kPasses, int kXLoads, bool kHostRanges, bool kOffset0>
__global__ void __launch_bounds__(kMaxThreads) __attribute__((amdgpu_waves_per_eu(4)))
gemv_kernel(const uint16_t* __restrict__ x, int32_t G, int32_t ri, int32_t rows_per_wg, int32_t opts,
            int32_t wb1, int32_t wb2, int32_t wb3, int32_t wb4, int32_t wb5, int32_t wb6, int32_t wb7,
            int32_t nthreads, const GemvArgs args) {
  // The table is the kernel's only static LDS, so it sits at LDS address 0
  // and a table address is just the perm result (no base to add).
  __shared__ __attribute__((aligned(16))) unsigned char lut[kLutBytes];
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int S = 2 * G;
  const int SP = padded_slots(S);
  const int segs = SP > 64 ? SP >> 6 : 1;   // waves per row
  const int K = G * kGroup;
  uint32_t* xsw = reinterpret_cast<uint32_t*>(smem);
  // Plane-0 sum of every (row, wave of the row), then two values per record
  // (its halves, 8-byte aligned).  Pointers derive from the LDS base by plain
  // offsets, so accesses stay LDS instructions.
  float* rowsum = reinterpret_cast<float*>(smem + 4 * kXStrideDw * G);
  float* recval = rowsum + ((rows_per_wg * segs + 1) & ~1);
  const int rec_cap = rows_per_wg * G;   // records a block can hold

  const int tid = threadIdx.x;
  const int T = nthreads;   // == blockDim.x, without a load of the dispatch packet
  // opts: bit 0 fp32 output; bits 16.. the first thread of the record waves
  // (0: no record waves, every thread takes records after plane 0).
  const int out_f32 = opts & 1;
  const int rec_tid0 = opts >> 16;

  // 1. x, first of all: it needs only preloaded arguments, so it goes out
  //    before the wait for the matrix record below.
  uint4 xv[kXLoads];
#pragma unroll
  for (int q = 0; q < kXLoads; ++q) xv[q] = reinterpret_cast<const uint4*>(x)[min(tid + q * T, K / 8 - 1)];
  // Keep the issue order: neither the optimiser nor the scheduler may move
  // loads across these points (no instruction emitted).
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);

  // Which matrix this workgroup serves: the first workgroups of matrices
  // 1..7 arrive in SGPRs (unused ones are INT32_MAX), so the matrix record
  // is one scalar load away.
  const int w = blockIdx.x;
  const int sel = __builtin_amdgcn_readfirstlane((w >= wb1) + (w >= wb2) + (w >= wb3) + (w >= wb4) + (w >= wb5) +
                                                 (w >= wb6) + (w >= wb7));
  // The whole record in one batch of scalar loads and one wait (left to
  // itself the compiler fetches fields at their first use, one round trip
  // each).
  const GemvMat M = args.m[sel];
  int hk0 = 0, hk1 = 0;
  if constexpr (kHostRanges) {
    hk0 = args.rec_begin[w + sel];
    hk1 = args.rec_begin[w + sel + 1];
  }
  __builtin_amdgcn_sched_barrier(0);
  // Every wave's x loads go out before any wave's weight loads: the CU
  // serves its waves' loads in issue order, and x is needed first (a bare
  // barrier, no wait for the loads; the record's scalar loads are already
  // on their way).
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::"s"(M.codes0), "s"(M.scale0), "s"(M.rowptr1), "s"(M.gidx1), "s"(M.codes1), "s"(M.offset1),
               "s"(M.scale1), "s"(M.offset0), "s"(M.y), "s"(M.n_out), "s"(M.nnz1), "s"(M.wg_begin), "s"(hk0),
               "s"(hk1));
  __builtin_amdgcn_sched_barrier(0);
  void* const yp = M.y;
  const int row_begin = (w - M.wg_begin) * rows_per_wg;
  const int row_end = min(M.n_out, row_begin + rows_per_wg);
  const int nrb = row_end - row_begin;

  const bool in_rows = tid < ri * SP;
  const int sl = in_rows ? tid % SP : 0;   // half-group slot within the row
  const bool active = in_rows && sl < S;
  const int g = active ? sl >> 1 : 0;
  const int h = sl & 1;
  const int rl = in_rows ? tid / SP : 0;
  const uint32_t slot = (uint32_t)(tid & (kRep - 1)) << 4;
  const bool has_rec = M.nnz1 > 0;

  // Loads, in the order their data is needed (each wait is then exact).
  // 2. The block's record range: from the arguments with host ranges, else
  //    its first and last row pointers.  Without records x stands in as a
  //    readable address.
  const int* rpb = has_rec ? M.rowptr1 + row_begin : reinterpret_cast<const int*>(x);
  int k0, k1;
  if constexpr (kHostRanges) {
    k0 = hk0;
    k1 = hk1;
  } else {
    k0 = rpb[0];
    k1 = rpb[has_rec ? nrb : 0];
  }
  // Record halves: two consecutive threads per record, so that the record
  // work occupies as few waves as possible (the record code costs a wave
  // the same time however few of its lanes have a record).
  // With record waves (threads rec_tid0 .., whole waves) only they take
  // records, from the start, while the other waves run plane 0.
  const bool rec_wave = rec_tid0 > 0 && tid >= rec_tid0;
  // (Plane-0 threads of such a launch load the block's first record, which
  // they never use: an index below the block's range would fetch other
  // blocks' records for nothing.)
  const int rt = rec_tid0 > 0 ? (rec_wave ? tid - rec_tid0 : 0) : tid;
  const int hh = rt & 1;
  const int kr = k0 + (rt >> 1);
  const int per_sweep = (rec_tid0 > 0 ? T - rec_tid0 : T) >> 1;
  // Without records, plane-0 arrays stand in as readable addresses (the
  // loaded values are ignored).
  RecSrc MR;
  MR.codes1 = has_rec ? M.codes1 : M.codes0;
  MR.nnz1 = has_rec ? (uint32_t)M.nnz1 : 0u;
  MR.gidx1 = has_rec ? M.gidx1 : M.scale0;
  MR.offset1 = has_rec ? M.offset1 : M.scale0;
  MR.scale1 = has_rec ? M.scale1 : M.scale0;
  const int kmax = has_rec ? M.nnz1 - 1 : 0;
  RecHalf rec;
  // Threads past the block's records reload its last record (no extra
  // cache lines); the values are ignored.
  auto rec_index = [&](int k) -> uint32_t { return (uint32_t)max(min(k, min(max(k1 - 1, k0), kmax)), 0); };
  // 3. With host ranges the first sweep of records needs no row pointer.
  if constexpr (kHostRanges) load_rec_half(rec, MR, rec_index(kr), has_rec ? hh : 0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  // 4. The first kAhead plane-0 passes of this lane; each later pass is
  //    issued once the pass kAhead before it has been computed.  Issuing
  //    every pass here would stall the waves at issue (the CU holds only so
  //    many loads in flight) and with them the set-up below.
  constexpr int kAhead = kPasses < kPrefetch ? kPasses : kPrefetch;
  const uint32_t ngroups = (uint32_t)M.n_out * (uint32_t)G;
  const uint8_t* body0 = M.codes0 + kHalfBytes * h;
  const uint8_t* tail0 = M.codes0 + (size_t)(kMainBytes * ngroups) + h;
  // A matrix without offsets in a launch with offsets reads its scales in
  // their place (the values are multiplied by zero).
  const bool has_off = kOffset0 && M.offset0 != nullptr;
  const uint16_t* off0 = has_off ? M.offset0 : M.scale0;
  Pass buf[kPasses];
  auto issue_pass = [&](int d) {
    const int r = min(row_begin + rl + d * ri, row_end - 1);
    // Multiply, then add: fused into a 64-bit multiply-add, the unused high
    // half of the addend can land on a register a load is still filling,
    // and the wait for that load would stall the issue here.
    uint32_t rg = (uint32_t)r * (uint32_t)G;
    asm volatile("" : "+v"(rg));
    load_pass<kOffset0>(buf[d], body0, tail0, M.scale0, off0, rg + (uint32_t)g);
  };
#pragma unroll
  for (int d = 0; d < kAhead; ++d) issue_pass(d);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  // 5. Thread t < nrb: the bounds of row t (it adds that row's records at
  //    the end).
  const int tr = has_rec ? min(tid, nrb - 1) : 0;
  const int rpa = rpb[tr];
  const int rpz = rpb[has_rec ? tr + 1 : 0];
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  // 6. Without host ranges: the first sweep of records once the range is
  //    known, when few passes leave registers to spare (else after plane 0).
  constexpr bool kPreRec = kHostRanges || kPasses <= 2;
  if constexpr (!kHostRanges && kPreRec) load_rec_half(rec, MR, rec_index(kr), has_rec ? hh : 0);

  // Set-up in LDS: the table first (it needs no loaded data, so it is built
  // while x is still in flight), then x.
  // One thread per code writes its 16 copies; at step q thread c writes copy
  // (q + c) % 16, so the 16 lanes of an LDS pass hit 16 different bank
  // quads.
  for (int c = tid; c < 256; c += T) {
    const uint4 e = lut_entry(c);
#pragma unroll
    for (int q = 0; q < kRep; ++q) reinterpret_cast<uint4*>(lut)[c * kRep + ((q + c) & (kRep - 1))] = e;
  }
#pragma unroll
  for (int q = 0; q < kXLoads; ++q) {
    // 8 inputs 8c .. 8c + 7 of group i / 16 (c = i % 16), as two 4-input
    // halves (neither straddles a part of the slot).  Unconditional (threads
    // past the end rewrite the last slot with the same data), so the load is
    // not sunk into a branch behind the weight loads.
    typedef uint32_t u2v __attribute__((ext_vector_type(2)));
    const int i = min(tid + q * T, K / 8 - 1);
    const int c = i & 15;
    uint32_t* xg = xsw + kXStrideDw * (i >> 4);
    *reinterpret_cast<u2v*>(xg + x_slot_dw(8 * c)) = u2v{xv[q].x, xv[q].y};
    *reinterpret_cast<u2v*>(xg + x_slot_dw(8 * c + 4)) = u2v{xv[q].z, xv[q].w};
  }
  __syncthreads();

  // This lane's activations.
  uint32_t xr[kXrRegs];
  load_xr(xr, xsw, g, h);
  // With offsets: the sum of this lane's activations (its half of the
  // group), in a fixed order, for the mu0 * sum(x) term of every pass.
  float xsum = 0.f;
  if constexpr (kOffset0) {
    typedef _Float16 h2v __attribute__((ext_vector_type(2)));
    const h2v ones = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
    for (int i = 0; i < kXrRegs; ++i) xsum = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2v, xr[i]), ones, xsum, false);
  }

  // Plane 0, one row per pass: s0 * sum_i t0 x over each half-group, summed
  // over the row's lanes of this wave.
  const int seg = SP < 64 ? SP : 64;
  if (!rec_wave) {
#pragma unroll
  for (int d = 0; d < kPasses; ++d) {
    const int row = rl + d * ri;
    pass_priority<kPasses>(d);
    float v = code_dot(lut, slot, buf[d].w, xr) * h2f(buf[d].sc);
    if constexpr (kOffset0) v = v + (has_off ? h2f(buf[d].mu) : 0.f) * xsum;
    // Pin the value here: otherwise the dot products sink into the guarded
    // store below while their table reads cannot, and the reads' results of
    // every pass stay live at once.
    asm volatile("" : "+v"(v));
    if (d + kAhead < kPasses) issue_pass(d + kAhead);
    v = (active && row < nrb) ? v : 0.f;
    const float sum = segment_sum(v, seg);
    if (in_rows && row < nrb && (sl & (seg - 1)) == seg - 1) rowsum[row * segs + (sl >> 6)] = sum;
    __builtin_amdgcn_sched_barrier(0);   // keep passes apart: bounds the LUT reads in flight
  }
  }

  __builtin_amdgcn_s_setprio(0);
  // Plane 1: each record half stores its value (records of a block are
  // contiguous, so a record's slot is its index in the block).
  if (has_rec && (rec_tid0 == 0 || rec_wave)) {
    for (int k = kr, first = 1; k < k1; k += per_sweep, first = 0) {
      if (!kPreRec || !first) load_rec_half(rec, MR, rec_index(k), hh);
      if (k >= 0 && k - k0 < rec_cap) recval[2 * (k - k0) + hh] = record_half_value(lut, slot, xsw, rec, hh, G);
    }
  }
  __syncthreads();

  // Row totals, one thread per row in a fixed order: the row's wave sums,
  // then its records (half 0 + half 1) in index order.
  if (tid < nrb) {
    float a = rowsum[tid * segs];
    for (int c = 1; c < segs; ++c) a += rowsum[tid * segs + c];
    if (has_rec) {
      // Eight records per step, all reads first (absent ones add +0).
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
    store_y(yp, row_begin + tid, a, out_f32);
  }
}

// ------------------------------------------------------ a few batch rows
// Y = X W^T for kB = 2..4 activation rows of one matrix: the GEMV above with
// kB activation rows held in registers (33 each), so every code byte is
// decoded once for all rows; for small batches this is cheaper than the
// MFMA path (which must widen each code byte to 8 k-slots).  Records use the
// host ranges and are taken by all threads after plane 0; X rows are staged
// in LDS one after another.  Y is [kB][N].
template <int kB>
constexpr int batch_max_threads() {
  return kB <= 2 ? 1024 : 512;   // 33 activation registers per row
}

template <int kPasses, int kXLoads, bool kOffset0, int kB>
__global__ void __launch_bounds__(batch_max_threads<kB>())
gemv_batch_kernel(const uint16_t* __restrict__ X, int32_t G, int32_t ri, int32_t rows_per_wg, int32_t out_f32,
                  int32_t rec_slots, int32_t nthreads, const GemvArgs args) {
  __shared__ __attribute__((aligned(16))) unsigned char lut[kLutBytes];
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int S = 2 * G;
  const int SP = padded_slots(S);
  const int segs = SP > 64 ? SP >> 6 : 1;
  const int K = G * kGroup;
  const int xslot = kXStrideDw * G;   // dwords per staged X row
  uint32_t* xsw = reinterpret_cast<uint32_t*>(smem);
  // Wave sums [row][wave of the row][batch row], then record values
  // [record][half][batch row].
  float* rowsum = reinterpret_cast<float*>(smem + 4 * (size_t)xslot * kB);
  float* recval = rowsum + ((rows_per_wg * segs * kB + 1) & ~1);
  const int tid = threadIdx.x;
  const int T = nthreads;

  // 1. X, first of all.
  uint4 xv[kB][kXLoads];
#pragma unroll
  for (int b = 0; b < kB; ++b)
#pragma unroll
    for (int q = 0; q < kXLoads; ++q)
      xv[b][q] = reinterpret_cast<const uint4*>(X + (size_t)b * K)[min(tid + q * T, K / 8 - 1)];
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  const int w = blockIdx.x;
  const GemvMat M = args.m[0];
  const int hk0 = args.rec_begin[w], hk1 = args.rec_begin[w + 1];
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("" ::"s"(M.codes0), "s"(M.scale0), "s"(M.rowptr1), "s"(M.gidx1), "s"(M.codes1), "s"(M.offset1),
               "s"(M.scale1), "s"(M.offset0), "s"(M.y), "s"(M.n_out), "s"(M.nnz1), "s"(hk0), "s"(hk1));
  __builtin_amdgcn_sched_barrier(0);
  const int row_begin = w * rows_per_wg;
  const int row_end = min(M.n_out, row_begin + rows_per_wg);
  const int nrb = row_end - row_begin;

  const bool in_rows = tid < ri * SP;
  const int sl = in_rows ? tid % SP : 0;
  const bool active = in_rows && sl < S;
  const int g = active ? sl >> 1 : 0;
  const int h = sl & 1;
  const int rl = in_rows ? tid / SP : 0;
  const uint32_t slot = (uint32_t)(tid & (kRep - 1)) << 4;
  const bool has_rec = M.nnz1 > 0;

  // 2. Records of this block (host ranges), first sweep.
  const int k0 = hk0, k1 = hk1;
  const int hh = tid & 1;
  const int kr = k0 + (tid >> 1);
  const int per_sweep = T >> 1;
  RecSrc MR;
  MR.codes1 = has_rec ? M.codes1 : M.codes0;
  MR.nnz1 = has_rec ? (uint32_t)M.nnz1 : 0u;
  MR.gidx1 = has_rec ? M.gidx1 : M.scale0;
  MR.offset1 = has_rec ? M.offset1 : M.scale0;
  MR.scale1 = has_rec ? M.scale1 : M.scale0;
  const int kmax = has_rec ? M.nnz1 - 1 : 0;
  RecHalf rec;
  auto rec_index = [&](int k) -> uint32_t { return (uint32_t)max(min(k, min(max(k1 - 1, k0), kmax)), 0); };
  load_rec_half(rec, MR, rec_index(kr), has_rec ? hh : 0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  // 3. The first passes of plane 0; later ones inside the pass loop.
  constexpr int kAhead = kPasses < kPrefetch ? kPasses : kPrefetch;
  const uint32_t ngroups = (uint32_t)M.n_out * (uint32_t)G;
  const uint8_t* body0 = M.codes0 + kHalfBytes * h;
  const uint8_t* tail0 = M.codes0 + (size_t)(kMainBytes * ngroups) + h;
  const bool has_off = kOffset0 && M.offset0 != nullptr;
  const uint16_t* off0 = has_off ? M.offset0 : M.scale0;
  Pass buf[kPasses];
  auto issue_pass = [&](int d) {
    const int r = min(row_begin + rl + d * ri, row_end - 1);
    uint32_t rg = (uint32_t)r * (uint32_t)G;
    asm volatile("" : "+v"(rg));
    load_pass<kOffset0>(buf[d], body0, tail0, M.scale0, off0, rg + (uint32_t)g);
  };
#pragma unroll
  for (int d = 0; d < kAhead; ++d) issue_pass(d);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  // 4. Row bounds for the row totals.
  const int* rpb = has_rec ? M.rowptr1 + row_begin : reinterpret_cast<const int*>(X);
  const int tr = has_rec ? min(tid, nrb - 1) : 0;
  const int rpa = rpb[tr];
  const int rpz = rpb[has_rec ? tr + 1 : 0];
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);

  // Set-up: the table, then the X rows.
  for (int c = tid; c < 256; c += T) {
    const uint4 e = lut_entry(c);
#pragma unroll
    for (int q = 0; q < kRep; ++q) reinterpret_cast<uint4*>(lut)[c * kRep + ((q + c) & (kRep - 1))] = e;
  }
#pragma unroll
  for (int b = 0; b < kB; ++b) {
#pragma unroll
    for (int q = 0; q < kXLoads; ++q) {
      typedef uint32_t u2v __attribute__((ext_vector_type(2)));
      const int i = min(tid + q * T, K / 8 - 1);
      const int c = i & 15;
      uint32_t* xg = xsw + xslot * b + kXStrideDw * (i >> 4);
      *reinterpret_cast<u2v*>(xg + x_slot_dw(8 * c)) = u2v{xv[b][q].x, xv[b][q].y};
      *reinterpret_cast<u2v*>(xg + x_slot_dw(8 * c + 4)) = u2v{xv[b][q].z, xv[b][q].w};
    }
  }
  __syncthreads();

  uint32_t xr[kB][kXrRegs];
#pragma unroll
  for (int b = 0; b < kB; ++b) load_xr(xr[b], xsw + xslot * b, g, h);
  float xsum[kB];
#pragma unroll
  for (int b = 0; b < kB; ++b) {
    xsum[b] = 0.f;
    if constexpr (kOffset0) {
      typedef _Float16 h2v __attribute__((ext_vector_type(2)));
      const h2v ones = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
      for (int i = 0; i < kXrRegs; ++i)
        xsum[b] = __builtin_amdgcn_fdot2(__builtin_bit_cast(h2v, xr[b][i]), ones, xsum[b], false);
    }
  }

  // Plane 0.
  const int seg = SP < 64 ? SP : 64;
#pragma unroll
  for (int d = 0; d < kPasses; ++d) {
    const int row = rl + d * ri;
    pass_priority<kPasses>(d);
    float v[kB];
    code_dot_rows<kB>(lut, slot, buf[d].w, xr, v);
    const float sc = h2f(buf[d].sc);
#pragma unroll
    for (int b = 0; b < kB; ++b) {
      v[b] = v[b] * sc;
      if constexpr (kOffset0) v[b] = v[b] + (has_off ? h2f(buf[d].mu) : 0.f) * xsum[b];
      asm volatile("" : "+v"(v[b]));
    }
    if (d + kAhead < kPasses) issue_pass(d + kAhead);
#pragma unroll
    for (int b = 0; b < kB; ++b) {
      const float vb = (active && row < nrb) ? v[b] : 0.f;
      const float sum = segment_sum(vb, seg);
      if (in_rows && row < nrb && (sl & (seg - 1)) == seg - 1) rowsum[(row * segs + (sl >> 6)) * kB + b] = sum;
    }
    __builtin_amdgcn_sched_barrier(0);
  }

  __builtin_amdgcn_s_setprio(0);
  // Plane 1, all threads, sweeps of T / 2 records.
  if (has_rec) {
    for (int k = kr, first = 1; k < k1; k += per_sweep, first = 0) {
      if (!first) load_rec_half(rec, MR, rec_index(k), hh);
      if (k >= 0 && k - k0 < rec_slots) {
        uint32_t xq[kB][kXrRegs];
        const int rg = min((int)rec.g, G - 1);
#pragma unroll
        for (int b = 0; b < kB; ++b) load_xr(xq[b], xsw + xslot * b, rg, hh);
        float p[kB];
        code_dot_rows<kB>(lut, slot, rec.w, xq, p);
#pragma unroll
        for (int b = 0; b < kB; ++b) {
          float s0 = 0.f, s1 = 0.f, s2 = 0.f;
#pragma unroll
          for (int i = 0; i < kXrRegs; i += 3) {
            s0 = fdot2(xq[b][i], 0x3C003C00u, s0);
            s1 = fdot2(xq[b][i + 1], 0x3C003C00u, s1);
            s2 = fdot2(xq[b][i + 2], 0x3C003C00u, s2);
          }
          const float xs = (s0 + s1) + s2;
          recval[(2 * (k - k0) + hh) * kB + b] = h2f(rec.s1) * p[b] + h2f(rec.mu) * xs;
        }
      }
    }
  }
  __syncthreads();

  // Row totals, one thread per row, every batch row in a fixed order.
  if (tid < nrb) {
    const int kb = has_rec ? max(rpa, k0) : 0, ke = has_rec ? min(min(rpz, k1), k0 + rec_slots) : 0;
#pragma unroll
    for (int b = 0; b < kB; ++b) {
      float a = rowsum[(tid * segs) * kB + b];
      for (int c = 1; c < segs; ++c) a += rowsum[(tid * segs + c) * kB + b];
      for (int k = kb; k < ke; ++k) a += recval[(2 * (k - k0)) * kB + b] + recval[(2 * (k - k0) + 1) * kB + b];
      store_y(M.y, b * M.n_out + row_begin + tid, a, out_f32);
    }
  }
}

typedef void (*GemvKernel)(const uint16_t*, int32_t, int32_t, int32_t, int32_t, int32_t, int32_t, int32_t, int32_t,
                           int32_t, int32_t, int32_t, int32_t, const GemvArgs);

constexpr int kPassChoices[] = {1, 2, 3, 4, 6, 8};
constexpr int kNumPass = 6;
constexpr int kXChoices[] = {1, 2, 4};

template <int PI, int XI, bool HR, bool OFF>
constexpr GemvKernel kernel_at() {
  return gemv_kernel<kPassChoices[PI], kXChoices[XI], HR, OFF>;
}

template <bool HR, bool OFF>
GemvKernel select_kernel_hr(int pi, int xi) {
  static const GemvKernel table[kNumPass][3] = {
      {kernel_at<0, 0, HR, OFF>(), kernel_at<0, 1, HR, OFF>(), kernel_at<0, 2, HR, OFF>()},
      {kernel_at<1, 0, HR, OFF>(), kernel_at<1, 1, HR, OFF>(), kernel_at<1, 2, HR, OFF>()},
      {kernel_at<2, 0, HR, OFF>(), kernel_at<2, 1, HR, OFF>(), kernel_at<2, 2, HR, OFF>()},
      {kernel_at<3, 0, HR, OFF>(), kernel_at<3, 1, HR, OFF>(), kernel_at<3, 2, HR, OFF>()},
      {kernel_at<4, 0, HR, OFF>(), kernel_at<4, 1, HR, OFF>(), kernel_at<4, 2, HR, OFF>()},
      {kernel_at<5, 0, HR, OFF>(), kernel_at<5, 1, HR, OFF>(), kernel_at<5, 2, HR, OFF>()},
  };
  return table[pi][xi];
}

struct DeviceInfo {
  int cus = 0;
  bool attr_set[2][2][kNumPass][3] = {};
};

DeviceInfo& device_info() {
  static thread_local DeviceInfo info[64];
  int dev = 0;
  (void)hipGetDevice(&dev);
  return info[dev & 63];
}

// LDS bytes of one workgroup: table, x, wave sums of every row, two values
// per record.
size_t lds_bytes(int G, int rows) {
  const int SP = padded_slots(2 * G);
  const int segs = SP > 64 ? SP / 64 : 1;
  return (size_t)kLutBytes + 4 * (size_t)kXStrideDw * G + 4 * (size_t)((rows * segs + 1) & ~1) + 8 * (size_t)rows * G;
}

}  // namespace

hipError_t launch_gemv(const MatDev* ms, void* const* ys, int n, const uint16_t* x, bool out_f32,
                       hipStream_t s) {
  DeviceInfo& di = device_info();
  if (di.cus == 0) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&di.cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
  }

  const int G = ms[0].n_groups;
  const int S = 2 * G;
  const int SP = padded_slots(S);
  // Launch shape: one workgroup per CU (the 64 KiB table leaves no room for
  // two), T threads (a multiple of SP and of 64, at least 256) and passes
  // per lane.  Chosen from measurements on MI355X: first one round of
  // workgroups, then the fewest rows per workgroup (the most CUs busy), then
  // the least of waves + 4 * passes (a wave's serial pass chain costs about
  // four times its share of the set-up).
  int T = 0, pi = -1;
  int64_t best_rounds = 0;
  int best_rows = 0, best_score = 0;
  for (int t = 256; t <= kMaxThreads; t += 64) {
    if (t % SP != 0 || (G * kGroup / 8 + t - 1) / t > kXChoices[2]) continue;
    const int r = t / SP;
    for (int p = 0; p < kNumPass; ++p) {
      const int rows = kPassChoices[p] * r;
      if (lds_bytes(G, rows) > 160 * 1024 || rows > t) break;   // one thread per row at the end
      int64_t nwg = 0;
      for (int i = 0; i < n; ++i) nwg += (ms[i].n_out + rows - 1) / rows;
      const int64_t rounds = (nwg + di.cus - 1) / di.cus;
      const int score = t / 64 + 4 * kPassChoices[p];
      if (pi < 0 || rounds < best_rounds ||
          (rounds == best_rounds && (rows < best_rows || (rows == best_rows && score < best_score)))) {
        T = t;
        pi = p;
        best_rounds = rounds;
        best_rows = rows;
        best_score = score;
      }
    }
  }
  if (pi < 0) return hipErrorInvalidValue;
  const int ri = T / SP;
  const int passes = kPassChoices[pi];
  const int rows_per_wg = passes * ri;

  GemvArgs A = {};
  int32_t wb[TQ_MAX_GROUPED];
  int wg = 0;
  for (int i = 0; i < TQ_MAX_GROUPED; ++i) {
    wb[i] = INT32_MAX;
    if (i >= n) continue;
    GemvMat& a = A.m[i];
    a.codes0 = ms[i].codes0;
    a.scale0 = ms[i].scale0;
    a.rowptr1 = ms[i].rowptr1;
    a.gidx1 = ms[i].gidx1;
    a.codes1 = ms[i].codes1;
    a.offset1 = ms[i].offset1;
    a.scale1 = ms[i].scale1;
    a.offset0 = ms[i].offset0;
    a.y = ys[i];
    a.n_out = ms[i].n_out;
    a.nnz1 = (int32_t)ms[i].nnz1;
    a.wg_begin = wg;
    wb[i] = wg;
    wg += (ms[i].n_out + rows_per_wg - 1) / rows_per_wg;
  }

  // Record ranges from the host copies of the row pointers, when every
  // matrix with records has one and the table fits.
  bool host_ranges = wg + n <= kMaxRangeEntries;
  for (int i = 0; i < n && host_ranges; ++i)
    if (ms[i].nnz1 > 0 && ms[i].rowptr1_host == nullptr) host_ranges = false;
  if (host_ranges) {
    for (int i = 0; i < n; ++i) {
      const int nwg = (ms[i].n_out + rows_per_wg - 1) / rows_per_wg;
      int32_t* t = A.rec_begin + A.m[i].wg_begin + i;
      const int64_t nnz = ms[i].nnz1;
      for (int j = 0; j <= nwg; ++j) {
        int64_t v = 0;
        if (nnz > 0) {
          const int64_t r = (int64_t)j * rows_per_wg < ms[i].n_out ? (int64_t)j * rows_per_wg : ms[i].n_out;
          v = ms[i].rowptr1_host[r];
          v = v < 0 ? 0 : (v > nnz ? nnz : v);   // in bounds whatever the host copy holds
        }
        t[j] = (int32_t)v;
      }
    }
  }

  // Record waves: with host ranges the largest record count of any
  // workgroup is known, and extra waves (up to the 1024-thread limit) take
  // the records while the others run plane 0, instead of the plane-0 waves
  // taking them afterwards.  Used when they need at most kMaxRecSweeps
  // sweeps.
  int rec_threads = 0;
  if (host_ranges) {
    int maxrec = 0;
    for (int i = 0; i < n; ++i) {
      const int nwg = (ms[i].n_out + rows_per_wg - 1) / rows_per_wg;
      const int32_t* t = A.rec_begin + A.m[i].wg_begin + i;
      for (int j = 0; j < nwg; ++j) maxrec = t[j + 1] - t[j] > maxrec ? t[j + 1] - t[j] : maxrec;
    }
    const int want = (2 * maxrec + 63) / 64 * 64;
    const int room = kMaxThreads - T;
    if (want > 0 && room > 0 && (want + room - 1) / room <= kMaxRecSweeps) rec_threads = want < room ? want : room;
  }
  const int Tt = T + rec_threads;
  const int xloads = (G * kGroup / 8 + Tt - 1) / Tt;
  const int xi = xloads <= 1 ? 0 : (xloads <= 2 ? 1 : 2);
  if (kXChoices[xi] < xloads) return hipErrorInvalidValue;
  const int opts = (out_f32 ? 1 : 0) | (rec_threads > 0 ? T << 16 : 0);

  const int hr = host_ranges ? 1 : 0;
  bool any_off = false;
  for (int i = 0; i < n; ++i) any_off = any_off || ms[i].offset0 != nullptr;
  const int oi = any_off ? 1 : 0;
  GemvKernel kern;
  if (host_ranges)
    kern = any_off ? select_kernel_hr<true, true>(pi, xi) : select_kernel_hr<true, false>(pi, xi);
  else
    kern = any_off ? select_kernel_hr<false, true>(pi, xi) : select_kernel_hr<false, false>(pi, xi);
  if (!di.attr_set[hr][oi][pi][xi]) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024 - kLutBytes);
    if (e != hipSuccess) return e;
    di.attr_set[hr][oi][pi][xi] = true;
  }
  hipLaunchKernelGGL(kern, dim3(wg), dim3(Tt), lds_bytes(G, rows_per_wg) - kLutBytes, s, x, G, ri, rows_per_wg,
                     opts, wb[1], wb[2], wb[3], wb[4], wb[5], wb[6], wb[7], Tt, A);
  return hipGetLastError();
}

namespace {

typedef void (*BatchKernel)(const uint16_t*, int32_t, int32_t, int32_t, int32_t, int32_t, int32_t, const GemvArgs);

template <int PI, int XI, bool OFF, int B>
constexpr BatchKernel batch_kernel_at() {
  return gemv_batch_kernel<kPassChoices[PI], kXChoices[XI], OFF, B>;
}

template <bool OFF, int B>
BatchKernel select_batch(int pi, int xi) {
  static const BatchKernel table[kNumPass][3] = {
      {batch_kernel_at<0, 0, OFF, B>(), batch_kernel_at<0, 1, OFF, B>(), batch_kernel_at<0, 2, OFF, B>()},
      {batch_kernel_at<1, 0, OFF, B>(), batch_kernel_at<1, 1, OFF, B>(), batch_kernel_at<1, 2, OFF, B>()},
      {batch_kernel_at<2, 0, OFF, B>(), batch_kernel_at<2, 1, OFF, B>(), batch_kernel_at<2, 2, OFF, B>()},
      {batch_kernel_at<3, 0, OFF, B>(), batch_kernel_at<3, 1, OFF, B>(), batch_kernel_at<3, 2, OFF, B>()},
      {batch_kernel_at<4, 0, OFF, B>(), batch_kernel_at<4, 1, OFF, B>(), batch_kernel_at<4, 2, OFF, B>()},
      {batch_kernel_at<5, 0, OFF, B>(), batch_kernel_at<5, 1, OFF, B>(), batch_kernel_at<5, 2, OFF, B>()},
  };
  return table[pi][xi];
}

struct BatchDeviceInfo {
  int cus = 0;
  bool attr_set[2][3][kNumPass][3] = {};
};

BatchDeviceInfo& batch_device_info() {
  static thread_local BatchDeviceInfo info[64];
  int dev = 0;
  (void)hipGetDevice(&dev);
  return info[dev & 63];
}

size_t batch_lds_bytes(int G, int B, int rows, int rec_slots) {
  const int SP = padded_slots(2 * G);
  const int segs = SP > 64 ? SP / 64 : 1;
  return (size_t)kLutBytes + 4 * (size_t)kXStrideDw * G * B + 4 * (size_t)((rows * segs * B + 1) & ~1) +
         8 * (size_t)B * rec_slots;
}

}  // namespace

bool gemv_batch_supported(const MatDev& m, int B) {
  return B >= 2 && B <= 4 && (m.nnz1 == 0 || m.rowptr1_host != nullptr);
}

hipError_t launch_gemv_batch(const MatDev& m, const uint16_t* X, int B, void* Y, bool out_f32, hipStream_t s) {
  if (!gemv_batch_supported(m, B)) return hipErrorNotSupported;
  BatchDeviceInfo& di = batch_device_info();
  if (di.cus == 0) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&di.cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
  }
  const int G = m.n_groups;
  const int SP = padded_slots(2 * G);
  const int tmax = B <= 2 ? 1024 : 512;
  // Records per workgroup for a given row count, from the host row pointers.
  auto max_records = [&](int rows) -> int {
    if (m.nnz1 == 0) return 0;
    int best = 0;
    for (int64_t r = 0; r < m.n_out; r += rows) {
      const int64_t e = r + rows < m.n_out ? r + rows : m.n_out;
      const int64_t c = (int64_t)m.rowptr1_host[e] - m.rowptr1_host[r];
      best = c > best ? (int)c : best;
    }
    return best;
  };
  // The GEMV's launch policy (one round of workgroups, then the fewest rows,
  // then the fewest waves + 4 * passes), within this kernel's LDS.
  int T = 0, pi = -1, rec_slots = 0;
  int64_t best_rounds = 0;
  int best_rows = 0, best_score = 0;
  for (int t = 256; t <= tmax; t += 64) {
    if (t % SP != 0 || (G * kGroup / 8 + t - 1) / t > kXChoices[2]) continue;
    const int r = t / SP;
    for (int p = 0; p < kNumPass; ++p) {
      const int rows = kPassChoices[p] * r;
      if (rows > t) break;
      const int64_t nwg = (m.n_out + rows - 1) / rows;
      if (nwg + 1 > kMaxRangeEntries) continue;
      const int mr = max_records(rows);
      if (batch_lds_bytes(G, B, rows, mr > 0 ? mr : 1) > 160 * 1024) break;
      const int64_t rounds = (nwg + di.cus - 1) / di.cus;
      const int score = t / 64 + 4 * kPassChoices[p];
      if (pi < 0 || rounds < best_rounds ||
          (rounds == best_rounds && (rows < best_rows || (rows == best_rows && score < best_score)))) {
        T = t;
        pi = p;
        rec_slots = mr > 0 ? mr : 1;
        best_rounds = rounds;
        best_rows = rows;
        best_score = score;
      }
    }
  }
  // Staged rows of x that do not fit beside the table (down, K = 12288, at
  // B = 4): the MFMA kernel takes the batch in one launch (16 us there,
  // against 20 us for two launches of two rows here).
  if (pi < 0) return hipErrorNotSupported;
  const int ri = T / SP;
  const int rows_per_wg = kPassChoices[pi] * ri;
  const int xloads = (G * kGroup / 8 + T - 1) / T;
  const int xi = xloads <= 1 ? 0 : (xloads <= 2 ? 1 : 2);
  const int nwg = (int)((m.n_out + rows_per_wg - 1) / rows_per_wg);

  GemvArgs A = {};
  GemvMat& a = A.m[0];
  a.codes0 = m.codes0;
  a.scale0 = m.scale0;
  a.rowptr1 = m.rowptr1;
  a.gidx1 = m.gidx1;
  a.codes1 = m.codes1;
  a.offset1 = m.offset1;
  a.scale1 = m.scale1;
  a.offset0 = m.offset0;
  a.y = Y;
  a.n_out = m.n_out;
  a.nnz1 = (int32_t)m.nnz1;
  a.wg_begin = 0;
  for (int j = 0; j <= nwg; ++j) {
    int64_t v = 0;
    if (m.nnz1 > 0) {
      const int64_t r = (int64_t)j * rows_per_wg < m.n_out ? (int64_t)j * rows_per_wg : m.n_out;
      v = m.rowptr1_host[r];
      v = v < 0 ? 0 : (v > m.nnz1 ? m.nnz1 : v);
    }
    A.rec_begin[j] = (int32_t)v;
  }
  const bool off = m.offset0 != nullptr;
  BatchKernel kern;
  if (B == 2) kern = off ? select_batch<true, 2>(pi, xi) : select_batch<false, 2>(pi, xi);
  else if (B == 3) kern = off ? select_batch<true, 3>(pi, xi) : select_batch<false, 3>(pi, xi);
  else kern = off ? select_batch<true, 4>(pi, xi) : select_batch<false, 4>(pi, xi);
  bool& set = di.attr_set[off ? 1 : 0][B - 2][pi][xi];
  if (!set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024 - kLutBytes);
    if (e != hipSuccess) return e;
    set = true;
  }
  hipLaunchKernelGGL(kern, dim3(nwg), dim3(T), batch_lds_bytes(G, B, rows_per_wg, rec_slots) - kLutBytes, s, X, G,
                     ri, rows_per_wg, out_f32 ? 1 : 0, rec_slots, T, A);
  return hipGetLastError();
}

}  // namespace tq
