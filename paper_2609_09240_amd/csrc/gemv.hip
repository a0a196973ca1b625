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
//   tail byte 24+h (inputs 120+5h ..).  A workgroup of T threads covers
//   RI = T / S rows per pass and thread t always owns half-group t % S, so its
//   activations stay in 39 VGPRs for the whole launch, laid out per code byte
//   j as the fp16 pairs (x5j, x5j+1), (x5j+2, x5j+3), (x5j+4, 0).
// * Decode.  A 256-entry table maps a code to the same three pairs of fp16
//   patterns (+1 = 0x3C00, -1 = 0xBC00, 0 = 0); three v_dot2_f32_f16 then
//   accumulate the sign-selected activations in fp32.  The table is
//   replicated kRep times in LDS (copy q of code c at byte 16 (kRep c + q)); a
//   lane reads copy lane % kRep, so lanes served in the same LDS cycle hit
//   different bank quads whatever codes they hold.  With kRep = 16 the table
//   address (c << 8) | 16 q is one v_perm_b32 of the code dword.
// * Loads.  Per pass a lane loads 12 body bytes (three dwords, 4-aligned in
//   the split layout), its tail byte and its group's scale; lanes of a row
//   read consecutive bytes, so every wave load is contiguous.  Loads run
//   kDepth passes ahead of the decode (register ring), and each thread's
//   first plane-1 record is loaded before the workgroup's set-up, so HBM
//   latency overlaps the set-up and the plane-0 pass.
// * Plane 1.  After the plane-0 pass over a block of rows has written
//   s0 * p0 for every (row, half-group) into LDS, the block's records are
//   processed densely (one per thread) and each adds
//   mu * sum(x_g) + s1 * sum(t1 * x_g) to its (row, group) slot.
// * Reduction.  Each row's S partials are summed by one thread in a fixed
//   order (four accumulators over 16-byte LDS reads; the partial rows are
//   padded so consecutive threads hit different bank quads).  The two halves
//   of a group exchange their activation sums with a DPP quad permute.  No
//   atomics: results are bit-identical run to run.

#include "tq_internal.h"

#ifndef TQ_GEMV_REP
#define TQ_GEMV_REP 4
#endif
#ifndef TQ_GEMV_EARLY
#define TQ_GEMV_EARLY 8
#endif

namespace tq {
namespace {

constexpr int kRep = TQ_GEMV_REP;              // LUT copies
constexpr int kLutBytes = 256 * kRep * 16;
// Plane-0 passes issued before the set-up wait; the rest follow the
// workgroup barrier, so that x and the CSR slice do not queue behind them.
constexpr int kEarlyMax = TQ_GEMV_EARLY;
constexpr int kMaxThreads = 1024;
constexpr int kHalfBytes = 12;                 // body bytes per half-group
constexpr int kLaneBytes = kHalfBytes + 1;     // + one tail byte
// x in LDS: group g at dword 65 g (130 halves).  The odd dword stride puts
// the 64 lanes of a wave (32 groups x 2 halves) on different banks when they
// read their activations.
constexpr int kXStrideDw = 65;

static_assert(kRep == 1 || kRep == 2 || kRep == 4 || kRep == 8 || kRep == 16, "kRep");

// ---------------------------------------------------------------- table
__device__ inline uint32_t trit_pattern(int t) { return t > 0 ? 0x3C00u : (t < 0 ? 0xBC00u : 0u); }

// Table entry of code c: fp16 patterns of (t0, t1), (t2, t3), (t4, 0);
// codes 243..255 map to zeros.  Computed in registers (no memory access).
__device__ inline uint4 lut_entry(int c) {
  uint32_t t[5];
  int d = c;
#pragma unroll
  for (int i = 0; i < 5; ++i) {
    t[i] = c < 243 ? trit_pattern(d % 3 - 1) : 0u;
    d /= 3;
  }
  return uint4{t[0] | (t[1] << 16), t[2] | (t[3] << 16), t[4], 0u};
}

// Row stride of the LDS partials in floats: at least S, a multiple of 4
// (16-byte rows), and an odd number of 16-byte slots so that the one-thread-
// per-row final sum reads different bank quads from consecutive rows.
__host__ __device__ inline int part_stride(int S) {
  int ps = ((S + 3) & ~3) + 4;
  if (((ps >> 2) & 1) == 0) ps += 4;
  return ps;
}

// ---------------------------------------------------------------- params
// Per-matrix launch record.  The kernel reads the one its workgroup serves
// straight from the kernel-argument segment (one scalar memory round trip);
// everything needed to find it is in the leading scalar arguments, which the
// build asks the hardware to preload into SGPRs.
struct GemvMat {
  const uint8_t* codes0;
  const uint16_t* scale0;
  const int32_t* rowptr1;
  const uint16_t* gidx1;
  const uint8_t* codes1;
  const uint16_t* offset1;
  const uint16_t* scale1;
  void* y;
  int32_t n_out;
  int32_t nnz1;       // < 2^31: the host caps code buffers at 2^32 bytes
  int32_t wg_begin;   // first workgroup of this matrix
  int32_t pad;
};
struct GemvMats {
  GemvMat m[TQ_MAX_GROUPED];
};

struct __attribute__((aligned(16))) U3 {
  uint32_t x, y, z;
};

__device__ inline float fdot2(uint32_t a, uint32_t b, float c) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, a), __builtin_bit_cast(h2, b), c, false);
}

__device__ inline float h2f(uint32_t b) { return (float)__builtin_bit_cast(_Float16, (uint16_t)b); }


// LDS byte address of this lane's table copy for byte B of dword w.
template <int B>
__device__ inline uint32_t lut_addr(uint32_t w, uint32_t slot) {
  if constexpr (kRep == 16) {
    // bytes [slot, code, 0, 0]: selector 4 picks byte 0 of `slot`, B byte B of w.
    return __builtin_amdgcn_perm(slot, w, 0x0C0C0004u | (B << 8));
  } else {
    constexpr int sh = 4 + (kRep == 8 ? 3 : kRep == 4 ? 2 : kRep == 2 ? 1 : 0);
    return (((w >> (8 * B)) & 0xFFu) << sh) | slot;
  }
}

// Dot product of NB code bytes (byte j in byte j % 4 of w[j / 4]) with the
// activation pairs xp(j, q).
template <int NB, typename W, typename XP>
__device__ __attribute__((always_inline)) inline float code_dot(const unsigned char* lut, uint32_t slot,
                                                                const W& w, XP xp) {
  float a0 = 0.f, a1 = 0.f, a2 = 0.f;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    uint32_t addr;
    switch (j & 3) {
      case 0: addr = lut_addr<0>(w[j >> 2], slot); break;
      case 1: addr = lut_addr<1>(w[j >> 2], slot); break;
      case 2: addr = lut_addr<2>(w[j >> 2], slot); break;
      default: addr = lut_addr<3>(w[j >> 2], slot); break;
    }
    const U3 p = *reinterpret_cast<const U3*>(lut + addr);
    a0 = fdot2(p.x, xp(j, 0), a0);
    a1 = fdot2(p.y, xp(j, 1), a1);
    a2 = fdot2(p.z, xp(j, 2), a2);
  }
  return (a0 + a1) + a2;
}

// One pass of plane 0 for one lane: 12 body bytes, 1 tail byte, 1 scale.
struct Pass {
  uint32_t w[4];   // w[0..2] body, w[3] tail byte
  uint32_t sc;     // scale bits
};

// Byte offsets fit in 32 bits (the host rejects larger code buffers), so
// every address is a 64-bit base plus a zero-extended 32-bit offset.
__device__ inline void load_pass(Pass& p, const uint8_t* body0, const uint8_t* tail0, const uint16_t* scale0,
                                 uint32_t f) {
  const uint32_t* b = reinterpret_cast<const uint32_t*>(body0 + (size_t)(kMainBytes * f));
  p.w[0] = __builtin_nontemporal_load(b);
  p.w[1] = __builtin_nontemporal_load(b + 1);
  p.w[2] = __builtin_nontemporal_load(b + 2);
  p.w[3] = __builtin_nontemporal_load(tail0 + (size_t)(2 * f));
  p.sc = __builtin_nontemporal_load(scale0 + (size_t)f);
}

// Half hh of a plane-1 record: 12 body bytes, its tail byte, and the
// record's group, offset and scale.
struct RecHalf {
  uint32_t w[4];   // w[0..2] body bytes 12 hh .., w[3] tail byte 24 + hh
  uint32_t g, mu, s1;
};

// Where a workgroup reads its records from.
struct RecSrc {
  const uint8_t* codes1;
  const uint16_t* gidx1;
  const uint16_t* offset1;
  const uint16_t* scale1;
  uint32_t nnz1;
};

__device__ inline void load_rec_half(RecHalf& r, const RecSrc& M, uint32_t k, int hh) {
  const uint32_t* b = reinterpret_cast<const uint32_t*>(M.codes1 + (size_t)(kMainBytes * k + kHalfBytes * hh));
  r.w[0] = b[0];
  r.w[1] = b[1];
  r.w[2] = b[2];
  r.w[3] = M.codes1[(size_t)(kMainBytes * M.nnz1 + 2 * k + hh)];
  r.g = M.gidx1[k];
  r.mu = M.offset1[k];
  r.s1 = M.scale1[k];
}

// Contribution of one record half: s1 * sum(t1 x) over the half, plus
// mu * sum(x_g) on half 0.  Activations come from LDS.
__device__ __attribute__((always_inline)) inline float record_half_value(const unsigned char* lut, uint32_t slot,
                                                                         const uint16_t* xs, const float* gsum,
                                                                         const RecHalf& r, int hh, int G) {
  const int gg = min((int)r.g, G - 1);
  const uint32_t* xd = reinterpret_cast<const uint32_t*>(xs) + kXStrideDw * gg + 30 * hh;   // inputs 60 hh ..
  const uint16_t* xt = xs + 2 * kXStrideDw * gg + 120 + 5 * hh;
  const float p1 = code_dot<kLaneBytes>(lut, slot, r.w, [&](int j, int q) -> uint32_t {
    if (j < kHalfBytes) {
      const int p = 5 * j + 2 * q;   // input offset within the half
      if ((p & 1) == 0) return q < 2 ? xd[p / 2] : (xd[p / 2] & 0xFFFFu);
      return q < 2 ? __builtin_amdgcn_alignbit(xd[(p + 1) / 2], xd[(p - 1) / 2], 16) : (xd[(p - 1) / 2] >> 16);
    }
    const int p = 2 * q;             // tail byte: inputs 120 + 5 hh + p
    const uint32_t a = 120 + 5 * hh + p < kGroup ? (uint32_t)xt[p] : 0u;
    const uint32_t b = (q < 2 && 121 + 5 * hh + p < kGroup) ? (uint32_t)xt[p + 1] : 0u;
    return a | (b << 16);
  });
  const float v = h2f(r.s1) * p1;
  return hh == 0 ? h2f(r.mu) * gsum[gg] + v : v;
}

// kPasses: plane-0 passes per lane, all loaded up front.  kXLoads: 16-byte
// loads of x per thread (ceil(K / 8 / T)).  Every global load of the
// preamble is unconditional (out-of-range lanes load a valid address and
// ignore it) and issued in the order the data is needed, so each wait is an
// exact vmcnt and one memory round trip covers the set-up while the plane-0
// bytes stream in behind it.
template <int kPasses, int kXLoads>
__global__ void __launch_bounds__(kMaxThreads) __attribute__((amdgpu_waves_per_eu(4)))
gemv_kernel(const uint16_t* __restrict__ x, int32_t G, int32_t ri, int32_t rows_per_wg, int32_t out_f32,
            int32_t wb1, int32_t wb2, int32_t wb3, int32_t wb4, int32_t wb5, int32_t wb6, int32_t wb7,
            int32_t nthreads, const GemvMats mats) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int S = 2 * G;
  const int K = G * kGroup;
  unsigned char* lut = smem;
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem + kLutBytes);
  uint32_t* xsw = reinterpret_cast<uint32_t*>(xs);
  float* gsum = reinterpret_cast<float*>(smem + kLutBytes + 4 * kXStrideDw * G);
  int* rp = reinterpret_cast<int*>(gsum + G);
  uint16_t* rowof = reinterpret_cast<uint16_t*>(rp + rows_per_wg + 1);   // record -> row in block
  const int rowof_cap = rows_per_wg * G;
  float* part = reinterpret_cast<float*>(
      (reinterpret_cast<uintptr_t>(rowof + rowof_cap) + 15) & ~static_cast<uintptr_t>(15));
  const int PS = part_stride(2 * G);

  const int tid = threadIdx.x;
  const int T = nthreads;   // == blockDim.x, without a load of the dispatch packet
  const int nw = T >> 6;

  // Which matrix this workgroup serves: the first workgroups of matrices
  // 1..7 arrive in SGPRs (unused ones are INT32_MAX), so the matrix record
  // is one scalar load away.
  const int w = blockIdx.x;
  const int sel = __builtin_amdgcn_readfirstlane((w >= wb1) + (w >= wb2) + (w >= wb3) + (w >= wb4) + (w >= wb5) +
                                                 (w >= wb6) + (w >= wb7));
  // The whole record in one batch of scalar loads and one wait (left to
  // itself the compiler fetches fields at their first use, one round trip
  // each).
  const GemvMat M = mats.m[sel];
  asm volatile("" ::"s"(M.codes0), "s"(M.scale0), "s"(M.rowptr1), "s"(M.gidx1), "s"(M.codes1), "s"(M.offset1),
               "s"(M.scale1), "s"(M.y), "s"(M.n_out), "s"(M.nnz1), "s"(M.wg_begin));
  __builtin_amdgcn_sched_barrier(0);
  void* const yp = M.y;
  const int row_begin = (w - M.wg_begin) * rows_per_wg;
  const int row_end = min(M.n_out, row_begin + rows_per_wg);
  const int nrb = row_end - row_begin;

  const bool active = tid < ri * S;
  const int sl = active ? tid % S : 0;   // half-group slot within the row
  const int g = sl >> 1;
  const int h = sl & 1;
  const int rl = active ? tid / S : 0;
  const uint32_t slot = (uint32_t)(tid & (kRep - 1)) << 4;
  const bool has_rec = M.nnz1 > 0;

  // 1. CSR slice and record range (loaded first: waiting for them waits for
  //    nothing else).  Without records, x stands in as a readable address.
  const int* rpp = has_rec ? M.rowptr1 + row_begin : reinterpret_cast<const int*>(x);
  const int rp_mine = rpp[has_rec ? min(tid, nrb) : 0];
  const int k0 = rpp[0];
  const int k1 = rpp[has_rec ? nrb : 0];
  // 2. x.
  uint4 xv[kXLoads];
#pragma unroll
  for (int q = 0; q < kXLoads; ++q) xv[q] = reinterpret_cast<const uint4*>(x)[min(tid + q * T, K / 8 - 1)];
  // Keep the issue order = the order of need: neither the optimiser nor the
  // scheduler may move loads across these points (no instruction emitted).
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  // 3. Every plane-0 pass of this lane.
  const uint32_t ngroups = (uint32_t)M.n_out * (uint32_t)G;
  const uint8_t* body0 = M.codes0 + kHalfBytes * h;
  const uint8_t* tail0 = M.codes0 + (size_t)(kMainBytes * ngroups) + h;
  constexpr int kEarly = kEarlyMax < kPasses ? kEarlyMax : kPasses;
  Pass buf[kPasses];
  auto issue_pass = [&](int d) {
    const int r = min(row_begin + rl + d * ri, row_end - 1);
    load_pass(buf[d], body0, tail0, M.scale0, (uint32_t)r * (uint32_t)G + (uint32_t)g);
  };
#pragma unroll
  for (int d = 0; d < kEarly; ++d) issue_pass(d);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  // 4. Record halves (two threads per record), spread across the waves:
  //    loaded here when few passes leave registers to spare, else after
  //    plane 0.
  constexpr bool kPreRec = kPasses <= 2;
  const int item = (tid & 63) * nw + (tid >> 6);
  const int hh = item & 1;
  const int kr = k0 + (item >> 1);
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
  const int k_last = min(max(k1 - 1, k0), kmax);
  if constexpr (kPreRec) load_rec_half(rec, MR, (uint32_t)max(min(kr, k_last), 0), has_rec ? hh : 0);

  // Set-up in LDS.
#pragma unroll
  for (int q = 0; q < kXLoads; ++q) {
    // 8 halves: group i / 16, dwords 4 (i % 16) ..  Unconditional (threads
    // past the end rewrite the last slot with the same data), so the load is
    // not sunk into a branch behind the weight loads.
    const int i = min(tid + q * T, K / 8 - 1);
    uint32_t* d = xsw + kXStrideDw * (i >> 4) + 4 * (i & 15);
    d[0] = xv[q].x;
    d[1] = xv[q].y;
    d[2] = xv[q].z;
    d[3] = xv[q].w;
  }
  if (tid < 256) {
    const uint4 e = lut_entry(tid);
#pragma unroll
    for (int q = 0; q < kRep; ++q) reinterpret_cast<uint4*>(lut)[tid * kRep + q] = e;
  }
  if (has_rec && tid <= nrb) rp[tid] = rp_mine;
  __syncthreads();
  if constexpr (kEarly < kPasses) {
    asm volatile("" ::: "memory");
#pragma unroll
    for (int d = kEarly; d < kPasses; ++d) issue_pass(d);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
  }

  // Row of every record of the block (replaces a search per record).
  if (has_rec && tid < nrb) {
    const int kb = max(rp[tid], k0), ke = min(rp[tid + 1], k1);
    for (int k = kb; k < ke && k - k0 < rowof_cap; ++k) rowof[k - k0] = (uint16_t)tid;
  }

  // This lane's activations: 12 body bytes (inputs 60h + 5j ..) and the tail
  // byte (inputs 120 + 5h ..), three fp16 pairs per byte.
  uint32_t xr[kLaneBytes][3];
  {
    const uint32_t* xd = xsw + kXStrideDw * g + 30 * h;   // inputs 60 h ..
#pragma unroll
    for (int j = 0; j < kHalfBytes; j += 2) {   // bytes j, j+1: inputs 5j .. 5j+9 = dwords 5j/2 ..
      const int q = 5 * j / 2;
      const uint32_t d0 = xd[q], d1 = xd[q + 1], d2 = xd[q + 2], d3 = xd[q + 3], d4 = xd[q + 4];
      xr[j][0] = d0;
      xr[j][1] = d1;
      xr[j][2] = d2 & 0xFFFFu;
      xr[j + 1][0] = __builtin_amdgcn_alignbit(d3, d2, 16);
      xr[j + 1][1] = __builtin_amdgcn_alignbit(d4, d3, 16);
      xr[j + 1][2] = d4 >> 16;
      __builtin_amdgcn_sched_barrier(0);
    }
    const uint16_t* xt = xs + 2 * kXStrideDw * g + 120 + 5 * h;
    uint32_t e[5];
#pragma unroll
    for (int i = 0; i < 5; ++i) e[i] = (120 + 5 * h + i < kGroup) ? (uint32_t)xt[i] : 0u;
    xr[kHalfBytes][0] = e[0] | (e[1] << 16);
    xr[kHalfBytes][1] = e[2] | (e[3] << 16);
    xr[kHalfBytes][2] = e[4];
  }
  // Group sums for the offsets: each lane sums its half, the pair combines
  // (half 0 first on both lanes, so both get the same bits).
  {
    float s0 = 0.f, s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int j = 0; j < kLaneBytes; ++j) {
      s0 = fdot2(xr[j][0], 0x3C003C00u, s0);
      s1 = fdot2(xr[j][1], 0x3C003C00u, s1);
      s2 = fdot2(xr[j][2], 0x3C003C00u, s2);
    }
    const float s = (s0 + s1) + s2;
    const float other = __builtin_bit_cast(   // lane ^ 1 (quad_perm 1,0,3,2)
        float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, s), 0xB1, 0xF, 0xF, false));
    const float tot = h == 0 ? s + other : other + s;
    if (active && rl == 0 && h == 0) gsum[g] = tot;
  }

  // Plane 0: part[row][slot] = s0 * sum_i t0 x over the half-group.
#pragma unroll
  for (int d = 0; d < kPasses; ++d) {
    const float p = code_dot<kLaneBytes>(lut, slot, buf[d].w, [&](int j, int q) { return xr[j][q]; });
    if (active && rl + d * ri < nrb) part[(rl + d * ri) * PS + sl] = p * h2f(buf[d].sc);
    __builtin_amdgcn_sched_barrier(0);   // keep passes apart: bounds the LUT reads in flight
  }
  // Plane-0 passes beyond kPasses (only when the host could not fit a
  // matrix into one round of workgroups with kPasses passes).
  for (int d = kPasses; active && rl + d * ri < nrb; ++d) {
    Pass q;
    load_pass(q, body0, tail0, M.scale0, (uint32_t)(row_begin + rl + d * ri) * (uint32_t)G + (uint32_t)g);
    const float p = code_dot<kLaneBytes>(lut, slot, q.w, [&](int j, int qq) { return xr[j][qq]; });
    part[(rl + d * ri) * PS + sl] = p * h2f(q.sc);
  }

  // Plane 1: each record half adds to its (row, half-group) slot.
  if (has_rec) {
    __syncthreads();   // plane-0 partials and group sums are in LDS
    const int per_sweep = T >> 1;
    for (int k = kr, first = 1; k < k1; k += per_sweep, first = 0) {
      if (!kPreRec || !first) load_rec_half(rec, MR, (uint32_t)min(max(k, 0), kmax), hh);
      if (k < 0 || k - k0 >= rowof_cap) continue;
      const int lo = min((int)rowof[k - k0], nrb - 1);
      const float v = record_half_value(lut, slot, xs, gsum, rec, hh, G);
      float* dst = part + lo * PS + 2 * min((int)rec.g, G - 1) + hh;
      *dst = *dst + v;
    }
  }
  __syncthreads();

  // Row sums: one thread per row, four independent accumulators over the
  // row's partials in a fixed order.
  for (int rr = tid; rr < nrb; rr += T) {
    const float4* pr = reinterpret_cast<const float4*>(part + rr * PS);
    float4 a = {0.f, 0.f, 0.f, 0.f};
    const int n4 = S >> 2;
    for (int c = 0; c < n4; ++c) {
      const float4 v = pr[c];
      a.x += v.x;
      a.y += v.y;
      a.z += v.z;
      a.w += v.w;
    }
    if (S & 2) {   // S = 2G is even: at most two trailing partials
      a.x += part[rr * PS + 4 * n4];
      a.y += part[rr * PS + 4 * n4 + 1];
    }
    const float sum = (a.x + a.y) + (a.z + a.w);
    if (out_f32)
      reinterpret_cast<float*>(yp)[row_begin + rr] = sum;
    else
      reinterpret_cast<uint16_t*>(yp)[row_begin + rr] = __builtin_bit_cast(uint16_t, (_Float16)sum);
  }
}

typedef void (*GemvKernel)(const uint16_t*, int32_t, int32_t, int32_t, int32_t, int32_t, int32_t, int32_t, int32_t,
                           int32_t, int32_t, int32_t, int32_t, const GemvMats);

constexpr int kPassChoices[] = {1, 2, 3, 4, 6, 8};
constexpr int kNumPass = 6;
constexpr int kXChoices[] = {1, 2, 4};

template <int PI, int XI>
constexpr GemvKernel kernel_at() {
  return gemv_kernel<kPassChoices[PI], kXChoices[XI]>;
}

GemvKernel select_kernel(int pi, int xi) {
  static const GemvKernel table[kNumPass][3] = {
      {kernel_at<0, 0>(), kernel_at<0, 1>(), kernel_at<0, 2>()},
      {kernel_at<1, 0>(), kernel_at<1, 1>(), kernel_at<1, 2>()},
      {kernel_at<2, 0>(), kernel_at<2, 1>(), kernel_at<2, 2>()},
      {kernel_at<3, 0>(), kernel_at<3, 1>(), kernel_at<3, 2>()},
      {kernel_at<4, 0>(), kernel_at<4, 1>(), kernel_at<4, 2>()},
      {kernel_at<5, 0>(), kernel_at<5, 1>(), kernel_at<5, 2>()},
  };
  return table[pi][xi];
}

struct DeviceInfo {
  int cus = 0;
  bool attr_set[kNumPass][3] = {};
};

DeviceInfo& device_info() {
  static thread_local DeviceInfo info[64];
  int dev = 0;
  (void)hipGetDevice(&dev);
  return info[dev & 63];
}

size_t lds_bytes(int G, int rb_max) {
  const size_t head = (size_t)kLutBytes + 4 * (size_t)kXStrideDw * G + 4 * (size_t)G + 4 * (size_t)(rb_max + 1) +
                      2 * (size_t)rb_max * G;
  return ((head + 15) & ~(size_t)15) + 4 * (size_t)rb_max * part_stride(2 * G);
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
  int64_t total_rows = 0;
  for (int i = 0; i < n; ++i) total_rows += ms[i].n_out;

  // LDS: table + x + group sums + CSR slice + partials.  Two workgroups per
  // CU when they fit in half of the 160 KiB (then at most 512 threads each,
  // 16 waves per CU in all); otherwise one of up to 1024 threads.
  const size_t fixed = lds_bytes(G, 0) + 16;   // + alignment of the partials
  const size_t per_row = 4 * (size_t)part_stride(S) + 2 * (size_t)G + 4;
  const size_t half_lds = 80 * 1024, full_lds = 160 * 1024;
  const int ri512 = 512 / S;
  const int wgs_per_cu = (ri512 >= 1 && fixed + per_row * ri512 <= half_lds) ? 2 : 1;
  const size_t budget = wgs_per_cu == 2 ? half_lds : full_lds;
  const int t_max = wgs_per_cu == 2 ? 512 : kMaxThreads;

  // Threads per workgroup: the multiple of 64 in [256, t_max] leaving the
  // fewest lanes without a half-group; the larger wins ties.
  int T = 0;
  double best = -1.0;
  for (int t = 256; t <= t_max; t += 64) {
    const double used = (double)((t / S) * S) / t;
    if (used >= best - 1e-9) {
      best = used;
      T = t;
    }
  }
  const int ri = T / S;

  // Passes per lane: enough for one round of workgroups, capped by the
  // compiled choices, by LDS for the partials and by one CSR entry per thread.
  int max_rows = (int)((budget - fixed) / per_row);
  if (max_rows > T - 1) max_rows = T - 1;
  const int max_pass = max_rows / ri < 1 ? 1 : max_rows / ri;
  const int64_t target_wgs = (int64_t)di.cus * wgs_per_cu;
  int want = (int)((total_rows + target_wgs * ri - 1) / (target_wgs * ri));
  if (want > max_pass) want = max_pass;
  int pi = 0;
  while (pi < kNumPass - 1 && kPassChoices[pi] < want) ++pi;
  int passes = kPassChoices[pi];
  if (passes > max_pass) {   // largest compiled choice that fits
    while (pi > 0 && kPassChoices[pi] > max_pass) --pi;
    passes = kPassChoices[pi];
  }
  const int rows_per_wg = passes * ri;
  const int xloads = (G * kGroup / 8 + T - 1) / T;
  const int xi = xloads <= 1 ? 0 : (xloads <= 2 ? 1 : 2);
  if (kXChoices[xi] < xloads) return hipErrorInvalidValue;

  const GemvKernel kern = select_kernel(pi, xi);
  if (!di.attr_set[pi][xi]) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    di.attr_set[pi][xi] = true;
  }

  GemvMats A = {};
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
    a.y = ys[i];
    a.n_out = ms[i].n_out;
    a.nnz1 = (int32_t)ms[i].nnz1;
    a.wg_begin = wg;
    wb[i] = wg;
    wg += (ms[i].n_out + rows_per_wg - 1) / rows_per_wg;
  }
  hipLaunchKernelGGL(kern, dim3(wg), dim3(T), lds_bytes(G, rows_per_wg), s, x, G, ri, rows_per_wg,
                     out_f32 ? 1 : 0, wb[1], wb[2], wb[3], wb[4], wb[5], wb[6], wb[7], T, A);
  return hipGetLastError();
}

}  // namespace tq
