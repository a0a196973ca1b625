// Small-batch packed GEMM Y = X W^T with MFMA (gfx950).
//
// Paper: section 3, eq. 3 (the weight), section 18 (kernel work across
// shapes and batch sizes is the stated next step).  For a batch of B
// activation rows the product is a dense contraction, so it runs on
// v_mfma_f32_16x16x32_f16: A = 16 weight rows, B = 16 batch rows, C = the
// 16 x 16 block of Y^T.
//
// Slot order.  MFMA sums over k in any order.  Each group's 128 inputs are
// laid out as 28 code bytes (26 real, 2 pad) of 8 slots each: byte j owns
// slots 8j .. 8j+7 holding inputs 5j .. 5j+4 and three zeros, so one MFMA
// k-step (32 slots) covers bytes 4s .. 4s+3 and lane block q of the A
// operand decodes exactly one code byte (4s + q).  The B operand gathers the
// same five activations from X (one 12-byte load, a half-word shift for odd
// bytes) and zeros the pad slots, so the slot order never reaches memory.
//
// Decode.  A code byte maps through an LDS table to five v_perm selectors;
// v_perm then picks each weight's fp16 bits from {-s0, +0, +s0} (plane 0)
// or {mu - s1, mu, mu + s1} (plane 1, rounded to fp16 once per record), so a
// weight costs no arithmetic.  On two-plane groups the two halves are added
// in fp16 (one more rounding; the result stays within the accuracy bound).
//
// Staging.  A workgroup owns 16 RT consecutive weight rows.  Their packed
// bytes (one contiguous span per buffer), scales and plane-1 records are
// loaded in one burst of coalesced loads and written to LDS as one 32-byte
// slot per (group, row).  Waves then own (row tile, K quarter) pairs; when a
// workgroup has fewer row tiles than waves, K is split across waves and the
// partial sums are added in a fixed order through LDS (bit-reproducible).
// Shapes whose staging does not fit (more than kMaxPairs (row, group) pairs
// per row tile) use the simple per-group kernel at the end of this file.

#include "tq_internal.h"

namespace tq {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float float4v __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

constexpr int kLutCopies = 8;                       // table copies (lane & 7)
constexpr int kLutEntries = 256;
constexpr int kMaxPairs = 1536;                     // staged (row, group) pairs per workgroup
constexpr int kSlotBytes = 32;
constexpr int kStepsPerGroup = 7;                   // 28 code bytes / 4 per k-step
constexpr int kRecBatch = 2;                        // plane-1 records loaded per thread per batch
constexpr int kLdsLimit = 160 * 1024;
constexpr int kLutBytes = kLutEntries * kLutCopies * 16;

// Dynamic LDS bytes for P staged pairs and R rows.
__host__ __device__ constexpr int staged_bytes(int P, int R) {
  return P * (2 * kSlotBytes + 2 + 2 + 1) + 4 * (R + 1);
}

struct SbArgs {
  MatDev m;
  const uint16_t* X;
  void* Y;
  int B;
  int out_f32;
};

// v_perm selector of one weight: digit d (t = d - 1) picks fp16 half d of
// the source pair {lo: halves 0, 1; hi: half 2}.
__device__ constexpr uint32_t digit_selector(int d) { return (uint32_t)(2 * d) | ((uint32_t)(2 * d + 1) << 8); }

__device__ inline float h2f(uint32_t b) { return (float)__builtin_bit_cast(_Float16, (uint16_t)b); }
__device__ inline uint32_t f2h(float a) { return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)a); }

// Quotient and remainder of i / d for 0 <= i < 2^24, d >= 1 (float estimate,
// corrected by one step).
__device__ inline int divide(int i, int d, float inv, int& rem) {
  int q = (int)((float)i * inv);
  int r = i - q * d;
  if (r < 0) { --q; r += d; }
  if (r >= d) { ++q; r -= d; }
  rem = r;
  return q;
}

template <int RT, int KS, int CT>
__global__ void __launch_bounds__(64 * RT * KS) sb_kernel(SbArgs a) {
  constexpr int T = 64 * RT * KS;
  constexpr int R = 16 * RT;
  constexpr int kPieces = (3 * kMaxPairs + T - 1) / T;     // 8-byte code pieces per thread
  constexpr int kPairsPerThread = (kMaxPairs + T - 1) / T;
  constexpr int D = CT == 1 ? 4 : (CT == 2 ? 2 : 1);       // groups per X gather stage

  __shared__ uint4 lut[kLutEntries * kLutCopies];
  extern __shared__ uint4 dyn[];

  const MatDev& m = a.m;
  const int G = m.n_groups;
  const int P = G * R;
  uint8_t* sbase = reinterpret_cast<uint8_t*>(dyn);
  uint32_t* w_s = reinterpret_cast<uint32_t*>(sbase);                        // [P][8] plane 0
  uint32_t* r_s = reinterpret_cast<uint32_t*>(sbase + P * kSlotBytes);       // [P][8] plane 1
  int* rowptr_s = reinterpret_cast<int*>(sbase + 2 * P * kSlotBytes);        // [R + 1]
  uint16_t* s0_s = reinterpret_cast<uint16_t*>(rowptr_s + R + 1);            // [P]
  uint16_t* m0_s = s0_s + P;                                                 // [P] per-group offsets
  uint8_t* hr_s = reinterpret_cast<uint8_t*>(m0_s + P);                      // [P] record present
  // Per-group offsets are optional; without them the scales stand in as a
  // readable address and the staged values are unused.
  const bool has_off = m.offset0 != nullptr;
  const uint16_t* off_src = has_off ? m.offset0 : m.scale0;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int row0 = blockIdx.x * R;
  const int nrows = min(R, m.n_out - row0);
  const int np = nrows * G;                      // pairs of this workgroup, f - f0 = row * G + g
  const int64_t f0 = (int64_t)row0 * G;
  const int64_t ngroups = (int64_t)m.n_out * G;
  const float invG = 1.0f / (float)G;
  const float inv3G = 1.0f / (float)(3 * G);

  // ---- 1. Loads, all issued before any wait, every one unconditional at a
  // clamped (in-bounds) address: a load whose destination is also written on
  // another path would force a wait for it.  Row pointers first, so the
  // first LDS writes wait for them alone.
  int kb = 0, ke = 0, rp = 0;
  if (m.nnz1 > 0) {
    kb = m.rowptr1[row0];
    ke = m.rowptr1[row0 + nrows];
    rp = m.rowptr1[row0 + min(tid, nrows)];
  }
  const uint64_t* mainp = reinterpret_cast<const uint64_t*>(m.codes0 + 24 * f0);
  const uint16_t* tailp = reinterpret_cast<const uint16_t*>(m.codes0 + 24 * ngroups) + f0;
  uint64_t pc[kPieces];
  uint32_t tl[kPairsPerThread], sc[kPairsPerThread], mo[kPairsPerThread];
#pragma unroll
  for (int u = 0; u < kPieces; ++u) pc[u] = mainp[min(tid + u * T, 3 * np - 1)];
#pragma unroll
  for (int u = 0; u < kPairsPerThread; ++u) {
    const int i = min(tid + u * T, np - 1);
    tl[u] = tailp[i];
    sc[u] = m.scale0[f0 + i];
    mo[u] = off_src[f0 + i];
  }

  // ---- 2. Selector table (one entry per thread, written to every copy).
  for (int c = tid; c < kLutEntries; c += T) {
    uint32_t sel[5];
    int cc = c;
#pragma unroll
    for (int i = 0; i < 5; ++i) {
      const int q = (cc * 171) >> 9;    // cc / 3 for cc < 256
      sel[i] = c < 243 ? digit_selector(cc - 3 * q) : 0x0C0Cu;   // invalid codes read as zeros
      cc = q;
    }
    const uint4 e = make_uint4(sel[0] | (sel[1] << 16), sel[2] | (sel[3] << 16), sel[4] | (0x0C0Cu << 16), 0u);
    // Every copy is identical; the rotation spreads one store instruction's
    // lanes over the banks.
#pragma unroll
    for (int k = 0; k < kLutCopies; ++k) lut[c * kLutCopies + ((k + c) & (kLutCopies - 1))] = e;
  }

  // ---- 3. Plane-0 data to LDS: slot (g, row) = bytes 0..23, tail bytes,
  // two pad codes 121 (zero trits).
  if (m.nnz1 > 0 && tid <= nrows) rowptr_s[tid] = rp;
#pragma unroll
  for (int u = 0; u < kPieces; ++u) {
    const int i = tid + u * T;
    if (i < 3 * np) {
      int rem;
      const int row = divide(i, 3 * G, inv3G, rem);
      const int g = rem / 3, part = rem - 3 * (rem / 3);
      uint32_t* d = w_s + 8 * (g * R + row) + 2 * part;
      d[0] = (uint32_t)pc[u];
      d[1] = (uint32_t)(pc[u] >> 32);
    }
  }
#pragma unroll
  for (int u = 0; u < kPairsPerThread; ++u) {
    const int i = tid + u * T;
    if (i < np) {
      int g;
      const int row = divide(i, G, invG, g);
      const int p = g * R + row;
      w_s[8 * p + 6] = tl[u] | 0x79790000u;
      s0_s[p] = (uint16_t)sc[u];
      m0_s[p] = (uint16_t)mo[u];
    }
  }
  for (int p = tid; p < P; p += T) hr_s[p] = 0;
  __syncthreads();

  // ---- 4. Plane-1 records of the workgroup's rows (CSR range kb..ke).
  if (ke > kb) {
    const uint64_t* rmain = reinterpret_cast<const uint64_t*>(m.codes1);
    const uint16_t* rtail = reinterpret_cast<const uint16_t*>(m.codes1 + 24 * m.nnz1);
    for (int k0 = kb; k0 < ke; k0 += kRecBatch * T) {
      uint64_t rpc[kRecBatch][3];
      uint32_t rt[kRecBatch], rm[kRecBatch];
      int rg[kRecBatch];
#pragma unroll
      for (int u = 0; u < kRecBatch; ++u) {
        const int k = min(k0 + tid + u * T, ke - 1);
#pragma unroll
        for (int part = 0; part < 3; ++part) rpc[u][part] = rmain[3 * (int64_t)k + part];
        rt[u] = rtail[k];
        rm[u] = (uint32_t)m.offset1[k] | ((uint32_t)m.scale1[k] << 16);
        rg[u] = (int)m.gidx1[k];
      }
#pragma unroll
      for (int u = 0; u < kRecBatch; ++u) {
        const int k = k0 + tid + u * T;
        if (k < ke && rg[u] < G) {
          // Row of record k: the last r with rowptr_s[r] <= k.
          int lo = 0, hi = nrows;
          while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (rowptr_s[mid] <= k) lo = mid; else hi = mid;
          }
          const int p = rg[u] * R + lo;
          uint32_t* d = r_s + 8 * p;
#pragma unroll
          for (int part = 0; part < 3; ++part) {
            d[2 * part] = (uint32_t)rpc[u][part];
            d[2 * part + 1] = (uint32_t)(rpc[u][part] >> 32);
          }
          d[6] = rt[u] | 0x79790000u;
          d[7] = rm[u];
          hr_s[p] = 1;
        }
      }
    }
  }
  __syncthreads();

  // ---- 5. Main loop: this wave's row tile over its K range.
  const int rt = wave % RT;
  const int ks = wave / RT;
  const int gper = (G + KS - 1) / KS;
  const int gb = ks * gper;
  const int ge = min(G, gb + gper);
  const int row_l = 16 * rt + (lane & 15);       // A operand row of this lane
  const int q = lane >> 4;                        // k block of this lane
  const uint32_t qsh = 8u * q;
  const int n = lane & 15;                        // B operand batch column
  const uint32_t xsh = (q & 1) ? 2u : 0u;         // odd code bytes start one half later
  const int copy = lane & (kLutCopies - 1);

  float4v acc[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) acc[c] = float4v{0.f, 0.f, 0.f, 0.f};

  // Each workgroup walks its K range from a different starting group, so the
  // workgroups of a chip do not all read the same slice of X at the same
  // time.  The order is fixed per workgroup, so results stay reproducible.
  const int nG = ge - gb;
  const int rot = nG > 0 ? (int)(blockIdx.x % (unsigned)nG) : 0;
  auto group_at = [&](int t) {   // t-th group visited; past the range: G - 1 (read, never used)
    if (t >= nG) return G - 1;
    const int u = t + rot;
    return gb + (u >= nG ? u - nG : u);
  };

  // X gathers, in stages of D groups loaded one stage ahead (ping-pong
  // buffers, so each wait covers exactly the stage being consumed).  Loads
  // are unconditional: a batch column past B reads row B - 1 (its column of C
  // is never stored) and a group past the range reads group G - 1.  Byte 25
  // (inputs 125..127) is loaded from input 122 and realigned when consumed;
  // pad bytes 26, 27 are zeroed then.
  typedef uint32_t XStage[D][CT][kStepsPerGroup][3];
  auto gather = [&](XStage& dst, int t_first) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int g = group_at(t_first + d);
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const int b = min(16 * c + n, a.B - 1);
        const uint16_t* xrow = a.X + (int64_t)b * (G * kGroup) + kGroup * g;
#pragma unroll
        for (int s = 0; s < kStepsPerGroup; ++s) {
          const int j = 4 * s + q;                  // code byte of this lane
          const int off = s < kStepsPerGroup - 1 ? 5 * j - (j & 1) : (q == 1 ? 122 : 120);
          const uint32_t* p = reinterpret_cast<const uint32_t*>(xrow + off);
          dst[d][c][s][0] = p[0];
          dst[d][c][s][1] = p[1];
          dst[d][c][s][2] = p[2];
        }
      }
    }
  };

  // Staged weights of one (group, row) pair: plane-0 code words, scale,
  // record flag and the record slot (read whether or not it is used).
  struct Slot {
    uint4 w0, w1, r0, r1;
    uint32_t s0, m0, hr;
  };
  auto read_slot = [&](int g) {
    const int p = g * R + row_l;
    Slot v;
    v.w0 = *reinterpret_cast<const uint4*>(w_s + 8 * p);
    v.w1 = *reinterpret_cast<const uint4*>(w_s + 8 * p + 4);
    v.r0 = *reinterpret_cast<const uint4*>(r_s + 8 * p);
    v.r1 = *reinterpret_cast<const uint4*>(r_s + 8 * p + 4);
    v.s0 = s0_s[p];
    v.m0 = m0_s[p];
    v.hr = hr_s[p];
    return v;
  };

  // One group: table reads for all seven k-steps first, then the products.
  auto consume = [&](const uint32_t (&xg)[CT][kStepsPerGroup][3], const Slot& cur) {
    u4v xo[CT][kStepsPerGroup];
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int s = 0; s < kStepsPerGroup; ++s) {
        uint32_t l0 = xg[c][s][0], l1 = xg[c][s][1], l2 = xg[c][s][2];
        if (s == kStepsPerGroup - 1) {
          if (q == 1) { l0 = l1; l1 = l2; l2 = 0u; }       // inputs 125..127 from 122..127
          else if (q >= 2) { l0 = 0u; l1 = 0u; l2 = 0u; }  // pad bytes
        }
        xo[c][s] = u4v{__builtin_amdgcn_alignbyte(l1, l0, xsh), __builtin_amdgcn_alignbyte(l2, l1, xsh),
                       (l2 >> (8 * xsh)) & 0xFFFFu, 0u};
      }
    const uint32_t sw[kStepsPerGroup] = {cur.w0.x, cur.w0.y, cur.w0.z, cur.w0.w, cur.w1.x, cur.w1.y, cur.w1.z};
    uint4 e[kStepsPerGroup];
#pragma unroll
    for (int s = 0; s < kStepsPerGroup; ++s) e[s] = lut[((sw[s] >> qsh) & 0xFFu) * kLutCopies + copy];
    // Halves {-s0, +0, +s0}; with per-group offsets {mu0 - s0, mu0, mu0 + s0},
    // each rounded once from fp32 as in the dense dequantisation.
    uint32_t lo0 = cur.s0 ^ 0x8000u, hi0 = cur.s0;
    if (has_off) {
      const float m0 = 0.0f + h2f(cur.m0), s0 = h2f(cur.s0);
      lo0 = f2h(m0 - s0) | (f2h(m0) << 16);
      hi0 = f2h(m0 + s0);
    }
    uint32_t av[kStepsPerGroup][3];
#pragma unroll
    for (int s = 0; s < kStepsPerGroup; ++s) {
      av[s][0] = __builtin_amdgcn_perm(hi0, lo0, e[s].x);
      av[s][1] = __builtin_amdgcn_perm(hi0, lo0, e[s].y);
      av[s][2] = __builtin_amdgcn_perm(hi0, lo0, e[s].z);
    }
    const bool rec = cur.hr != 0;
    if (__ballot(rec) != 0) {
      // Plane 1 (lanes without a record add zeros): halves {mu - s1, mu, mu + s1}.
      const uint32_t ms = cur.r1.w;
      const float mu = h2f(ms & 0xFFFFu), s1 = h2f(ms >> 16);
      const uint32_t lo1 = rec ? (f2h(mu - s1) | ((ms & 0xFFFFu) << 16)) : 0u;
      const uint32_t hi1 = rec ? f2h(mu + s1) : 0u;
      const uint32_t rw[kStepsPerGroup] = {cur.r0.x, cur.r0.y, cur.r0.z, cur.r0.w, cur.r1.x, cur.r1.y, cur.r1.z};
      uint4 e1[kStepsPerGroup];
#pragma unroll
      for (int s = 0; s < kStepsPerGroup; ++s) e1[s] = lut[((rw[s] >> qsh) & 0xFFu) * kLutCopies + copy];
#pragma unroll
      for (int s = 0; s < kStepsPerGroup; ++s) {
        const uint32_t b1[3] = {__builtin_amdgcn_perm(hi1, lo1, e1[s].x), __builtin_amdgcn_perm(hi1, lo1, e1[s].y),
                                __builtin_amdgcn_perm(hi1, lo1, e1[s].z)};
#pragma unroll
        for (int i = 0; i < 3; ++i)
          av[s][i] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, av[s][i]) + __builtin_bit_cast(half2v, b1[i]));
      }
    }
#pragma unroll
    for (int s = 0; s < kStepsPerGroup; ++s) {
      const half8 A = __builtin_bit_cast(half8, u4v{av[s][0], av[s][1], av[s][2], 0u});
#pragma unroll
      for (int c = 0; c < CT; ++c)
        acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, __builtin_bit_cast(half8, xo[c][s]), acc[c], 0, 0, 0);
    }
  };

  XStage xa, xb;
  gather(xa, 0);
  Slot cur = read_slot(group_at(0));
  auto run_stage = [&](const XStage& xs, int t_first) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int t = t_first + d;
      const Slot nxt = read_slot(group_at(t + 1));   // next group's slot, read one group ahead
      if (t < nG) consume(xs[d], cur);
      cur = nxt;
    }
  };
  for (int t0 = 0; t0 < nG; t0 += 2 * D) {
    gather(xb, t0 + D);
    run_stage(xa, t0);
    gather(xa, t0 + 2 * D);
    run_stage(xb, t0 + D);
  }

  // ---- 6. K-split partial sums, added in a fixed order, then Y.
  if constexpr (KS > 1) {
    __syncthreads();                              // staging buffers are free now
    float4v* red = reinterpret_cast<float4v*>(sbase);
    if (ks > 0) {
#pragma unroll
      for (int c = 0; c < CT; ++c) red[(((rt * (KS - 1)) + ks - 1) * CT + c) * 64 + lane] = acc[c];
    }
    __syncthreads();
    if (ks == 0) {
#pragma unroll
      for (int k2 = 1; k2 < KS; ++k2)
#pragma unroll
        for (int c = 0; c < CT; ++c) acc[c] += red[(((rt * (KS - 1)) + k2 - 1) * CT + c) * 64 + lane];
    }
  }
  if (ks == 0) {
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      const int b = 16 * c + n;
      if (b < a.B) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = 16 * rt + 4 * q + i;
          if (r < nrows) {
            const int64_t o = (int64_t)b * m.n_out + row0 + r;
            if (a.out_f32)
              reinterpret_cast<float*>(a.Y)[o] = acc[c][i];
            else
              reinterpret_cast<uint16_t*>(a.Y)[o] = (uint16_t)f2h(acc[c][i]);
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Fallback for shapes whose staging does not fit: per 128-wide K step, 64
// rows are decoded into an fp16 LDS tile in a 6-slots-per-byte order (the X
// tile uses the same order) and multiplied with MFMA for every 16-column
// slice of the batch.
// ---------------------------------------------------------------------------

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;   // fallback kernel
constexpr int kRows = 16 * kWaves;      // W rows per workgroup
constexpr int kSlots = 160;             // k slots per 128-wide step
constexpr int kStride = 168;            // LDS row stride in halves
constexpr int kMaxColTiles = TQ_MAX_BATCH / 16;


__device__ inline uint32_t trit_pattern(int t) {
  return t > 0 ? 0x3C00u : (t < 0 ? 0xBC00u : 0u);
}


__device__ inline int64_t byte_offset(int64_t f, int j, int64_t n) {
  return j < kMainBytes ? f * kMainBytes + j : (int64_t)kMainBytes * n + 2 * f + (j - kMainBytes);
}

__global__ void __launch_bounds__(kThreads) fallback_kernel(MatDev m, const uint16_t* __restrict__ X, int B,
                                                        void* __restrict__ Y, int out_f32) {
  __shared__ __attribute__((aligned(16))) uint4 lut[256];
  __shared__ __attribute__((aligned(16))) uint16_t ws[kRows * kStride];
  __shared__ __attribute__((aligned(16))) uint16_t xs[TQ_MAX_BATCH * kStride];
  __shared__ int recs[kRows];
  __shared__ int cursor[kRows];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int G = m.n_groups;
  const int K = G * kGroup;
  const int64_t ngroups = (int64_t)m.n_out * G;
  const int row0 = blockIdx.x * kRows;
  const int nrows = min(kRows, m.n_out - row0);
  const int ncol_tiles = (B + 15) / 16;

  for (int c = tid; c < 256; c += kThreads) {
    uint4 v = {0u, 0u, 0u, 0u};
    if (c < 243) {
      int cc = c, t[5];
      for (int i = 0; i < 5; ++i) {
        t[i] = cc % 3 - 1;
        cc /= 3;
      }
      v.x = trit_pattern(t[0]) | (trit_pattern(t[1]) << 16);
      v.y = trit_pattern(t[2]) | (trit_pattern(t[3]) << 16);
      v.z = trit_pattern(t[4]);
    }
    lut[c] = v;
  }
  if (tid < kRows) cursor[tid] = (m.nnz1 > 0 && tid < nrows) ? m.rowptr1[row0 + tid] : 0;
  // Zero the X tile once: pad slots and absent batch rows stay zero.
  for (int i = tid; i < TQ_MAX_BATCH * kStride / 2; i += kThreads) reinterpret_cast<uint32_t*>(xs)[i] = 0u;
  for (int i = tid; i < kRows * kStride / 2; i += kThreads) reinterpret_cast<uint32_t*>(ws)[i] = 0u;

  float4v acc[kMaxColTiles];
#pragma unroll
  for (int c = 0; c < kMaxColTiles; ++c) acc[c] = float4v{0.f, 0.f, 0.f, 0.f};

  for (int g = 0; g < G; ++g) {
    __syncthreads();   // previous step's MFMA reads are done; cursors visible
    if (tid < kRows) {
      int rec = -1;
      if (m.nnz1 > 0 && tid < nrows) {
        const int cur = cursor[tid];
        if (cur < m.rowptr1[row0 + tid + 1] && (int)m.gidx1[cur] == g) {
          rec = cur;
          cursor[tid] = cur + 1;
        }
      }
      recs[tid] = rec;
    }
    // X tile: batch row b, code byte j -> slots 6j .. 6j+4.
    for (int it = tid; it < B * kGroupBytes; it += kThreads) {
      const int b = it / kGroupBytes;
      const int j = it - b * kGroupBytes;
      const uint16_t* xp = X + (int64_t)b * K + kGroup * g + 5 * j;
      uint16_t* dst = xs + b * kStride + 6 * j;
#pragma unroll
      for (int i = 0; i < 5; ++i) dst[i] = (5 * j + i < kGroup) ? xp[i] : (uint16_t)0;
    }
    __syncthreads();   // recs visible
    // W tile: row r, code byte j -> slots 6j .. 6j+5.
    for (int it = tid; it < kRows * kGroupBytes; it += kThreads) {
      const int r = it / kGroupBytes;
      const int j = it - r * kGroupBytes;
      uint32_t o0 = 0u, o1 = 0u, o2 = 0u;
      if (r < nrows) {
        const int64_t f = (int64_t)(row0 + r) * G + g;
        const int c0 = m.codes0[byte_offset(f, j, ngroups)];
        const uint16_t s0b = m.scale0[f];
        const int k = recs[r];
        const uint4 p = lut[c0];
        const bool off = m.offset0 != nullptr;
        if (k < 0 && !off) {
          const half2v s2 = {__builtin_bit_cast(_Float16, s0b), __builtin_bit_cast(_Float16, s0b)};
          o0 = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, p.x) * s2);
          o1 = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, p.y) * s2);
          o2 = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, p.z) * s2);
        } else {
          // a = +0; a += mu0; a += mu; a += s0*t0; a += s1*t1 (the terms
          // that exist), rounded once.
          const int c1 = k >= 0 ? m.codes1[byte_offset(k, j, m.nnz1)] : 121;
          const float s0 = h2f(s0b);
          const float mu0 = off ? h2f(m.offset0[f]) : 0.0f;
          const float mu = k >= 0 ? h2f(m.offset1[k]) : 0.0f, s1 = k >= 0 ? h2f(m.scale1[k]) : 0.0f;
          int d0 = c0, d1 = c1;
          uint16_t h[5];
#pragma unroll
          for (int i = 0; i < 5; ++i) {
            float a = 0.0f;
            if (off) a = a + mu0;
            if (k >= 0) a = a + mu;
            a = a + s0 * (float)(d0 % 3 - 1);
            if (k >= 0) a = a + s1 * (float)(d1 % 3 - 1);
            h[i] = __builtin_bit_cast(uint16_t, (_Float16)a);
            d0 /= 3;
            d1 /= 3;
          }
          o0 = h[0] | ((uint32_t)h[1] << 16);
          o1 = h[2] | ((uint32_t)h[3] << 16);
          o2 = h[4];
        }
      }
      uint32_t* dst = reinterpret_cast<uint32_t*>(ws + r * kStride + 6 * j);
      dst[0] = o0;
      dst[1] = o1;
      dst[2] = o2;
    }
    __syncthreads();
    // MFMA: this wave's 16 rows against every 16-column slice of the batch.
    const uint16_t* arow = ws + (wave * 16 + (lane & 15)) * kStride + 8 * (lane >> 4);
#pragma unroll
    for (int ks = 0; ks < kSlots / 32; ++ks) {
      const half8 a = *reinterpret_cast<const half8*>(arow + 32 * ks);
#pragma unroll
      for (int c = 0; c < kMaxColTiles; ++c) {
        if (c < ncol_tiles) {
          const uint16_t* brow = xs + (16 * c + (lane & 15)) * kStride + 8 * (lane >> 4) + 32 * ks;
          const half8 bv = *reinterpret_cast<const half8*>(brow);
          acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bv, acc[c], 0, 0, 0);
        }
      }
    }
  }

  // acc[c][i] is C[row = 4*(lane/16) + i][col = lane % 16] of this wave's tile.
#pragma unroll
  for (int c = 0; c < kMaxColTiles; ++c) {
    if (c < ncol_tiles) {
      const int b = 16 * c + (lane & 15);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = wave * 16 + 4 * (lane >> 4) + i;
        if (b < B && r < nrows) {
          const int64_t o = (int64_t)b * m.n_out + row0 + r;
          if (out_f32)
            reinterpret_cast<float*>(Y)[o] = acc[c][i];
          else
            reinterpret_cast<uint16_t*>(Y)[o] = __builtin_bit_cast(uint16_t, (_Float16)acc[c][i]);
        }
      }
    }
  }
}


typedef void (*SbKernel)(SbArgs);

SbKernel sb_select(int RT, int ci) {
  static const SbKernel table[4][3] = {
      {sb_kernel<1, 4, 1>, sb_kernel<1, 4, 2>, sb_kernel<1, 4, 4>},
      {sb_kernel<2, 2, 1>, sb_kernel<2, 2, 2>, sb_kernel<2, 2, 4>},
      {sb_kernel<3, 1, 1>, sb_kernel<3, 1, 2>, sb_kernel<3, 1, 4>},
      {sb_kernel<4, 1, 1>, sb_kernel<4, 1, 2>, sb_kernel<4, 1, 4>},
  };
  return table[RT - 1][ci];
}

struct SbDeviceInfo {
  bool attr_set[4][3] = {};
};

SbDeviceInfo& sb_device_info() {
  static thread_local SbDeviceInfo info[64];
  int dev = 0;
  (void)hipGetDevice(&dev);
  return info[dev & 63];
}

}  // namespace

hipError_t launch_gemm_smallbatch(const MatDev& m, const uint16_t* X, int B, void* Y, bool out_f32,
                                  hipStream_t s) {
  const int G = m.n_groups;
  // Rows per workgroup: about one workgroup per CU (256), at most 4 row
  // tiles, and a staging that fits.
  int RT = (m.n_out + 16 * 256 - 1) / (16 * 256);
  RT = RT < 1 ? 1 : (RT > 4 ? 4 : RT);
  while (RT > 1 && G * 16 * RT > kMaxPairs) --RT;
  if (G * 16 * RT > kMaxPairs) {
    const int wgs = (m.n_out + kRows - 1) / kRows;
    hipLaunchKernelGGL(fallback_kernel, dim3(wgs), dim3(kThreads), 0, s, m, X, B, Y, out_f32 ? 1 : 0);
    return hipGetLastError();
  }
  const int KS = RT == 1 ? 4 : (RT == 2 ? 2 : 1);
  const int ci = B <= 16 ? 0 : (B <= 32 ? 1 : 2);
  const int CT = 1 << ci;
  const int R = 16 * RT;
  const int staged = staged_bytes(G * R, R);
  const int red = RT * (KS - 1) * CT * 64 * 16;
  const int dyn = staged > red ? staged : red;
  const SbKernel kern = sb_select(RT, ci);
  SbDeviceInfo& di = sb_device_info();
  if (!di.attr_set[RT - 1][ci]) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsLimit - kLutBytes);
    if (e != hipSuccess) return e;
    di.attr_set[RT - 1][ci] = true;
  }
  SbArgs args{m, X, Y, B, out_f32 ? 1 : 0};
  const int wgs = (m.n_out + R - 1) / R;
  hipLaunchKernelGGL(kern, dim3(wgs), dim3(64 * RT * KS), dyn, s, args);
  return hipGetLastError();
}

}  // namespace tq
