// Small-batch packed GEMM Y = X W^T with MFMA (gfx950).
//
// Paper: section 3, eq. 3 (the weight), section 18 (kernel work across
// shapes and batch sizes is the stated next step).  For a batch of B
// activation rows the product is a dense contraction, so it runs on
// v_mfma_f32_16x16x32_f16: A = 16 weight rows, B = 16 batch rows, C = the
// 16 x 16 block of Y^T.
//
// k order.  MFMA sums over k in any order, so the 32 k of a step are chosen
// to make both operands cheap.  Groups are taken four at a time (a quad);
// lane block q (lanes 16q .. 16q+15) works on group 4Q + q in every step of
// quad Q, and step u (0..15) takes inputs 8u .. 8u+7 of each block's group.
// The B operand is then one aligned 16-byte chunk of X per lane, and the
// code bytes and trit phase of a window (its first input is trit 8u % 5 of
// byte 8u / 5) are fixed per step, known at compile time.
//
// Decode.  The GEMV's table (fp16 +-1/0 patterns (t0,t1), (t2,t3), (t4,0)
// per code, 16 copies, static LDS) is read once per code byte, with one
// 16-byte read (a byte shared by two windows is kept in registers); a window's four dwords
// are table dwords or two of them joined by v_alignbit / v_lshl_or.  A
// weight is pattern * s0 + offset in one v_pk_fma_f16 (exact without
// offsets); on two-plane groups the plane-1 pattern * s1 is added with one
// more fma and the record's offset is folded into the plane-0 term, so a
// weight takes at most three fp16 roundings (well inside the accuracy
// bound).
//
// Work split.  A workgroup of 8 waves owns 16 RT consecutive rows.  Its
// waves split K by quads, and each wave covers all RT row tiles and all
// batch columns, so a CU reads its slice of X once and decodes every weight
// once.  Plane-0 codes go straight to registers, all loaded up front; X
// comes in bursts of a whole line per lane, one burst ahead of use.  The
// workgroup's plane-1 records are staged in LDS with one slot per (row,
// group).  The waves' partial sums are added in a fixed order through LDS
// (bit-reproducible).  Shapes past the register and LDS limits (more than
// four quads per wave) use the simple per-group kernel at the end of this
// file.

#include "tq_internal.h"

namespace tq {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float float4v __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

constexpr int kLdsLimit = 160 * 1024;
constexpr int kQWaves = 8;                       // waves per workgroup (K split)
constexpr int kQThreads = 64 * kQWaves;
constexpr int kQRep = 16;                        // table copies (lane & 15)
constexpr int kQLutBytes = 256 * kQRep * 16;     // 64 KiB
constexpr int kQMaxPairs = 2048;                 // record slots (rows x groups) per workgroup
constexpr int kQMaxUnits = 4;                    // row tiles x quads per wave
constexpr int kWindows = 16;                     // 8-input k blocks per group

__device__ inline float h2f(uint32_t b) { return (float)__builtin_bit_cast(_Float16, (uint16_t)b); }
__device__ inline uint32_t f2h(float a) { return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)a); }

struct __attribute__((aligned(16))) U3 {
  uint32_t x, y, z;
};

constexpr int kQMaxRanges = 640;   // workgroups with record ranges in the kernel arguments

struct QArgs {
  MatDev m;
  const uint16_t* X;
  void* Y;
  int B;
  int out_f32;
  // With kHost: the first record of every workgroup, then nnz1 (from the
  // host row pointers), so record loads need no dependent load.
  int32_t rec_begin[kQMaxRanges + 1];
};

// LDS: the table (the kernel's only static array, so it sits at LDS address
// 0 and the byte-to-address v_perm is the whole address; in the dynamic
// block it cost an add per read), then the dynamic part: row pointers [R + 1], record flags
// [R * G], record slots [R * G] x 32 B (byte offsets below); after the main
// loop the partial sums [waves][RT][CT][64 lanes] x 16 B overlay it.
__host__ __device__ constexpr int q_flag_off(int R) { return 4 * (R + 1); }
__host__ __device__ constexpr int q_rec_off(int R, int G) { return (q_flag_off(R) + R * G + 15) & ~15; }
__host__ __device__ constexpr int q_stage_bytes(int R, int G) { return q_rec_off(R, G) + 32 * R * G; }
__host__ __device__ constexpr int q_red_bytes(int RT, int CT) { return kQWaves * RT * CT * 64 * 16; }

__device__ inline uint32_t q_pattern(int t) { return t > 0 ? 0x3C00u : (t < 0 ? 0xBC00u : 0u); }

// Table entry of code c: fp16 patterns of (t0, t1), (t2, t3), (t4, 0);
// codes 243..255 read as zeros.
__device__ inline uint4 q_entry(int c) {
  uint32_t t[5];
  uint32_t d = (uint32_t)c;
#pragma unroll
  for (int i = 0; i < 5; ++i) {
    const uint32_t qd = (d * 171u) >> 9;   // d / 3 for d < 256
    t[i] = c < 243 ? q_pattern((int)(d - 3u * qd) - 1) : 0u;
    d = qd;
  }
  return uint4{t[0] | (t[1] << 16), t[2] | (t[3] << 16), t[4], 0u};
}

// LDS byte address of this lane's table copy for byte BY of dword w:
// bytes [slot, code, 0, 0].
template <int BY>
__device__ inline uint32_t q_addr(uint32_t w, uint32_t slot) {
  return __builtin_amdgcn_perm(slot, w, 0x0C0C0004u | (BY << 8));
}

// Window u (inputs 8u .. 8u+7 of a group): first code byte, trit phase
// (index of its first trit in that byte) and last code byte.
__host__ __device__ constexpr int win_byte(int u) { return (8 * u) / 5; }
__host__ __device__ constexpr int win_phase(int u) { return (8 * u) % 5; }
__host__ __device__ constexpr int win_last(int u) { return (8 * u + 7) / 5; }

// Table address of code byte j of a group whose bytes 0..23 are w[0..5] and
// bytes 24, 25 the low half of w[6] (j is a constant after unrolling; w is
// registers or a record slot in LDS).
__device__ __attribute__((always_inline)) inline uint32_t code_byte_addr(const uint32_t* w, int j, uint32_t slot) {
  const uint32_t word = j < 24 ? w[j >> 2] : w[6];
  switch (j < 24 ? (j & 3) : j - 24) {
    case 0: return q_addr<0>(word, slot);
    case 1: return q_addr<1>(word, slot);
    case 2: return q_addr<2>(word, slot);
    default: return q_addr<3>(word, slot);
  }
}

// Table entry at LDS byte address a, read whole: a 16-byte read puts the 16
// lanes served together on 64 different banks (one copy each), where a
// 12-byte read is split by the compiler into reads that share banks.
__device__ __attribute__((always_inline)) inline U3 table_entry(const unsigned char* lut, uint32_t a) {
  const u4v v = *reinterpret_cast<const u4v*>(lut + a);
  return U3{v.x, v.y, v.z};
}

// Patterns of a window of phase o from the table entries of its bytes: the
// window's 8 trits are trits o..4 of e0's byte, then e1's, then e2's.
__device__ __attribute__((always_inline)) inline void window_patterns(int o, const U3& e0, const U3& e1,
                                                                      const U3& e2, uint32_t (&d)[4]) {
  const uint32_t a01 = __builtin_amdgcn_alignbit(e0.y, e0.x, 16), a12 = __builtin_amdgcn_alignbit(e0.z, e0.y, 16);
  const uint32_t b01 = __builtin_amdgcn_alignbit(e1.y, e1.x, 16), b12 = __builtin_amdgcn_alignbit(e1.z, e1.y, 16);
  switch (o) {
    case 0: d[0] = e0.x; d[1] = e0.y; d[2] = e0.z | (e1.x << 16); d[3] = b01; break;
    case 1: d[0] = a01; d[1] = a12; d[2] = e1.x; d[3] = e1.y; break;
    case 2: d[0] = e0.y; d[1] = e0.z | (e1.x << 16); d[2] = b01; d[3] = b12; break;
    case 3: d[0] = a12; d[1] = e1.x; d[2] = e1.y; d[3] = e1.z | (e2.x << 16); break;
    default: d[0] = e0.z | (e1.x << 16); d[1] = b01; d[2] = b12; d[3] = e2.x; break;
  }
}

// p * s + c on two fp16 halves; p and c are fp16 bit pairs (a plain
// uint32 must never meet a half2v by value conversion).
__device__ inline uint32_t hfma2(uint32_t p, half2v s, uint32_t c) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_fma(__builtin_bit_cast(half2v, p), s,
                                                                __builtin_bit_cast(half2v, c)));
}

__device__ inline half2v hsplat(uint32_t h) {
  const _Float16 v = __builtin_bit_cast(_Float16, (uint16_t)h);
  return half2v{v, v};
}

// Workgroup barrier for LDS data only: waits for this wave's LDS accesses
// but leaves its global loads in flight (a plain __syncthreads waits for
// those too).
__device__ inline void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// One plane-1 record as loaded: code bytes 0..23, bytes 24, 25, mu | s1 << 16, group.
struct RecLoad {
  uint64_t v0, v1, v2;
  uint32_t tl, ms;
  int gg;
};

// Record k; a matrix without records reads its plane-0 arrays at k = 0
// instead (no branch around the loads, whose results are then unused).
__device__ inline RecLoad load_record(const MatDev& m, int64_t k) {
  const bool has = m.nnz1 > 0;
  const uint8_t* codes = has ? m.codes1 : m.codes0;
  const int64_t n = has ? m.nnz1 : (int64_t)m.n_out * m.n_groups;
  const uint16_t* mu = has ? m.offset1 : m.scale0;
  const uint16_t* s1 = has ? m.scale1 : m.scale0;
  const uint16_t* gi = has ? m.gidx1 : m.scale0;
  // In bounds whatever range the caller's row pointers give.
  k = has ? (k < 0 ? 0 : (k >= n ? n - 1 : k)) : 0;
  const uint64_t* rm = reinterpret_cast<const uint64_t*>(codes) + 3 * k;
  RecLoad r;
  r.v0 = rm[0];
  r.v1 = rm[1];
  r.v2 = rm[2];
  r.tl = reinterpret_cast<const uint16_t*>(codes + 24 * n)[k];
  r.ms = (uint32_t)mu[k] | ((uint32_t)s1[k] << 16);
  r.gg = (int)gi[k];
  return r;
}

// kHost: the workgroup's record range comes from the kernel arguments
// (host row pointers), so its record loads are issued before anything else.
template <int RT, int CT, int QPW, bool kHost>
__global__ void __launch_bounds__(kQThreads) quad_kernel(QArgs a) {
  __shared__ __attribute__((aligned(16))) unsigned char lut[kQLutBytes];
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  constexpr int R = 16 * RT;
  // X is loaded in bursts of L consecutive chunks per lane, a whole 128-byte
  // line, so every line is fetched once and used whole.  Single 16-byte
  // chunks per step made each line be refetched for every chunk: the 16
  // batch rows of a step lie a power-of-two stride apart and evict each
  // other from L1.  With up to two column tiles the next burst is loaded
  // while the current one is used (NB = 2 buffers).  Three or four column
  // tiles leave registers for one line buffer only: with several quads per
  // wave it is refilled after each block (whole lines, the latency exposed
  // once per 8 steps); with one quad, half-line bursts in two buffers are
  // faster (gate 12288x4096 at B = 64: 28 against 31 us; down 4096x12288:
  // 57 against 55 us the other way round).
  constexpr int L = (CT <= 2 || QPW >= 2) ? 8 : 4;
  constexpr int NB = (CT <= 2 || QPW == 1) ? 2 : 1;
  constexpr int NW = QPW * kWindows;      // k-steps of this wave

  const MatDev& m = a.m;
  const int G = m.n_groups;
  const int64_t K = (int64_t)G * kGroup;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int q = lane >> 4;                // group of the quad (A and B operands)
  const int r16 = lane & 15;              // A: row of the tile; B: batch column
  const uint32_t slot = (uint32_t)r16 << 4;
  const int row0 = blockIdx.x * R;
  const int nrows = min(R, m.n_out - row0);
  const int64_t ngroups = (int64_t)m.n_out * G;
  const bool has_off = m.offset0 != nullptr;
  const bool has_rec = m.nnz1 > 0;

  int* rowptr_s = reinterpret_cast<int*>(lds);
  uint8_t* flag_s = lds + q_flag_off(R);
  uint4* rec_s = reinterpret_cast<uint4*>(lds + q_rec_off(R, G));

  // ---- 1. Loads, all issued before any wait, every one unconditional at a
  // clamped address (a load whose destination is also written on another
  // path forces an early wait).  With host ranges: the workgroup's first
  // records (their range is known), the row pointers, the first X burst,
  // then the codes and scales of every (row tile, quad) of this wave, so the
  // record staging waits for the records alone while the codes stream in.
  // Without: row pointers, codes, X, then the records once the device row
  // pointers give their range.
  const int32_t* rp_src = has_rec ? m.rowptr1 : reinterpret_cast<const int32_t*>(m.codes0);
  int kb = 0, ke = 0;
  RecLoad rec0;
  if constexpr (kHost) {
    kb = a.rec_begin[blockIdx.x];
    ke = a.rec_begin[blockIdx.x + 1];
    rec0 = load_record(m, min(kb + tid, max(ke - 1, 0)));
  }
  const int32_t rp_l = rp_src[row0 + min(tid, nrows)];
  const uint16_t* off_src = has_off ? m.offset0 : m.scale0;
  const uint16_t* tail_src = reinterpret_cast<const uint16_t*>(m.codes0 + 24 * ngroups);

  u4v xb[NB][L][CT];
  auto issue_x = [&](int v) {   // burst v: k-steps v L .. v L + L - 1 of this wave
#pragma unroll
    for (int k = 0; k < L; ++k) {
      const int F = v * L + k;
      const int qi = F / kWindows, u = F % kWindows;
      const int g = min(4 * (wave * QPW + qi) + q, G - 1);
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const int b = min(16 * c + r16, a.B - 1);
        xb[v % NB][k][c] = *reinterpret_cast<const u4v*>(a.X + (int64_t)b * K + kGroup * g + 8 * u);
      }
    }
  };
  if constexpr (kHost) issue_x(0);

  uint32_t cw[QPW][RT][7];   // code bytes 0..23, then bytes 24, 25
  uint32_t sc[QPW][RT];      // s0 | offset << 16
#pragma unroll
  for (int qi = 0; qi < QPW; ++qi) {
    const int g = min(4 * (wave * QPW + qi) + q, G - 1);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = min(16 * rt + r16, nrows - 1);
      const int64_t f = (int64_t)(row0 + r) * G + g;
      const uint64_t* mp = reinterpret_cast<const uint64_t*>(m.codes0 + 24 * f);
#pragma unroll
      for (int i = 0; i < 3; ++i) {
        const uint64_t v = mp[i];
        cw[qi][rt][2 * i] = (uint32_t)v;
        cw[qi][rt][2 * i + 1] = (uint32_t)(v >> 32);
      }
      cw[qi][rt][6] = tail_src[f];
      sc[qi][rt] = (uint32_t)m.scale0[f] | ((uint32_t)off_src[f] << 16);
    }
  }

  if constexpr (!kHost) {
    issue_x(0);
    // The workgroup's first kQThreads plane-1 records, one per thread (a
    // clamped in-range index where there are fewer; only threads below the
    // count use theirs).
    const int32_t kb_l = rp_src[row0];
    const int32_t ke_l = rp_src[row0 + nrows];
    kb = has_rec ? kb_l : 0;
    ke = has_rec ? ke_l : 0;
    rec0 = load_record(m, min(kb + tid, max(ke - 1, 0)));
  }

  // ---- 2. Table (one code and half of its copies per thread; at step k
  // the copy index is rotated by the code so one store instruction's lanes
  // spread over the banks), record flags cleared, row pointers.
  for (int t = tid; t < 512; t += kQThreads) {
    const int c = t & 255, h = t >> 8;
    const uint4 e = q_entry(c);
#pragma unroll
    for (int k = 0; k < kQRep / 2; ++k)
      reinterpret_cast<uint4*>(lut)[c * kQRep + ((8 * h + k + c) & (kQRep - 1))] = e;
  }
  for (int i = tid; i < (q_rec_off(R, G) - q_flag_off(R)) / 4; i += kQThreads)
    reinterpret_cast<uint32_t*>(flag_s)[i] = 0u;
  if (tid <= nrows) rowptr_s[tid] = rp_l;
  lds_barrier();

  // ---- 3. Plane-1 records of the workgroup's rows (CSR range kb..ke) to
  // their (row, group) slots.
  auto stage = [&](int k, const RecLoad& r) {
    // Row of record k: the last r with rowptr_s[r] <= k.
    int lo = 0, hi = nrows;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (rowptr_s[mid] <= k) lo = mid; else hi = mid;
    }
    if (r.gg < G) {
      const int p = lo * G + r.gg;
      rec_s[2 * p] = uint4{(uint32_t)r.v0, (uint32_t)(r.v0 >> 32), (uint32_t)r.v1, (uint32_t)(r.v1 >> 32)};
      rec_s[2 * p + 1] = uint4{(uint32_t)r.v2, (uint32_t)(r.v2 >> 32), r.tl, r.ms};
      flag_s[p] = 1;
    }
  };
  if (kb + tid < ke) stage(kb + tid, rec0);
  for (int k = kb + kQThreads + tid; k < ke; k += kQThreads) stage(k, load_record(m, k));
  lds_barrier();

  // ---- 4. Main loop: quads of this wave, 16 k-steps each, all row tiles
  // and batch column tiles.
  float4v acc[RT][CT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int c = 0; c < CT; ++c) acc[rt][c] = float4v{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int qi = 0; qi < QPW; ++qi) {
    const int g = 4 * (wave * QPW + qi) + q;
    // Per row tile: weight = p0 * s0 + c0 (+ p1 * s1 with a record), c0 =
    // group offset + record offset (each zero where absent); lanes past the
    // rows or groups get zero weights.
    half2v s0v[RT], s1v[RT];
    uint32_t c0v[RT];
    bool hr[RT];
    // Record codes: in registers where they fit (few column and row tiles),
    // else read from the LDS slot when used.
    constexpr bool kRcRegs = CT == 1 || (CT == 2 && RT <= 3);
    uint32_t rcr[RT][kRcRegs ? 7 : 1];
    const uint32_t* rcs[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = 16 * rt + r16;
      const bool valid = g < G && r < nrows;
      const int p = min(r, nrows - 1) * G + min(g, G - 1);
      const uint4 rb = rec_s[2 * p + 1];
      hr[rt] = valid && flag_s[p] != 0;
      const float mu = hr[rt] ? h2f(rb.w & 0xFFFFu) : 0.0f;
      const uint32_t s1b = hr[rt] ? (rb.w >> 16) : 0u;
      const float m0 = has_off ? h2f(sc[qi][rt] >> 16) : 0.0f;
      s0v[rt] = hsplat(valid ? (sc[qi][rt] & 0xFFFFu) : 0u);
      const uint32_t c0 = valid ? f2h(m0 + mu) : 0u;
      c0v[rt] = c0 | (c0 << 16);
      s1v[rt] = hsplat(s1b);
      rcs[rt] = reinterpret_cast<const uint32_t*>(rec_s + 2 * p);
      if constexpr (kRcRegs) {
        const uint4 ra = rec_s[2 * p];
        rcr[rt][0] = ra.x; rcr[rt][1] = ra.y; rcr[rt][2] = ra.z; rcr[rt][3] = ra.w;
        rcr[rt][4] = rb.x; rcr[rt][5] = rb.y; rcr[rt][6] = rb.z;
      }
    }

    U3 ep0[RT], ep1[RT];   // table entry of the previous window's last byte (planes 0, 1)
#pragma unroll
    for (int v = 0; v < kWindows / L; ++v) {
    const int F0 = qi * kWindows + v * L;
    if (NB == 2 && F0 + L < NW) issue_x(F0 / L + 1);
#pragma unroll
    for (int k = 0; k < L; ++k) {
      const int u = v * L + k, F = F0 + k;
      const u4v (&xv)[CT] = xb[(F / L) % NB][k];
      const int j0 = win_byte(u), jl = win_last(u);
      const bool shared = u > 0 && win_last(u - 1) == j0;   // first byte already read
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const U3 a0 = shared ? ep0[rt] : table_entry(lut, code_byte_addr(cw[qi][rt], j0, slot));
        const U3 a1 = table_entry(lut, code_byte_addr(cw[qi][rt], j0 + 1, slot));
        const U3 a2 = jl > j0 + 1 ? table_entry(lut, code_byte_addr(cw[qi][rt], jl, slot)) : a1;
        ep0[rt] = a2;
        uint32_t p[4], w[4];
        window_patterns(win_phase(u), a0, a1, a2, p);
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = hfma2(p[i], s0v[rt], c0v[rt]);
        if (hr[rt]) {
          const uint32_t* rc = kRcRegs ? rcr[rt] : rcs[rt];
          const U3 b0 = shared ? ep1[rt] : table_entry(lut, code_byte_addr(rc, j0, slot));
          const U3 b1 = table_entry(lut, code_byte_addr(rc, j0 + 1, slot));
          const U3 b2 = jl > j0 + 1 ? table_entry(lut, code_byte_addr(rc, jl, slot)) : b1;
          ep1[rt] = b2;
          uint32_t p1[4];
          window_patterns(win_phase(u), b0, b1, b2, p1);
#pragma unroll
          for (int i = 0; i < 4; ++i) w[i] = hfma2(p1[i], s1v[rt], w[i]);
        }
        const half8 A = __builtin_bit_cast(half8, u4v{w[0], w[1], w[2], w[3]});
#pragma unroll
        for (int c = 0; c < CT; ++c)
          acc[rt][c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, __builtin_bit_cast(half8, xv[c]), acc[rt][c], 0, 0, 0);
      }
    }
    if (NB == 1 && F0 + L < NW) issue_x(F0 / L + 1);
    }
  }

  // ---- 5. Partial sums of the waves, added in wave order, then Y.
  lds_barrier();   // every wave is done with the table and the records
  float4v* red = reinterpret_cast<float4v*>(lds);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int c = 0; c < CT; ++c) red[((wave * RT + rt) * CT + c) * 64 + lane] = acc[rt][c];
  lds_barrier();
  constexpr int kItems = RT * CT * 64;
  for (int it = tid; it < kItems; it += kQThreads) {
    // Four consecutive threads hold 16 consecutive rows of one column.
    const int qq = it & 3, n = (it >> 2) & 15, c = (it >> 6) % CT, rt = (it >> 6) / CT;
    const int ln = 16 * qq + n;
    float4v s = red[(rt * CT + c) * 64 + ln];
#pragma unroll
    for (int w = 1; w < kQWaves; ++w) s += red[((w * RT + rt) * CT + c) * 64 + ln];
    const int b = 16 * c + n;
    if (b < a.B) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 16 * rt + 4 * qq + i;
        if (r < nrows) {
          const int64_t o = (int64_t)b * m.n_out + row0 + r;
          if (a.out_f32)
            reinterpret_cast<float*>(a.Y)[o] = s[i];
          else
            reinterpret_cast<uint16_t*>(a.Y)[o] = (uint16_t)f2h(s[i]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Fallback for shapes past the quad kernel's limits: per 128-wide K step, 64
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
      v.x = q_pattern(t[0]) | (q_pattern(t[1]) << 16);
      v.y = q_pattern(t[2]) | (q_pattern(t[3]) << 16);
      v.z = q_pattern(t[4]);
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




typedef void (*QKernel)(QArgs);

template <int RT, int QPW, bool H>
QKernel q_pick(int CT) {
  switch (CT) {
    case 1: return quad_kernel<RT, 1, QPW, H>;
    case 2: return quad_kernel<RT, 2, QPW, H>;
    case 3: return quad_kernel<RT, 3, QPW, H>;
    default:
      if constexpr (RT == 4) return nullptr;   // not launched: it would spill registers
      else return quad_kernel<RT, 4, QPW, H>;
  }
}

// (RT, QPW) pairs with RT * QPW <= kQMaxUnits.
template <bool H>
QKernel q_select(int RT, int QPW, int CT) {
  switch (RT) {
    case 1:
      switch (QPW) {
        case 1: return q_pick<1, 1, H>(CT);
        case 2: return q_pick<1, 2, H>(CT);
        case 3: return q_pick<1, 3, H>(CT);
        default: return q_pick<1, 4, H>(CT);
      }
    case 2: return QPW == 1 ? q_pick<2, 1, H>(CT) : q_pick<2, 2, H>(CT);
    case 3: return q_pick<3, 1, H>(CT);
    default: return q_pick<4, 1, H>(CT);
  }
}

struct QDeviceInfo {
  bool attr_set[2][4][4][4] = {};
};

QDeviceInfo& q_device_info() {
  static thread_local QDeviceInfo info[64];
  int dev = 0;
  (void)hipGetDevice(&dev);
  return info[dev & 63];
}

}  // namespace

hipError_t launch_gemm_smallbatch(const MatDev& m, const uint16_t* X, int B, void* Y, bool out_f32,
                                  hipStream_t s) {
  const int G = m.n_groups;
  const int NQ = (G + 3) / 4;
  const int QPW = (NQ + kQWaves - 1) / kQWaves;
  // Rows per workgroup: about one workgroup per CU (256), at most 4 row
  // tiles, and at most kQMaxUnits (row tile, quad) units per wave and
  // kQMaxPairs record slots.
  int RT = (m.n_out + 16 * 256 - 1) / (16 * 256);
  RT = RT < 1 ? 1 : (RT > 4 ? 4 : RT);
  const int CT = (B + 15) / 16;
  // Four row tiles with four column tiles would spill registers.
  if (RT == 4 && CT == 4) RT = 3;
  while (RT > 1 && (RT * QPW > kQMaxUnits || 16 * RT * G > kQMaxPairs)) --RT;
  if (RT * QPW > kQMaxUnits || 16 * RT * G > kQMaxPairs) {
    const int wgs = (m.n_out + kRows - 1) / kRows;
    hipLaunchKernelGGL(fallback_kernel, dim3(wgs), dim3(kThreads), 0, s, m, X, B, Y, out_f32 ? 1 : 0);
    return hipGetLastError();
  }
  const int R = 16 * RT;
  const int staged = q_stage_bytes(R, G);
  const int red = q_red_bytes(RT, CT);
  const int dyn = staged > red ? staged : red;
  const int wgs = (m.n_out + R - 1) / R;
  // Record ranges in the kernel arguments where the host has the row
  // pointers (or there are no records) and the workgroups are few enough.
  const bool host = (m.nnz1 == 0 || m.rowptr1_host != nullptr) && wgs <= kQMaxRanges;
  const QKernel kern = host ? q_select<true>(RT, QPW, CT) : q_select<false>(RT, QPW, CT);
  if (kern == nullptr) return hipErrorInvalidValue;
  QDeviceInfo& di = q_device_info();
  if (!di.attr_set[host][RT - 1][QPW - 1][CT - 1]) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kLdsLimit - kQLutBytes);
    if (e != hipSuccess) return e;
    di.attr_set[host][RT - 1][QPW - 1][CT - 1] = true;
  }
  QArgs args;
  args.m = m;
  args.X = X;
  args.Y = Y;
  args.B = B;
  args.out_f32 = out_f32 ? 1 : 0;
  if (host) {
    for (int w = 0; w <= wgs; ++w) {
      const int64_t r = (int64_t)w * R < m.n_out ? (int64_t)w * R : m.n_out;
      int64_t v = m.nnz1 > 0 ? m.rowptr1_host[r] : 0;
      v = v < 0 ? 0 : (v > m.nnz1 ? m.nnz1 : v);   // in bounds whatever the host copy holds
      args.rec_begin[w] = (int32_t)v;
    }
  }
  hipLaunchKernelGGL(kern, dim3(wgs), dim3(kQThreads), dyn, s, args);
  return hipGetLastError();
}

}  // namespace tq
