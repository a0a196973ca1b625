// Decode helpers shared by the batch-1 GEMV kernels (gemv.hip) and the
// decode-step chain kernel (chain.hip): the 16-copy LDS table of fp16 sign
// patterns, the staged layout of x, one half-group's dot product, the loads
// of a pass and of a record half, and the fixed-order DPP segment sums.
// Included inside namespace tq's anonymous namespace of each file (internal
// linkage per translation unit).
#pragma once

constexpr int kRep = 16;                       // LUT copies
constexpr int kLutBytes = 256 * kRep * 16;
constexpr int kMaxThreads = 1024;
constexpr int kHalfBytes = 12;                 // body bytes per half-group
constexpr int kLaneBytes = kHalfBytes + 1;     // + one tail byte
// x in LDS: group g at dword 68 g, inputs 0..59 at dwords 0..29, inputs
// 60..119 at 32..61, inputs 120..127 at 62..65 (dwords 30, 31, 66, 67
// unused).  Each half's 30 body dwords then start 16-byte aligned, and the
// 16 lanes that one 16-byte LDS read serves together (8 groups x 2 halves)
// cover the 64 banks exactly once.
constexpr int kXStrideDw = 68;
constexpr int kXHalfDw = 32;   // dword offset of half 1's body
constexpr int kXTailDw = 62;   // dword offset of inputs 120..127

// Dword offset within a group's slot of inputs i .. i+3 (i % 4 == 0).
__device__ inline int x_slot_dw(int i) {
  return i < 60 ? i / 2 : (i < 120 ? kXHalfDw + (i - 60) / 2 : kXTailDw + (i - 120) / 2);
}

static_assert(kRep == 16, "the table addressing assumes 16 copies");

// Lanes per row: S itself when it is a multiple of 64, else S rounded up to
// a power of two (S < 64) or to a multiple of 64 (S > 64).
__host__ __device__ inline int padded_slots(int S) {
  if ((S & 63) == 0) return S;
  if (S < 64) {
    int p = 2;
    while (p < S) p <<= 1;
    return p;
  }
  return (S + 63) & ~63;
}

// ---------------------------------------------------------------- table
__device__ inline uint32_t trit_pattern(int t) { return t > 0 ? 0x3C00u : (t < 0 ? 0xBC00u : 0u); }

// Table entry of code c: fp16 patterns of (t0, t1), (t2, t3), (t4, 0),
// (0, t4); codes 243..255 map to zeros.  Computed in registers.
__device__ inline uint4 lut_entry(int c) {
  uint32_t t[5];
  uint32_t d = (uint32_t)c;
#pragma unroll
  for (int i = 0; i < 5; ++i) {
    const uint32_t q = (d * 171u) >> 9;   // d / 3 for d < 256
    t[i] = c < 243 ? trit_pattern((int)(d - 3u * q) - 1) : 0u;
    d = q;
  }
  return uint4{t[0] | (t[1] << 16), t[2] | (t[3] << 16), t[4], t[4] << 16};
}

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
  // bytes [slot, code, 0, 0]: selector 4 picks byte 0 of `slot`, B byte B of w.
  return __builtin_amdgcn_perm(slot, w, 0x0C0C0004u | (B << 8));
}

// Activation registers of a half-group: 6 pairs of code bytes x 5 dwords,
// then 3 for the tail byte.
constexpr int kXrRegs = 33;

// LDS byte address of this lane's table copy for code byte j of w.
__device__ __attribute__((always_inline)) inline uint32_t code_addr(const uint32_t (&w)[4], int j, uint32_t slot) {
  switch (j & 3) {
    case 0: return lut_addr<0>(w[j >> 2], slot);
    case 1: return lut_addr<1>(w[j >> 2], slot);
    case 2: return lut_addr<2>(w[j >> 2], slot);
    default: return lut_addr<3>(w[j >> 2], slot);
  }
}

// Dot product of the 13 code bytes of a half-group (byte j in byte j % 4 of
// w[j / 4]) with its activation registers.
__device__ __attribute__((always_inline)) inline float code_dot(const unsigned char* lut, uint32_t slot,
                                                                const uint32_t (&w)[4],
                                                                const uint32_t (&xr)[kXrRegs]) {
  typedef uint32_t u4v __attribute__((ext_vector_type(4)));
  float a0 = 0.f, a1 = 0.f, a2 = 0.f;
#pragma unroll
  for (int m = 0; m < kHalfBytes / 2; ++m) {
    // Full 16-byte reads: the 16 lanes served together cover the 64 banks
    // exactly once, and the fourth dword carries t4 in the high half.
    const u4v e0 = *reinterpret_cast<const u4v*>(lut + code_addr(w, 2 * m, slot));
    const u4v e1 = *reinterpret_cast<const u4v*>(lut + code_addr(w, 2 * m + 1, slot));
    a0 = fdot2(e0.x, xr[5 * m], a0);
    a1 = fdot2(e0.y, xr[5 * m + 1], a1);
    a0 = fdot2(e1.x, xr[5 * m + 2], a0);
    a1 = fdot2(e1.y, xr[5 * m + 3], a1);
    a2 = fdot2(e0.z | e1.w, xr[5 * m + 4], a2);
  }
  const U3 e = *reinterpret_cast<const U3*>(lut + code_addr(w, kHalfBytes, slot));
  a0 = fdot2(e.x, xr[30], a0);
  a1 = fdot2(e.y, xr[31], a1);
  a2 = fdot2(e.z, xr[32], a2);
  return (a0 + a1) + a2;
}

// code_dot for kB activation rows at once: the table reads are shared, each
// row keeps its own accumulators (same order as code_dot for each row).
template <int kB>
__device__ __attribute__((always_inline)) inline void code_dot_rows(const unsigned char* lut, uint32_t slot,
                                                                   const uint32_t (&w)[4],
                                                                   const uint32_t (&xr)[kB][kXrRegs],
                                                                   float (&out)[kB]) {
  typedef uint32_t u4v __attribute__((ext_vector_type(4)));
  float a0[kB], a1[kB], a2[kB];
#pragma unroll
  for (int b = 0; b < kB; ++b) a0[b] = a1[b] = a2[b] = 0.f;
#pragma unroll
  for (int m = 0; m < kHalfBytes / 2; ++m) {
    const u4v e0 = *reinterpret_cast<const u4v*>(lut + code_addr(w, 2 * m, slot));
    const u4v e1 = *reinterpret_cast<const u4v*>(lut + code_addr(w, 2 * m + 1, slot));
    const uint32_t t4 = e0.z | e1.w;
#pragma unroll
    for (int b = 0; b < kB; ++b) {
      a0[b] = fdot2(e0.x, xr[b][5 * m], a0[b]);
      a1[b] = fdot2(e0.y, xr[b][5 * m + 1], a1[b]);
      a0[b] = fdot2(e1.x, xr[b][5 * m + 2], a0[b]);
      a1[b] = fdot2(e1.y, xr[b][5 * m + 3], a1[b]);
      a2[b] = fdot2(t4, xr[b][5 * m + 4], a2[b]);
    }
  }
  const U3 e = *reinterpret_cast<const U3*>(lut + code_addr(w, kHalfBytes, slot));
#pragma unroll
  for (int b = 0; b < kB; ++b) {
    a0[b] = fdot2(e.x, xr[b][30], a0[b]);
    a1[b] = fdot2(e.y, xr[b][31], a1[b]);
    a2[b] = fdot2(e.z, xr[b][32], a2[b]);
    out[b] = (a0[b] + a1[b]) + a2[b];
  }
}

// Activations of half h of group g from the LDS copy of x: 12 body bytes
// (inputs 60h + 5j ..) and the tail byte (inputs 120 + 5h ..); inputs past
// the group (pad digits) are zero.  Seven 16-byte reads, one 8-byte read for
// the body and two for the tail.
__device__ __attribute__((always_inline)) inline void load_xr(uint32_t (&xr)[kXrRegs], const uint32_t* xsw, int g,
                                                              int h) {
  typedef uint32_t u4v __attribute__((ext_vector_type(4)));
  typedef uint32_t u2v __attribute__((ext_vector_type(2)));
  const uint32_t* xg = xsw + kXStrideDw * g;
  const uint32_t* xd = xg + kXHalfDw * h;   // inputs 60 h ..
  uint32_t D[30];
#pragma unroll
  for (int q = 0; q < 7; ++q) {
    const u4v v = *reinterpret_cast<const u4v*>(xd + 4 * q);
    D[4 * q] = v.x;
    D[4 * q + 1] = v.y;
    D[4 * q + 2] = v.z;
    D[4 * q + 3] = v.w;
  }
  const u2v b = *reinterpret_cast<const u2v*>(xd + 28);
  D[28] = b.x;
  D[29] = b.y;
  const u2v t0 = *reinterpret_cast<const u2v*>(xg + kXTailDw);       // inputs 120..123
  const u2v t1 = *reinterpret_cast<const u2v*>(xg + kXTailDw + 2);   // inputs 124..127
#pragma unroll
  for (int m = 0; m < kHalfBytes / 2; ++m) {   // bytes 2m, 2m+1: inputs 10m .. 10m+9 = dwords 5m ..
    const uint32_t d2 = D[5 * m + 2], d3 = D[5 * m + 3], d4 = D[5 * m + 4];
    xr[5 * m] = D[5 * m];
    xr[5 * m + 1] = D[5 * m + 1];
    xr[5 * m + 2] = __builtin_amdgcn_alignbit(d3, d2, 16);
    xr[5 * m + 3] = __builtin_amdgcn_alignbit(d4, d3, 16);
    xr[5 * m + 4] = __builtin_amdgcn_perm(d4, d2, 0x07060100u);   // (low half of d2, high half of d4)
  }
  // Half 0: (x120, x121), (x122, x123), (x124, 0).  Half 1: (x125, x126),
  // (x127, 0), (0, 0).
  xr[30] = h ? __builtin_amdgcn_alignbit(t1.y, t1.x, 16) : t0.x;
  xr[31] = h ? t1.y >> 16 : t0.y;
  xr[32] = h ? 0u : t1.x & 0xFFFFu;
}

// One pass of plane 0 for one lane: 12 body bytes, 1 tail byte, 1 scale.
struct Pass {
  uint32_t w[4];   // w[0..2] body, w[3] tail byte
  uint32_t sc;     // scale bits
  uint32_t mu;     // per-group offset bits (with offsets)
};

// Byte offsets fit in 32 bits (the host rejects larger code buffers), so
// every address is a 64-bit base plus a zero-extended 32-bit offset.
template <bool kOffset0>
__device__ inline void load_pass(Pass& p, const uint8_t* body0, const uint8_t* tail0, const uint16_t* scale0,
                                 const uint16_t* offset0, uint32_t f) {
  const uint32_t* b = reinterpret_cast<const uint32_t*>(body0 + (size_t)(kMainBytes * f));
  p.w[0] = __builtin_nontemporal_load(b);
  p.w[1] = __builtin_nontemporal_load(b + 1);
  p.w[2] = __builtin_nontemporal_load(b + 2);
  p.w[3] = __builtin_nontemporal_load(tail0 + (size_t)(2 * f));
  p.sc = __builtin_nontemporal_load(scale0 + (size_t)f);
  if constexpr (kOffset0) p.mu = __builtin_nontemporal_load(offset0 + (size_t)f);
}

// Where a workgroup reads its records from.
struct RecSrc {
  const uint8_t* codes1;
  const uint16_t* gidx1;
  const uint16_t* offset1;
  const uint16_t* scale1;
  uint32_t nnz1;
};

// Half hh of a plane-1 record: 12 body bytes, its tail byte, and the
// record's group, offset and scale.
struct RecHalf {
  uint32_t w[4];   // w[0..2] body bytes 12 hh .., w[3] tail byte 24 + hh
  uint32_t g, mu, s1;
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

// Contribution of one record half: s1 * sum(t1 x) + mu * sum(x) over the
// half-group (the two halves together give mu * sum(x_g) + s1 * sum(t1 x_g)).
__device__ __attribute__((always_inline)) inline float record_half_value(const unsigned char* lut, uint32_t slot,
                                                                         const uint32_t* xsw, const RecHalf& r,
                                                                         int hh, int G) {
  uint32_t xr[kXrRegs];
  load_xr(xr, xsw, min((int)r.g, G - 1), hh);
  float s0 = 0.f, s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int i = 0; i < kXrRegs; i += 3) {
    s0 = fdot2(xr[i], 0x3C003C00u, s0);
    s1 = fdot2(xr[i + 1], 0x3C003C00u, s1);
    s2 = fdot2(xr[i + 2], 0x3C003C00u, s2);
  }
  const float xsum = (s0 + s1) + s2;
  const float p1 = code_dot(lut, slot, r.w, xr);
  return h2f(r.s1) * p1 + h2f(r.mu) * xsum;
}

// Wave priority for plane-0 pass d of n: high for early passes, falling to
// 0 for the last.  The CU issues for its oldest waves first, so without it
// the youngest waves of a workgroup start their passes last and finish
// long after the others, with fewer and fewer waves left to keep the LDS
// busy; by pass, the waves that are behind are served first.
template <int kPasses>
__device__ __attribute__((always_inline)) inline void pass_priority(int d) {
  switch ((kPasses - 1 - d) * 4 / kPasses) {
    case 3: __builtin_amdgcn_s_setprio(3); break;
    case 2: __builtin_amdgcn_s_setprio(2); break;
    case 1: __builtin_amdgcn_s_setprio(1); break;
    default: __builtin_amdgcn_s_setprio(0); break;
  }
}

// Sum of v over aligned segments of seg lanes (seg a power of two <= 64),
// exact in the last lane of each segment (and in every lane for seg <= 16).
// Butterflies inside 16-lane rows, then row broadcasts: a fixed order, so
// the result is bit-reproducible.
__device__ __attribute__((always_inline)) inline float segment_sum(float v, int seg) {
  auto shuffled = [](float a, int ctrl, int row_mask) -> float {
    const int x = __builtin_bit_cast(int, a);
    int r;
    switch (ctrl) {
      case 0: r = __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false); break;    // quad_perm [1,0,3,2]
      case 1: r = __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false); break;    // quad_perm [2,3,0,1]
      case 2: r = __builtin_amdgcn_update_dpp(0, x, 0x141, 0xF, 0xF, false); break;   // half-row mirror
      case 3: r = __builtin_amdgcn_update_dpp(0, x, 0x140, 0xF, 0xF, false); break;   // row mirror
      case 4: r = __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false); break;   // row_bcast:15 -> rows 1, 3
      default: r = __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false); break;  // row_bcast:31 -> rows 2, 3
    }
    (void)row_mask;
    return __builtin_bit_cast(float, r);
  };
  if (seg >= 2) v = v + shuffled(v, 0, 0xF);
  if (seg >= 4) v = v + shuffled(v, 1, 0xF);
  if (seg >= 8) v = v + shuffled(v, 2, 0xF);
  if (seg >= 16) v = v + shuffled(v, 3, 0xF);
  if (seg >= 32) v = v + shuffled(v, 4, 0xA);   // rows 1, 3: + the row before (lanes 31, 63 final for 32)
  if (seg >= 64) v = v + shuffled(v, 5, 0xC);   // rows 2, 3: + lane 31 (lane 63 final for 64)
  return v;
}

__device__ inline void store_y(void* y, int i, float v, int out_f32) {
  if (out_f32)
    reinterpret_cast<float*>(y)[i] = v;
  else
    reinterpret_cast<uint16_t*>(y)[i] = __builtin_bit_cast(uint16_t, (_Float16)v);
}
