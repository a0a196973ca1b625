// E2M-ATQ group ternarisation (gfx950): the step that produces the planes
// and scales the packed format stores.
//
// Paper: section 4.2 (E2M-ATQ), eqs. 4-6, for the representation of section
// 3, eq. 3.  Per 128-weight group:
//
// * one plane (no stored offset): T0 = +-1 where |w| exceeds 0.75 mean|w|,
//   s0 = <T0, w> / <T0, T0> (the least-squares scale, 0 on an empty
//   support);
// * two planes: mu = mean(w), T0 and s0 from w - mu as above, T1 and s1 from
//   the residual w - mu - s0 T0 the same way, then `iters` sweeps updating
//   mu, s0, s1 in turn with the supports fixed (block coordinate descent on
//   the squared error);
// * for every group, the residual energy ||w - s0 T0||^2 of the one-plane
//   fit, which ranks groups for the second plane;
// * with an offset on every group (the paper's own representation), the
//   one-plane fit also takes mu = mean(w), thresholds w - mu and refines mu
//   and s0; two-plane groups store their mu as the group's offset and 0 as
//   the record's.
//
// Two launches: every group's one-plane fit (and its energy), then the
// two-plane groups alone, one thread per record.  A thread owns one group
// and works in fp64 with every sum taken in index order 0..127, so each
// threshold decision and each stored value is a deterministic function of
// the group's 128 inputs.  Sums of 128 fp16 values
// and of their centred magnitudes are exact in fp64 for |w| < 2^10, so the
// plane-0 decisions do not depend on the summation order at all.  The stored
// mu, s0, s1 are rounded from fp64 to fp16 once, to nearest even.

#include "tq_internal.h"

// Products and sums are rounded as written: no fused multiply-add.
#pragma clang fp contract(off)

namespace tq {
namespace {

constexpr int kThreads = 128;
constexpr int64_t kMaxBlocks = 1 << 16;
constexpr double kThreshold = 0.75;

// fp64 -> fp16 bits, rounded once to nearest even (overflow to inf, NaN to
// the quiet NaN 0x7E00).
__device__ inline uint16_t f64_to_f16(double d) {
  const uint64_t b = __builtin_bit_cast(uint64_t, d);
  const uint32_t sign = (uint32_t)(b >> 48) & 0x8000u;
  const uint64_t a = b & 0x7FFFFFFFFFFFFFFFull;
  if (a >= 0x7FF0000000000000ull) return (uint16_t)(sign | (a > 0x7FF0000000000000ull ? 0x7E00u : 0x7C00u));
  if (a == 0) return (uint16_t)sign;
  int e = (int)(a >> 52) - 1023;
  uint64_t m = a & 0x000FFFFFFFFFFFFFull;
  if ((a >> 52) == 0) {   // fp64 subnormal: far below the fp16 range
    return (uint16_t)sign;
  }
  m |= 1ull << 52;                      // 53-bit significand, value m * 2^(e - 52)
  const int q = e < -14 ? -24 : e - 10; // fp16 quantum at this magnitude
  const int drop = q - (e - 52);        // significand bits below the quantum
  if (drop > 53) return (uint16_t)sign; // below half the smallest subnormal
  uint64_t sig = m >> drop;
  const uint64_t rem = m & ((1ull << drop) - 1);
  const uint64_t half = 1ull << (drop - 1);
  if (rem > half || (rem == half && (sig & 1))) ++sig;
  uint32_t bits;
  if (q == -24) {
    bits = (uint32_t)sig;               // subnormal (1024 reads as the smallest normal)
  } else {
    bits = ((uint32_t)(e + 15) << 10) + (uint32_t)(sig - 1024);   // sig == 2048 carries into the exponent
  }
  if (bits >= 0x7C00u) bits = 0x7C00u;
  return (uint16_t)(sign | bits);
}

__device__ inline double h2d(uint32_t bits) { return (double)__builtin_bit_cast(_Float16, (uint16_t)bits); }

// A thread's group lives in LDS transposed, element i of thread t at
// [i * kThreads + t], so the lanes of a wave touch consecutive addresses:
// the fp16 weights and the int8 trits of both supports.
struct GroupView {
  const uint16_t* w;
  int8_t* t0;
  int8_t* t1;
  int tid;
  __device__ double wat(int i) const { return h2d(w[i * kThreads + tid]); }
  __device__ double t0at(int i) const { return (double)t0[i * kThreads + tid]; }
  __device__ double t1at(int i) const { return (double)t1[i * kThreads + tid]; }
};

__device__ inline int8_t threshold(double v, double delta) { return v > delta ? 1 : (v < -delta ? -1 : 0); }

__device__ inline double ls_ratio(double num, int n) { return n > 0 ? num / (double)n : 0.0; }

// Writes 128 int8 trits (16-byte aligned destination) from the transposed
// LDS copy.
__device__ inline void store_trits(int8_t* dst, const int8_t* t, int tid) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    uint32_t wds[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      uint32_t v = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) v |= (uint32_t)(uint8_t)t[(16 * c + 4 * k + b) * kThreads + tid] << (8 * b);
      wds[k] = v;
    }
    reinterpret_cast<uint4*>(dst)[c] = make_uint4(wds[0], wds[1], wds[2], wds[3]);
  }
}

// Loads group f into this thread's LDS column.
__device__ inline void load_group(uint16_t* w_s, const uint16_t* __restrict__ w, int64_t f, int tid) {
  const uint4* src = reinterpret_cast<const uint4*>(w + f * kGroup);
#pragma unroll
  for (int c = 0; c < 16; ++c) {
    const uint4 v = src[c];
    const uint32_t d[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 8; ++k) w_s[(8 * c + k) * kThreads + tid] = (uint16_t)(d[k >> 1] >> (16 * (k & 1)));
  }
}

// Pass 1, every group: the one-plane fit (stored for one-plane groups) and
// its residual energy.  A two-plane group instead leaves its own index in
// the first 8 bytes of its record's t1 row, which pass 2 reads and then
// overwrites, so pass 2 can run over the records alone (no wave then mixes
// the two fits).
__global__ void __launch_bounds__(kThreads) one_plane_kernel(const uint16_t* __restrict__ w, int64_t n,
                                                             const int32_t* __restrict__ rec_index, int64_t nnz,
                                                             int iters, int8_t* __restrict__ t0_out,
                                                             uint16_t* __restrict__ s0_out, int8_t* __restrict__ t1_out,
                                                             uint16_t* __restrict__ off0_out,
                                                             double* __restrict__ energy_out) {
  __shared__ uint16_t w_s[kGroup * kThreads];
  __shared__ int8_t t0_s[kGroup * kThreads];
  const int tid = threadIdx.x;
  const GroupView g{w_s, t0_s, nullptr, tid};
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  // Threads share no LDS data (each reads back only its own column), so no
  // barrier is needed.
  for (int64_t f = (int64_t)blockIdx.x * kThreads + tid; f < n; f += stride) {
    load_group(w_s, w, f, tid);
    int64_t k = rec_index != nullptr ? (int64_t)rec_index[f] : -1;
    if (k >= nnz) k = -1;
    // Without group offsets mu stays 0 (the raw weights are thresholded);
    // with them mu starts at the mean and is refined with s0.
    double mu = 0.0;
    if (off0_out != nullptr) {
      double sw = 0.0;
      for (int i = 0; i < kGroup; ++i) sw = sw + g.wat(i);
      mu = sw / kGroup;
    }
    const double mu_c = mu;
    double sabs = 0.0;
    for (int i = 0; i < kGroup; ++i) sabs = sabs + fabs(g.wat(i) - mu_c);
    const double delta = kThreshold * (sabs / kGroup);
    int n_one = 0;
    double num = 0.0;
    for (int i = 0; i < kGroup; ++i) {
      const double v = g.wat(i) - mu_c;
      const int8_t t = threshold(v, delta);
      t0_s[i * kThreads + tid] = t;
      n_one += t != 0;
      num = num + (double)t * v;
    }
    double s0_one = ls_ratio(num, n_one);
    if (off0_out != nullptr) {
      for (int it = 0; it < iters; ++it) {
        double a = 0.0;
        for (int i = 0; i < kGroup; ++i) a = a + (g.wat(i) - s0_one * g.t0at(i));
        mu = a / kGroup;
        double b = 0.0;
        for (int i = 0; i < kGroup; ++i) b = b + g.t0at(i) * (g.wat(i) - mu);
        s0_one = ls_ratio(b, n_one);
      }
    }
    if (energy_out != nullptr) {
      double e = 0.0;
      for (int i = 0; i < kGroup; ++i) {
        const double d = (g.wat(i) - mu) - s0_one * g.t0at(i);
        e = e + d * d;
      }
      energy_out[f] = e;
    }
    if (k < 0) {
      store_trits(t0_out + f * kGroup, t0_s, tid);
      s0_out[f] = f64_to_f16(s0_one);
      if (off0_out != nullptr) off0_out[f] = f64_to_f16(mu);
    } else {
      *reinterpret_cast<int64_t*>(t1_out + k * kGroup) = f;
    }
  }
}

// Pass 2, one thread per record: the two-plane fit of the group that named
// it (a record no group names, or one named twice, is skipped).
__global__ void __launch_bounds__(kThreads) two_plane_kernel(const uint16_t* __restrict__ w, int64_t n,
                                                             const int32_t* __restrict__ rec_index, int64_t nnz,
                                                             int iters, int8_t* __restrict__ t0_out,
                                                             uint16_t* __restrict__ s0_out, int8_t* __restrict__ t1_out,
                                                             uint16_t* __restrict__ mu_out, uint16_t* __restrict__ s1_out,
                                                             uint16_t* __restrict__ off0_out) {
  __shared__ uint16_t w_s[kGroup * kThreads];
  __shared__ int8_t t0_s[kGroup * kThreads];
  __shared__ int8_t t1_s[kGroup * kThreads];
  const int tid = threadIdx.x;
  const GroupView g{w_s, t0_s, t1_s, tid};
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t k = (int64_t)blockIdx.x * kThreads + tid; k < nnz; k += stride) {
    const int64_t f = *reinterpret_cast<const int64_t*>(t1_out + k * kGroup);
    if (f < 0 || f >= n || (int64_t)rec_index[f] != k) continue;
    load_group(w_s, w, f, tid);

    // Offset, centred first support, residual second support.
    double sw = 0.0;
    for (int i = 0; i < kGroup; ++i) sw = sw + g.wat(i);
    double mu = sw / kGroup;
    const double mu_c = mu;
    double sc = 0.0;
    for (int i = 0; i < kGroup; ++i) sc = sc + fabs(g.wat(i) - mu_c);
    const double delta0 = kThreshold * (sc / kGroup);
    int c0 = 0;
    double n0 = 0.0;
    for (int i = 0; i < kGroup; ++i) {
      const double v = g.wat(i) - mu_c;
      const int8_t t = threshold(v, delta0);
      t0_s[i * kThreads + tid] = t;
      c0 += t != 0;
      n0 = n0 + (double)t * v;
    }
    double s0 = ls_ratio(n0, c0);
    const double s0_c = s0;
    double sr = 0.0;
    for (int i = 0; i < kGroup; ++i) sr = sr + fabs((g.wat(i) - mu_c) - s0_c * g.t0at(i));
    const double delta1 = kThreshold * (sr / kGroup);
    int c1 = 0;
    double n1 = 0.0;
    for (int i = 0; i < kGroup; ++i) {
      const double v = (g.wat(i) - mu_c) - s0_c * g.t0at(i);
      const int8_t t = threshold(v, delta1);
      t1_s[i * kThreads + tid] = t;
      c1 += t != 0;
      n1 = n1 + (double)t * v;
    }
    double s1 = ls_ratio(n1, c1);
    // Refinement with the supports fixed.
    for (int it = 0; it < iters; ++it) {
      double a = 0.0;
      for (int i = 0; i < kGroup; ++i) a = a + ((g.wat(i) - s0 * g.t0at(i)) - s1 * g.t1at(i));
      mu = a / kGroup;
      double b = 0.0;
      for (int i = 0; i < kGroup; ++i) b = b + g.t0at(i) * ((g.wat(i) - mu) - s1 * g.t1at(i));
      s0 = ls_ratio(b, c0);
      double c = 0.0;
      for (int i = 0; i < kGroup; ++i) c = c + g.t1at(i) * ((g.wat(i) - mu) - s0 * g.t0at(i));
      s1 = ls_ratio(c, c1);
    }
    store_trits(t0_out + f * kGroup, t0_s, tid);
    s0_out[f] = f64_to_f16(s0);
    store_trits(t1_out + k * kGroup, t1_s, tid);
    if (off0_out != nullptr) {   // the offset belongs to the group; the record's is 0
      off0_out[f] = f64_to_f16(mu);
      mu_out[k] = 0;
    } else {
      mu_out[k] = f64_to_f16(mu);
    }
    s1_out[k] = f64_to_f16(s1);
  }
}

}  // namespace

hipError_t launch_ternarize(const uint16_t* w, int64_t n, const int32_t* rec_index, int64_t nnz, int iters,
                            int8_t* t0, uint16_t* s0, int8_t* t1, uint16_t* mu, uint16_t* s1, uint16_t* off0,
                            double* energy, hipStream_t s) {
  auto blocks_for = [](int64_t work) {
    const int64_t b = (work + kThreads - 1) / kThreads;
    return (unsigned)(b < 1 ? 1 : (b > kMaxBlocks ? kMaxBlocks : b));
  };
  const bool two = rec_index != nullptr && nnz > 0;
  hipLaunchKernelGGL(one_plane_kernel, dim3(blocks_for(n)), dim3(kThreads), 0, s, w, n, two ? rec_index : nullptr,
                     two ? nnz : 0, iters, t0, s0, t1, off0, energy);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !two) return e;
  hipLaunchKernelGGL(two_plane_kernel, dim3(blocks_for(nnz)), dim3(kThreads), 0, s, w, n, rec_index, nnz, iters, t0,
                     s0, t1, mu, s1, off0);
  return hipGetLastError();
}

}  // namespace tq
