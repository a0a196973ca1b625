// Lattice-code kernels: pack, unpack, validate and dense fp16 dequantisation.
//
// Paper: section 12 (the packed format persists the discrete supports and
// re-encodes them losslessly) and section 3, eq. 3 (the affine two-plane
// weight).  Code byte j of a group holds trits 5j..5j+4 as
// sum_i (t + 1) 3^i; bytes 0..23 of group f sit at 24 f, bytes 24..25 at
// 24 n + 2 f (the split layout declared in tq.h).
//
// These kernels move a few bytes per thread and are HBM-bound; each thread
// owns one code byte (pack, unpack, validate) or one 16-byte run of the
// dense output (unpack_fp16), so consecutive lanes touch consecutive bytes.

#include "tq_internal.h"

namespace tq {
namespace {

constexpr int kThreads = 256;
constexpr int64_t kMaxBlocks = 1 << 16;

__host__ __device__ inline int64_t grid_for(int64_t work) {
  int64_t b = (work + kThreads - 1) / kThreads;
  return b < 1 ? 1 : (b > kMaxBlocks ? kMaxBlocks : b);
}

// Group index and byte index of storage position `pos` in a buffer of n groups.
__device__ inline void locate(int64_t pos, int64_t n, int64_t& f, int& j) {
  int64_t main_bytes = (int64_t)kMainBytes * n;
  if (pos < main_bytes) {
    f = pos / kMainBytes;
    j = (int)(pos - f * kMainBytes);
  } else {
    int64_t q = pos - main_bytes;
    f = q >> 1;
    j = kMainBytes + (int)(q & 1);
  }
}

// Storage offset of byte j of group f in a buffer of n groups.
__device__ inline int64_t byte_offset(int64_t f, int j, int64_t n) {
  return j < kMainBytes ? f * kMainBytes + j : (int64_t)kMainBytes * n + 2 * f + (j - kMainBytes);
}

__device__ inline void count_error(int32_t* d_err, bool bad) {
  // One atomic per wave that saw errors (vector memory atomic).
  uint64_t m = __ballot(bad);
  if (m != 0 && d_err != nullptr) {
    int lane = __lane_id();
    int first = __builtin_ctzll(m);
    if (lane == first) atomicAdd(d_err, (int32_t)__popcll(m));
  }
}

__global__ void __launch_bounds__(kThreads) pack_kernel(const int8_t* __restrict__ trits, int64_t n,
                                                        uint8_t* __restrict__ codes, int32_t* d_err) {
  const int64_t total = (int64_t)kGroupBytes * n;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t base = (int64_t)blockIdx.x * kThreads; base < total; base += stride) {
    int64_t pos = base + threadIdx.x;
    bool bad = false;
    if (pos < total) {
      int64_t f;
      int j;
      locate(pos, n, f, j);
      const int8_t* t = trits + f * kGroup + 5 * j;
      int code = 0, mul = 1;
#pragma unroll
      for (int i = 0; i < 5; ++i) {
        int v = (5 * j + i < kGroup) ? (int)t[i] : 0;   // the two pad trits are 0
        bad |= (v < -1) | (v > 1);
        code += (v + 1) * mul;
        mul *= 3;
      }
      codes[pos] = bad ? (uint8_t)0xFF : (uint8_t)code;
    }
    count_error(d_err, bad);
  }
}

__global__ void __launch_bounds__(kThreads) unpack_kernel(const uint8_t* __restrict__ codes, int64_t n,
                                                          int8_t* __restrict__ trits, int32_t* d_err) {
  const int64_t total = (int64_t)kGroupBytes * n;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t base = (int64_t)blockIdx.x * kThreads; base < total; base += stride) {
    int64_t pos = base + threadIdx.x;
    bool bad = false;
    if (pos < total) {
      int64_t f;
      int j;
      locate(pos, n, f, j);
      int c = codes[pos];
      bad = c > 242;
      if (bad) c = 121;                      // five zero trits
      int8_t* t = trits + f * kGroup + 5 * j;
#pragma unroll
      for (int i = 0; i < 5; ++i) {
        if (5 * j + i < kGroup) t[i] = (int8_t)(c % 3 - 1);
        c /= 3;
      }
    }
    count_error(d_err, bad);
  }
}

__global__ void __launch_bounds__(kThreads) validate_kernel(const uint8_t* __restrict__ codes, int64_t n,
                                                            int32_t* d_err) {
  const int64_t total = (int64_t)kGroupBytes * n;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t base = (int64_t)blockIdx.x * kThreads; base < total; base += stride) {
    int64_t pos = base + threadIdx.x;
    bool bad = false;
    if (pos < total) {
      int64_t f;
      int j;
      locate(pos, n, f, j);
      int c = codes[pos];
      bad = c > 242;
      if (!bad && j == kGroupBytes - 1) bad = (c / 27) != 4;   // pad digits 3, 4 must be 1
    }
    count_error(d_err, bad);
  }
}

// Record index of (row r, group g) in the CSR of plane 1, or -1.
__device__ inline int64_t find_record(const MatDev& m, int64_t r, int g) {
  if (m.nnz1 == 0) return -1;
  int64_t lo = m.rowptr1[r], hi = m.rowptr1[r + 1];
  while (lo < hi) {
    int64_t mid = (lo + hi) >> 1;
    if ((int)m.gidx1[mid] < g) lo = mid + 1; else hi = mid;
  }
  return (lo < m.rowptr1[r + 1] && (int)m.gidx1[lo] == g) ? lo : -1;
}

__device__ inline float half_bits_to_float(uint16_t b) {
  return (float)__builtin_bit_cast(_Float16, b);
}

// One thread writes 8 consecutive fp16 weights (16 bytes) of one group.
__global__ void __launch_bounds__(kThreads) unpack_fp16_kernel(MatDev m, uint16_t* __restrict__ w) {
  const int64_t n = (int64_t)m.n_out * m.n_groups;
  const int64_t total = n * 16;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t id = (int64_t)blockIdx.x * kThreads + threadIdx.x; id < total; id += stride) {
    const int64_t f = id >> 4;
    const int c = (int)(id & 15);
    const int64_t r = f / m.n_groups;
    const int g = (int)(f - r * m.n_groups);
    const int64_t k = find_record(m, r, g);
    const float s0 = half_bits_to_float(m.scale0[f]);
    float mu = 0.f, s1 = 0.f;
    if (k >= 0) {
      mu = half_bits_to_float(m.offset1[k]);
      s1 = half_bits_to_float(m.scale1[k]);
    }
    const int p0 = 8 * c;
    const int j0 = p0 / 5;
    int b0[3], b1[3];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      int j = j0 + q;
      j = j < kGroupBytes ? j : kGroupBytes - 1;
      b0[q] = m.codes0[byte_offset(f, j, n)];
      b1[q] = k >= 0 ? m.codes1[byte_offset(k, j, m.nnz1)] : 121;
    }
    uint32_t outw[4];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int p = p0 + e;
      const int q = p / 5 - j0;
      const int d = p % 5;
      int c0 = b0[q], c1 = b1[q];
      for (int i = 0; i < d; ++i) { c0 /= 3; c1 /= 3; }
      const float t0 = (float)(c0 % 3 - 1);
      const float t1 = (float)(c1 % 3 - 1);
      float a = 0.0f;
      if (k >= 0) a = a + mu;
      a = a + s0 * t0;                  // s0*t0 is exact: one rounding
      if (k >= 0) a = a + s1 * t1;
      const uint16_t h = __builtin_bit_cast(uint16_t, (_Float16)a);   // RNE
      if (e & 1) outw[e >> 1] |= (uint32_t)h << 16; else outw[e >> 1] = h;
    }
    uint4 v;
    v.x = outw[0]; v.y = outw[1]; v.z = outw[2]; v.w = outw[3];
    reinterpret_cast<uint4*>(w)[id] = v;
  }
}

}  // namespace

hipError_t launch_pack(const int8_t* trits, int64_t n, uint8_t* codes, int32_t* d_err, hipStream_t s) {
  hipLaunchKernelGGL(pack_kernel, dim3((unsigned)grid_for(kGroupBytes * n)), dim3(kThreads), 0, s,
                     trits, n, codes, d_err);
  return hipGetLastError();
}

hipError_t launch_unpack(const uint8_t* codes, int64_t n, int8_t* trits, int32_t* d_err, hipStream_t s) {
  hipLaunchKernelGGL(unpack_kernel, dim3((unsigned)grid_for(kGroupBytes * n)), dim3(kThreads), 0, s,
                     codes, n, trits, d_err);
  return hipGetLastError();
}

hipError_t launch_validate(const uint8_t* codes, int64_t n, int32_t* d_err, hipStream_t s) {
  hipLaunchKernelGGL(validate_kernel, dim3((unsigned)grid_for(kGroupBytes * n)), dim3(kThreads), 0, s,
                     codes, n, d_err);
  return hipGetLastError();
}

hipError_t launch_unpack_fp16(const MatDev& m, uint16_t* w, hipStream_t s) {
  const int64_t work = (int64_t)m.n_out * m.n_groups * 16;
  hipLaunchKernelGGL(unpack_fp16_kernel, dim3((unsigned)grid_for(work)), dim3(kThreads), 0, s, m, w);
  return hipGetLastError();
}

}  // namespace tq
