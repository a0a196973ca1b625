// Packed ternary GEMV y = W^ x for gfx950 (batch 1), and its grouped form.
//
// Paper: section 3, eq. 3 (W^ = (mu + a0 T0 + a1 T1) (.) M, T_i in
// {-1, 0, +1}; per-group offsets/scales on a salience-selected subset), A16
// activations (section 3), packed supports (section 12).  The paper's own
// kernel (section 13) is a prototype for another GPU and gives no design;
// this one is built for CDNA4:
//
// * Lane ownership.  A workgroup of T threads covers RI = T / G rows per
//   pass; thread t always owns group column g = t % G, so the 128
//   activations of its group live in 78 VGPRs for the whole launch, laid out
//   per code byte j as the fp16 pairs (x5j, x5j+1), (x5j+2, x5j+3),
//   (x5j+4, 0).
// * Decode.  A 256-entry table maps a code byte to the same three pairs of
//   fp16 patterns (+1 = 0x3C00, -1 = 0xBC00, 0 = 0); three v_dot2_f32_f16
//   then accumulate the sign-selected activations in fp32.  The table is
//   replicated 16 times in LDS, copy q at byte offset 16 q of every 256-byte
//   row, and lane t reads copy t % 16: the 16 lanes served together always
//   hit 16 different bank quads, whatever codes they hold.
// * Loads.  Group bodies (24 bytes, 8-aligned) arrive as three dwordx2
//   loads, the two tail bytes as one ushort, the scale as one ushort; lanes
//   of a row read consecutive groups, so every wave load is contiguous.
// * Plane 1.  After the plane-0 pass over a block of rows has written
//   s0 * p0 for every (row, group) into LDS, the block's two-plane records
//   are processed densely (one record per thread) and each adds
//   mu * sum(x_g) + s1 * sum(t1 * x_g) to its own (row, group) slot.
// * Reduction.  Each row's G partials are summed by one wave: a fixed
//   strided sum per lane, then an xor butterfly of ds_swizzle steps and a
//   cross-half readlane.  No atomics: results are bit-identical run to run.

#include "tq_internal.h"

namespace tq {
namespace {

constexpr int kRep = 16;                       // LUT copies (one per bank quad)
constexpr int kLutEntries = 256 * kRep;        // 16-byte entries
constexpr int kLutBytes = kLutEntries * 16;    // 64 KiB
constexpr int kMaxThreads = 512;

struct GemvParams {
  MatDev m[TQ_MAX_GROUPED];
  void* y[TQ_MAX_GROUPED];
  int32_t wg_begin[TQ_MAX_GROUPED + 1];
  int32_t rows_per_wg;
  int32_t n_mats;
  int32_t G;        // groups per row, shared by all matrices
  int32_t ri;       // rows per pass = T / G
  int32_t rb_max;   // rows per LDS block
  int32_t out_f32;
};

struct __attribute__((aligned(16))) U3 {
  uint32_t x, y, z;
};

__device__ inline uint32_t trit_pattern(int t) {
  return t > 0 ? 0x3C00u : (t < 0 ? 0xBC00u : 0u);
}

// Entry e = code * kRep + copy, 16 bytes each: byte address code*256 + copy*16.
__device__ inline void build_lut(uint4* lut, int tid, int nthreads) {
  for (int e = tid; e < kLutEntries; e += nthreads) {
    const int code = e / kRep;
    uint4 v = {0u, 0u, 0u, 0u};
    if (code < 243) {
      int c = code, t[5];
#pragma unroll
      for (int i = 0; i < 5; ++i) {
        t[i] = c % 3 - 1;
        c /= 3;
      }
      v.x = trit_pattern(t[0]) | (trit_pattern(t[1]) << 16);
      v.y = trit_pattern(t[2]) | (trit_pattern(t[3]) << 16);
      v.z = trit_pattern(t[4]);
    }
    lut[e] = v;
  }
}

__device__ inline float fdot2(uint32_t a, uint32_t b, float c) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(h2, a), __builtin_bit_cast(h2, b), c, false);
}

__device__ inline float h2f(uint16_t b) { return (float)__builtin_bit_cast(_Float16, b); }

// Sum over the 64 lanes of a wave; every lane returns the same value.
__device__ inline float wave_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x041F));
  v += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x081F));
  v += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x101F));
  v += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x201F));
  v += __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x401F));
  const float lo = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
  const float hi = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
  return lo + hi;
}

// Code byte j (0..25) of a group whose body dwords are w[0..5] and whose two
// tail bytes are the low half of w[6].
__device__ inline uint32_t code_of(const uint32_t (&w)[7], int j) {
  return (w[j >> 2] >> (8 * (j & 3))) & 0xFFu;
}

// Dot product of one group's trits (code dwords w) with activations laid
// out as three fp16 pairs per code byte.
template <typename XPairs>
__device__ __attribute__((always_inline)) inline float group_dot(const unsigned char* lut_bytes, uint32_t slot16,
                                  const uint32_t (&w)[7], XPairs xp) {
  float a0 = 0.f, a1 = 0.f, a2 = 0.f;
#pragma unroll
  for (int j = 0; j < kGroupBytes; ++j) {
    const uint32_t addr = (code_of(w, j) << 8) | slot16;
    const U3 p = *reinterpret_cast<const U3*>(lut_bytes + addr);
    a0 = fdot2(p.x, xp(j, 0), a0);
    a1 = fdot2(p.y, xp(j, 1), a1);
    a2 = fdot2(p.z, xp(j, 2), a2);
  }
  return (a0 + a1) + a2;
}

__device__ inline void load_group(const uint8_t* body, const uint8_t* tail, uint32_t (&w)[7]) {
  const uint2* b = reinterpret_cast<const uint2*>(body);
  const uint2 w0 = b[0], w1 = b[1], w2 = b[2];
  w[0] = w0.x; w[1] = w0.y; w[2] = w1.x; w[3] = w1.y; w[4] = w2.x; w[5] = w2.y;
  w[6] = *reinterpret_cast<const uint16_t*>(tail);
}

__global__ void __launch_bounds__(kMaxThreads) gemv_kernel(const GemvParams P, const uint16_t* __restrict__ x) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int G = P.G;
  const int K = G * kGroup;
  unsigned char* lut_bytes = smem;
  uint16_t* xs = reinterpret_cast<uint16_t*>(smem + kLutBytes);
  float* gsum = reinterpret_cast<float*>(smem + kLutBytes + 2 * K);
  int* rp = reinterpret_cast<int*>(gsum + G);
  float* part = reinterpret_cast<float*>(rp + P.rb_max + 1);

  const int tid = threadIdx.x;
  const int T = blockDim.x;

  // Which matrix this workgroup serves (constant indices only, so the
  // parameter block is never copied to scratch).
  int mi = 0;
#pragma unroll
  for (int i = 1; i < TQ_MAX_GROUPED; ++i)
    if (i < P.n_mats && (int)blockIdx.x >= P.wg_begin[i]) mi = i;
  MatDev M = P.m[0];
  void* yp = P.y[0];
  int wgb = P.wg_begin[0];
#pragma unroll
  for (int i = 1; i < TQ_MAX_GROUPED; ++i)
    if (i == mi) {
      M = P.m[i];
      yp = P.y[i];
      wgb = P.wg_begin[i];
    }
  const int row_begin = ((int)blockIdx.x - wgb) * P.rows_per_wg;
  const int row_end = min(M.n_out, row_begin + P.rows_per_wg);

  // Stage x and the decode table.
  for (int i = tid; i < K / 8; i += T)
    reinterpret_cast<uint4*>(xs)[i] = reinterpret_cast<const uint4*>(x)[i];
  build_lut(reinterpret_cast<uint4*>(lut_bytes), tid, T);
  __syncthreads();
  for (int g = tid; g < G; g += T) {
    float s = 0.f;
    for (int i = 0; i < kGroup; ++i) s += h2f(xs[kGroup * g + i]);
    gsum[g] = s;
  }

  const int ri = P.ri;
  const bool active = tid < ri * G;
  const int g = active ? tid % G : 0;
  const int rl = active ? tid / G : 0;
  const uint32_t slot16 = (uint32_t)(tid & (kRep - 1)) << 4;

  // This thread's activations as three fp16 pairs per code byte.
  uint32_t xr[kGroupBytes][3];
  {
    const uint16_t* xg = xs + kGroup * g;
#pragma unroll
    for (int j = 0; j < kGroupBytes; ++j) {
#pragma unroll
      for (int q = 0; q < 3; ++q) {
        const int p = 5 * j + 2 * q;
        const uint32_t lo = p < kGroup ? xg[p] : 0u;
        const uint32_t hi = (q < 2 && p + 1 < kGroup) ? xg[p + 1] : 0u;
        xr[j][q] = lo | (hi << 16);
      }
    }
  }
  __syncthreads();

  const int64_t ngroups = (int64_t)M.n_out * G;
  const uint8_t* tails0 = M.codes0 + (int64_t)kMainBytes * ngroups;
  const uint8_t* tails1 = M.codes1 + (int64_t)kMainBytes * M.nnz1;

  for (int rb0 = row_begin; rb0 < row_end; rb0 += P.rb_max) {
    const int rb1 = min(row_end, rb0 + P.rb_max);
    const int nrb = rb1 - rb0;

    // Plane 0: part[row][g] = s0 * sum_i t0 x.
    if (active) {
      for (int r = rb0 + rl; r < rb1; r += ri) {
        const int64_t f = (int64_t)r * G + g;
        uint32_t w[7];
        load_group(M.codes0 + (int64_t)kMainBytes * f, tails0 + 2 * f, w);
        const float s0 = h2f(M.scale0[f]);
        const float p = group_dot(lut_bytes, slot16, w, [&](int j, int q) { return xr[j][q]; });
        part[(r - rb0) * G + g] = p * s0;
      }
    }

    // Plane 1: one record per thread, added to its own (row, group) slot.
    if (M.nnz1 > 0) {
      for (int i = tid; i <= nrb; i += T) rp[i] = M.rowptr1[rb0 + i];
      __syncthreads();
      // Clamped so that a malformed CSR cannot index outside the buffers.
      const int k0 = max(rp[0], 0);
      const int k1 = (int)min((int64_t)rp[nrb], M.nnz1);
      for (int k = k0 + tid; k < k1; k += T) {
        int lo = 0, hi = nrb - 1;   // last row whose first record is <= k
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (rp[mid] <= k) lo = mid; else hi = mid - 1;
        }
        const int gg = min((int)M.gidx1[k], G - 1);
        uint32_t w[7];
        load_group(M.codes1 + (int64_t)kMainBytes * k, tails1 + 2 * (int64_t)k, w);
        const float mu = h2f(M.offset1[k]);
        const float s1 = h2f(M.scale1[k]);
        const uint16_t* xg = xs + kGroup * gg;
        const float p1 = group_dot(lut_bytes, slot16, w, [&](int j, int q) {
          const int p = 5 * j + 2 * q;
          const uint32_t lo2 = p < kGroup ? xg[p] : 0u;
          const uint32_t hi2 = (q < 2 && p + 1 < kGroup) ? xg[p + 1] : 0u;
          return lo2 | (hi2 << 16);
        });
        float* slot = part + lo * G + gg;
        *slot = *slot + (mu * gsum[gg] + s1 * p1);
      }
    }
    __syncthreads();

    // Row sums: one wave per row.
    const int lane = tid & 63;
    const int nw = T >> 6;
    for (int rr = tid >> 6; rr < nrb; rr += nw) {
      float s = 0.f;
      for (int q = lane; q < G; q += 64) s += part[rr * G + q];
      s = wave_sum(s);
      if (lane == 0) {
        if (P.out_f32)
          reinterpret_cast<float*>(yp)[rb0 + rr] = s;
        else
          reinterpret_cast<uint16_t*>(yp)[rb0 + rr] = __builtin_bit_cast(uint16_t, (_Float16)s);
      }
    }
    __syncthreads();
  }
}

struct DeviceInfo {
  int cus = 0;
  bool attr_set = false;
};

DeviceInfo& device_info() {
  static thread_local DeviceInfo info[64];
  int dev = 0;
  (void)hipGetDevice(&dev);
  return info[dev & 63];
}

size_t lds_bytes(int G, int rb_max) {
  const int K = G * kGroup;
  return (size_t)kLutBytes + 2 * (size_t)K + 4 * (size_t)G + 4 * (size_t)(rb_max + 1) +
         4 * (size_t)rb_max * G;
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
  if (!di.attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(gemv_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e != hipSuccess) return e;
    di.attr_set = true;
  }

  GemvParams P = {};
  const int G = ms[0].n_groups;
  // Threads per workgroup: the multiple of 64 in [256, 512] that leaves the
  // fewest lanes without a group column.
  int T = 256, best_used = -1;
  for (int t = 256; t <= kMaxThreads; t += 64) {
    const int used = (t / G) * G;
    if (used * (int64_t)T > (int64_t)best_used * t) {
      best_used = used;
      T = t;
    }
  }
  const int ri = T / G;
  int64_t total_rows = 0;
  for (int i = 0; i < n; ++i) total_rows += ms[i].n_out;

  // LDS block: as many rows as fit beside the fixed arrays, preferring two
  // workgroups per CU when they fit.
  const size_t fixed = lds_bytes(G, 0);
  const size_t per_row = 4 * (size_t)G + 4;
  const size_t two_per_cu = 80 * 1024, one_per_cu = 160 * 1024;
  const int wgs_per_cu = fixed + per_row * ri <= two_per_cu ? 2 : 1;
  const size_t budget = wgs_per_cu == 2 ? two_per_cu : one_per_cu;
  const int target_wgs = di.cus * wgs_per_cu;
  int rows_per_wg = (int)((total_rows + target_wgs - 1) / target_wgs);
  rows_per_wg = ((rows_per_wg + ri - 1) / ri) * ri;
  int rb_max = (int)((budget - fixed) / per_row);
  rb_max = rb_max / ri * ri;
  if (rb_max < ri) rb_max = ri;
  if (rb_max > rows_per_wg) rb_max = rows_per_wg;

  int wg = 0;
  for (int i = 0; i < n; ++i) {
    P.m[i] = ms[i];
    P.y[i] = ys[i];
    P.wg_begin[i] = wg;
    wg += (ms[i].n_out + rows_per_wg - 1) / rows_per_wg;
  }
  P.wg_begin[n] = wg;
  P.rows_per_wg = rows_per_wg;
  P.n_mats = n;
  P.G = G;
  P.ri = ri;
  P.rb_max = rb_max;
  P.out_f32 = out_f32 ? 1 : 0;
  hipLaunchKernelGGL(gemv_kernel, dim3(wg), dim3(T), lds_bytes(G, rb_max), s, P, x);
  return hipGetLastError();
}

}  // namespace tq
