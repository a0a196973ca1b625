// Small-batch packed GEMM Y = X W^T on LDS-decoded tiles with MFMA (gfx950).
//
// Paper: section 3, eq. 3 (the weight), section 18 (kernel work across
// shapes and batch sizes is the stated next step).  For a batch of B
// activation rows the product is a genuine dense contraction, so each
// 128-wide K step is decoded once into an fp16 tile in LDS and consumed by
// v_mfma_f32_16x16x32_f16 for every 16-column slice of the batch.
//
// Tile layout ("slot" order).  MFMA sums over k in any order, so a K step is
// laid out per code byte: byte j of a group fills slots 6j .. 6j+5 with the
// weights of inputs 5j .. 5j+4 and one zero slot; 26 bytes give 156 slots,
// padded to 160 = 5 MFMA k-steps.  The X tile uses the same slot order (x of
// input 5j+i at slot 6j+i, zero at every pad slot), so pad slots contribute
// nothing.  Rows are 168 halves apart (336 bytes) so that the 16 rows read by
// one MFMA operand load land on 16 different bank quads.
//
// Weights: one-plane groups decode to s0 * t exactly (fp16 pattern times the
// scale with v_pk_mul_f16); two-plane groups are evaluated in fp32 as
// ((0 + mu) + s0 t0) + s1 t1 and rounded once to fp16.

#include "tq_internal.h"

namespace tq {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kRows = 16 * kWaves;      // W rows per workgroup
constexpr int kSlots = 160;             // k slots per 128-wide step
constexpr int kStride = 168;            // LDS row stride in halves
constexpr int kMaxColTiles = TQ_MAX_BATCH / 16;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float float4v __attribute__((ext_vector_type(4)));

__device__ inline uint32_t trit_pattern(int t) {
  return t > 0 ? 0x3C00u : (t < 0 ? 0xBC00u : 0u);
}

__device__ inline float h2f(uint16_t b) { return (float)__builtin_bit_cast(_Float16, b); }

__device__ inline int64_t byte_offset(int64_t f, int j, int64_t n) {
  return j < kMainBytes ? f * kMainBytes + j : (int64_t)kMainBytes * n + 2 * f + (j - kMainBytes);
}

__global__ void __launch_bounds__(kThreads) gemm_kernel(MatDev m, const uint16_t* __restrict__ X, int B,
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
        if (k < 0) {
          const half2v s2 = {__builtin_bit_cast(_Float16, s0b), __builtin_bit_cast(_Float16, s0b)};
          o0 = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, p.x) * s2);
          o1 = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, p.y) * s2);
          o2 = __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2v, p.z) * s2);
        } else {
          const int c1 = m.codes1[byte_offset(k, j, m.nnz1)];
          const float s0 = h2f(s0b), mu = h2f(m.offset1[k]), s1 = h2f(m.scale1[k]);
          int d0 = c0, d1 = c1;
          uint16_t h[5];
#pragma unroll
          for (int i = 0; i < 5; ++i) {
            float a = 0.0f;
            a = a + mu;
            a = a + s0 * (float)(d0 % 3 - 1);
            a = a + s1 * (float)(d1 % 3 - 1);
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

}  // namespace

hipError_t launch_gemm_smallbatch(const MatDev& m, const uint16_t* X, int B, void* Y, bool out_f32,
                                  hipStream_t s) {
  const int wgs = (m.n_out + kRows - 1) / kRows;
  hipLaunchKernelGGL(gemm_kernel, dim3(wgs), dim3(kThreads), 0, s, m, X, B, Y, out_f32 ? 1 : 0);
  return hipGetLastError();
}

}  // namespace tq
