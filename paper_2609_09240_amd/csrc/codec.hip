// Lattice-code kernels: pack, unpack, validate and dense fp16 dequantisation.
//
// Paper: section 12 (the packed format persists the discrete supports and
// re-encodes them losslessly) and section 3, eq. 3 (the affine two-plane
// weight).  Code byte j of a group holds trits 5j..5j+4 as
// sum_i (t + 1) 3^i; bytes 0..23 of group f sit at 24 f, bytes 24..25 at
// 24 n + 2 f (the split layout declared in tq.h).
//
// All of these are HBM-bound streams.  Pack and unpack give each group three
// threads (part p owns main code bytes 8p..8p+7, part 2 also the two tail
// bytes), so every thread moves 8 code bytes and 40-48 trit bytes with vector
// loads and stores and consecutive lanes touch consecutive memory.  A trit
// buffer that is not 16-byte aligned takes a one-byte-per-thread kernel.
// Validate reads the code buffer in flat 16-byte chunks.  The fp16
// dequantisation stages blocks of rows in LDS with coalesced loads, gives
// each thread 8-weight items and writes them with 16-byte nontemporal stores;
// persistent workgroups load the next block while storing the current one.

#include <type_traits>

#include "tq_internal.h"

namespace tq {
namespace {

constexpr int64_t kMaxBlocks = 1 << 16;

constexpr int kPartThreads = 192;   // three threads per group
constexpr int kPartGroups = 64;     // groups per workgroup pass
constexpr int kPartMaxBlocks = 2048;

constexpr int kByteThreads = 256;


inline int64_t clamp_blocks(int64_t b, int64_t cap) { return b < 1 ? 1 : (b > cap ? cap : b); }

// Adds the wave's number of bad bytes to *d_err: one vector atomic per wave
// that saw any.  Every lane of the wave must call it.
__device__ inline void count_errors(int32_t* d_err, int nbad) {
  if (d_err == nullptr || __ballot(nbad != 0) == 0) return;
  for (int off = 32; off > 0; off >>= 1) nbad += __shfl_xor(nbad, off);
  if (__lane_id() == 0) atomicAdd(d_err, nbad);
}

// ---------------------------------------------------------------------------
// Pack.
// ---------------------------------------------------------------------------

// Signed trit byte b of a little-endian word array.
__device__ inline int trit_at(const uint32_t* w, int b) { return (int)(int8_t)(w[b >> 2] >> (8 * (b & 3))); }

// Code of the trits w[b .. b+nt-1] (digits nt..4 are pad zeros, digit 1);
// 0xFF and one bad byte if any trit is outside {-1, 0, +1}.
__device__ inline uint32_t encode(const uint32_t* w, int b, int nt, int& nbad) {
  uint32_t code = 0, top = 0;
#pragma unroll
  for (int k = 4; k >= 0; --k) {
    const uint32_t u = k < nt ? (uint32_t)(trit_at(w, b + k) + 1) : 1u;
    top = u > top ? u : top;
    code = code * 3u + u;
  }
  const bool bad = top > 2u;
  nbad += bad;
  return bad ? 0xFFu : code;
}

__global__ void __launch_bounds__(kPartThreads) pack_kernel(const int8_t* __restrict__ trits, int64_t n,
                                                            uint8_t* __restrict__ codes, int32_t* d_err) {
  const int part = threadIdx.x % 3;
  const int slot = threadIdx.x / 3;
  const int first = part == 0 ? 0 : (part == 1 ? 32 : 80);   // first trit loaded (16-byte aligned)
  for (int64_t base = (int64_t)blockIdx.x * kPartGroups; base < n; base += (int64_t)gridDim.x * kPartGroups) {
    const int64_t f = base + slot;
    int nbad = 0;
    if (f < n) {
      const uint4* src = reinterpret_cast<const uint4*>(trits + f * kGroup + first);
      const uint4 a = src[0], b = src[1], c = src[2];
      const uint32_t raw[12] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w, c.x, c.y, c.z, c.w};
      // Trit 40*part at w[0]: part 1 loaded from trit 32, two words early.
      uint32_t w[12];
#pragma unroll
      for (int d = 0; d < 10; ++d) w[d] = part == 1 ? raw[d + 2] : raw[d];
      w[10] = raw[10];
      w[11] = raw[11];
      uint32_t out[2] = {0u, 0u};
#pragma unroll
      for (int i = 0; i < 8; ++i) out[i >> 2] |= encode(w, 5 * i, 5, nbad) << (8 * (i & 3));
      *reinterpret_cast<uint2*>(codes + 24 * f + 8 * part) = make_uint2(out[0], out[1]);
      if (part == 2) {   // bytes 24 and 25: trits 120..124 and 125..127
        const uint32_t c24 = encode(w, 40, 5, nbad), c25 = encode(w, 45, 3, nbad);
        *reinterpret_cast<uint16_t*>(codes + (int64_t)kMainBytes * n + 2 * f) = (uint16_t)(c24 | (c25 << 8));
      }
    }
    count_errors(d_err, nbad);
  }
}

// ---------------------------------------------------------------------------
// Unpack.
// ---------------------------------------------------------------------------

// The five trit bytes (t as int8) of a code, bytes 0..3 in .x and 4 in .y;
// codes above 242 decode to five zeros.  (c * 171) >> 9 == c / 3 for c < 256.
__device__ inline uint2 trit_bytes(int c) {
  if (c > 242) c = 121;
  uint32_t lo = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int q = (c * 171) >> 9;
    lo |= (uint32_t)(uint8_t)(c - 3 * q - 1) << (8 * k);
    c = q;
  }
  return make_uint2(lo, (uint32_t)(uint8_t)(c - 1));
}

// ORs the trit bytes e of one code into out[] at byte offset o (bytes past
// `limit` dropped).
template <int o, int limit>
__device__ inline void place(uint32_t* out, uint2 e) {
  constexpr int d = o >> 2, s = 8 * (o & 3);
  out[d] |= e.x << s;
  if constexpr (d + 1 < limit / 4) {
    if constexpr (s == 0) out[d + 1] |= e.y;
    else out[d + 1] |= (e.x >> (32 - s)) | (e.y << s);
  }
}

__global__ void __launch_bounds__(kPartThreads) unpack_kernel(const uint8_t* __restrict__ codes, int64_t n,
                                                              int8_t* __restrict__ trits, int32_t* d_err) {
  __shared__ uint2 table[256];
  // The pass's 64 groups of trits, written back with 16-byte lanes over
  // consecutive addresses (per-thread stores would cut every line in pieces).
  __shared__ uint4 tile[kPartGroups * kGroup / 16];
  for (int c = threadIdx.x; c < 256; c += kPartThreads) table[c] = trit_bytes(c);
  __syncthreads();
  const int part = threadIdx.x % 3;
  const int slot = threadIdx.x / 3;
  uint8_t* tile_b = reinterpret_cast<uint8_t*>(tile) + slot * kGroup;
  for (int64_t base = (int64_t)blockIdx.x * kPartGroups; base < n; base += (int64_t)gridDim.x * kPartGroups) {
    const int64_t f = base + slot;
    int nbad = 0;
    if (f < n) {
      const uint2 cw = *reinterpret_cast<const uint2*>(codes + 24 * f + 8 * part);
      uint32_t tail = 0;
      if (part == 2) tail = *reinterpret_cast<const uint16_t*>(codes + (int64_t)kMainBytes * n + 2 * f);
      uint32_t cb[10];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        cb[i] = (cw.x >> (8 * i)) & 0xFFu;
        cb[4 + i] = (cw.y >> (8 * i)) & 0xFFu;
      }
      cb[8] = tail & 0xFFu;
      cb[9] = tail >> 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) nbad += cb[i] > 242u;
      if (part == 2) nbad += (cb[8] > 242u) + (cb[9] > 242u);
      uint32_t out[12] = {};
      place<0, 48>(out, table[cb[0]]);
      place<5, 48>(out, table[cb[1]]);
      place<10, 48>(out, table[cb[2]]);
      place<15, 48>(out, table[cb[3]]);
      place<20, 48>(out, table[cb[4]]);
      place<25, 48>(out, table[cb[5]]);
      place<30, 48>(out, table[cb[6]]);
      place<35, 48>(out, table[cb[7]]);
      if (part == 1) {   // trits 40..79
        *reinterpret_cast<uint2*>(tile_b + 40) = make_uint2(out[0], out[1]);
        *reinterpret_cast<uint4*>(tile_b + 48) = make_uint4(out[2], out[3], out[4], out[5]);
        *reinterpret_cast<uint4*>(tile_b + 64) = make_uint4(out[6], out[7], out[8], out[9]);
      } else if (part == 0) {   // trits 0..39
        *reinterpret_cast<uint4*>(tile_b) = make_uint4(out[0], out[1], out[2], out[3]);
        *reinterpret_cast<uint4*>(tile_b + 16) = make_uint4(out[4], out[5], out[6], out[7]);
        *reinterpret_cast<uint2*>(tile_b + 32) = make_uint2(out[8], out[9]);
      } else {   // trits 80..127: bytes 24 (5 trits) and 25 (3 trits) fill 40..47
        place<40, 48>(out, table[cb[8]]);
        place<45, 48>(out, table[cb[9]]);
        *reinterpret_cast<uint4*>(tile_b + 80) = make_uint4(out[0], out[1], out[2], out[3]);
        *reinterpret_cast<uint4*>(tile_b + 96) = make_uint4(out[4], out[5], out[6], out[7]);
        *reinterpret_cast<uint4*>(tile_b + 112) = make_uint4(out[8], out[9], out[10], out[11]);
      }
    }
    count_errors(d_err, nbad);
    __syncthreads();
    const int64_t left = n - base;
    const int chunks = (int)(left < kPartGroups ? left : kPartGroups) * (kGroup / 16);
    uint4* dst = reinterpret_cast<uint4*>(trits + base * kGroup);
    for (int i = threadIdx.x; i < chunks; i += kPartThreads) dst[i] = tile[i];
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// One-byte-per-thread pack and unpack, for trit buffers that are not 16-byte
// aligned.
// ---------------------------------------------------------------------------

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

__global__ void __launch_bounds__(kByteThreads) pack_bytes_kernel(const int8_t* __restrict__ trits, int64_t n,
                                                                  uint8_t* __restrict__ codes, int32_t* d_err) {
  const int64_t total = (int64_t)kGroupBytes * n;
  const int64_t stride = (int64_t)gridDim.x * kByteThreads;
  for (int64_t base = (int64_t)blockIdx.x * kByteThreads; base < total; base += stride) {
    int64_t pos = base + threadIdx.x;
    int nbad = 0;
    if (pos < total) {
      int64_t f;
      int j;
      locate(pos, n, f, j);
      const int8_t* t = trits + f * kGroup + 5 * j;
      bool bad = false;
      int code = 0, mul = 1;
#pragma unroll
      for (int i = 0; i < 5; ++i) {
        int v = (5 * j + i < kGroup) ? (int)t[i] : 0;   // the two pad trits are 0
        bad |= (v < -1) | (v > 1);
        code += (v + 1) * mul;
        mul *= 3;
      }
      codes[pos] = bad ? (uint8_t)0xFF : (uint8_t)code;
      nbad = bad;
    }
    count_errors(d_err, nbad);
  }
}

__global__ void __launch_bounds__(kByteThreads) unpack_bytes_kernel(const uint8_t* __restrict__ codes, int64_t n,
                                                                    int8_t* __restrict__ trits, int32_t* d_err) {
  const int64_t total = (int64_t)kGroupBytes * n;
  const int64_t stride = (int64_t)gridDim.x * kByteThreads;
  for (int64_t base = (int64_t)blockIdx.x * kByteThreads; base < total; base += stride) {
    int64_t pos = base + threadIdx.x;
    int nbad = 0;
    if (pos < total) {
      int64_t f;
      int j;
      locate(pos, n, f, j);
      int c = codes[pos];
      nbad = c > 242;
      if (nbad) c = 121;                      // five zero trits
      int8_t* t = trits + f * kGroup + 5 * j;
#pragma unroll
      for (int i = 0; i < 5; ++i) {
        if (5 * j + i < kGroup) t[i] = (int8_t)(c % 3 - 1);
        c /= 3;
      }
    }
    count_errors(d_err, nbad);
  }
}

// ---------------------------------------------------------------------------
// Validate: flat 16-byte chunks (8-byte chunks when the buffer is only
// 8-byte aligned).  In the main region (24 n bytes) a byte is bad if it is
// above 242, counted four bytes at a time; in the tail region odd bytes are
// byte 25, whose pad digits 3 and 4 must be 1 (108 <= c <= 134).
// ---------------------------------------------------------------------------

// Bytes above 242 in a word: b >= 243 iff its top bit is set and its low
// seven bits plus 13 reach 128 (no carry leaves a byte).
__device__ inline int bad_main(uint32_t w) {
  const uint32_t t = ((w & 0x7F7F7F7Fu) + 0x0D0D0D0Du) & w & 0x80808080u;
  return __builtin_popcount(t);
}

// One byte at storage position pos.
__device__ inline int bad_byte(uint32_t c, int64_t pos, int64_t main_bytes) {
  if (pos < main_bytes) return c > 242u;
  return ((pos - main_bytes) & 1) ? (c < 108u || c > 134u) : (c > 242u);
}

template <int W>   // chunk bytes: 16 or 8
__global__ void __launch_bounds__(kByteThreads) validate_kernel(const uint8_t* __restrict__ codes, int64_t n,
                                                                int32_t* d_err) {
  typedef typename std::conditional<W == 16, uint4, uint2>::type Chunk;
  constexpr int kWords = W / 4;
  const int64_t total = (int64_t)kGroupBytes * n;
  const int64_t main_bytes = (int64_t)kMainBytes * n;
  const int64_t chunks = (total + W - 1) / W;
  const int64_t stride = (int64_t)gridDim.x * kByteThreads;
  for (int64_t base = (int64_t)blockIdx.x * kByteThreads; base < chunks; base += stride) {
    const int64_t i = base + threadIdx.x;
    int nbad = 0;
    if (i < chunks) {
      const int64_t pos = (int64_t)W * i;
      uint32_t w[kWords];
      if (pos + W <= total) {
        const Chunk v = *reinterpret_cast<const Chunk*>(codes + pos);
        w[0] = v.x;
        w[1] = v.y;
        if constexpr (W == 16) {
          w[2] = reinterpret_cast<const uint4&>(v).z;
          w[3] = reinterpret_cast<const uint4&>(v).w;
        }
      } else {   // last, partial chunk: missing bytes read as 121 (valid everywhere)
#pragma unroll
        for (int k = 0; k < kWords; ++k) {
          uint32_t x = 0;
#pragma unroll
          for (int b = 0; b < 4; ++b) x |= (pos + 4 * k + b < total ? (uint32_t)codes[pos + 4 * k + b] : 121u) << (8 * b);
          w[k] = x;
        }
      }
      if (pos + W <= main_bytes) {
#pragma unroll
        for (int k = 0; k < kWords; ++k) nbad += bad_main(w[k]);
      } else {
#pragma unroll
        for (int k = 0; k < kWords; ++k)
#pragma unroll
          for (int b = 0; b < 4; ++b) nbad += bad_byte((w[k] >> (8 * b)) & 0xFFu, pos + 4 * k + b, main_bytes);
      }
    }
    count_errors(d_err, nbad);
  }
}

// ---------------------------------------------------------------------------
// Dense fp16 dequantisation.
// ---------------------------------------------------------------------------

// Base-3 digits of a code in 2-bit fields (digit k at bits 2k, 2k+1); codes
// above 242 read as 121 (the kernel's output for invalid codes is unspecified).
__device__ inline uint32_t digit_fields(int c) {
  if (c > 242) c = 121;
  uint32_t v = 0;
#pragma unroll
  for (int k = 0; k < 5; ++k) {
    const int q = (c * 171) >> 9;
    v |= (uint32_t)(c - 3 * q) << (2 * k);
    c = q;
  }
  return v;
}

__device__ inline float half_bits_to_float(uint32_t b) { return (float)__builtin_bit_cast(_Float16, (uint16_t)b); }

__device__ inline uint32_t float_to_half_bits(float a) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)a);   // nearest-even
}

// v_perm selectors for two weights of one plane with digits (u_a, u_b) =
// (e & 3, e >> 2), picking from S = s0 | (s0 ^ 0x8000) << 16: digit 0 (t = -1)
// takes bytes 0 and 3 (-s0), digit 2 (t = +1) bytes 0 and 1 (s0), digit 1
// (t = 0) selector 12, a zero byte.
__device__ inline uint32_t pair_selector(int e) {
  const uint32_t sel[4] = {0x0300u, 0x0C0Cu, 0x0100u, 0x0C0Cu};
  return sel[e & 3] | (sel[(e >> 2) & 3] << 16);
}

// Work split: a workgroup of 256 threads takes a block of RB whole rows
// (ng = RB * G <= 256 groups) and every thread owns 8-weight items of it
// (16 output bytes; 16 lanes per group, so a wave's store covers 1 KiB of
// consecutive output).  The block's plane-0 bytes arrive with coalesced dword
// loads and are staged in LDS, 8 words per group: bytes 0..23, the two tail
// bytes, and s0 | mu0 << 16.  Thread q of the block loads the block's q-th
// plane-1 record (rows' records are consecutive in the CSR arrays) into an
// LDS slot and points the group's entry of a map at it.
//
// Workgroups are persistent (a few per CU) and pipelined: while a block is
// decoded and stored, the loads of the next block (plane-0 words, records)
// and the row pointers of the one after are already in flight.  They are all
// issued before the current block's stores, and every load is unconditional
// (clamped to valid addresses), so waiting for them never waits for a store.
// With kExact every thread stores exactly kItems items per block (the host
// picks RB and kItems so that 16 * RB * G = 256 * kItems and RB divides N);
// the general variant bounds-checks its items instead.
constexpr int kDqThreads = 256;
constexpr int kDqMaxRows = 8;        // rows per block (small G)
constexpr int kDqBlocksPerCU = 4;    // persistent workgroups per CU
constexpr int kDqGeneralItems = 8;   // items per thread per pass, general variant

__host__ __device__ constexpr int dq_general_rows(int G) {
  return 16 * G >= kDqThreads * kDqGeneralItems
             ? 1
             : (kDqThreads * kDqGeneralItems / (16 * G) < kDqMaxRows ? kDqThreads * kDqGeneralItems / (16 * G)
                                                                      : kDqMaxRows);
}

template <bool kRec, bool kOff, int kItems, bool kExact>
__global__ void __launch_bounds__(kDqThreads) unpack_fp16_kernel(MatDev m, uint16_t* __restrict__ w, int RB) {
  static_assert(kDqThreads == 256 && kDqThreads >= TQ_MAX_GROUPS_PER_ROW,
                "one digit-table entry per thread; a block's groups and records fit one per thread");
  __shared__ uint32_t digits[256];
  __shared__ uint32_t selector[16];
  __shared__ int32_t rec_s[2][TQ_MAX_GROUPS_PER_ROW];            // group -> record slot, or -1 (two blocks)
  __shared__ uint32_t grp_s[8 * TQ_MAX_GROUPS_PER_ROW];          // staged plane-0 words
  __shared__ uint32_t rcd_s[kRec ? 8 * TQ_MAX_GROUPS_PER_ROW : 8];   // staged records: 6 code words, tail, mu | s1 << 16
  constexpr int kBlockItems = kDqThreads * kItems;
  const int G = m.n_groups;
  const int tid = threadIdx.x;
  const int64_t n = (int64_t)m.n_out * G;
  const int64_t n_blocks = ((int64_t)m.n_out + RB - 1) / RB;
  const uint32_t* c0 = reinterpret_cast<const uint32_t*>(m.codes0);
  const uint16_t* t0 = reinterpret_cast<const uint16_t*>(m.codes0 + (int64_t)kMainBytes * n);
  const uint32_t* c1 = reinterpret_cast<const uint32_t*>(m.codes1);
  const uint16_t* t1 = reinterpret_cast<const uint16_t*>(m.codes1 + (int64_t)kMainBytes * m.nnz1);
  const int64_t kmax = m.nnz1 > 0 ? m.nnz1 - 1 : 0;
  const int64_t b0 = blockIdx.x, gs = gridDim.x;
  if (b0 >= n_blocks) return;
  digits[tid] = digit_fields(tid);
  if (tid < 16) selector[tid] = pair_selector(tid);

  // Registers of the block being staged.
  uint32_t mw[6], tl, sc, mo;   // plane-0: 6 main words, tail, s0, mu0
  uint32_t rv[8];               // this thread's record: 6 code words, tail, mu | s1 << 16
  int rg = G, rslot = 0;        // its group in the row (G: none) and slot
  int rpv = 0;                  // lane j < 16: rowptr1[r0 + min(j, nr)]
  auto rows = [&](int64_t b, int& r0, int& nr) {
    b = b < n_blocks ? b : n_blocks - 1;   // past the end: the last block again (loads only)
    r0 = (int)(b * RB);
    nr = m.n_out - r0 < RB ? m.n_out - r0 : RB;
  };
  auto load_plane0 = [&](int64_t b) {
    int r0, nr;
    rows(b, r0, nr);
    const int ng = nr * G;
    const int64_t f0 = (int64_t)r0 * G;
#pragma unroll
    for (int u = 0; u < 6; ++u) {
      int i = u * kDqThreads + tid;
      i = i < 6 * ng ? i : 6 * ng - 1;
      mw[u] = c0[6 * f0 + i];
    }
    const int gt = tid < ng ? tid : ng - 1;
    tl = t0[f0 + gt];
    sc = m.scale0[f0 + gt];
    mo = kOff ? m.offset0[f0 + gt] : 0u;
  };
  auto load_rowptr = [&](int64_t b) {
    int r0, nr;
    rows(b, r0, nr);
    const int j = (tid & 15) < nr ? (tid & 15) : nr;
    rpv = m.rowptr1[r0 + j];
  };
  auto load_records = [&](int64_t b) {   // rpv holds block b's row pointers
    int r0, nr;
    rows(b, r0, nr);
    int rp[kDqMaxRows + 1];
#pragma unroll
    for (int j = 0; j <= kDqMaxRows; ++j) rp[j] = __builtin_amdgcn_readlane(rpv, j);
    // Record k = rp[0] + tid lies in row rr (rp[rr] <= k < rp[rr + 1]) at
    // position q; a row keeps at most G records, and k stays in [0, nnz1).
    const int k = rp[0] + tid;
    int rr = 0, lo_k = rp[0], hi_k = rp[1];
#pragma unroll
    for (int j = 1; j < kDqMaxRows; ++j)
      if (j < nr && rp[j] <= k) {
        rr = j;
        lo_k = rp[j];
        hi_k = rp[j + 1];
      }
    const int q = k - lo_k;
    const bool have = k >= 0 && k < m.nnz1 && k < hi_k && q >= 0 && q < G;
    const int64_t kc = have ? k : kmax;
    const int gi = m.gidx1[kc];
#pragma unroll
    for (int e = 0; e < 6; ++e) rv[e] = c1[6 * kc + e];
    rv[6] = t1[kc];
    rv[7] = (uint32_t)m.offset1[kc] | ((uint32_t)m.scale1[kc] << 16);
    rg = have ? gi : G;
    rslot = rr * G + q;
  };
  auto clear_map = [&](int64_t b, int par) {
    int r0, nr;
    rows(b, r0, nr);
    if (tid < nr * G) rec_s[par][tid] = -1;
  };

  auto step = [&](int64_t b, int par) {
    int r0, nr;
    rows(b, r0, nr);
    const int ng = nr * G;
    const int64_t f0 = (int64_t)r0 * G;
    // Stage block b from registers.
#pragma unroll
    for (int u = 0; u < 6; ++u) {
      const int i = u * kDqThreads + tid;
      if (i < 6 * ng) grp_s[8 * (i / 6) + i % 6] = mw[u];
    }
    if (tid < ng) {
      grp_s[8 * tid + 6] = tl;
      grp_s[8 * tid + 7] = sc | (mo << 16);
    }
    if (kRec && rg < G) {
#pragma unroll
      for (int e = 0; e < 8; ++e) rcd_s[8 * rslot + e] = rv[e];
      rec_s[par][rslot - rslot % G + rg] = rslot;
    }
    // The next block's loads and the row pointers of the one after.
    if (kRec) load_records(b + gs);
    load_plane0(b + gs);
    if (kRec) {
      load_rowptr(b + 2 * gs);
      clear_map(b + gs, par ^ 1);
    }
    __syncthreads();
    const int n_items = 16 * ng;
    auto pass = [&](const int it0) {
#pragma unroll
      for (int u = 0; u < kItems; ++u) {
        const int item = it0 + u * kDqThreads + tid;
        if (!kExact && item >= n_items) break;
        const int gl = item >> 4, i = item & 15;
        const int p0 = 8 * i;   // first of the 8 weights
        const int j0 = p0 / 5, d0 = p0 - 5 * j0;
        const int wb = j0 >> 2;
        // Code bytes j0..j0+2 of the group (for j0 = 24: the tail word; bytes
        // past 25 are zero or the next word's and their digits are unused).
        const uint32_t* gw = grp_s + 8 * gl;
        const uint32_t bytes = (uint32_t)((((uint64_t)gw[wb + 1] << 32) | gw[wb]) >> (8 * (j0 & 3)));
        uint32_t D0 = digits[bytes & 0xFFu] | (digits[(bytes >> 8) & 0xFFu] << 10) |
                      (digits[(bytes >> 16) & 0xFFu] << 20);
        D0 >>= 2 * d0;   // digit e of the 8 weights at bits 2e, 2e+1
        const uint32_t w7 = gw[7];
        const uint32_t s0 = w7 & 0xFFFFu;
        const int sl = kRec ? rec_s[par][gl] : -1;
        uint32_t o[4];
        if (!kOff && sl < 0 && (s0 & 0x7FFFu) != 0 && (s0 & 0x7C00u) != 0x7C00u) {
          // One plane, finite nonzero scale: +0 + s0*t is exactly +0 or +-s0.
          const uint32_t S = s0 | ((s0 ^ 0x8000u) << 16);
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = __builtin_amdgcn_perm(S, S, selector[(D0 >> (4 * q)) & 15u]);
        } else {
          // a = +0; a += mu0; a += mu; a += s0*t0; a += s1*t1 in fp32 (each
          // product exact), rounded once.
          const float s0f = half_bits_to_float(s0);
          const float mu0 = half_bits_to_float(w7 >> 16);
          float mu = 0.0f, s1f = 0.0f;
          uint32_t D1 = 0;
          if (kRec && sl >= 0) {
            const uint32_t* rw = rcd_s + 8 * sl;
            mu = half_bits_to_float(rw[7] & 0xFFFFu);
            s1f = half_bits_to_float(rw[7] >> 16);
            const uint32_t rb = (uint32_t)((((uint64_t)rw[wb + 1] << 32) | rw[wb]) >> (8 * (j0 & 3)));
            D1 = digits[rb & 0xFFu] | (digits[(rb >> 8) & 0xFFu] << 10) | (digits[(rb >> 16) & 0xFFu] << 20);
            D1 >>= 2 * d0;
          }
          uint32_t h[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float tz = (float)((int)((D0 >> (2 * e)) & 3u) - 1);
            float a = 0.0f;
            if (kOff) a = a + mu0;
            if (kRec && sl >= 0) a = a + mu;
            a = a + s0f * tz;
            if (kRec && sl >= 0) {
              const float t1v = (float)((int)((D1 >> (2 * e)) & 3u) - 1);
              a = a + s1f * t1v;
            }
            h[e] = float_to_half_bits(a);
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = h[2 * q] | (h[2 * q + 1] << 16);
        }
        // Streaming output: nontemporal 16-byte store.
        typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 ov = {o[0], o[1], o[2], o[3]};
        __builtin_nontemporal_store(ov, reinterpret_cast<u32x4*>(w + (f0 + gl) * kGroup + p0));
      }
    };
    if (kExact) {
      pass(0);   // straight-line, so the stores are always the newest memory operations
    } else {
      for (int it0 = 0; it0 < n_items; it0 += kBlockItems) pass(it0);
    }
  };

  // Prologue: the first block in registers, the second block's row pointers
  // in flight.  The first step is peeled so that the loop is entered only
  // after a step's stores.
  if (kRec) {
    load_rowptr(b0);
    load_records(b0);
    clear_map(b0, 0);
  }
  load_plane0(b0);
  if (kRec) load_rowptr(b0 + gs);
  __syncthreads();
  step(b0, 0);
  int par = 1;
  for (int64_t b = b0 + gs; b < n_blocks; b += gs) {
    __syncthreads();   // the previous block's LDS reads are done
    step(b, par);
    par ^= 1;
  }
}

}  // namespace

hipError_t launch_pack(const int8_t* trits, int64_t n, uint8_t* codes, int32_t* d_err, hipStream_t s) {
  if ((reinterpret_cast<uintptr_t>(trits) & 15) == 0) {
    const int64_t blocks = clamp_blocks((n + kPartGroups - 1) / kPartGroups, kPartMaxBlocks);
    hipLaunchKernelGGL(pack_kernel, dim3((unsigned)blocks), dim3(kPartThreads), 0, s, trits, n, codes, d_err);
  } else {
    const int64_t blocks = clamp_blocks((kGroupBytes * n + kByteThreads - 1) / kByteThreads, kMaxBlocks);
    hipLaunchKernelGGL(pack_bytes_kernel, dim3((unsigned)blocks), dim3(kByteThreads), 0, s, trits, n, codes, d_err);
  }
  return hipGetLastError();
}

hipError_t launch_unpack(const uint8_t* codes, int64_t n, int8_t* trits, int32_t* d_err, hipStream_t s) {
  if ((reinterpret_cast<uintptr_t>(trits) & 15) == 0) {
    const int64_t blocks = clamp_blocks((n + kPartGroups - 1) / kPartGroups, kPartMaxBlocks);
    hipLaunchKernelGGL(unpack_kernel, dim3((unsigned)blocks), dim3(kPartThreads), 0, s, codes, n, trits, d_err);
  } else {
    const int64_t blocks = clamp_blocks((kGroupBytes * n + kByteThreads - 1) / kByteThreads, kMaxBlocks);
    hipLaunchKernelGGL(unpack_bytes_kernel, dim3((unsigned)blocks), dim3(kByteThreads), 0, s, codes, n, trits,
                       d_err);
  }
  return hipGetLastError();
}

hipError_t launch_validate(const uint8_t* codes, int64_t n, int32_t* d_err, hipStream_t s) {
  const bool wide = (reinterpret_cast<uintptr_t>(codes) & 15) == 0;
  const int W = wide ? 16 : 8;
  const int64_t chunks = (kGroupBytes * n + W - 1) / W;
  const int64_t blocks = clamp_blocks((chunks + kByteThreads - 1) / kByteThreads, kMaxBlocks);
  if (wide)
    hipLaunchKernelGGL(validate_kernel<16>, dim3((unsigned)blocks), dim3(kByteThreads), 0, s, codes, n, d_err);
  else
    hipLaunchKernelGGL(validate_kernel<8>, dim3((unsigned)blocks), dim3(kByteThreads), 0, s, codes, n, d_err);
  return hipGetLastError();
}

hipError_t launch_unpack_fp16(const MatDev& m, uint16_t* w, hipStream_t s) {
  static int cus_of[64];   // CUs per device, read once
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  int& cus = cus_of[dev & 63];
  if (cus == 0) {
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
  }
  // An exact fit: 16 * RB * G = 256 * items with RB | N, the most items first.
  const int G = m.n_groups;
  int RB = 0, items = 0;
  for (int c : {8, 6, 5}) {
    const int rb = 16 * c / G;
    if ((16 * c) % G == 0 && rb >= 1 && rb <= kDqMaxRows && m.n_out % rb == 0) {
      RB = rb;
      items = c;
      break;
    }
  }
  const bool rec = m.nnz1 > 0, off = m.offset0 != nullptr;
  void (*kernel)(MatDev, uint16_t*, int);
#define TQ_DQ_PICK(I, E)                                                                     \
  (rec ? (off ? unpack_fp16_kernel<true, true, I, E> : unpack_fp16_kernel<true, false, I, E>) \
       : (off ? unpack_fp16_kernel<false, true, I, E> : unpack_fp16_kernel<false, false, I, E>))
  if (items == 8) {
    kernel = TQ_DQ_PICK(8, true);
  } else if (items == 6) {
    kernel = TQ_DQ_PICK(6, true);
  } else if (items == 5) {
    kernel = TQ_DQ_PICK(5, true);
  } else {
    kernel = TQ_DQ_PICK(kDqGeneralItems, false);
    RB = dq_general_rows(G);
  }
#undef TQ_DQ_PICK
  const int64_t blocks = clamp_blocks(((int64_t)m.n_out + RB - 1) / RB, (int64_t)kDqBlocksPerCU * cus);
  hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(kDqThreads), 0, s, m, w, RB);
  return hipGetLastError();
}

}  // namespace tq
