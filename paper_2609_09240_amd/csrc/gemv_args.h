// Launch arguments of the batch-1 GEMV kernels (gemv.hip):
// the matrix records of a grouped launch and the record-range table, read
// by the kernels straight from the kernel-argument segment.  Included inside
// namespace tq's anonymous namespace of each file.
//
// Budget: 8 records of 88 bytes plus 768 range entries come to 3776 bytes;
// with the leading scalar arguments a launch passes about 3.8 KiB of the
// 4 KiB that a kernel's arguments may take.  A new field, a larger
// TQ_MAX_GROUPED or a longer range table has to give room elsewhere first.
#pragma once

// Record-range table entries passed with a launch (host ranges).
constexpr int kMaxRangeEntries = 768;

struct GemvMat {
  const uint8_t* codes0;
  const uint16_t* scale0;
  const int32_t* rowptr1;
  const uint16_t* gidx1;
  const uint8_t* codes1;
  const uint16_t* offset1;
  const uint16_t* scale1;
  const uint16_t* offset0;   // per-group offsets on every group, or NULL
  void* y;
  int32_t n_out;
  int32_t nnz1;       // < 2^31: the host caps code buffers at 2^32 bytes
  int32_t wg_begin;   // first workgroup of this matrix
  int32_t pad;
};
struct GemvArgs {
  GemvMat m[TQ_MAX_GROUPED];
  // With host ranges: the first record of every workgroup, matrix by
  // matrix, each matrix closed by its nnz1 (entry of workgroup w of matrix
  // i is rec_begin[w + i]).
  int32_t rec_begin[kMaxRangeEntries];
};
static_assert(sizeof(GemvArgs) == 3776, "launch argument budget");
