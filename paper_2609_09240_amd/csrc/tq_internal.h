// Internal interface between the host entry points (tq_api.hip) and the
// kernel launchers (codec.hip, gemv.hip, gemm.hip, quantize.hip).  Every
// launcher assumes its arguments were already checked on the host and
// returns the status of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/tq.h"

namespace tq {

constexpr int kGroup = TQ_GROUP;            // trits per group
constexpr int kGroupBytes = TQ_GROUP_BYTES; // code bytes per group
constexpr int kMainBytes = 24;              // bytes 0..23 (main region)

// Device-side view of one packed linear (row counts fit in int32 here; the
// host rejects larger matrices).
struct MatDev {
  const uint8_t* codes0;
  const uint16_t* scale0;
  const int32_t* rowptr1;
  const uint16_t* gidx1;
  const uint8_t* codes1;
  const uint16_t* offset1;
  const uint16_t* scale1;
  const int32_t* rowptr1_host;   // host memory, may be NULL
  const uint16_t* offset0;       // per-group offsets on every group, may be NULL
  int64_t nnz1;
  int32_t n_out;
  int32_t n_groups;   // groups per row, K / 128
};

hipError_t launch_pack(const int8_t* trits, int64_t n_groups, uint8_t* codes,
                       int32_t* d_err, hipStream_t s);
hipError_t launch_unpack(const uint8_t* codes, int64_t n_groups, int8_t* trits,
                         int32_t* d_err, hipStream_t s);
hipError_t launch_validate(const uint8_t* codes, int64_t n_groups,
                           int32_t* d_err, hipStream_t s);
hipError_t launch_unpack_fp16(const MatDev& m, uint16_t* w, hipStream_t s);

// n matrices sharing x (all with the same n_groups).
hipError_t launch_gemv(const MatDev* ms, void* const* ys, int n,
                       const uint16_t* x, bool out_f32, hipStream_t s);

// A few batch rows (2..4) through the GEMV's decode, each code byte decoded
// once for all rows; needs the host row pointers when the matrix has
// records.  Returns hipErrorNotSupported where it does not apply.
bool gemv_batch_supported(const MatDev& m, int B);
hipError_t launch_gemv_batch(const MatDev& m, const uint16_t* X, int B, void* Y, bool out_f32, hipStream_t s);

hipError_t launch_gemm_smallbatch(const MatDev& m, const uint16_t* X, int B,
                                  void* Y, bool out_f32, hipStream_t s);

hipError_t launch_ternarize(const uint16_t* w, int64_t n_groups, const int32_t* rec_index, int64_t nnz,
                            int iters, int8_t* t0, uint16_t* s0, int8_t* t1, uint16_t* offset1,
                            uint16_t* scale1, uint16_t* offset0, double* energy, hipStream_t s);

// Two-plane selection and plane-1 CSR (select.hip); workspace of
// select_workspace_bytes(n_out * G) bytes, 256-byte aligned.
size_t select_workspace_bytes(int64_t n_groups);
hipError_t launch_select(const double* energy, int64_t n_out, int32_t G, int64_t nnz, int32_t* rec_index,
                         int32_t* rowptr1, uint16_t* gidx1, void* workspace, hipStream_t s);
// The same with the library's static per-device scratch (no allocation).
hipError_t launch_select_noalloc(const double* energy, int64_t n_out, int32_t G, int64_t nnz, int32_t* rec_index,
                                 int32_t* rowptr1, uint16_t* gidx1, hipStream_t s);

// ---- Decode-step chain (chain.hip).
// Work of one workgroup in one stage: rows [row_begin, row_end) of one
// matrix (none when row_end <= row_begin), read by the kernel from the
// device copy of the plan.
struct alignas(128) ChainWork {
  const uint8_t* codes0;
  const uint16_t* scale0;
  const int32_t* rowptr1;
  const uint16_t* gidx1;
  const uint8_t* codes1;
  const uint16_t* offset1;
  const uint16_t* scale1;
  const uint16_t* offset0;
  const uint16_t* x;
  void* y;
  int32_t n_out;
  int32_t nnz1;
  int32_t row_begin;
  int32_t row_end;
  int32_t rec_begin;   // records of the rows; -1: from the device row pointers
  int32_t rec_end;
  int32_t G;           // groups per row
  int32_t flags;       // bit 0: fp32 output; bits 8..15: plane-0 passes
};
static_assert(sizeof(ChainWork) == 128, "plan record size");

struct ChainStageDev {
  MatDev m[TQ_MAX_GROUPED];
  void* ys[TQ_MAX_GROUPED];
  const uint16_t* x;
  int n;
  bool out_f32;
};

int chain_lds_limit();
int chain_sync_head_bytes();
int chain_flag_stride_bytes();
hipError_t chain_workgroups(int* nwg);
bool plan_stage(const MatDev* ms, int n, int nwg, int* rows_per_wg, int* passes, int* used);
hipError_t chain_plan_fill(const ChainStageDev* st, int n_stages, int nwg, ChainWork* plan, int64_t* max_lds);
hipError_t launch_chain_clear(void* sync, int64_t bytes, hipStream_t s);
hipError_t launch_chain(const ChainWork* plan, int n_stages, int nwg, int lds_dyn, void* sync, hipStream_t s);

}  // namespace tq
