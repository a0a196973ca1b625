// Host entry points of libtq.so (declared in include/tq.h): argument checks
// on the host, then one asynchronous launch on the caller's stream.
//
// Every check runs before the first HIP call, so an argument error is
// returned synchronously and touches neither the device nor the stream.

#include <stdint.h>

#include <memory>
#include <new>

#include "tq_internal.h"

namespace {

using tq::MatDev;

inline bool misaligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; }

inline tq_status from_hip(hipError_t e) { return e == hipSuccess ? TQ_OK : TQ_ERR_HIP; }

tq_status check_codes_call(const void* codes, const void* other, int64_t n_groups, int32_t group) {
  if (group != TQ_GROUP) return TQ_ERR_UNSUPPORTED;
  if (n_groups < 0) return TQ_ERR_SHAPE;
  if (n_groups > (INT64_MAX / 256)) return TQ_ERR_SHAPE;
  if (n_groups == 0) return TQ_OK;
  if (codes == nullptr || other == nullptr) return TQ_ERR_NULL;
  if (misaligned(codes, 8)) return TQ_ERR_ALIGN;
  return TQ_OK;
}

// Checks one matrix view and fills its device-side form.
tq_status check_matrix(const tq_matrix* m, MatDev* d) {
  if (m == nullptr) return TQ_ERR_NULL;
  if (m->group != TQ_GROUP) return TQ_ERR_UNSUPPORTED;
  if (m->reserved != 0) return TQ_ERR_SHAPE;
  if (m->n_out < 1 || m->n_out > INT32_MAX) return TQ_ERR_SHAPE;
  if (m->n_in < TQ_GROUP || m->n_in % TQ_GROUP != 0) return TQ_ERR_SHAPE;
  const int64_t G = m->n_in / TQ_GROUP;
  if (G > TQ_MAX_GROUPS_PER_ROW) return TQ_ERR_UNSUPPORTED;
  // Kernels address code buffers with 32-bit byte offsets.
  if ((int64_t)TQ_GROUP_BYTES * m->n_out * G > (int64_t)UINT32_MAX) return TQ_ERR_UNSUPPORTED;
  if (m->codes0 == nullptr || m->scale0 == nullptr) return TQ_ERR_NULL;
  if (misaligned(m->codes0, 8) || misaligned(m->scale0, 2) || misaligned(m->offset0, 2)) return TQ_ERR_ALIGN;
  if (m->nnz1 < 0 || m->nnz1 > m->n_out * G) return TQ_ERR_SHAPE;
  if (m->nnz1 > 0) {
    if (m->rowptr1 == nullptr || m->gidx1 == nullptr || m->codes1 == nullptr || m->offset1 == nullptr ||
        m->scale1 == nullptr)
      return TQ_ERR_NULL;
    if (misaligned(m->rowptr1, 4) || misaligned(m->gidx1, 2) || misaligned(m->codes1, 8) ||
        misaligned(m->offset1, 2) || misaligned(m->scale1, 2))
      return TQ_ERR_ALIGN;
  }
  d->codes0 = m->codes0;
  d->scale0 = m->scale0;
  d->nnz1 = m->nnz1;
  d->rowptr1 = m->nnz1 > 0 ? m->rowptr1 : nullptr;
  d->gidx1 = m->nnz1 > 0 ? m->gidx1 : nullptr;
  d->codes1 = m->nnz1 > 0 ? m->codes1 : nullptr;
  d->offset1 = m->nnz1 > 0 ? m->offset1 : nullptr;
  d->scale1 = m->nnz1 > 0 ? m->scale1 : nullptr;
  d->rowptr1_host = m->nnz1 > 0 ? m->rowptr1_host : nullptr;
  d->offset0 = m->offset0;
  d->n_out = (int32_t)m->n_out;
  d->n_groups = (int32_t)G;
  return TQ_OK;
}

// Arguments shared by both selection entry points (not the workspace).
tq_status check_select(const double* energy, int64_t n_out, int32_t G, int64_t nnz, const int32_t* rec_index,
                       const int32_t* rowptr1, const uint16_t* gidx1) {
  if (n_out < 1 || G < 1 || G > TQ_MAX_GROUPS_PER_ROW) return TQ_ERR_SHAPE;
  if (n_out > (int64_t)INT32_MAX / G) return TQ_ERR_SHAPE;
  const int64_t n = n_out * G;
  if (nnz < 0 || nnz > n) return TQ_ERR_SHAPE;
  if (energy == nullptr || rec_index == nullptr || rowptr1 == nullptr) return TQ_ERR_NULL;
  if (nnz > 0 && gidx1 == nullptr) return TQ_ERR_NULL;
  if (misaligned(energy, 8) || misaligned(rec_index, 4) || misaligned(rowptr1, 4) ||
      (gidx1 != nullptr && misaligned(gidx1, 2)))
    return TQ_ERR_ALIGN;
  return TQ_OK;
}

tq_status check_flags(int32_t flags) {
  return (flags == TQ_OUT_FP16 || flags == TQ_OUT_FP32) ? TQ_OK : TQ_ERR_UNSUPPORTED;
}

}  // namespace

extern "C" {

int tq_abi_version(void) { return TQ_ABI_VERSION; }

const char* tq_status_string(tq_status s) {
  switch (s) {
    case TQ_OK: return "TQ_OK";
    case TQ_ERR_NULL: return "TQ_ERR_NULL: a required pointer is NULL";
    case TQ_ERR_SHAPE: return "TQ_ERR_SHAPE: a size is out of range or inconsistent";
    case TQ_ERR_ALIGN: return "TQ_ERR_ALIGN: a pointer is not aligned as required";
    case TQ_ERR_UNSUPPORTED: return "TQ_ERR_UNSUPPORTED: request not supported by this build";
    case TQ_ERR_HIP: return "TQ_ERR_HIP: the HIP runtime reported an error";
  }
  return "unknown tq_status";
}

tq_status tq_pack(const int8_t* trits, int64_t n_groups, int32_t group, uint8_t* codes, int32_t* d_err,
                  void* stream) {
  tq_status st = check_codes_call(codes, trits, n_groups, group);
  if (st != TQ_OK || n_groups == 0) return st;
  return from_hip(tq::launch_pack(trits, n_groups, codes, d_err, (hipStream_t)stream));
}

tq_status tq_unpack(const uint8_t* codes, int64_t n_groups, int32_t group, int8_t* trits, int32_t* d_err,
                    void* stream) {
  tq_status st = check_codes_call(codes, trits, n_groups, group);
  if (st != TQ_OK || n_groups == 0) return st;
  return from_hip(tq::launch_unpack(codes, n_groups, trits, d_err, (hipStream_t)stream));
}

tq_status tq_validate(const uint8_t* codes, int64_t n_groups, int32_t group, int32_t* d_err, void* stream) {
  tq_status st = check_codes_call(codes, d_err, n_groups, group);
  if (st != TQ_OK || n_groups == 0) return st;
  if (misaligned(d_err, 4)) return TQ_ERR_ALIGN;
  return from_hip(tq::launch_validate(codes, n_groups, d_err, (hipStream_t)stream));
}

tq_status tq_unpack_fp16(const tq_matrix* m, uint16_t* w, void* stream) {
  MatDev d;
  tq_status st = check_matrix(m, &d);
  if (st != TQ_OK) return st;
  if (w == nullptr) return TQ_ERR_NULL;
  if (misaligned(w, 16)) return TQ_ERR_ALIGN;
  return from_hip(tq::launch_unpack_fp16(d, w, (hipStream_t)stream));
}

tq_status tq_gemv(const tq_matrix* m, const uint16_t* x, void* y, int32_t flags, void* stream) {
  MatDev d;
  tq_status st = check_matrix(m, &d);
  if (st != TQ_OK) return st;
  if ((st = check_flags(flags)) != TQ_OK) return st;
  if (x == nullptr || y == nullptr) return TQ_ERR_NULL;
  if (misaligned(x, 16) || misaligned(y, 4)) return TQ_ERR_ALIGN;
  void* ys[1] = {y};
  return from_hip(tq::launch_gemv(&d, ys, 1, x, flags == TQ_OUT_FP32, (hipStream_t)stream));
}

tq_status tq_gemv_grouped(const tq_matrix* ms, int32_t n, const uint16_t* x, void* const* ys, int32_t flags,
                          void* stream) {
  if (ms == nullptr || ys == nullptr || x == nullptr) return TQ_ERR_NULL;
  if (n < 1 || n > TQ_MAX_GROUPED) return TQ_ERR_SHAPE;
  tq_status st = check_flags(flags);
  if (st != TQ_OK) return st;
  MatDev d[TQ_MAX_GROUPED];
  int64_t total_rows = 0;
  for (int i = 0; i < n; ++i) {
    if ((st = check_matrix(&ms[i], &d[i])) != TQ_OK) return st;
    if (ms[i].n_in != ms[0].n_in) return TQ_ERR_SHAPE;
    if (ys[i] == nullptr) return TQ_ERR_NULL;
    if (misaligned(ys[i], 4)) return TQ_ERR_ALIGN;
    total_rows += ms[i].n_out;
  }
  if (total_rows > INT32_MAX) return TQ_ERR_SHAPE;
  if (misaligned(x, 16)) return TQ_ERR_ALIGN;
  return from_hip(tq::launch_gemv(d, ys, n, x, flags == TQ_OUT_FP32, (hipStream_t)stream));
}

tq_status tq_gemm_smallbatch(const tq_matrix* m, const uint16_t* X, int32_t B, void* Y, int32_t flags,
                             void* stream) {
  MatDev d;
  tq_status st = check_matrix(m, &d);
  if (st != TQ_OK) return st;
  if ((st = check_flags(flags)) != TQ_OK) return st;
  if (X == nullptr || Y == nullptr) return TQ_ERR_NULL;
  if (B < 1 || B > TQ_MAX_BATCH) return TQ_ERR_SHAPE;
  if (misaligned(X, 16) || misaligned(Y, 4)) return TQ_ERR_ALIGN;
  if (B == 1) {
    void* ys[1] = {Y};
    return from_hip(tq::launch_gemv(&d, ys, 1, X, flags == TQ_OUT_FP32, (hipStream_t)stream));
  }
  if (tq::gemv_batch_supported(d, B)) {
    // A few rows: the GEMV's decode with one accumulator set per row, where
    // its launch fits; otherwise the MFMA path below.
    const hipError_t e = tq::launch_gemv_batch(d, X, B, Y, flags == TQ_OUT_FP32, (hipStream_t)stream);
    if (e != hipErrorNotSupported) return from_hip(e);
  }
  return from_hip(tq::launch_gemm_smallbatch(d, X, B, Y, flags == TQ_OUT_FP32, (hipStream_t)stream));
}

tq_status tq_ternarize(const uint16_t* w, int64_t n_groups, int32_t group, const int32_t* rec_index, int64_t nnz,
                       int32_t iters, int8_t* t0, uint16_t* s0, int8_t* t1, uint16_t* offset1, uint16_t* scale1,
                       uint16_t* offset0, double* energy, void* stream) {
  if (group != TQ_GROUP) return TQ_ERR_UNSUPPORTED;
  if (n_groups < 0 || nnz < 0 || n_groups > (INT64_MAX / 256) || iters < 0 || iters > 1024) return TQ_ERR_SHAPE;
  if (n_groups == 0) return TQ_OK;
  if (w == nullptr || t0 == nullptr || s0 == nullptr) return TQ_ERR_NULL;
  if (nnz > 0 && (t1 == nullptr || offset1 == nullptr || scale1 == nullptr)) return TQ_ERR_NULL;
  if (misaligned(w, 16) || misaligned(t0, 16) || misaligned(s0, 2)) return TQ_ERR_ALIGN;
  if (rec_index != nullptr && misaligned(rec_index, 4)) return TQ_ERR_ALIGN;
  if (nnz > 0 && (misaligned(t1, 16) || misaligned(offset1, 2) || misaligned(scale1, 2))) return TQ_ERR_ALIGN;
  if (energy != nullptr && misaligned(energy, 8)) return TQ_ERR_ALIGN;
  if (offset0 != nullptr && misaligned(offset0, 2)) return TQ_ERR_ALIGN;
  return from_hip(tq::launch_ternarize(w, n_groups, rec_index, nnz, iters, t0, s0, t1, offset1, scale1, offset0,
                                       energy, (hipStream_t)stream));
}

size_t tq_select_workspace_bytes(int64_t n_groups) {
  if (n_groups < 0) return 0;
  return tq::select_workspace_bytes(n_groups);
}

tq_status tq_select_two_plane(const double* energy, int64_t n_out, int32_t groups_per_row, int64_t nnz,
                              int32_t* rec_index, int32_t* rowptr1, uint16_t* gidx1, void* workspace,
                              size_t workspace_bytes, void* stream) {
  tq_status st = check_select(energy, n_out, groups_per_row, nnz, rec_index, rowptr1, gidx1);
  if (st != TQ_OK) return st;
  if (workspace == nullptr) return TQ_ERR_NULL;
  if (workspace_bytes < tq::select_workspace_bytes(n_out * groups_per_row)) return TQ_ERR_SHAPE;
  if (misaligned(workspace, 256)) return TQ_ERR_ALIGN;
  return from_hip(tq::launch_select(energy, n_out, groups_per_row, nnz, rec_index, rowptr1, gidx1, workspace,
                                    (hipStream_t)stream));
}

tq_status tq_select_two_plane_noalloc(const double* energy, int64_t n_out, int32_t groups_per_row, int64_t nnz,
                                      int32_t* rec_index, int32_t* rowptr1, uint16_t* gidx1, void* stream) {
  tq_status st = check_select(energy, n_out, groups_per_row, nnz, rec_index, rowptr1, gidx1);
  if (st != TQ_OK) return st;
  if (n_out * groups_per_row > TQ_SELECT_NOALLOC_MAX_GROUPS) return TQ_ERR_UNSUPPORTED;
  return from_hip(tq::launch_select_noalloc(energy, n_out, groups_per_row, nnz, rec_index, rowptr1, gidx1,
                                            (hipStream_t)stream));
}

tq_status tq_chain_plan(const tq_stage* stages, int32_t n_stages, tq_chain_info* info, void* plan_host,
                        size_t plan_host_bytes) {
  if (stages == nullptr || info == nullptr) return TQ_ERR_NULL;
  if (n_stages < 1) return TQ_ERR_SHAPE;
  tq::ChainStageDev* st = new (std::nothrow) tq::ChainStageDev[n_stages];
  if (st == nullptr) return TQ_ERR_SHAPE;
  std::unique_ptr<tq::ChainStageDev[]> keep(st);
  tq_status r;
  for (int s = 0; s < n_stages; ++s) {
    const tq_stage& S = stages[s];
    if (S.mats == nullptr || S.ys == nullptr || S.x == nullptr) return TQ_ERR_NULL;
    if (S.n < 1 || S.n > TQ_MAX_GROUPED) return TQ_ERR_SHAPE;
    if ((r = check_flags(S.flags)) != TQ_OK) return r;
    if (misaligned(S.x, 16)) return TQ_ERR_ALIGN;
    st[s].n = S.n;
    st[s].out_f32 = S.flags == TQ_OUT_FP32;
    st[s].x = S.x;
    for (int i = 0; i < S.n; ++i) {
      if ((r = check_matrix(&S.mats[i], &st[s].m[i])) != TQ_OK) return r;
      if (S.mats[i].n_in != S.mats[0].n_in) return TQ_ERR_SHAPE;
      if (S.ys[i] == nullptr) return TQ_ERR_NULL;
      if (misaligned(S.ys[i], 4)) return TQ_ERR_ALIGN;
      st[s].ys[i] = S.ys[i];
    }
  }
  int nwg = 0;
  if (tq::chain_workgroups(&nwg) != hipSuccess) return TQ_ERR_HIP;
  for (int s = 0; s < n_stages; ++s) {
    int rpw, passes, used;
    if (!tq::plan_stage(st[s].m, st[s].n, nwg, &rpw, &passes, &used)) return TQ_ERR_UNSUPPORTED;
  }
  info->n_stages = n_stages;
  info->n_workgroups = nwg;
  info->reserved = 0;
  info->plan_bytes = (int64_t)sizeof(tq::ChainWork) * n_stages * nwg;
  info->sync_bytes = tq::chain_sync_head_bytes() + (int64_t)tq::chain_flag_stride_bytes() * nwg;
  // The plan also decides the LDS: fill it into a scratch table when the
  // caller asks only for the sizes.
  std::unique_ptr<tq::ChainWork[]> tmp;
  tq::ChainWork* out = static_cast<tq::ChainWork*>(plan_host);
  if (out == nullptr) {
    tmp.reset(new (std::nothrow) tq::ChainWork[(size_t)n_stages * nwg]);
    if (!tmp) return TQ_ERR_SHAPE;
    out = tmp.get();
  } else if (plan_host_bytes < (size_t)info->plan_bytes) {
    return TQ_ERR_SHAPE;
  } else if (misaligned(plan_host, 8)) {
    return TQ_ERR_ALIGN;
  }
  int64_t lds = 0;
  if (tq::chain_plan_fill(st, n_stages, nwg, out, &lds) != hipSuccess) return TQ_ERR_UNSUPPORTED;
  if (lds > tq::chain_lds_limit()) return TQ_ERR_UNSUPPORTED;
  info->lds_bytes = (int32_t)((lds + 15) & ~(int64_t)15);
  return TQ_OK;
}

static tq_status check_chain_info(const tq_chain_info* info) {
  if (info == nullptr) return TQ_ERR_NULL;
  if (info->n_stages < 1 || info->n_workgroups < 1 || info->lds_bytes < 0 ||
      info->lds_bytes > tq::chain_lds_limit() ||
      info->plan_bytes != (int64_t)sizeof(tq::ChainWork) * info->n_stages * info->n_workgroups ||
      info->sync_bytes != tq::chain_sync_head_bytes() + (int64_t)tq::chain_flag_stride_bytes() * info->n_workgroups)
    return TQ_ERR_SHAPE;
  return TQ_OK;
}

tq_status tq_chain_sync_init(void* sync, const tq_chain_info* info, void* stream) {
  tq_status r = check_chain_info(info);
  if (r != TQ_OK) return r;
  if (sync == nullptr) return TQ_ERR_NULL;
  if (misaligned(sync, 256)) return TQ_ERR_ALIGN;
  return from_hip(tq::launch_chain_clear(sync, info->sync_bytes, (hipStream_t)stream));
}

tq_status tq_gemv_chain(const void* plan, void* sync, const tq_chain_info* info, void* stream) {
  tq_status r = check_chain_info(info);
  if (r != TQ_OK) return r;
  if (plan == nullptr || sync == nullptr) return TQ_ERR_NULL;
  if (misaligned(plan, 128) || misaligned(sync, 256)) return TQ_ERR_ALIGN;
  int nwg = 0;
  if (tq::chain_workgroups(&nwg) != hipSuccess) return TQ_ERR_HIP;
  if (nwg != info->n_workgroups) return TQ_ERR_SHAPE;   // planned for another device
  return from_hip(tq::launch_chain(static_cast<const tq::ChainWork*>(plan), info->n_stages, info->n_workgroups,
                                   info->lds_bytes, sync, (hipStream_t)stream));
}

}  // extern "C"
