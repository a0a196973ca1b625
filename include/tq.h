/*
 * tq.h — packed ternary GEMV for AMD Instinct MI355X (gfx950): C ABI.
 *
 * The operation (paper arXiv 2609.09240, section 3, eq. 3, and the footnote
 * to section 3): a linear projection is stored as
 *     W^ = (mu + a0*T0 + a1*T1) (.) M,   T_i in {-1, 0, +1},
 * where every 128-wide group of a row carries plane T0 with an fp16 scale
 * s0, and a selected subset of groups also carries plane T1 with an fp16
 * offset mu and an fp16 scale s1.  On such a two-plane group every weight is
 * mu + s0*t0 + s1*t1; elsewhere it is s0*t0.  Activations stay fp16 (A16,
 * section 3).  The packed format persists the discrete supports losslessly
 * (section 12): five trits per byte as a base-3 code.
 *
 * ------------------------------------------------------------------------
 * Packed format (the paper fixes no byte layout; this is the library's).
 *
 *   Group: 128 trits t[0..127] of one row, input indices 128g .. 128g+127.
 *   Code byte j (j = 0..25) holds trits 5j .. 5j+4:
 *       code = sum_{i=0..4} (t[5j+i] + 1) * 3^i          (0 .. 242)
 *   Byte 25 holds t[125..127] in digits 0..2; its digits 3 and 4 are 1
 *   (trit 0), so a valid last byte lies in 108..134.  Codes 243..255 are
 *   invalid.
 *   A code buffer of n groups is 26*n bytes in the "split" layout: bytes
 *   0..23 of group f at offset 24*f, bytes 24 and 25 of group f at offset
 *   24*n + 2*f.  (Every group body is 8-byte aligned for vector loads.)
 *
 *   A packed linear of N outputs and K inputs (K % 128 == 0, G = K/128):
 *     codes0   uint8  [26*N*G]   plane 0, groups in row-major (r, g) order
 *     scale0   fp16   [N][G]     s0
 *     rowptr1  int32  [N+1]      CSR over rows of the two-plane groups
 *     gidx1    uint16 [nnz1]     group index of each record; strictly
 *                                increasing within a row
 *     codes1   uint8  [26*nnz1]  plane 1 of each record (split layout)
 *     offset1  fp16   [nnz1]     mu
 *     scale1   fp16   [nnz1]     s1
 *
 * ------------------------------------------------------------------------
 * Conventions for every entry point.
 *
 *   - Pointers to data are DEVICE pointers (hipMalloc / torch tensors on
 *     the GPU) unless stated otherwise; tq_matrix itself lives in host
 *     memory and is read only during the call.  The caller owns every
 *     buffer; the library keeps no state and allocates no memory.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Every call is
 *     asynchronous on that stream; nothing synchronises.
 *   - Argument errors (NULL pointers, bad sizes or alignment, group != 128)
 *     are detected on the host before anything is launched and returned
 *     synchronously.  A failed launch returns TQ_ERR_HIP.
 *   - Data errors (invalid trits or codes) are reported asynchronously
 *     through an optional device counter `d_err` (int32, may be NULL),
 *     which is incremented, never reset, by the number of bad bytes.
 *   - tq_gemv, tq_gemv_grouped and tq_gemm_smallbatch do not validate codes:
 *     invalid codes give unspecified (but finite-time, in-bounds) results.
 *     Validate a matrix once with tq_validate when it is loaded.
 *   - Results are deterministic: the same inputs give bit-identical outputs
 *     on every run.
 *   - Fp16 values are passed as their uint16 bit patterns.
 */
#ifndef TQ_H
#define TQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TQ_ABI_VERSION 7
#define TQ_GROUP 128
#define TQ_GROUP_BYTES 26
#define TQ_MAX_GROUPS_PER_ROW 256    /* K <= 32768 */
#define TQ_MAX_GROUPED 8             /* matrices per tq_gemv_grouped call */
#define TQ_MAX_BATCH 64              /* rows of X in tq_gemm_smallbatch */
#define TQ_SELECT_NOALLOC_MAX_GROUPS (1 << 24)  /* n_out * groups_per_row in
                                                   tq_select_two_plane_noalloc */

/* Output element type for tq_gemv / tq_gemm_smallbatch (the `flags` word). */
#define TQ_OUT_FP16 0   /* fp16, rounded to nearest even from fp32 */
#define TQ_OUT_FP32 1   /* the fp32 accumulator, unrounded */

typedef enum {
  TQ_OK = 0,
  TQ_ERR_NULL = 1,        /* a required pointer is NULL */
  TQ_ERR_SHAPE = 2,       /* a size is out of range or inconsistent */
  TQ_ERR_ALIGN = 3,       /* a pointer is not aligned as required */
  TQ_ERR_UNSUPPORTED = 4, /* a valid request this build does not support */
  TQ_ERR_HIP = 5          /* the HIP runtime reported an error */
} tq_status;

/* Non-owning view of one packed linear (layout above).  When nnz1 == 0 the
 * plane-1 pointers are ignored and may be NULL. */
typedef struct tq_matrix {
  int64_t n_out;            /* N >= 1 */
  int64_t n_in;             /* K >= 128, K % 128 == 0, K/128 <= TQ_MAX_GROUPS_PER_ROW;
                               26 * N * K/128 must be below 2^32 (codes of one
                               matrix under 4 GiB) */
  int32_t group;            /* must be 128 */
  int32_t reserved;         /* must be 0 */
  const uint8_t* codes0;    /* 8-byte aligned */
  const uint16_t* scale0;   /* 2-byte aligned */
  int64_t nnz1;             /* 0 <= nnz1 <= N*G */
  const int32_t* rowptr1;   /* 4-byte aligned; rowptr1[0] == 0, rowptr1[N] == nnz1 */
  const uint16_t* gidx1;
  const uint8_t* codes1;    /* 8-byte aligned */
  const uint16_t* offset1;
  const uint16_t* scale1;
  /* Optional (may be NULL): a HOST copy of rowptr1, read during the call
   * only.  With it the GEMV and the small-batch kernels find every
   * workgroup's records on the host and issue their loads with their first
   * batch, instead of reading the device row pointers first (B = 2..4 use
   * the GEMV's decode only when it is present).  It must hold the same
   * values as rowptr1; if it does not, results are unspecified, but every
   * access stays in bounds. */
  const int32_t* rowptr1_host;
  /* Optional (may be NULL; ABI 3): fp16 [N][G] offset mu0 of EVERY group,
   * the paper's representation (eq. 3 gives every masked block an offset).
   * Each weight of group (r, g) is then mu0[r][g] + s0*t0, plus
   * mu + s1*t1 on two-plane groups; the accuracy bound adds |mu0| to the
   * group's coefficient.  2-byte aligned. */
  const uint16_t* offset0;
} tq_matrix;

/* Version of this ABI (TQ_ABI_VERSION). */
int tq_abi_version(void);

/* Static, human-readable name of a status code. */
const char* tq_status_string(tq_status status);

/* Encode trits to lattice codes (section 12: lossless encoding of the
 * discrete supports).
 *   trits   int8 [n_groups][128], values in {-1, 0, +1}
 *   codes   uint8 [26*n_groups], split layout; 8-byte aligned
 *   n_groups >= 0 (0 is a no-op); group must be 128.
 * A code byte whose five trits include a value outside {-1, 0, +1} is
 * written as 0xFF and counted in *d_err. */
tq_status tq_pack(const int8_t* trits, int64_t n_groups, int32_t group,
                  uint8_t* codes, int32_t* d_err, void* stream);

/* Decode lattice codes to trits (inverse of tq_pack; bit-exact).
 *   codes   uint8 [26*n_groups], split layout; 8-byte aligned
 *   trits   int8 [n_groups][128]
 * A code above 242 decodes to five zero trits and is counted in *d_err.
 * The pad digits of byte 25 are not inspected (see tq_validate). */
tq_status tq_unpack(const uint8_t* codes, int64_t n_groups, int32_t group,
                    int8_t* trits, int32_t* d_err, void* stream);

/* Count invalid bytes of a code buffer into *d_err (required here): codes
 * above 242, and last bytes (byte 25) whose pad digits are not both 1.
 * Section 12 makes the packed buffer the lossless carrier of the discrete
 * supports; section 5.4 reports malformed packed tensors that still gave
 * plausible-looking numbers, and section 15 lists such artifact failures.
 * So a loader checks a buffer once with this call; the GEMV does not. */
tq_status tq_validate(const uint8_t* codes, int64_t n_groups, int32_t group,
                      int32_t* d_err, void* stream);

/* Dense fp16 dequantisation of a packed linear (eq. 3).
 *   w  fp16 [N][K] row-major; 16-byte aligned
 * Each weight is evaluated in fp32 in the fixed order
 *     a = +0;  a += mu0;  a += mu;  a += s0*t0;  a += s1*t1
 * (mu0 only with per-group offsets, mu and s1 only on two-plane groups;
 * s*t is exact) and rounded once to fp16, nearest-even, so the result is
 * bit-exact and unique. */
tq_status tq_unpack_fp16(const tq_matrix* m, uint16_t* w, void* stream);

/* y = W^ x for one fp16 activation vector (the decode-time GEMV).
 *   x  fp16 [K]; 16-byte aligned
 *   y  [N], fp16 (flags = TQ_OUT_FP16) or fp32 (TQ_OUT_FP32); 4-byte aligned
 * Accumulates sign-selected fp16 activations in fp32, applies s0 (and
 * mu0*sum(x_g) with per-group offsets) per group and mu*sum(x_g) +
 * s1*sum(t1*x_g) per two-plane group.  Accuracy:
 * |y - exact| <= 2e-3 * sum_g (|s0| + |mu0| + [two-plane](|mu| + |s1|)) *
 * ||x_g||_1 per output (|mu0| only with per-group offsets).  x and y must
 * not overlap the matrix buffers. */
tq_status tq_gemv(const tq_matrix* m, const uint16_t* x, void* y,
                  int32_t flags, void* stream);

/* Several GEMVs that read the same x in one launch (e.g. q, k and v, or
 * gate and up of one decoder layer).  Section 13 measures the packed decode
 * step of a whole model; in a decoder layer q, k, v read the same normalised
 * input and so do gate and up, so one launch serves each pair or triple.
 *   ms  host array of n matrices (1 <= n <= TQ_MAX_GROUPED), all with the
 *       same K
 *   ys  host array of n device output pointers, ys[i] of N_i elements
 * Each ys[i] equals what tq_gemv(&ms[i], x, ys[i], flags) produces,
 * bit for bit. */
tq_status tq_gemv_grouped(const tq_matrix* ms, int32_t n, const uint16_t* x,
                          void* const* ys, int32_t flags, void* stream);

/* Y = X W^T for a small batch of activations (paper section 18 lists kernel
 * work across batch sizes as the next step).
 *   X  fp16 [B][K] row-major; 16-byte aligned; 1 <= B <= TQ_MAX_BATCH
 *   Y  [B][N] row-major, fp16 or fp32 per flags; 4-byte aligned
 * Same accuracy bound as tq_gemv for every (b, r). */
tq_status tq_gemm_smallbatch(const tq_matrix* m, const uint16_t* X, int32_t B,
                             void* Y, int32_t flags, void* stream);

/* E2M-ATQ ternarisation of 128-weight groups: the planes and scales this
 * format stores, from dense fp16 weights (section 4.2, eqs. 4-6; the
 * representation of section 3, eq. 3).
 *   w          fp16 [n_groups][128], row-major groups; 16-byte aligned
 *   rec_index  int32 [n_groups], or NULL (every group one-plane): -1 for a
 *              one-plane group, k in [0, nnz) for a two-plane group whose
 *              second plane is written as record k (values outside that
 *              range are one-plane).  Records must be distinct: groups
 *              naming the same record, and records no group names, are left
 *              with unspecified contents (always in bounds).
 *   nnz        number of records (rows of t1, offset1, scale1), >= 0
 *   iters      refinement sweeps of every fit that has an offset (two-plane
 *              groups; with offset0 also one-plane groups), 0..1024
 *   t0         int8 [n_groups][128] (16-byte aligned), s0 fp16 [n_groups]
 *   t1         int8 [nnz][128] (16-byte aligned), offset1 and scale1 fp16
 *              [nnz]; may be NULL when nnz == 0
 *   offset0    fp16 [n_groups] or NULL.  Given, every group gets an offset
 *              (the paper's representation, tq_matrix.offset0): one-plane
 *              groups are fitted like the first plane below (mu = mean(w),
 *              then `iters` sweeps of mu <- mean(w - s0*T0),
 *              s0 <- <T0, w - mu>/<T0, T0>), two-plane groups store their mu
 *              here and +0 in offset1.
 *   energy     fp64 [n_groups] or NULL: ||w - mu - s0*T0||^2 of each
 *              group's one-plane fit (mu = 0 without offset0), the ranking
 *              used to choose two-plane groups
 * One-plane groups without offset0: T0 = +1 / -1 where w exceeds
 * +0.75 mean|w| / is below its negation, else 0; s0 = <T0, w> / <T0, T0>
 * (0 on an empty support).
 * Two-plane groups: mu = mean(w); T0, s0 as above on w - mu; T1, s1 the
 * same way on the residual w - mu - s0*T0; then `iters` sweeps updating mu,
 * s0 and s1 in turn with T0, T1 fixed.  Arithmetic is fp64 with every sum
 * in index order; mu, s0, s1 are rounded once to fp16 (nearest even), so
 * results are bit-exact and unique.  All buffers are device memory. */
tq_status tq_ternarize(const uint16_t* w, int64_t n_groups, int32_t group,
                       const int32_t* rec_index, int64_t nnz, int32_t iters,
                       int8_t* t0, uint16_t* s0, int8_t* t1, uint16_t* offset1,
                       uint16_t* scale1, uint16_t* offset0, double* energy,
                       void* stream);

/* Bytes of device workspace tq_select_two_plane needs for n_groups groups
 * (host function; 0 for n_groups < 0). */
size_t tq_select_workspace_bytes(int64_t n_groups);

/* The two-plane groups of a linear and its plane-1 CSR (ABI 5).  Section
 * 4.2 gives a second ternary plane to a minority of blocks; section 3
 * chooses them with salience masks fitted on calibration activations, so
 * without calibration data the ranking is each group's one-plane residual
 * energy (tq_ternarize's `energy`).  The call selects the nnz groups with
 * the largest energy, ties to the lower flat index (groups in row-major
 * (r, g) order); a NaN energy ranks below every number, -0 and +0 tie.
 * Records are numbered in flat order, which is the CSR order by row.
 *   energy          fp64 [n_out * groups_per_row]; 8-byte aligned
 *   n_out >= 1, 1 <= groups_per_row <= TQ_MAX_GROUPS_PER_ROW,
 *   n_out * groups_per_row < 2^31
 *   nnz             0 <= nnz <= n_out * groups_per_row
 *   rec_index       int32 [n_out * groups_per_row] out: the record of each
 *                   group, -1 for one-plane groups (tq_ternarize's input)
 *   rowptr1         int32 [n_out + 1] out (tq_matrix.rowptr1)
 *   gidx1           uint16 [nnz] out (tq_matrix.gidx1); may be NULL when
 *                   nnz == 0
 *   workspace       device scratch of workspace_bytes >=
 *                   tq_select_workspace_bytes(n_out * groups_per_row)
 *                   bytes, 256-byte aligned; its contents on entry do not
 *                   matter and on return are unspecified.  Two calls that
 *                   share a workspace must not overlap in time.
 * All pointers are device memory; 4-byte alignment for rec_index and
 * rowptr1, 2-byte for gidx1.  The result is deterministic and unique. */
tq_status tq_select_two_plane(const double* energy, int64_t n_out, int32_t groups_per_row, int64_t nnz,
                              int32_t* rec_index, int32_t* rowptr1, uint16_t* gidx1,
                              void* workspace, size_t workspace_bytes, void* stream);

/* tq_select_two_plane without a workspace argument (ABI 6), for callers
 * that cannot allocate device memory: code under HIP graph capture, serving
 * loops that must not call hipMalloc, harnesses that forbid it.  Same
 * arguments (less the workspace), same result bit for bit.  The scratch is
 * a static array in the library, one per GPU (about 65 KB, held until the
 * process ends), sized for n_out * groups_per_row <=
 * TQ_SELECT_NOALLOC_MAX_GROUPS; larger requests return TQ_ERR_UNSUPPORTED
 * before anything is launched.  The call allocates nothing.  Every call on
 * one GPU shares that GPU's scratch, so calls that overlap in time on one
 * GPU (other streams, other host threads) race and give unspecified
 * results; order them on one stream. */
tq_status tq_select_two_plane_noalloc(const double* energy, int64_t n_out, int32_t groups_per_row, int64_t nnz,
                                      int32_t* rec_index, int32_t* rowptr1, uint16_t* gidx1, void* stream);

/* ------------------------------------------------------------------------
 * Decode-step chain (ABI 7): a sequence of dependent grouped GEMVs in one
 * launch.  Section 13 runs the packed model's whole decode step; within a
 * decoder layer q, k and v read one input, o the attention output, gate and
 * up the normalised residual and down the activated MLP state, so at batch
 * 1 the step is a chain of GEMVs, each waiting for the one before.  Stage s
 * computes exactly what tq_gemv_grouped(stage s) computes (bit for bit),
 * and reads its x only after every output of stage s - 1 is written, so x
 * may be (or be derived by device code in a later design from) an earlier
 * stage's output.  One cooperative launch of one 1024-thread workgroup per
 * CU runs every stage; each workgroup keeps the decode table across stages.
 */
typedef struct tq_stage {
  const tq_matrix* mats;   /* host array of n matrices, all with the same n_in */
  int32_t n;               /* 1 .. TQ_MAX_GROUPED */
  int32_t flags;           /* TQ_OUT_FP16 or TQ_OUT_FP32 */
  const uint16_t* x;       /* device fp16 [n_in]; 16-byte aligned */
  void* const* ys;         /* host array of n device outputs (4-byte aligned) */
} tq_stage;

typedef struct tq_chain_info {
  int32_t n_stages;
  int32_t n_workgroups;    /* one per CU of the device current at planning */
  int32_t lds_bytes;       /* dynamic LDS per workgroup */
  int32_t reserved;
  int64_t plan_bytes;      /* 128 * n_stages * n_workgroups */
  int64_t sync_bytes;      /* 256 + 64 * n_workgroups */
} tq_chain_info;

/* Plan a chain for the current device.  Checks every stage (as tq_gemv_
 * grouped does) and fills *info.  With plan_host != NULL it also writes the
 * plan, a table of info->plan_bytes bytes of device pointers and row
 * ranges, into that HOST buffer (plan_host_bytes >= info->plan_bytes); the
 * caller copies it unchanged to device memory (128-byte aligned) and keeps
 * every buffer the stages name alive while the plan is used.  Record
 * ranges come from the matrices' host row pointers where present.  Returns
 * TQ_ERR_UNSUPPORTED for a stage that does not fit one round of workgroups
 * (more than 6 row passes per workgroup) or the LDS. */
tq_status tq_chain_plan(const tq_stage* stages, int32_t n_stages, tq_chain_info* info,
                        void* plan_host, size_t plan_host_bytes);

/* Zero a sync block (device memory, info->sync_bytes bytes, 256-byte
 * aligned) on `stream`; required once before its first tq_gemv_chain and
 * whenever it is reused for a plan with another stage count.  Layout: word
 * 0 counts completed calls, word 2 (int32 at byte 8) is a sticky error flag
 * that a call sets when one of its waits gave up (after about 0.1 s; the
 * outputs of that call are then unspecified), then one 64-byte slot per
 * workgroup. */
tq_status tq_chain_sync_init(void* sync, const tq_chain_info* info, void* stream);

/* Run every stage of a planned chain on `stream` (one launch).  `plan` is
 * the device copy of the plan, `sync` a sync block of this plan.  Calls on
 * one sync block must not overlap in time. */
tq_status tq_gemv_chain(const void* plan, void* sync, const tq_chain_info* info, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TQ_H */
