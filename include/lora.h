/*
 * lora.h -- C ABI of the mixed-adapter LoRA layer for AMD Instinct MI355X (gfx950).
 *
 * What it computes.  For a batch of n token rows, each carrying an adapter id,
 * the residual term of the adapted linear layer of the paper's Section 3.4
 * (LoRA layer equation  y = x W^T + s_a (x A_a^T) B_a^T,  with
 * A_a in R^{r_a x d_in}, B_a in R^{d_out x r_a}, s_a = alpha_a / r_a):
 *
 *   forward   Y[t, :] += s_a * (X[t, :] A_a^T) B_a^T        for every row t with id a >= 0
 *   backward  dB_a = s_a * dY_m^T (X_m A_a^T)      [d_out, r_a]
 *             dA_a = s_a * (dY_m B_a)^T X_m        [r_a, d_in]
 *
 * where X_m, dY_m are the rows of adapter a whose loss mask is nonzero.  The
 * forward follows the gather-group-compute-scatter structure of Section 3.4 and
 * Figure 2: rows are grouped by adapter id (the "plan"), the per-group residual
 * Delta_a = s_a (X_a A_a^T) B_a^T is computed and added back to the original
 * rows.  The dense base term x W^T is not part of this library: Y arrives
 * holding it.  The backward is the chain rule on the same equation, with the
 * explicit loss mask of Section 3.3 and the adapter-local gradients of
 * Section 3.5 ("Batch routing").
 *
 * Conventions (every entry point).
 *  - Matrices are row-major; leading dimensions are in elements.
 *    X [n, ldx >= d_in], Y and dY [n, ld >= d_out], H [n, ldh >= r_max] (float).
 *    A_a [r_a, d_in] and B_a [d_out, r_a] are dense row-major (leading dim d_in, r_a).
 *  - Every device buffer, including workspaces, is allocated by the caller.
 *    The library never allocates device memory.  Host objects (lora_table,
 *    lora_plan) are allocated by the library and freed by *_destroy.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Every op is
 *    asynchronous on that stream; only lora_plan_export and lora_plan_check
 *    wait for it.
 *  - Argument errors are detected on the host before anything is enqueued, so a
 *    call that returns an error has written nothing.  Data errors that only the
 *    device can see (bad ids, malformed segments) set a sticky flag in the plan
 *    workspace; the offending rows are treated as having no adapter, and
 *    lora_plan_check reports the flag.
 *  - Device pointers must be 16-byte aligned; d_in and d_out must be multiples
 *    of 8, leading dimensions multiples of 8 (elements).
 *  - X / Y, dY / dA / dB and H must not overlap each other.
 *  - Results are deterministic: the same inputs give the same bytes, run to run.
 */
#ifndef LORA_MI355X_H
#define LORA_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LORA_ABI_VERSION 1
#define LORA_MAX_RANK    128        /* 1 <= r_a <= LORA_MAX_RANK */
#define LORA_MAX_SLOTS   1024       /* table slots per layer */
#define LORA_MAX_ROWS    (1 << 22)  /* rows per batch */
#define LORA_MAX_DIM     65536      /* d_in, d_out */

typedef enum lora_status {
  LORA_OK = 0,
  LORA_ERR_NULL = 1,        /* a required pointer is NULL */
  LORA_ERR_SHAPE = 2,       /* a size or leading dimension is out of range */
  LORA_ERR_DTYPE = 3,       /* dtype combination not supported */
  LORA_ERR_ALIGN = 4,       /* pointer or leading dimension misaligned */
  LORA_ERR_RANK = 5,        /* rank outside [1, LORA_MAX_RANK] */
  LORA_ERR_SLOT = 6,        /* slot index outside [0, num_slots) */
  LORA_ERR_DATA = 7,        /* the device flagged bad ids or segments (lora_plan_check) */
  LORA_ERR_WORKSPACE = 8,   /* workspace too small */
  LORA_ERR_HIP = 9,         /* a HIP runtime call failed */
  LORA_ERR_VALUE = 10,      /* a hyperparameter or step number is out of range */
  LORA_ERR_ALIAS = 11       /* debug build: an output overlaps an input or another output
                               (the call enqueued nothing) */
} lora_status;

typedef enum lora_dtype { LORA_F32 = 0, LORA_BF16 = 1 } lora_dtype;

/* bits of the device data-error flag (lora_plan_check, lora_plan_export) */
#define LORA_DATA_BAD_ID       1u   /* an id outside [-1, num_slots) */
#define LORA_DATA_EMPTY_SLOT   2u   /* an id naming a slot with no adapter */
#define LORA_DATA_BAD_SEGMENTS 4u   /* seg_offsets not 0 = o_0 <= o_1 <= ... = n */
#define LORA_DATA_BOUNDS       8u   /* debug build: a kernel read a plan value (row id,
                                       adapter id) outside its bound; it used an in-range
                                       value instead, so that call's results are void */

typedef struct lora_table lora_table;
typedef struct lora_plan lora_plan;

/* ---- library ----------------------------------------------------------- */
int32_t     lora_abi_version(void);
const char* lora_status_string(lora_status s);
/* Human-readable detail of the last error returned on this thread. */
const char* lora_last_error(void);

/* ---- debug build ---------------------------------------------------------
 * The library is also built as liblora_mi355x_debug.so: the same entry points
 * and results, plus checks that the release library leaves out.
 *  - Before enqueuing anything, every op checks that its outputs overlap
 *    neither its inputs (row-indexed matrices, the table's adapter weights,
 *    the id array) nor each other nor the workspace, and returns
 *    LORA_ERR_ALIAS if they do (X / Y, dY / dA / dB and H must be disjoint;
 *    the release library leaves the result of an overlapping call undefined).
 *  - Every kernel that reads the plan checks each row id and adapter id it
 *    takes from it against [0, n) and [0, num_slots) before using it as an
 *    index; a value out of range sets LORA_DATA_BOUNDS in the plan's data flag
 *    (read by lora_plan_check) and is replaced by 0, so that no access leaves
 *    the caller's buffers.
 * lora_build_flags returns LORA_BUILD_DEBUG in the debug library, 0 in the
 * release one. */
#define LORA_BUILD_DEBUG 1
int32_t     lora_build_flags(void);
/* Test hook of the debug library: overwrite entry `index` of one plan array
 * of row ids with `value`, after the work already on `stream` and before any
 * later work (the call waits for the stream), so that a test can check that
 * the kernels' bounds checks catch a bad plan.  Arrays: LORA_PLAN_PERM, the
 * active rows in group order [n]; LORA_PLAN_M_PERM, the trainable rows [n];
 * LORA_PLAN_SMALL_ROW, row index % 16 of small-group record index / 16.  The
 * release library returns LORA_ERR_VALUE and writes nothing.  Errors: NULL,
 * VALUE (unknown array, index past the array's capacity), HIP. */
#define LORA_PLAN_PERM      0
#define LORA_PLAN_M_PERM    1
#define LORA_PLAN_SMALL_ROW 2
lora_status lora_debug_plan_poke(lora_plan* p, int32_t array, int32_t index, int32_t value,
                                 void* stream);

/* ---- adapter table (Section 3.4, "Adapter table") -----------------------
 * One table per adapted layer.  A slot holds one pinned adapter version: its
 * rank, scale and layer-local A/B pointers.  The identity / version ->
 * slot mapping and residency belong to the caller.  Slot contract (the
 * paper's refresh rule for the adapter table): new weights go into a free slot,
 * and a slot that some plan still references is not set, cleared or uploaded
 * until every launch using that plan has finished.
 *
 * dev_meta: caller device memory of lora_table_device_bytes(num_slots) bytes
 * that receives the slot metadata on lora_table_upload.  It must outlive the
 * table and every plan built on it.  w_dtype is the storage type of every A_a
 * and B_a (LORA_BF16 or LORA_F32).  Errors: NULL, SHAPE (num_slots not in
 * [1, LORA_MAX_SLOTS], d_in / d_out not in [8, LORA_MAX_DIM] or not multiples
 * of 8), DTYPE, ALIGN, WORKSPACE (dev_meta_bytes too small). */
size_t      lora_table_device_bytes(int32_t num_slots);
lora_status lora_table_create(int32_t num_slots, int32_t d_in, int32_t d_out,
                              lora_dtype w_dtype, void* dev_meta, size_t dev_meta_bytes,
                              lora_table** out);
/* Host-side update of one slot; takes effect on the device at the next
 * lora_table_upload.  A: device [rank, d_in], B: device [d_out, rank], both
 * 16-byte aligned and owned by the caller.  Errors: NULL, SLOT, RANK, ALIGN. */
lora_status lora_table_set(lora_table* t, int32_t slot, int32_t rank, float scale,
                           const void* A, const void* B);
/* Mark a slot empty (rows naming it are a data error).  Errors: NULL, SLOT. */
lora_status lora_table_clear(lora_table* t, int32_t slot);
/* Stream-ordered copy of the host metadata into dev_meta.  The host copy may be
 * changed again as soon as this returns. */
lora_status lora_table_upload(lora_table* t, void* stream);
void        lora_table_destroy(lora_table* t);

/* ---- plan: grouping of rows by adapter (Section 3.4 gather step, Figure 2;
 *      Section 3.5 routing by adapter identity) ---------------------------
 * Built on the device, with no host synchronisation.  For S = num_slots it
 * produces, in the caller's workspace `ws` (lora_plan_workspace_bytes bytes):
 *   counts[a]          rows with id a
 *   offsets[0..S]      exclusive prefix sum of counts
 *   perm[0..n_act)     row indices grouped by adapter, ascending inside a group
 *   runs               maximal runs [start, start+len) of one adapter id >= 0
 *   m_counts, m_offsets, m_perm   the same grouping over rows with mask != 0
 *                      (mask == NULL: every row)
 * plus the tile lists the ops launch over.  An id outside [-1, S), or naming an
 * empty slot, sets the data flag and the row is treated as id -1.
 *
 * idx: device int32 [n], -1 = no adapter.  mask: device uint8 [n] or NULL;
 * nonzero = the row's target token is trainable.  The explicit mask is kept
 * apart from the learning signal (Section 3.3): a trainable row whose dY is zero
 * still counts.  The table, idx, mask and ws must stay valid until every op
 * using the plan has finished.  A plan records the table's slot contents
 * (weight pointers, ranks, scales) as uploaded when it is built: after
 * lora_table_set / lora_table_clear + lora_table_upload, build the plan again
 * before using it.  Errors: NULL, SHAPE (n not in [0, LORA_MAX_ROWS]), ALIGN,
 * WORKSPACE, HIP. */
size_t      lora_plan_workspace_bytes(int32_t n, int32_t num_slots);
lora_status lora_plan_build(const lora_table* t, int32_t n, const int32_t* idx,
                            const uint8_t* mask, void* ws, size_t ws_bytes, void* stream,
                            lora_plan** out);
/* The same plan from contiguous segments: rows [seg_offsets[s], seg_offsets[s+1])
 * carry id seg_adapter[s] (device int32 arrays of num_segs+1 and num_segs
 * entries).  Adjacent segments of one adapter merge into one run; empty
 * segments are allowed.  If seg_offsets is not 0 = o_0 <= ... <= o_S = n, the
 * LORA_DATA_BAD_SEGMENTS flag is set and every row is treated as id -1. */
lora_status lora_plan_build_segments(const lora_table* t, int32_t n, int32_t num_segs,
                                     const int32_t* seg_offsets, const int32_t* seg_adapter,
                                     const uint8_t* mask, void* ws, size_t ws_bytes,
                                     void* stream, lora_plan** out);
/* Path selection (testing and tuning).  Every op picks its kernels from the
 * plan and the shapes; a policy given to lora_plan_build_policy replaces those
 * choices for every op run on that plan.  -1 in a field keeps the library's
 * choice (lora_policy_init sets every field to -1).  No setting changes what is
 * computed, only which kernels compute it: results agree within each op's
 * floating-point tolerance, and bit for bit on integer-exact inputs.  The
 * library reads no environment variables and has no process-wide settings.
 * Errors: VALUE (a field outside its range), and those of lora_plan_build. */
typedef struct lora_policy {
  int32_t small_max;     /* groups of <= small_max rows take the small-group kernels, >= 0
                            (-1: every group when n <= 1024; groups of <= 32 rows when
                            n < 64 x num_slots; none otherwise) */
  int32_t small_split;   /* small groups: 0 = one fused kernel, 1 = shrink per d-slice + expand
                            (-1: split when d_in >= 1024) */
  int32_t split_slices;  /* d-slices of the split small-group shrink, 1..8 (-1: min(4, d_in / 256)) */
  int32_t small_chunks;  /* output-column chunks per small group, 1..16 (-1: ceil(d_out / 1024)) */
  int32_t fork;          /* mixed batch in lora_apply: 0 = one stream, 1 = small groups on the
                            second stream (-1: when n < 64 x num_slots) */
  int32_t grad_splits;   /* most d-slices of the gradient's first stage, 1..8
                            (-1: ceil(min(d_in, d_out) / 512)) */
  int32_t block_rows;    /* rows per block of the large groups, 64 or 256 (-1: 64 when
                            n < 12288, else 256); only that size's kernels are launched */
} lora_policy;
void        lora_policy_init(lora_policy* q);
lora_status lora_plan_build_policy(const lora_table* t, int32_t n, const int32_t* idx,
                                   const uint8_t* mask, const lora_policy* policy, void* ws,
                                   size_t ws_bytes, void* stream, lora_plan** out);
/* Copy the plan arrays to host memory (each pointer may be NULL to skip it) and
 * wait for the stream.  Sizes: counts, m_counts [S]; offsets, m_offsets [S+1];
 * perm, m_perm, run_start, run_len, run_adapter [n] (only the first n_act /
 * m_n_act / n_runs entries are meaningful); scalars [1]. */
lora_status lora_plan_export(const lora_plan* p, int32_t* counts, int32_t* offsets,
                             int32_t* perm, int32_t* n_runs, int32_t* run_start,
                             int32_t* run_len, int32_t* run_adapter, int32_t* m_counts,
                             int32_t* m_offsets, int32_t* m_perm, uint32_t* data_flags,
                             void* stream);
/* Wait for the stream and read the sticky data flag (LORA_DATA_* bits) into
 * *data_flags (nullable).  Returns LORA_ERR_DATA if any bit is set. */
lora_status lora_plan_check(const lora_plan* p, uint32_t* data_flags, void* stream);
void        lora_plan_destroy(lora_plan* p);

/* ---- forward ops (Section 3.4: LoRA layer equation, Delta_a) ------------
 * dtypes: X and the table weights are both LORA_BF16 (matrix-core path) or any
 * mix of LORA_BF16 / LORA_F32 (vector path); Y is LORA_BF16 or LORA_F32.
 * Arithmetic: products of the stored values, accumulated in float32; the
 * intermediate H = X A_a^T is kept in float32 (split into two bfloat16 terms
 * when it feeds a bfloat16 matrix product); s_a is applied once to the float32
 * accumulator; a bfloat16 Y is rounded to nearest even once, at the store.
 * Rows with id -1 are neither read nor written.  Row-indexed matrices (X, Y,
 * H, dY, H_saved) are device pointers with leading dimension a multiple of 8
 * and 16-byte alignment; for a plan with n = 0 they are never touched and may
 * be NULL.  Errors: NULL, DTYPE, SHAPE, ALIGN, WORKSPACE, HIP. */

/* lora_shrink (gather + shrink): H[t, 0:r_a] = X[t, :] A_a^T (unscaled) for
 * every row t with id a >= 0.  H is float32 [n, ldh], ldh >= max rank over the
 * table; columns >= r_a and rows with id -1 are left untouched. */
lora_status lora_shrink(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                        float* H, int64_t ldh, void* stream);
/* lora_expand (expand + scatter-add): Y[t, :] += s_a * H[t, 0:r_a] B_a^T for every
 * row t with id a >= 0, in the original row order. */
lora_status lora_expand(const lora_plan* p, const float* H, int64_t ldh, void* Y,
                        lora_dtype y_dtype, int64_t ldy, void* stream);
/* lora_apply: shrink and expand in one call, Y[t] += s_a (X[t] A_a^T) B_a^T.
 * Small adapter groups (decode rows) run either a shrink per d-slice plus an
 * expand, with partial H in the workspace (d_in >= 1024), or one fused kernel
 * that keeps H on chip; larger groups (prefill segments) run a grouped
 * matrix-core shrink and expand through the workspace.  ws: device,
 * lora_apply_workspace_bytes(p) bytes, 16-byte aligned; it may be NULL only
 * when every group is small (the fused kernel then runs).  A batch with fewer
 * than 64 rows per table slot that has large groups runs its small-group
 * kernels on a library-owned second stream of the current device, forked from
 * and joined back into `stream` with events (so later work on `stream` and a
 * graph captured from it see the whole update); concurrent calls on one
 * device take a host mutex around that sequence. */
size_t      lora_apply_workspace_bytes(const lora_plan* p);
lora_status lora_apply(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                       void* Y, lora_dtype y_dtype, int64_t ldy, void* ws, size_t ws_bytes,
                       void* stream);

/* lora_apply without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same kernels and the same result as lora_apply, bit
 * for bit, always on `stream` alone (no second stream).  The workspace is a
 * fixed array of LORA_NOALLOC_SCRATCH_BYTES in the library's code object, one
 * per GPU, held until the process ends; its device address is looked up on the
 * first call on each device.  The call allocates nothing: no hipMalloc,
 * hipFree or allocating library routine.  Every call on one GPU shares that
 * GPU's array, so calls that overlap on one GPU (concurrent streams, or
 * replays of graphs holding this call that overlap) race and give undefined
 * results; calls ordered on one stream are safe (nothing is carried from one
 * call to the next: every byte the kernels read is written earlier in the same
 * call).  Errors: those of lora_apply, and LORA_ERR_WORKSPACE when
 * lora_apply_workspace_bytes(p) exceeds LORA_NOALLOC_SCRATCH_BYTES (nothing
 * is enqueued then). */
#define LORA_NOALLOC_SCRATCH_BYTES (32u << 20)
lora_status lora_apply_noalloc(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                               void* Y, lora_dtype y_dtype, int64_t ldy, void* stream);

/* lora_apply_ids: lora_apply for a small batch without a plan (the decode
 * step of Section 3.4: every row's adapter residual with its rows grouped by
 * adapter, here inside the kernels).  Two launches and nothing before them:
 * a shrink per (slot, d-slice) into the workspace's partial H planes and an
 * expand per (slot, output-column chunk); each workgroup finds the rows
 * T_a = {t : idx[t] = a} of its slot by scanning idx (ascending t).  Y[t] +=
 * s_a (X[t] A_a^T) B_a^T for every row whose id names a slot with an adapter;
 * rows with id -1, an id outside [-1, num_slots) or an id of an empty slot are
 * left unchanged (as lora_apply treats them; lora_plan_build and
 * lora_plan_export report such ids).  Arithmetic and result: those of
 * lora_apply's split small-group path.  idx: device int32 [n], 4-byte aligned;
 * 0 <= n <= LORA_APPLY_IDS_MAX_ROWS.  X bfloat16 [n, ldx], weights bfloat16
 * (else LORA_ERR_DTYPE); Y float32 or bfloat16 [n, ldy], updated in place.
 * ws: device, lora_apply_ids_workspace_bytes(t, n) bytes (0 when n = 0 or no
 * slot holds an adapter), 16-byte aligned.  The table's metadata must have been
 * uploaded.  Errors: NULL, SHAPE (n out of range), DTYPE, ALIGN, WORKSPACE,
 * HIP; nothing is enqueued on an error. */
#define LORA_APPLY_IDS_MAX_ROWS 1024
size_t      lora_apply_ids_workspace_bytes(const lora_table* t, int32_t n);
lora_status lora_apply_ids(const lora_table* t, int32_t n, const int32_t* idx, const void* X,
                           lora_dtype x_dtype, int64_t ldx, void* Y, lora_dtype y_dtype,
                           int64_t ldy, void* ws, size_t ws_bytes, void* stream);

/* ---- the whole adapted layer (Section 3.4: LoRA layer equation, with the
 *      base projection shared by every row and the residual added per group) --
 *   Y[t, :] = X[t, :] W^T + s_a (X[t, :] A_a^T) B_a^T     for a row with adapter a,
 *   Y[t, :] = X[t, :] W^T                                  for a row with id -1.
 * W: device bfloat16 [d_out, ldw >= d_in] row-major (the base layer's weight,
 * one for every row).  X: bfloat16 [n, ldx].  Y: float32 or bfloat16 [n, ldy],
 * written (not accumulated; one rounding per element for bfloat16) and not
 * read; it must not overlap X or W.  The table's adapter weights must be
 * bfloat16.  Arithmetic: bfloat16 products accumulated in float32; the
 * residual's H = X A_a^T is kept in float32 and split into two bfloat16 terms
 * before it meets B_a, with s_a applied to it first.  Two launches: the
 * grouped shrink (H of every adapter row, into the workspace) and one
 * matrix-core GEMM whose epilogue adds the residual of each maximal run of
 * one adapter crossing a 256-row tile (it is built for segment batches:
 * a tile crossed by many runs, as in a decode batch, pays one rank step per
 * run).  ws: lora_linear_workspace_bytes(p) bytes, 16-byte aligned.  Errors:
 * NULL, DTYPE (anything but bfloat16 X, W, weights), SHAPE (ldw < d_in, Y
 * overlapping X or W, a leading dimension above 2^21 elements), ALIGN,
 * WORKSPACE, HIP. */
size_t      lora_linear_workspace_bytes(const lora_plan* p);
lora_status lora_linear(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                        const void* W, lora_dtype w_dtype, int64_t ldw, void* Y,
                        lora_dtype y_dtype, int64_t ldy, void* ws, size_t ws_bytes,
                        void* stream);

/* ---- measurement utility (not part of the layer) ---------------------------
 * A register-only loop of bf16 matrix-core products: `workgroups` x 4 waves,
 * each running iters x 16 independent v_mfma_f32_32x32x16_bf16 (32768 flops
 * each), so one call performs workgroups * 4 * iters * 16 * 32768 flops.  Its
 * timed rate is the achieved matrix-core peak on the device (the benchmark's
 * calibration).  out: device float [workgroups * 256] (receives the sums, so the
 * products are not optimised away).  Errors: SHAPE, NULL, HIP. */
lora_status lora_calibrate_mfma(int32_t workgroups, int32_t iters, float* out, void* stream);

/* ---- backward (Sections 3.3 and 3.5: masked, adapter-local gradients) ----
 * For every slot a with dA[a] / dB[a] not NULL, over the rows T_a^m of the
 * plan's mask (mask == NULL at build time: every row of adapter a):
 *   dB_a = s_a dY_m^T H,  dA_a = s_a (dY_m B_a)^T X_m,  H = X_m A_a^T (or H_saved).
 * Rows outside T_a^m are never read, so they contribute exactly zero even if
 * they hold NaN or Inf.  accumulate = 0: overwrite (slots with no trainable row
 * get +0.0); accumulate != 0: add to the existing values.
 * dA, dB: HOST arrays of num_slots DEVICE pointers to float32 [r_a, d_in] and
 * [d_out, r_a] buffers (NULL = skip that slot).  The pointer arrays are copied
 * before the call returns.  H_saved: float32 [n, ldh] from lora_shrink, or NULL
 * to recompute.  x_dtype and dy_dtype must equal each other; the matrix-core
 * path needs LORA_BF16 inputs and weights.  ws: lora_grad_workspace_bytes(p).
 * The reduction over rows runs in a fixed order (no floating-point atomics). */
size_t      lora_grad_workspace_bytes(const lora_plan* p);
lora_status lora_grad(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                      const void* dY, lora_dtype dy_dtype, int64_t lddy, const float* H_saved,
                      int64_t ldh, float* const* dA, float* const* dB, int32_t accumulate,
                      void* ws, size_t ws_bytes, void* stream);

/* Input gradient through the adapter residual (the chain rule on the LoRA
 * layer equation of Section 3.4 with respect to x; same masked rows T_a^m as
 * lora_grad, Sections 3.3 and 3.5):
 *     dX[t] += s_a (dY[t] B_a) A_a      for every t in T_a^m,
 * every other row of dX untouched (rows with mask 0 or id -1 are never read).
 * dY: device [n, lddy] bfloat16 (the table's weights must be bfloat16 too);
 * dX: device [n, lddx] float32 or bfloat16, updated in place (one rounding
 * per element for bfloat16).  ws: lora_grad_x_workspace_bytes(p) bytes,
 * 16-byte aligned.  Errors: LORA_ERR_DTYPE for other dtypes, and the common
 * argument errors.  Asynchronous on stream. */
size_t      lora_grad_x_workspace_bytes(const lora_plan* p);
lora_status lora_grad_x(const lora_plan* p, const void* dY, lora_dtype dy_dtype, int64_t lddy,
                        void* dX, lora_dtype dx_dtype, int64_t lddx, void* ws, size_t ws_bytes,
                        void* stream);

/* Both gradients of one backward step in one call: lora_grad's dA_a / dB_a
 * and lora_grad_x's dX, with exactly their results (same kernels, same
 * arguments and semantics as the two calls).  The input gradient runs on a
 * library-owned second stream of the stream's device, forked from and joined
 * back into `stream` with events, beside the adapter gradients; both read the
 * plan and dY as they are when the call is made.  ws:
 * lora_backward_workspace_bytes(p) bytes, 16-byte aligned.  Needs bfloat16 dY
 * and weights (the input gradient's matrix-core path).  Errors: those of the
 * two calls, all checked before anything is enqueued. */
size_t      lora_backward_workspace_bytes(const lora_plan* p);
lora_status lora_backward(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                          const void* dY, lora_dtype dy_dtype, int64_t lddy, const float* H_saved,
                          int64_t ldh, float* const* dA, float* const* dB, int32_t accumulate,
                          void* dX, lora_dtype dx_dtype, int64_t lddx, void* ws, size_t ws_bytes,
                          void* stream);

/* ---- adapter-local optimizer step (Section 3.5: gradients, optimizer
 *      moments and step counters stay local to the owning policy, and each
 *      policy issues its own optimizer step) ------------------------------
 * The paper names no optimizer; the update is the published AdamW (Adam's
 * bias-corrected moment estimates, weight decay decoupled from the gradient),
 * elementwise over one tensor's fp32 state, with t = step:
 *     m <- beta1 m + (1 - beta1) g
 *     v <- beta2 v + (1 - beta2) g^2
 *     p <- p - lr (mhat / (sqrt(vhat) + eps) + weight_decay p),
 *     mhat = m / (1 - beta1^t),  vhat = v / (1 - beta2^t)
 * (the decay uses p before the step).  Arithmetic is fp32, with the per-step
 * constants 1 - lr wd, lr / (1 - beta1^t) and 1 / sqrt(1 - beta2^t) formed in
 * double on the host.  One call updates any number of tensors (e.g. every
 * dA_a and dB_a of the adapters that stepped, each with its own moments, step
 * count and hyperparameters) in one launch per 32 tensors. */
typedef struct lora_adamw_tensor {
  float* p;             /* device [n] fp32 master values, updated in place */
  float* m;             /* device [n] first moment, updated in place (zeros before step 1) */
  float* v;             /* device [n] second moment, updated in place (zeros before step 1) */
  const float* g;       /* device [n] gradient, e.g. dA_a or dB_a from lora_grad (same layout as p) */
  void* p_bf16;         /* nullable device [n] bfloat16: receives p after the update, rounded
                           to nearest even (e.g. the table's A_a or B_a) */
  int64_t n;            /* elements (0: the tensor is skipped) */
  int32_t step;         /* t >= 1: this update's number in this tensor's own count */
  float lr;             /* >= 0 */
  float beta1, beta2;   /* in [0, 1) */
  float eps;            /* > 0 */
  float weight_decay;   /* >= 0 */
} lora_adamw_tensor;

/* tensors: host array of `count` records (count >= 0), read before return.
 * p, m, v, g and p_bf16 must be 16-byte aligned; no two of one record's arrays
 * may overlap, and no array may overlap another record's.  Non-finite
 * gradients propagate into p, m and v.  Errors: NULL (tensors, or an array of
 * a record with n > 0), SHAPE (count < 0, n < 0, overlapping arrays, except
 * gradients shared read-only), ALIGN, VALUE (step < 1,
 * a hyperparameter out of its range or not finite), HIP.  Nothing is enqueued
 * unless every record is valid.  Asynchronous on stream. */
lora_status lora_adamw_step(const lora_adamw_tensor* tensors, int32_t count, void* stream);

/* ---- masked token-level losses -> gradient at the logits (Section 3.3: SFT
 *      weights w_t on the target-token axis; for RL the explicit action mask
 *      m_t, rollout log-probabilities l_old, advantages A_t and optional
 *      correction weights c_t on the same axis; Section 3.5, "Forward/backward
 *      path": cross-entropy, importance-sampling and PPO-style objectives) -----
 * The paper names the objectives; their forms here are the standard ones,
 * summed over positions (advantages arrive already normalised by the response
 * length, as the paper's data path sends them).  For row t with logits z_t:
 *     logp_t = z_t[y_t] - log sum_v exp(z_t[v])
 *     LORA_LOSS_CE:  L_t = -w_t logp_t                          (row active iff w_t != 0)
 *     LORA_LOSS_IS:  L_t = -m_t c_t A_t rho_t,  rho_t = exp(logp_t - l_old_t)
 *     LORA_LOSS_PPO: L_t = -m_t c_t min(rho_t A_t, clip(rho_t, 1 - clip_lo, 1 + clip_hi) A_t)
 *                    (IS / PPO rows active iff m_t != 0; mask NULL = every row)
 *     dlogits_t = dL_t / dz_t = g_t (softmax(z_t) - onehot(y_t)),  g_t = -dL_t / dlogp_t
 *     (PPO: g_t = m_t c_t A_t rho_t where the unclipped term is the minimum,
 *     ties included, else 0).
 * Inactive rows: their logits are never read, loss = logp = 0, and their
 * gradient row is written as zeros.  An active row whose target is outside
 * [0, vocab) gets NaN loss, logp and gradient row.
 * logits: device [n, ldz] float32 or bfloat16 (ldz >= vocab, a multiple of 8,
 * 16-byte aligned; the padding of each row up to the next multiple of 8 is
 * read, never used).  target: device int32 [n].  weight: device float32 [n]
 * (CE only, required).  mask: device uint8 [n] (IS / PPO, nullable).
 * old_logp, adv: device float32 [n] (IS / PPO, required).  corr: device float32
 * [n] (IS / PPO, nullable = 1).  clip_lo, clip_hi >= 0 (PPO).
 * loss: device float32 [n] (required); logp: device float32 [n] (nullable).
 * dlogits: device [n, ldd] float32 or bfloat16, written for columns < vocab of
 * every row; it must not overlap logits.  Errors: NULL, SHAPE (n or vocab out
 * of range), DTYPE, ALIGN, VALUE (unknown kind, negative or non-finite clip).
 * Asynchronous on stream. */
typedef enum lora_loss_kind { LORA_LOSS_CE = 0, LORA_LOSS_IS = 1, LORA_LOSS_PPO = 2 } lora_loss_kind;
#define LORA_MAX_VOCAB (1 << 24)
lora_status lora_token_loss(lora_loss_kind kind, int32_t n, int32_t vocab, const void* logits,
                            lora_dtype logits_dtype, int64_t ldz, const int32_t* target,
                            const float* weight, const uint8_t* mask, const float* old_logp,
                            const float* adv, const float* corr, float clip_lo, float clip_hi,
                            float* loss, float* logp, void* dlogits, lora_dtype dlogits_dtype,
                            int64_t ldd, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LORA_MI355X_H */
