// Internal definitions shared by the host runtime (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "lora.h"

namespace lora {

// One table slot as the kernels read it (32 bytes, in caller device memory).
struct SlotMeta {
  const void* A;     // [rank, d_in] row-major
  const void* B;     // [d_out, rank] row-major
  int32_t rank;      // 0 = empty slot
  float scale;       // s_a
  int32_t pad[2];
};
static_assert(sizeof(SlotMeta) == 32, "slot metadata layout");

// Plan header words (int32) at the start of the plan workspace.
enum : int {
  HDR_FLAGS = 0,      // LORA_DATA_* bits
  HDR_NACT = 1,       // rows with an adapter
  HDR_NRUNS = 2,      // maximal runs
  HDR_MNACT = 3,      // trainable rows with an adapter
  HDR_NRB_LARGE = 4,  // row-block entries of large groups (grouped matrix-core path)
  HDR_NRB_TOTAL = 5,  // all entries: large-group blocks, then small-group entries
  HDR_NMRB = 6,       // trainable row-block entries (gradient path)
  HDR_NSMALL = 7,     // small-group records (fused path); equals NRB_TOTAL - NRB_LARGE
  HDR_RB_ROWS = 8,    // rows per large-group block of this plan: RB_ROWS or RB_FINE
  HDR_WORDS = 64
};
static_assert(HDR_FLAGS == 0, "the debug build's bounds checks set bits of header word 0");
static_assert(LORA_DATA_BOUNDS == 8u, "device_common.h's DATA_BOUNDS_BIT");

constexpr int RB_ROWS = 256;     // rows per large-group row block
constexpr int RB_FINE = 64;      // ... when the batch has fewer than FINE_BELOW x RB_ROWS rows
constexpr int FINE_BELOW = 48;
constexpr int SHRINK_KS_MAX = 4; // most d-slices of the grouped shrink inside lora_apply
constexpr int SMALL_ROWS = 16;   // rows per small-group entry (one matrix-core column tile)
constexpr int IDS_MAX_ROWS = 1024;  // most rows of a plan-free (lora_apply_ids) batch
constexpr int MRB_ROWS = 64;     // trainable rows per gradient row block
constexpr int PLAN_THREADS = 1024;
constexpr int PLAN_WAVES = PLAN_THREADS / 64;
// batches of (PLAN_THREADS, PLAN_MULTI_MAX] rows are grouped by two launches over
// chunks of PLAN_THREADS rows; longer ones by one workgroup
constexpr int PLAN_MULTI_MAX = 65536;

// One small-group entry as the fused kernel reads it: everything a workgroup
// needs in one 128-byte line, so the kernel's first memory round trip already
// yields the weight pointers and the row ids.  row[i] for i >= rows repeats the
// last row (a real row, so padding lanes read valid memory).
struct SmallRec {
  const void* A;
  const void* B;
  int32_t rows;
  int32_t rank;
  float scale;
  int32_t adapter;
  int32_t row[SMALL_ROWS];
  int32_t pad[8];
};
static_assert(sizeof(SmallRec) == 128, "small-group record layout");

// Byte offsets of the plan arrays inside the caller's workspace.
struct PlanLayout {
  size_t hdr, counts, offsets, perm, run_start, run_end, run_adapter;
  size_t m_counts, m_offsets, m_perm, m_blk, rb, mrb, srec, seg_ids;
  size_t ch_hist, ch_mhist, ch_runs, ch_flags, minfo, total;   // chunked grouping
  int32_t rb_max, mrb_max, srec_max, chunks;
};

// Device pointers into one plan workspace.
struct PlanDev {
  int32_t* hdr;
  int32_t* counts;
  int32_t* offsets;
  int32_t* perm;
  int32_t* run_start;
  int32_t* run_end;    // last row of each run (lora_plan_export turns it into a length)
  int32_t* run_adapter;
  int32_t* m_counts;
  int32_t* m_offsets;
  int32_t* m_perm;
  int32_t* m_blk;  // first trainable row block of each adapter
  int4* rb;     // {adapter, first index into perm, rows, 0}
  int4* mrb;    // {adapter, first index into m_perm, rows, 0}
  SmallRec* srec;  // small-group records, in the order of the small rb entries
  int32_t* seg_ids;   // packed ids (one workgroup), or per-row id and rank (chunked)
  int32_t* ch_hist;   // chunked grouping: [chunk][adapter] row counts
  int32_t* ch_mhist;  //   ... of trainable rows
  int32_t* ch_runs;   //   [chunk] run starts
  int32_t* ch_flags;  //   [chunk] data flags
  int32_t* minfo;     //   per-row trainable id and rank
  int32_t chunks;     //   chunks of PLAN_THREADS rows (0: not chunked)
};

// Device address of this GPU's fixed scratch array (lora_apply_noalloc),
// looked up once per device: the device of `stream` (NULL: the current one).
hipError_t noalloc_scratch(hipStream_t stream, void** out);

// Groups of at most this many rows take the fused small-group path, and the
// large-group block size (true: RB_FINE rows) of a batch of n rows over S slots.
int32_t small_max_policy(int32_t n, int32_t S);
bool fine_policy(int32_t n);
PlanLayout plan_layout(int32_t n, int32_t num_slots);

// ---- launchers (defined in the .hip files) --------------------------------

struct PlanLaunch {
  PlanDev d;
  const int32_t* idx;           // per-row ids, or nullptr in segment mode
  const int32_t* seg_offsets;   // segment mode
  const int32_t* seg_adapter;
  int32_t num_segs;
  const uint8_t* mask;          // nullable
  const SlotMeta* meta;
  int32_t n, num_slots;
  int32_t small_max;            // groups with <= small_max rows go to the fused small-group path
  int32_t fine;                 // large-group blocks of RB_FINE rows (else RB_ROWS)
};
hipError_t launch_plan(const PlanLaunch& a, hipStream_t s);

// Common description of an op launch.
struct OpLaunch {
  const int32_t* hdr;
  const int4* rb;
  const SmallRec* srec;
  const int32_t* perm;
  const SlotMeta* meta;
  int32_t n, d_in, d_out, num_slots;
  int32_t r_max;
  bool rank8;                   // every live rank is a multiple of 8
  int32_t rb_ub;                // host upper bound of the entry count
  int32_t coarse_ub, fine_ub;   // ... when the plan chose RB_ROWS / RB_FINE blocks (grouped kernels)
  int count_word;               // header word holding the entry count
  int first_word;               // header word holding the first entry (-1: 0)
};

// d-slices of the grouped shrink over `count` entries: enough (entry, slice)
// units to cover the chip once, at most ks_max (the workspace holds that many
// partial planes).  Every reader of the planes uses the same count.
__host__ __device__ __forceinline__ int shrink_slices(int ks_max, int count) {
  const int c = count > 1 ? count : 1;
  const int q = 256 / c;
  const int k = ks_max < q ? ks_max : q;
  return k > 1 ? k : 1;
}

// H[t, :r] = X[t] A^T over entries [first, count) (bf16 X and weights, matrix
// cores).  With ks_max > 1 the kernel may split d_in into up to ks_max slices
// and write one partial plane per slice, plane k at H + k * hp_stride; the
// expand given the same (ks_max, hp_stride) and entries sums them.
hipError_t launch_shrink_mfma(const OpLaunch& o, const void* X, int64_t ldx, float* H,
                              int64_t ldh, int32_t ks_max, int64_t hp_stride, hipStream_t s);
// Y[t] += s H[t, :r] B^T over entries (bf16 weights, matrix cores, hi/lo split of H)
hipError_t launch_expand_mfma(const OpLaunch& o, const float* H, int64_t ldh, int32_t ks_max,
                              int64_t hp_stride, void* Y, lora_dtype y_dtype, int64_t ldy,
                              hipStream_t s);
// input gradient dX += s G A_a with G = dY B_a, over the entries o describes
// (the plan's masked blocks); H holds SHRINK_KS_MAX partial planes
hipError_t launch_grad_x_mfma(const OpLaunch& o, const void* dY, int64_t lddy, float* H, int64_t ldh,
                              int64_t hp_stride, void* dX, lora_dtype dx_dtype, int64_t lddx,
                              hipStream_t s);
// plan-free small batch (lora_apply_ids): shrink per (slot, d-slice) into
// partial planes H [slices][n][16 t] floats (t = 1, 2, 4 or 8 the rank tiles of
// r_max), then expand per (slot, column chunk); every workgroup finds its
// slot's rows in ids itself
struct IdsLaunch {
  const SlotMeta* meta;
  int32_t num_slots, d_in, d_out, r_max;
  bool rank8, y_bf16;
  const int32_t* ids;
  int32_t n;
  const void* X;
  int64_t ldx;
  void* Y;
  int64_t ldy;
  float* H;
  int32_t slices, n_chunks;
};
hipError_t launch_ids_mfma(const IdsLaunch& l, hipStream_t s);
// fused small-group kernel: shrink into LDS + expand, entries [first, count)
hipError_t launch_bgmv_mfma(const OpLaunch& o, const void* X, int64_t ldx, void* Y,
                            lora_dtype y_dtype, int64_t ldy, int32_t n_chunks, hipStream_t s);

// split small-group path: shrink per (record, d-slice) into partial planes
// (part: SPLIT_SLICES_MAX x records x 16 x 16 t floats, t = 1, 2, 4 or 8 the
// rank tiles of r_max), then expand
// per (record, column chunk)
constexpr int SPLIT_SLICES_MAX = 8;
hipError_t launch_small_split_mfma(const OpLaunch& o, const void* X, int64_t ldx, void* Y,
                                   lora_dtype y_dtype, int64_t ldy, int32_t n_chunks,
                                   int32_t slices, float* part, hipStream_t s);

// the whole adapted layer Y = X W^T + s_a (X A_a^T) B_a^T (bf16 X, W and
// weights): one GEMM whose epilogue adds the residual of every run crossing a
// tile, from H = the grouped shrink's ks_max-sliced partial planes
struct LinearLaunch {
  const void* X;
  int64_t ldx;
  const void* W;
  int64_t ldw;
  void* Y;
  int64_t ldy;
  bool y_bf16;
  const int32_t* run_start;
  const int32_t* run_end;
  const int32_t* run_adapter;
  const float* H;
  int64_t ldh;
  int64_t hp_stride;
  int32_t ks_max;
  uint16_t* Hs;        // [n][2 linear_rank_cols(r_max)] bf16: the packed s_a H (rank multiple of 8)
};
int32_t linear_rank_cols(int32_t r_max);

// register-only matrix-core loop (measurement utility): workgroups x 4 waves,
// each iters x 16 v_mfma_f32_32x32x16_bf16; out: workgroups x 256 floats
hipError_t launch_calib_mfma(int32_t workgroups, int32_t iters, float* out, hipStream_t s);
hipError_t launch_linear_mfma(const OpLaunch& o, const LinearLaunch& l, hipStream_t s);

// vector-ALU kernels for any mix of f32 / bf16 storage
hipError_t launch_shrink_valu(const OpLaunch& o, const void* X, lora_dtype x_dtype,
                              int64_t ldx, lora_dtype w_dtype, float* H, int64_t ldh,
                              hipStream_t s);
hipError_t launch_expand_valu(const OpLaunch& o, const float* H, int64_t ldh,
                              lora_dtype w_dtype, void* Y, lora_dtype y_dtype, int64_t ldy,
                              hipStream_t s);

// gradient path
constexpr int GRAD_SLOT_GROUP = 64;   // output pointers passed per launch
constexpr int GRAD_SPLITS_MAX = 8;    // most d-slices (partial planes) of the first stage
struct GradLaunch {
  OpLaunch o;                    // o.rb / o.rb_ub describe the trainable row blocks
  const int32_t* m_perm;
  const int32_t* m_offsets;
  const int32_t* m_counts;
  const int32_t* m_blk;
  const void* X;
  int64_t ldx;
  const void* dY;
  int64_t lddy;
  const float* H_saved;
  int64_t ldh;
  float* const* dA;              // host array [num_slots] of device pointers (nullable entries)
  float* const* dB;
  int32_t accumulate;
  float* hg;                     // workspace: partial H^T and G^T
  int32_t k_splits;
  int32_t p_stride;              // row stride (elements) of the H^T / G^T planes
  int32_t r_pad;                 // rank padding of the planes
  uint16_t* fin;                 // workspace: summed planes, bf16 hi / lo
};

// Byte offsets of the gradient workspace parts.
struct GradLayout {
  size_t partial, fin, total;
};
GradLayout grad_layout(int32_t mrb_ub, int32_t r_max);
hipError_t launch_grad_mfma(const GradLaunch& g, hipStream_t s);
hipError_t launch_grad_valu(const GradLaunch& g, lora_dtype x_dtype, lora_dtype w_dtype,
                            hipStream_t s);

// adapter-local optimizer step: one launch per group of up to ADAMW_GROUP
// tensors, each with the per-step constants the host derives in double
constexpr int ADAMW_GROUP = 32;
struct AdamwLaunch {
  float* p;
  float* m;
  float* v;
  const float* g;
  void* p_bf16;          // nullable
  int64_t n;
  float decay;           // 1 - lr wd
  float step_size;       // lr / (1 - beta1^t)
  float inv_sqrt_bc2;    // 1 / sqrt(1 - beta2^t)
  float eps, beta1, omb1, beta2, omb2;
};
hipError_t launch_adamw(const AdamwLaunch* t, int32_t count, hipStream_t s);

// masked token-level loss and its gradient at the logits, one workgroup per row
struct LossLaunch {
  int32_t kind, n, vocab;
  const void* logits;
  bool logits_bf16;
  int64_t ldz;
  const int32_t* target;
  const float* weight;
  const uint8_t* mask;
  const float* old_logp;
  const float* adv;
  const float* corr;
  float clip_lo, clip_hi;
  float* loss;
  float* logp;
  void* dlogits;
  bool dlogits_bf16;
  int64_t ldd;
};
hipError_t launch_token_loss(const LossLaunch& l, hipStream_t s);

}  // namespace lora
