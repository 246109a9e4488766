// The whole adapted layer of Section 3.4 (LoRA layer equation), for bfloat16
// X, W and adapter weights:
//
//   Y[t] = X[t] W^T + s_a (X[t] A_a^T) B_a^T     (a row with no adapter: X[t] W^T)
//
// The base projection is shared by every row and computed once for all of
// them; the adapter residual is added per group, as the paper structures the
// layer.  Two launches: the grouped shrink writes H = X A_a^T (float32, in
// d-sliced partial planes) for the rows of every adapter group; then one
// matrix-core GEMM computes X W^T tile by tile and, before its store, adds
// s_a H B_a^T for each maximal run of one adapter that crosses the tile, as
// extra rank steps on the same accumulators (H enters the bfloat16 matrix core
// as hi + lo terms).  The output Y is written once; nothing is read back.
//
// GEMM: 256 x 256 output tiles, 4 waves, each wave 128 x 128 as 4 x 4 tiles of
// v_mfma_f32_32x32x16_bf16.  K advances 64 at a time: both operand tiles of a
// step (256 rows of X and 256 rows of W, 64 bf16 each) go straight from global
// memory into LDS (global_load_lds_dwordx4, no registers), double buffered, one
// barrier per step.  Rows are stored 128 bytes apart with the eight 16-byte
// chunks of row R permuted by XOR with f(R) = (R & 7) ^ ((R >> 3) & 1), so that
// the 16 lanes of a fragment read (16 consecutive rows, one chunk) hit 16
// distinct 16-byte bank groups.
//
// Matrix core: lane l holds row l % 32 of the A operand and column l % 32 of
// the B operand, eight consecutive K values at K offset 8 (l / 32); the 16
// accumulator values of lane l sit at rows 8 (v / 4) + 4 (l / 32) + v % 4,
// column l % 32.
#include <algorithm>

#include "device_common.h"
#include "lora_internal.h"

namespace lora {

#ifndef LINEAR_KS
#define LINEAR_KS 64
#define LINEAR_NS 2
#define LINEAR_NTS 1
#define LINEAR_DMA 1
#endif

namespace {

constexpr int LT_M = 256, LT_N = 256;
constexpr int LT_GM = 4;                        // row tiles per group of the tile order
constexpr int LT_SST = 132;                     // row stride (floats) of the store staging

typedef __attribute__((ext_vector_type(16))) float f32x16;

// instruction classes of __builtin_amdgcn_sched_group_barrier
constexpr int SG_MFMA = 0x008, SG_VMEM = 0x010, SG_DS_READ = 0x100;

struct LinArgs {
  const uint16_t* X;
  int64_t ldx;
  const uint16_t* W;
  int64_t ldw;
  void* Y;
  int64_t ldy;
  int32_t n, d_in, d_out;
  int32_t num_slots;
  int32_t m_tiles, n_tiles;
  const int32_t* hdr;
  const int32_t* run_start;
  const int32_t* run_end;       // last row of each run
  const int32_t* run_adapter;
  const SlotMeta* meta;
  const float* H;               // partial planes of the grouped shrink
  int64_t ldh;
  int64_t hp_stride;
  int32_t ks_max;
  const int4* rb;               // plan entries {adapter, first index into perm, rows, 0}
  const int32_t* perm;
  uint16_t* Hs;                 // packed s_a H: per row [hi 0..rp) [lo 0..rp), bf16
  int32_t rp;                   // rank columns per half of an Hs row
  int32_t spr;                  // K steps per run: 2 rp / KS
};

__device__ __forceinline__ f32x16 mfma_32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Staging of one K step of KS columns: every operand row is KS bf16 = KS / 8
// chunks of 16 bytes, chunk c of row R stored at physical chunk c ^ f(R), so
// that the 16 lanes of a fragment read (16 consecutive rows, one chunk) hit 16
// distinct 16-byte bank groups: KS = 64 (128-byte rows, 2 rows per 256 bytes):
// f(R) = (R & 7) ^ ((R >> 3) & 1); KS = 32 (64-byte rows): f(R) = (R >> 2) & 3.
template <int KS>
struct Stage {
  static constexpr int ROW = KS * 2;                 // bytes per staged row
  static constexpr int CH = KS / 8;                  // chunks per row
  static constexpr int OP = LT_M * ROW;              // bytes per operand tile
  static constexpr int RPI = 1024 / ROW;             // rows per direct load (1 KB per wave)
  static constexpr int IPW = LT_M / RPI / 4;         // direct loads per wave and operand
  static constexpr int SUB = KS / 16;                // matrix-core sub-steps
  __device__ static __forceinline__ int swz(int row) {
    return KS == 64 ? ((row & 7) ^ ((row >> 3) & 1)) : ((row >> 2) & 3);
  }
};

// Per-lane source offsets of one operand's direct loads.  Load i of wave w
// fills LDS bytes [(IPW w + i) 1024, +1024): row R = (IPW w + i) RPI + lane / CH,
// physical chunk lane % CH, so logical chunk (lane % CH) ^ f(R).  For both
// staging widths that chunk depends on the lane and on i & 1 only, and the rows
// of load i are RPI i past those of load 0 (a wave-uniform step, which goes into
// the scalar offset with the step's K).
template <int KS>
struct StageMap {
  uint32_t off[2];     // lane offset at k = 0 for even / odd i
  int chunk[2];
  uint32_t step;       // bytes of RPI rows
};

template <int KS>
__device__ __forceinline__ StageMap<KS> lt_map(int64_t ld, int w, int lane) {
  using S = Stage<KS>;
  StageMap<KS> m;
  m.step = (uint32_t)S::RPI * (uint32_t)ld * 2u;
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int row = (S::IPW * w + e) * S::RPI + lane / S::CH;
    m.chunk[e] = (lane % S::CH) ^ S::swz(row);
    m.off[e] = (uint32_t)(row - e * S::RPI) * (uint32_t)ld * 2u + (uint32_t)m.chunk[e] * 16u;
  }
  return m;
}

// One direct load of 16 bytes per lane into LDS (byte offsets voff + soff of
// the resource).  Not a template: the host compilation pass cannot resolve the
// target builtin inside a template body.
__device__ __forceinline__ void lt_dma16(rsrc_t src, uint8_t* lds, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (__attribute__((address_space(3))) void*)lds, 16,
                                           voff, soff, 0, 0);
}

// One 16-byte store per lane through a buffer resource (offsets past it are
// dropped); `nt` marks it non-temporal.
__device__ __forceinline__ void lt_st16(rsrc_t dst, u32x4 v, uint32_t voff, bool nt) {
  if (nt) __builtin_amdgcn_raw_buffer_store_b128(v, dst, voff, 0, 2);
  else __builtin_amdgcn_raw_buffer_store_b128(v, dst, voff, 0, 0);
}

// One 16-byte load per lane into registers (the staging-through-registers path).
__device__ __forceinline__ u32x4 lt_ld16(rsrc_t src, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(src, voff, soff, 0);
}

// Where the loads of one K step go: straight into LDS (DMA), or into the
// registers R (2 IPW per lane) to be written to LDS one step later.
template <int KS, bool DMA>
struct Sink {
  u32x4 (&R)[2 * Stage<KS>::IPW];
  __device__ __forceinline__ void put(int k, rsrc_t src, uint8_t* lds, uint32_t voff, uint32_t soff) {
    if (DMA) lt_dma16(src, lds, voff, soff);
    else R[k] = lt_ld16(src, voff, soff);
  }
};

// Registers of one K step into its LDS slot: load k of wave w sits at bytes
// (IPW w + k) 1024 + 16 lane of the A tile (k < IPW) or the B tile.
template <int KS>
__device__ __forceinline__ void lt_write(const u32x4 (&R)[2 * Stage<KS>::IPW], uint8_t* slot, int w,
                                         int lane) {
  using S = Stage<KS>;
#pragma unroll
  for (int k = 0; k < 2 * S::IPW; ++k) {
    uint8_t* d = slot + (k < S::IPW ? 0 : S::OP) + (S::IPW * w + (k % S::IPW)) * 1024 + lane * 16;
    *reinterpret_cast<u32x4*>(d) = R[k];
  }
}

// One operand tile of one K step into LDS, through a buffer resource whose base
// is the tile's first row and whose size covers its valid rows: offsets past
// it read zeros (the rows past n or d_out of the last tiles), and chunks past
// d_in are sent past it (the K tail reads zeros).
template <int KS, bool DMA>
__device__ __forceinline__ void lt_stage(Sink<KS, DMA> sk, int k_base, const uint16_t* base,
                                         uint32_t bytes, const StageMap<KS>& m, int k0, int d_in,
                                         uint8_t* lds, int w) {
  using S = Stage<KS>;
  const rsrc_t src = make_rsrc(base, bytes);
  const int left = d_in - k0;          // valid K columns from k0 on
  const uint32_t v0 = 8 * m.chunk[0] < left ? m.off[0] : 0x80000000u;
  const uint32_t v1 = 8 * m.chunk[1] < left ? m.off[1] : 0x80000000u;
#pragma unroll
  for (int i = 0; i < S::IPW; ++i)
    sk.put(k_base + i, src, lds + (S::IPW * w + i) * 1024, (i & 1) ? v1 : v0,
           (uint32_t)k0 * 2u + (uint32_t)i * m.step);
}

template <int KS>
__device__ __forceinline__ bf16x8 lt_frag(const uint8_t* lds, int row, int chunk) {
  using S = Stage<KS>;
  return *reinterpret_cast<const bf16x8*>(lds + row * S::ROW + ((chunk ^ S::swz(row)) << 4));
}

// Fragments of one 16-wide K sub-step: 4 A (rows) and 4 B (columns) per wave.
struct Frags {
  bf16x8 a[4], b[4];
};

template <int KS>
__device__ __forceinline__ void lt_read(Frags& f, const uint8_t* sa, const uint8_t* sb, int kk,
                                        int wm, int wn, int lane) {
  const int rl = lane & 31, ch = lane >> 5;
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) f.a[mb] = lt_frag<KS>(sa, wm * 128 + mb * 32 + rl, 2 * kk + ch);
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) f.b[nb] = lt_frag<KS>(sb, wn * 128 + nb * 32 + rl, 2 * kk + ch);
}

__device__ __forceinline__ void lt_mma(const Frags& f, f32x16 (&acc)[4][4]) {
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = mfma_32x32x16(f.a[mb], f.b[nb], acc[mb][nb]);
}

// Wait until at most N of this wave's vector memory operations are
// outstanding and its LDS reads have completed, then meet the other waves.
// In one asm statement with a memory clobber, so that no memory operation
// moves across it (a plain barrier intrinsic does not order memory).
template <int N>
__device__ __forceinline__ void lt_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// One K step of the residual of one run: A = packed s_a H rows of the tile
// (rows outside the run [rs, re] are sent past the resource: zeros), B = the
// run's B_a rows for the tile's output columns, each staged K column k' of the
// step read at rank column (j KS + k') mod rp (hi and lo halves meet the same
// B_a), zero past r_a.  Rank a multiple of 8, so every 16-byte chunk of a B_a
// row is aligned and lies wholly inside or outside [0, r_a).
template <int KS, bool DMA>
__device__ __forceinline__ void lt_stage_lora(Sink<KS, DMA> sk, const LinArgs& p, const StageMap<KS>& hm,
                                              int r0, int n0, int j, int rs, int re, const uint16_t* Ba,
                                              int r, uint8_t* lds, int w, int lane) {
  using S = Stage<KS>;
  const rsrc_t ha = make_rsrc(p.Hs + (int64_t)r0 * (2 * p.rp),
                              (uint32_t)min(LT_M, p.n - r0) * (uint32_t)(2 * p.rp) * 2u);
  const rsrc_t bb = make_rsrc(Ba + (int64_t)n0 * r, (uint32_t)min(LT_N, p.d_out - n0) * (uint32_t)r * 2u);
  const int lr = lane / S::CH;                         // row of load i: (IPW w + i) RPI + lr
  uint32_t bo[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int jj = (j * KS + 8 * hm.chunk[e]) % p.rp;
    bo[e] = jj < r ? ((uint32_t)lr * (uint32_t)r + (uint32_t)jj) * 2u : 0x80000000u;
  }
#pragma unroll
  for (int i = 0; i < S::IPW; ++i) {
    const int row = (S::IPW * w + i) * S::RPI + lr;
    const bool in = r0 + row >= rs && r0 + row <= re;
    sk.put(i, ha, lds + (S::IPW * w + i) * 1024, in ? hm.off[i & 1] : 0x80000000u,
           (uint32_t)(j * KS) * 2u + (uint32_t)i * hm.step);
  }
#pragma unroll
  for (int i = 0; i < S::IPW; ++i)
    sk.put(S::IPW + i, bb, lds + S::OP + (S::IPW * w + i) * 1024, bo[i & 1],
           (uint32_t)((S::IPW * w + i) * S::RPI) * (uint32_t)r * 2u);
}

// Packs the residual's left operand once per call: for every row t of an
// adapter group, Hs[t][j] = bf16(s_a h_j) and Hs[t][rp + j] = bf16(s_a h_j - hi),
// j < rp (zeros past r_a), h = the shrink's slice planes summed in slice order.
// One workgroup per plan entry; a thread per (row, 8 rank columns).
__global__ __launch_bounds__(256) void linear_hpack_kernel(LinArgs p) {
  const int count = p.hdr[HDR_NRB_TOTAL];
  const int nks = shrink_slices(p.ks_max, count);
  const int g8 = p.rp / 8;
  for (int e = blockIdx.x; e < count; e += gridDim.x) {
    const int4 en = load_entry(p.rb, e);
    const int a = ck_slot(p.hdr, en.x, p.num_slots), p0 = en.y, rows = en.z;
    const Slot sm = load_slot(p.meta, a);
    const int r = sm.rank;
    for (int q = threadIdx.x; q < rows * g8; q += 256) {
      const int i = q / g8, j = (q - i * g8) * 8;
      const int t = ck_row(p.hdr, p.perm[p0 + i], p.n);
      float h[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) h[k] = 0.0f;
      if (j < r) {
        for (int sl = 0; sl < nks; ++sl) {
          const float* hp = p.H + (int64_t)sl * p.hp_stride + (int64_t)t * p.ldh + j;
          const float4 x0 = ldg_f4(hp), x1 = ldg_f4(hp + 4);
          h[0] += x0.x; h[1] += x0.y; h[2] += x0.z; h[3] += x0.w;
          h[4] += x1.x; h[5] += x1.y; h[6] += x1.z; h[7] += x1.w;
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) h[k] *= sm.scale;
      }
      bf16x8 hi, lo;
      split_hi_lo(h, hi, lo);
      uint16_t* dst = p.Hs + (int64_t)t * (2 * p.rp) + j;
      stg16(dst, __builtin_bit_cast(uint4, hi));
      stg16(dst + p.rp, __builtin_bit_cast(uint4, lo));
    }
  }
}

// Tile of this workgroup.  Workgroup g runs on XCD g % 8; XCD x takes a
// contiguous range of the tile order, which walks groups of LT_GM row tiles
// with the column tile outer and the row tile inner, so the tiles resident on
// one XCD at a time share their X rows and W rows in that XCD's L2.
__device__ __forceinline__ bool lt_tile(const LinArgs& p, int& m, int& nt) {
  const int total = p.m_tiles * p.n_tiles;
  const XcdRange xr = xcd_range(total);
  const int lin = xr.first;
  if (lin >= xr.end) return false;
  const int grp = lin / (LT_GM * p.n_tiles), rem = lin - grp * (LT_GM * p.n_tiles);
  const int gm = min(LT_GM, p.m_tiles - grp * LT_GM);
  nt = rem / gm;
  m = grp * LT_GM + (rem - nt * gm);
  return true;
}

// KS: K columns per step; NS: steps staged in LDS at once; NTS: non-temporal
// stores of Y; DMA: operands go straight from memory to LDS (NS - 1 steps in
// flight while one is multiplied), else through registers (NS = 2: one step in
// LDS being multiplied, the next in LDS, the one after in registers).
template <bool YBF16, bool RANK8, int KS, int NS, bool NTS, bool DMA>
__global__ __launch_bounds__(256, 1) void linear_kernel(LinArgs p) {
  using S = Stage<KS>;
  static_assert(DMA || NS == 2, "register staging keeps two LDS slots");
  // ring of NS steps, each [A | B][256 rows x S::ROW bytes]
  constexpr int BUFB = 2 * S::OP;
  static_assert(NS * BUFB <= 160 * 1024, "LDS");
  static_assert(NS * BUFB >= 4 * 32 * LT_SST * 4, "store staging fits in the ring");
  __shared__ __align__(1024) uint8_t s_lds[NS * BUFB];
  int m, nt;
  if (!lt_tile(p, m, nt)) return;
  const int lane = threadIdx.x & 63, w = wave_id();
  const int wm = w >> 1, wn = w & 1;
  const int rl = lane & 31, ch = lane >> 5;
  const int r0 = m * LT_M, n0 = nt * LT_N;

  f32x16 acc[4][4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[mb][nb][v] = 0.0f;

  // ---- X W^T ---------------------------------------------------------------
  const int nk = (p.d_in + KS - 1) / KS;
  const uint16_t* xs = p.X + (int64_t)r0 * p.ldx;
  const uint32_t xb = (uint32_t)min(LT_M, p.n - r0) * (uint32_t)p.ldx * 2u;
  const uint16_t* ws = p.W + (int64_t)n0 * p.ldw;
  const uint32_t wb = (uint32_t)min(LT_N, p.d_out - n0) * (uint32_t)p.ldw * 2u;
  const StageMap<KS> xm = lt_map<KS>(p.ldx, w, lane), wmap = lt_map<KS>(p.ldw, w, lane);
  // Pipeline: steps 0 .. NS - 1 are requested up front.  Step ks multiplies
  // ring slot ks % NS in SUB sub-steps, each reading the next sub-step's
  // fragments into the other register set before its own products.  After the
  // reads of the last sub-step the wave waits for step ks + 1's loads (steps
  // ks + 2 .. ks + NS - 1 may still be in flight) and meets the others at the
  // barrier (every wave has then read all of slot ks % NS); it requests step
  // ks + NS into that slot and reads step ks + 1's first sub-step, and only
  // then runs the products of the last sub-step, which cover the barrier and
  // the read latency.  Loads past the last step read zeros into slots nobody
  // reads, so no memory operation sits behind a branch.
  constexpr int LPS = 2 * S::IPW;                // direct loads per wave and step
  // Step sequence: the nk steps of X W^T, then (rank a multiple of 8) spr steps
  // per run of one adapter crossing the tile, which add s_a H B_a^T to the same
  // accumulators; past the end, steps read zeros.
  int nrt = 0, k_first = 0;
  if (RANK8) {
    const int nr = p.hdr[HDR_NRUNS];
    int lo = 0, hi = nr;           // first run whose last row is >= r0
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (p.run_end[mid] < r0) lo = mid + 1;
      else hi = mid;
    }
    k_first = uni(lo);
    while (k_first + nrt < nr && uni(p.run_start[k_first + nrt]) < r0 + LT_M) ++nrt;
  }
  const int T = nk + nrt * p.spr;
  const StageMap<KS> hm = lt_map<KS>(2 * p.rp, w, lane);
  int cur_run = -1, rs = 0, re = -1, rr = 8;
  const uint16_t* Ba = p.W;
  u32x4 R[2 * S::IPW];
  const Sink<KS, DMA> sk{R};
  auto issue = [&](int st, uint8_t* dst) {
    if (st < nk || st >= T) {
      lt_stage(sk, 0, xs, xb, xm, st * KS, p.d_in, dst, w);
      lt_stage(sk, S::IPW, ws, wb, wmap, st * KS, p.d_in, dst + S::OP, w);
    } else {
      const int q = st - nk, kr = q / p.spr;
      if (kr != cur_run) {
        cur_run = kr;
        rs = uni(p.run_start[k_first + kr]);
        re = uni(p.run_end[k_first + kr]);
        const Slot sm = load_slot(p.meta, ck_slot(p.hdr, uni(p.run_adapter[k_first + kr]), p.num_slots));
        Ba = static_cast<const uint16_t*>(sm.B);
        rr = sm.rank;
      }
      lt_stage_lora(sk, p, hm, r0, n0, q - kr * p.spr, rs, re, Ba, rr, dst, w, lane);
    }
  };
  if (DMA) {
#pragma unroll
    for (int j = 0; j < NS; ++j) issue(j, s_lds + j * BUFB);
    lt_barrier<(NS - 1) * LPS>();
  } else {
    issue(0, s_lds);
    lt_write<KS>(R, s_lds, w, lane);
    issue(1, s_lds + BUFB);
    lt_barrier<LPS>();
  }
  Frags f0, f1;
  lt_read<KS>(f0, s_lds, s_lds + S::OP, 0, wm, wn, lane);
  // one step: its products, with the loads of step ks + NS (ks + 2 through
  // the registers) issued at its end through `load`
  auto step = [&](int ks, auto load) {
    const int slot = ks % NS;
    uint8_t* cur = s_lds + slot * BUFB;
    uint8_t* nxt = s_lds + (slot + 1 == NS ? 0 : slot + 1) * BUFB;
#pragma unroll
    for (int kk = 0; kk + 1 < S::SUB; ++kk) {
      lt_read<KS>((kk & 1) ? f0 : f1, cur, cur + S::OP, kk + 1, wm, wn, lane);
      lt_mma((kk & 1) ? f1 : f0, acc);
      // one fragment read after each of the first 8 products, so the reads
      // issue while the matrix core is busy
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
        __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(SG_MFMA, 8, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (DMA) {
      lt_barrier<(NS - 2) * LPS>();
      load(ks + NS, cur);
    } else {
      // step ks + 1 from the registers into the other slot (last read in step
      // ks - 1, before the previous barrier), then step ks + 2 into the
      // registers; the barrier waits for the writes, not for those loads
      lt_write<KS>(R, nxt, w, lane);
      load(ks + 2, nxt);
      lt_barrier<LPS>();
    }
    lt_read<KS>(f0, nxt, nxt + S::OP, 0, wm, wn, lane);
    lt_mma(f1, acc);           // the last sub-step (SUB is even: its fragments are in f1)
    if (DMA) {
      // the step's loads two per product, then the next step's first reads one
      // per product: the matrix core stays busy while they issue
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
        __builtin_amdgcn_sched_group_barrier(SG_VMEM, LPS / 8, 0);
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
        __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // steps whose loads are all of X W^T run without a branch in the loop body;
  // the rest (the last steps of X W^T and the run steps) take the general loader
  const int lead = DMA ? NS : 2;
  const int n_plain = max(0, nk - lead);
  auto plain = [&](int st, uint8_t* dst) {
    lt_stage(sk, 0, xs, xb, xm, st * KS, p.d_in, dst, w);
    lt_stage(sk, S::IPW, ws, wb, wmap, st * KS, p.d_in, dst + S::OP, w);
  };
  for (int ks = 0; ks < n_plain; ++ks) step(ks, plain);
  for (int ks = n_plain; ks < T; ++ks) step(ks, issue);

  // ---- ranks not a multiple of 8: + s_a H B_a^T for each run crossing the
  // tile, from the slice planes, after the main loop --------------------------
  if (!RANK8) {
  const int nr = p.hdr[HDR_NRUNS];
  const int nks = shrink_slices(p.ks_max, p.hdr[HDR_NRB_TOTAL]);
  int lo = 0, hi = nr;           // first run whose last row is >= r0
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (p.run_end[mid] < r0) lo = mid + 1;
    else hi = mid;
  }
  for (int k = uni(lo); k < nr; ++k) {
    const int rs = uni(p.run_start[k]);
    if (rs >= r0 + LT_M) break;
    const int re = uni(p.run_end[k]);
    const Slot sm = load_slot(p.meta, ck_slot(p.hdr, uni(p.run_adapter[k]), p.num_slots));
    const int r = sm.rank;
    const rsrc_t Bw = make_rsrc(sm.B, (uint32_t)p.d_out * (uint32_t)r * 2u);
    for (int j0 = 0; j0 < r; j0 += 16) {
      const int jj = j0 + 8 * ch;
      bf16x8 bo[4];
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int o = min(n0 + wn * 128 + nb * 32 + rl, p.d_out - 1);
        bo[nb] = sel(jj < r, wrow8<RANK8>(Bw, (uint32_t)o * (uint32_t)r, jj, r));
      }
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const int row = r0 + wm * 128 + mb * 32 + rl;
        const bool in = row >= rs && row <= re;
        const int rc = min(max(row, rs), re);
        float h[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) h[i] = 0.0f;
        for (int sl = 0; sl < nks; ++sl) {
          const float* hp = p.H + (int64_t)sl * p.hp_stride + (int64_t)rc * p.ldh;
          if (RANK8) {
            const int jc = jj < r ? jj : r - 8;
            const float4 x0 = ldg_f4(hp + jc), x1 = ldg_f4(hp + jc + 4);
            h[0] += x0.x; h[1] += x0.y; h[2] += x0.z; h[3] += x0.w;
            h[4] += x1.x; h[5] += x1.y; h[6] += x1.z; h[7] += x1.w;
          } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) h[i] += ldg(hp + min(jj + i, r - 1));
          }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) h[i] = (in && jj + i < r) ? sm.scale * h[i] : 0.0f;
        bf16x8 hh, hl;
        split_hi_lo(h, hh, hl);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) {
          acc[mb][nb] = mfma_32x32x16(hh, bo[nb], acc[mb][nb]);
          acc[mb][nb] = mfma_32x32x16(hl, bo[nb], acc[mb][nb]);
        }
      }
    }
  }
  }
  mfma_fence();

  // ---- store -----------------------------------------------------------------
  // One 32-row block of the wave's 128 x 128 at a time through the wave's own
  // LDS area (32 rows of 128 floats, stride LT_SST), then back as 16-byte
  // vectors of whole rows: each store instruction writes four 256-byte row
  // pieces (bfloat16) or two 512-byte ones (float32).  The stores go through a
  // resource covering the tile's valid rows, with columns past d_out sent past
  // it, so none sits behind a branch.
  lt_barrier<0>();     // the unused loads past the last step have landed; all LDS reads done
  float* st = reinterpret_cast<float*>(s_lds) + w * (32 * LT_SST);
  constexpr uint32_t ES = YBF16 ? 2u : 4u;
  const rsrc_t yr = make_rsrc(static_cast<char*>(p.Y) + ((int64_t)r0 * p.ldy + n0) * ES,
                              (uint32_t)min(LT_M, p.n - r0) * (uint32_t)p.ldy * ES);
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) {
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        st[(8 * (v >> 2) + 4 * ch + (v & 3)) * LT_SST + nb * 32 + rl] = acc[mb][nb][v];
    const int row_base = wm * 128 + mb * 32;       // tile-local
    if (YBF16) {
      // lane: row 4 q + lane / 16 of each group of 4 rows, columns 8 (lane % 16) ..
      const int c8 = wn * 128 + (lane & 15) * 8;
      const bool col_ok = n0 + c8 < p.d_out;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int rr = 4 * q + (lane >> 4);
        const float* sp = st + rr * LT_SST + (lane & 15) * 8;
        const float4 a0 = *reinterpret_cast<const float4*>(sp);
        const float4 a1 = *reinterpret_cast<const float4*>(sp + 4);
        const u32x4 o = {pack2_bf16(a0.x, a0.y), pack2_bf16(a0.z, a0.w),
                         pack2_bf16(a1.x, a1.y), pack2_bf16(a1.z, a1.w)};
        const uint32_t off = col_ok ? ((uint32_t)(row_base + rr) * (uint32_t)p.ldy + (uint32_t)c8) * ES
                                    : 0x80000000u;
        lt_st16(yr, o, off, NTS);
      }
    } else {
      const int c4 = wn * 128 + (lane & 31) * 4;
      const bool col_ok = n0 + c4 < p.d_out;
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int rr = 2 * q + (lane >> 5);
        const float4 a = *reinterpret_cast<const float4*>(st + rr * LT_SST + (lane & 31) * 4);
        const u32x4 o = {__float_as_uint(a.x), __float_as_uint(a.y), __float_as_uint(a.z),
                         __float_as_uint(a.w)};
        const uint32_t off = col_ok ? ((uint32_t)(row_base + rr) * (uint32_t)p.ldy + (uint32_t)c4) * ES
                                    : 0x80000000u;
        lt_st16(yr, o, off, NTS);
      }
    }
  }
}

}  // namespace

int32_t linear_rank_cols(int32_t r_max) {
  // the run steps cover 2 rp K columns: a whole number of KS-wide steps
  const int32_t r = std::max(r_max, 1);
  return LINEAR_KS == 64 ? std::max(32, (r + 31) / 32 * 32) : (r + 15) / 16 * 16;
}

hipError_t launch_linear_mfma(const OpLaunch& o, const LinearLaunch& l, hipStream_t s) {
  LinArgs a{};
  a.X = static_cast<const uint16_t*>(l.X);
  a.ldx = l.ldx;
  a.W = static_cast<const uint16_t*>(l.W);
  a.ldw = l.ldw;
  a.Y = l.Y;
  a.ldy = l.ldy;
  a.n = o.n;
  a.num_slots = o.num_slots;
  a.d_in = o.d_in;
  a.d_out = o.d_out;
  a.m_tiles = (o.n + LT_M - 1) / LT_M;
  a.n_tiles = (o.d_out + LT_N - 1) / LT_N;
  a.hdr = o.hdr;
  a.run_start = l.run_start;
  a.run_end = l.run_end;
  a.run_adapter = l.run_adapter;
  a.meta = o.meta;
  a.H = l.H;
  a.ldh = l.ldh;
  a.hp_stride = l.hp_stride;
  a.ks_max = l.ks_max;
  a.rb = o.rb;
  a.perm = o.perm;
  a.Hs = l.Hs;
  a.rp = linear_rank_cols(o.r_max);
  a.spr = 2 * a.rp / LINEAR_KS;
  const long long total = (long long)a.m_tiles * a.n_tiles;
  if (total <= 0) return hipSuccess;
  const int grid = (int)(8 * ((total + 7) / 8));
  if (o.rank8 && o.r_max > 0 && o.rb_ub > 0) {
    hipLaunchKernelGGL(linear_hpack_kernel, dim3(std::min(o.rb_ub, 4096)), dim3(256), 0, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const bool yb = l.y_bf16;
  constexpr int KS = LINEAR_KS, NS = LINEAR_NS;
  constexpr bool NTS = LINEAR_NTS, DMA = LINEAR_DMA;
  if (yb && o.rank8) hipLaunchKernelGGL((linear_kernel<true, true, KS, NS, NTS, DMA>), dim3(grid), dim3(256), 0, s, a);
  else if (yb) hipLaunchKernelGGL((linear_kernel<true, false, KS, NS, NTS, DMA>), dim3(grid), dim3(256), 0, s, a);
  else if (o.rank8) hipLaunchKernelGGL((linear_kernel<false, true, KS, NS, NTS, DMA>), dim3(grid), dim3(256), 0, s, a);
  else hipLaunchKernelGGL((linear_kernel<false, false, KS, NS, NTS, DMA>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace lora
