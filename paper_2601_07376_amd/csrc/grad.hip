// Masked, adapter-local LoRA gradients (Section 3.3 for the explicit loss mask,
// Section 3.5 for gradients kept local to the owning adapter).  The paper does
// not write the backward; it is the chain rule on the LoRA layer equation of
// Section 3.4 restricted to the trainable rows T_a^m of adapter a:
//
//   H = X_m A_a^T,  G = dY_m B_a,  dB_a = s_a dY_m^T H,  dA_a = s_a G^T X_m.
//
// Matrix-core path, three launches:
//  1. per trainable row block (<= 64 rows) and d-slice: partial H and G over
//     the slice, written transposed into fp32 "planes" [j][column], where row i
//     of block e sits in column 64 e + i.  G's second operand is gathered from
//     B_a as stored ([d_out][r], eight 2-byte loads per lane and k-step).
//  2. the slice planes summed in slice order and split into bf16 hi + lo.
//  3. per adapter and 256-wide column tile of dB or dA: a fixed-order
//     reduction over the adapter's trainable rows, one 64-row block per step;
//     the row tile is transposed through LDS and meets the hi / lo planes on
//     the matrix cores.
// Rows outside T_a^m are never read.  No floating-point atomics anywhere, so
// the result is the same bytes run to run.
#include <algorithm>

#include "device_common.h"
#include "lora_internal.h"

namespace lora {

namespace {

struct GradArgs {
  const int32_t* hdr;
  const int4* mrb;
  const int32_t* m_perm;
  const int32_t* m_offsets;
  const int32_t* m_counts;
  const int32_t* m_blk;
  const SlotMeta* meta;
  int32_t d_in, d_out, num_slots;
  int32_t n_rows;                         // rows of the batch: the bound of every row id read from the plan
  const void* X;
  int64_t ldx;
  const void* dY;
  int64_t lddy;
  const float* H_saved;
  int64_t ldh;
  int32_t accumulate;
  int32_t slot_base, slot_count;          // slots of this launch's output pointers
  float* dA[GRAD_SLOT_GROUP];             // [r_a, d_in] per slot, nullptr = skip
  float* dB[GRAD_SLOT_GROUP];             // [d_out, r_a] per slot
  float* hg;
  int32_t ks;
  int32_t p_stride;
  int32_t r_pad;
  uint16_t* fin;            // summed planes, bf16: [which][hi, lo][j][column]
};

__device__ __forceinline__ uint16_t* fin_plane(const GradArgs& g, int which, int hl) {
  return g.fin + ((int64_t)(which * 2 + hl) * g.r_pad) * g.p_stride;
}

__device__ __forceinline__ float* plane(const GradArgs& g, int which, int ks) {
  return g.hg + ((int64_t)(which * g.ks + ks) * g.r_pad) * g.p_stride;
}

// d-slices actually used: enough (row block, slice) tiles to cover the chip
// once (about 256), at most g.ks (the workspace holds g.ks slice planes)
__device__ __forceinline__ int active_splits(const GradArgs& g, int n_blocks) {
  return max(1, min(g.ks, 256 / max(n_blocks, 1)));
}

// slice of a dimension for split ks, in multiples of 128
__device__ __forceinline__ void slice(int d, int nks, int ks, int& b, int& e) {
  const int w = ((d + nks - 1) / nks + 127) / 128 * 128;
  b = min(d, ks * w);
  e = min(d, b + w);
}

// ---------------------------------------------------------------------------
// stage 1 (matrix cores): partial H and G for one (row block, slice).  Both are
// shrink-shaped products (rows x d-slice times rank x d-slice), streamed with
// double-buffered 16-byte loads.
// ---------------------------------------------------------------------------
// acc_h += rows(xr) W1^T over k in [k1b, k1e) and acc_g += rows(yr) W2^T over
// k in [k2b, k2e), both with k-steps kb + w * 32 + i * 128.  Each round requests
// one batch of U k-steps of both products (every load unconditional, from a
// clamped address) and then feeds the matrix cores, so the second product's
// loads overlap the first one's arithmetic and nothing waits behind a branch.
// Every tile is computed (tiles past the rows or the rank are never stored).
template <int MT, int NT, int U, bool DB>
__device__ __forceinline__ void rows_times_w2(f32x4 (&acc_h)[MT * NT], f32x4 (&acc_g)[MT * NT],
                                              const uint16_t* (&xr)[MT], rsrc_t W1,
                                              const uint32_t (&wr1)[NT], int k1b, int k1e,
                                              const uint16_t* (&yr)[MT], rsrc_t W2,
                                              const uint32_t (&wr2)[NT], int k2b, int k2e,
                                              int r2) {
  const int kg = ((threadIdx.x & 63) >> 4) * 8 + wave_id() * 32;
  struct Buf {
    bf16x8 x[U][MT];
    bf16x8 w[U][NT];
    uint32_t e[U][NT][8];   // gathered values, packed only when multiplied
    bool kv[U];
  };
  // gather = false: W is [rows][K] (K contiguous), wr[nt] the row offset;
  // gather = true:  W is [K][r] (B_a as stored), wr[nt] the column, and the
  //                 eight K values of a lane are eight 2-byte loads r apart
  auto load = [&](Buf& b, const uint16_t* (&rr)[MT], rsrc_t W, const uint32_t (&wr)[NT], int kb,
                  int ke, bool gather) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kb + u * 128 + kg;
      b.kv[u] = k < ke;
      const int kk = k < ke ? k : ke - 8;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) b.x[u][mt] = as_bf16x8(ldg16(rr[mt] + kk));
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        if (!gather) {
          b.w[u][nt] = as_bf16x8(bload16(W, (wr[nt] + (uint32_t)kk) * 2u));
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i)
            b.e[u][nt][i] = bload_u16(W, ((uint32_t)(kk + i) * (uint32_t)r2 + wr[nt]) * 2u);
        }
      }
    }
  };
  auto compute = [&](const Buf& b, f32x4 (&acc)[MT * NT], bool gather) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      bf16x8 wv[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) wv[nt] = gather ? pack_bf16x8(b.e[u][nt]) : b.w[u][nt];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const bf16x8 xo = sel(b.kv[u], b.x[u][mt]);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          acc[mt * NT + nt] = mfma_16x16x32(xo, wv[nt], acc[mt * NT + nt]);
      }
    }
  };
  const int n1 = max(0, (k1e - k1b + U * 128 - 1) / (U * 128));
  const int n2 = max(0, (k2e - k2b + U * 128 - 1) / (U * 128));
  const int rounds = max(n1, n2);
  const int e1 = max(k1e, 8), e2 = max(k2e, 8);
  if (DB) {
    // rounds double buffered in registers: round i + 1 is requested before
    // round i is multiplied, so the memory stream never pauses for the
    // arithmetic (rounds past the end read clamped addresses and add zeros);
    // one exit, at the end of a pair of rounds
    Buf h0, g0, h1, g1;
    load(h0, xr, W1, wr1, k1b, e1, false);
    load(g0, yr, W2, wr2, k2b, e2, true);
    for (int i = 0; i < rounds; i += 2) {
      load(h1, xr, W1, wr1, k1b + (i + 1) * U * 128, e1, false);
      load(g1, yr, W2, wr2, k2b + (i + 1) * U * 128, e2, true);
      __builtin_amdgcn_sched_barrier(0);
      compute(h0, acc_h, false);
      compute(g0, acc_g, true);
      load(h0, xr, W1, wr1, k1b + (i + 2) * U * 128, e1, false);
      load(g0, yr, W2, wr2, k2b + (i + 2) * U * 128, e2, true);
      __builtin_amdgcn_sched_barrier(0);
      compute(h1, acc_h, false);
      compute(g1, acc_g, true);
      // wait states on the back edge between the last product and the loop
      // head, where the compiler may read an accumulator register
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_nop 7");
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
    for (int i = 0; i < rounds; ++i) {
      Buf bh, bg;
      load(bh, xr, W1, wr1, k1b + i * U * 128, e1, false);
      load(bg, yr, W2, wr2, k2b + i * U * 128, e2, true);
      // keep the whole round's loads ahead of its arithmetic (the scheduler
      // would otherwise interleave them to save registers, and wait on each)
      __builtin_amdgcn_sched_barrier(0);
      compute(bh, acc_h, false);
      compute(bg, acc_g, true);
    }
  }
  mfma_fence();
}

// Sum the four waves' accumulators in the fixed order ((w0 + w2) + (w1 + w3)),
// leaving the total in wave 0: waves 1-3 park CH accumulators at a time in
// s_red (3 x CH x 64 f32x4), one barrier per chunk.  The first barrier also
// orders this tile's writes after the previous tile's reads of s_red.
template <int N, int CH>
__device__ __forceinline__ void reduce_waves3(f32x4 (&acc)[N], f32x4* s_red) {
  const int lane = threadIdx.x & 63, w = wave_id();
#pragma unroll
  for (int c0 = 0; c0 < N; c0 += CH) {
    __syncthreads();
    if (w > 0) {
#pragma unroll
      for (int i = 0; i < CH; ++i)
        if (c0 + i < N) s_red[((w - 1) * CH + i) * 64 + lane] = acc[c0 + i];
    }
    __syncthreads();
    if (w == 0) {
#pragma unroll
      for (int i = 0; i < CH; ++i)
        if (c0 + i < N) {
          const f32x4 a1 = s_red[(0 * CH + i) * 64 + lane];
          const f32x4 a2 = s_red[(1 * CH + i) * 64 + lane];
          const f32x4 a3 = s_red[(2 * CH + i) * 64 + lane];
          acc[c0 + i] = (acc[c0 + i] + a2) + (a1 + a3);
        }
    }
  }
}

#ifndef HG_U
#define HG_U 1
#endif
template <int NT>
__global__ __launch_bounds__(256) void hg_kernel(GradArgs g) {
  constexpr int MT = MRB_ROWS / 16;                      // row tiles per block
  constexpr int U = HG_U > 0 ? HG_U : 1;                 // k-steps per wave and round
  constexpr bool DB = NT <= 4;                           // double-buffered rounds
  constexpr int N = 2 * MT * NT, CH = N < 16 ? N : 16;
  constexpr int OS = MRB_ROWS + 1;                       // LDS row stride of the plane tile
  constexpr int RED = 3 * CH * 64, PL = NT * 16 * OS, OUT = (2 * PL + 3) / 4;
  __shared__ f32x4 s_red[RED > OUT ? RED : OUT];
  const int lane = threadIdx.x & 63, w = wave_id();
  const int n_blocks = g.hdr[HDR_NMRB];
  const int nks = active_splits(g, n_blocks);
  const XcdRange xr = xcd_range(n_blocks * nks);
  const uint16_t* X = reinterpret_cast<const uint16_t*>(g.X);
  const uint16_t* dY = reinterpret_cast<const uint16_t*>(g.dY);
  for (int tile = xr.first; tile < xr.end; tile += xr.step) {
    const int e = tile / nks, ks = tile - e * nks;
    const int4 en = load_entry(g.mrb, e);
    const int a = ck_slot(g.hdr, en.x, g.num_slots), p0 = en.y, rows = en.z;
    const Slot m = load_slot(g.meta, a);
    const int r = m.rank;
    const rsrc_t Aw = make_rsrc(m.A, (uint32_t)r * (uint32_t)g.d_in * 2u);
    const rsrc_t Bw = make_rsrc(m.B, (uint32_t)g.d_out * (uint32_t)r * 2u);
    const uint16_t* xrow[MT];
    const uint16_t* yrow[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int i = mt * 16 + (lane & 15);
      const int t = ck_row(g.hdr, g.m_perm[p0 + (i < rows ? i : rows - 1)], g.n_rows);
      xrow[mt] = X + (int64_t)t * g.ldx;
      yrow[mt] = dY + (int64_t)t * g.lddy;
    }
    uint32_t arow[NT], brow[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int j = nt * 16 + (lane & 15);
      arow[nt] = (uint32_t)(j < r ? j : r - 1) * (uint32_t)g.d_in;
      brow[nt] = (uint32_t)(j < r ? j : r - 1);
    }
    // acc[0 .. MT NT) : H tiles (mt, nt); acc[MT NT .. 2 MT NT) : G tiles
    f32x4 acc[N];
#pragma unroll
    for (int i = 0; i < N; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 (&acc_h)[MT * NT] = *reinterpret_cast<f32x4(*)[MT * NT]>(&acc[0]);
    f32x4 (&acc_g)[MT * NT] = *reinterpret_cast<f32x4(*)[MT * NT]>(&acc[MT * NT]);
    {
      int kb, ke, ob, oe;
      slice(g.d_in, nks, ks, kb, ke);
      slice(g.d_out, nks, ks, ob, oe);
      if (g.H_saved != nullptr) ke = kb;          // H comes from the caller
      rows_times_w2<MT, NT, U, DB>(acc_h, acc_g, xrow, Aw, arow, kb, ke, yrow, Bw, brow, ob, oe, r);
    }
    vmem_drained();
    reduce_waves3<N, CH>(acc, s_red);
    // wave 0 holds the totals; both planes' tiles [j][64 columns] are staged
    // in LDS together and leave as whole 256-byte row pieces (one barrier, so
    // no wave waits for the first plane's stores)
    float* s_o = reinterpret_cast<float*>(s_red);
    const int col0 = e * MRB_ROWS;
    if (w == 0) {
#pragma unroll
      for (int which = 0; which < 2; ++which)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int i = mt * 16 + (lane >> 4) * 4 + v, j = nt * 16 + (lane & 15);
              s_o[which * PL + j * OS + i] = i < rows ? acc[which * MT * NT + mt * NT + nt][v] : 0.0f;
            }
    }
    __syncthreads();
#pragma unroll
    for (int which = 0; which < 2; ++which) {
      if (which == 1 || g.H_saved == nullptr) {
        float* pl = plane(g, which, ks);
        for (int q = threadIdx.x; q < g.r_pad * (MRB_ROWS / 4); q += 256) {
          const int j = q / (MRB_ROWS / 4), c4 = (q - j * (MRB_ROWS / 4)) * 4;
          const float* so = s_o + which * PL + j * OS + c4;
          stg_f4(pl + (int64_t)j * g.p_stride + col0 + c4, make_float4(so[0], so[1], so[2], so[3]));
        }
      }
    }
    if (g.H_saved != nullptr && w == 0) {
      float* ph = plane(g, 0, ks);
      for (int q = lane; q < MRB_ROWS * g.r_pad; q += 64) {
        const int i = q / g.r_pad, j = q - i * g.r_pad;
        float h = 0.0f;
        if (ks == 0 && i < rows && j < r) h = g.H_saved[(int64_t)ck_row(g.hdr, g.m_perm[p0 + i], g.n_rows) * g.ldh + j];
        ph[(int64_t)j * g.p_stride + col0 + i] = h;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// stage 2: planes summed in slice order, split into bf16 hi / lo (8 columns per
// thread)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void hgsum_kernel(GradArgs g) {
  const int n_blocks = g.hdr[HDR_NMRB];
  const int nks = active_splits(g, n_blocks);
  const int n8 = n_blocks * (MRB_ROWS / 8);           // 8-column groups per plane row
  const int64_t per = (int64_t)g.r_pad * n8;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < 2 * per;
       q += (int64_t)gridDim.x * 256) {
    const int which = (int)(q / per);
    const int64_t u = q - which * per;
    const int j = (int)(u / n8), c = (int)(u - (int64_t)j * n8) * 8;
    // every slice requested at once (slices past nks read the last one again
    // and are not added), then summed in slice order
    float4 x0[GRAD_SPLITS_MAX], x1[GRAD_SPLITS_MAX];
#pragma unroll
    for (int ks = 0; ks < GRAD_SPLITS_MAX; ++ks) {
      const float* p = plane(g, which, min(ks, nks - 1)) + (int64_t)j * g.p_stride + c;
      x0[ks] = ldg_f4(p);
      x1[ks] = ldg_f4(p + 4);
    }
    float h[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < GRAD_SPLITS_MAX; ++ks) {
      if (ks >= nks) break;
      h[0] += x0[ks].x; h[1] += x0[ks].y; h[2] += x0[ks].z; h[3] += x0[ks].w;
      h[4] += x1[ks].x; h[5] += x1[ks].y; h[6] += x1[ks].z; h[7] += x1[ks].w;
    }
    bf16x8 hi, lo;
    split_hi_lo(h, hi, lo);
    stg16(fin_plane(g, which, 0) + (int64_t)j * g.p_stride + c, __builtin_bit_cast(uint4, hi));
    stg16(fin_plane(g, which, 1) + (int64_t)j * g.p_stride + c, __builtin_bit_cast(uint4, lo));
  }
}

// ---------------------------------------------------------------------------
// stage 3 (matrix cores): one workgroup per (slot, dB or dA, 256-column tile).
// A step is one 64-row gradient block of the slot: every thread loads eight
// rows x 8 columns of dY (for dB) or X (for dA), transposes them in registers
// and writes 8 columns x 8 rows into LDS as 16-byte units, next to the step's
// hi / lo plane columns; the next step's loads are in flight meanwhile and LDS
// is double buffered with one barrier per step.
//   dB[o][j] = s sum_t dY[t][o] H[t][j]:  A operand = dY^T tile, B = H plane
//   dA[j][k] = s sum_t G[t][j] X[t][k]:   A operand = G plane, B = X^T tile
// ---------------------------------------------------------------------------
// tile columns: 256, or 128 for ranks above 64 (register budget)
constexpr int dt_ct(int NT) { return NT <= 4 ? 256 : 128; }
constexpr int DT_ROWS = MRB_ROWS;     // rows per step: one trainable row block
constexpr int DT_WIN = 1024;          // row ids staged per window

// LDS slot of 16-byte unit g (rows 8 g .. 8 g + 7 of a step) of column `col`
// (a tile column, or a plane row j).  Two columns share each 256-byte line
// and the units are permuted inside it, so that the 16 lanes of a transposing
// write (columns 8 apart) and of a matrix-core read (16 consecutive columns)
// both fall in 16 distinct 16-byte bank groups.
__device__ __forceinline__ int dt_unit(int col, int g) {
  const int r = col >> 1;
  const int f = (r & 7) ^ ((r >> 3) & 3) ^ (((r >> 5) & 1) << 3);
  return r * 16 + ((((col & 1) << 3) | g) ^ f);
}

// One (slot, column tile) of dB (IS_B) or dA: the whole reduction over the
// slot's trainable rows, then the scaled store.
template <int NT, bool IS_B>
__device__ __forceinline__ void dadb_tile(const GradArgs& g, int sl, int c0, uint16_t (*s_t)[dt_ct(NT) * DT_ROWS],
                                          uint16_t (*s_p)[2 * NT * 16 * DT_ROWS], int* s_rows) {
  constexpr int CT = dt_ct(NT);
  constexpr int PSEG = 2 * NT * 16 * (DT_ROWS / 8);   // 16-byte plane units per step
  constexpr int PPT = PSEG / 256;                     // per thread
  constexpr int CSN = CT / 8, I4 = CT / 64;     // loader column segments; 16-column tiles per wave
  static_assert(PSEG % 256 == 0, "plane units per thread");
  const int lane = threadIdx.x & 63, w = wave_id(), tid = threadIdx.x;
  // loader: columns 8 cs .., rows 8 tq ..; with 128-column tiles the upper
  // half of the threads repeats the lower half (same values, same addresses)
  const int cs = tid % CSN, tq = (tid / CSN) & 7;
  const int a = g.slot_base + sl;
  const Slot m = load_slot(g.meta, a);
  const int r = m.rank;
  float* out = IS_B ? g.dB[sl] : g.dA[sl];
  const int dcol = IS_B ? g.d_out : g.d_in;
  const int moff = uni(g.m_offsets[a]), blk0 = uni(g.m_blk[a]);
  const int mc = ck_count(g.hdr, moff, uni(g.m_counts[a]), g.n_rows);
  const float s = m.scale;
  const uint16_t* src = reinterpret_cast<const uint16_t*>(IS_B ? g.dY : g.X);
  const int64_t ld = IS_B ? g.lddy : g.ldx;
  const uint16_t* fin0 = fin_plane(g, IS_B ? 0 : 1, 0);
  const uint16_t* fin1 = fin_plane(g, IS_B ? 0 : 1, 1);
  const int lcol = c0 + cs * 8 < dcol ? c0 + cs * 8 : dcol - 8;   // clamped loader column
  const bool lcol_ok = c0 + cs * 8 < dcol;

  f32x4 acc[I4][NT];
#pragma unroll
  for (int i = 0; i < I4; ++i)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[i][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nch = (mc + DT_ROWS - 1) / DT_ROWS;
  for (int w0 = 0; w0 < nch; w0 += DT_WIN / DT_ROWS) {
    const int wch = min(DT_WIN / DT_ROWS, nch - w0);
    __syncthreads();
    for (int i = tid; i < DT_WIN; i += 256) {
      const int p = w0 * DT_ROWS + i;
      s_rows[i] = ck_row(g.hdr, g.m_perm[moff + (p < mc ? p : mc - 1)], g.n_rows);
    }
    __syncthreads();

    struct Step {
      uint4 t[8];
      uint4 p[PPT];
    };
    // raw loads of step cc (clamped to the window's last step; steps past it
    // are staged as zero rows).  Step cc is row block blk0 + w0 + cc, so its
    // plane columns are that block's 64 columns.
    auto load = [&](Step& q, int cc) {
      cc = min(cc, wch - 1);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        q.t[i] = ldg16(src + (int64_t)s_rows[cc * DT_ROWS + tq * 8 + i] * ld + lcol);
      const int col0 = (blk0 + w0 + cc) * DT_ROWS;
#pragma unroll
      for (int h = 0; h < PPT; ++h) {
        const int u = tid + 256 * h, jr = u >> 3, gg = u & 7;
        const int hl = jr / (NT * 16), j = jr - hl * (NT * 16);
        q.p[h] = ldg16((hl ? fin1 : fin0) + (int64_t)j * g.p_stride + col0 + gg * 8);
      }
    };
    auto stage = [&](const Step& q, int cc, int buf) {
      const int rows_left = mc - (w0 + cc) * DT_ROWS;
      uint32_t v[8][4];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const bool ok = lcol_ok && tq * 8 + i < rows_left;
        v[i][0] = ok ? q.t[i].x : 0u;
        v[i][1] = ok ? q.t[i].y : 0u;
        v[i][2] = ok ? q.t[i].z : 0u;
        v[i][3] = ok ? q.t[i].w : 0u;
      }
      // 8 rows x 8 columns -> 8 columns x 8 rows (bf16 pairs through byte permutes)
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
        uint4 o;
        o.x = __builtin_amdgcn_perm(v[1][c >> 1], v[0][c >> 1], sel);
        o.y = __builtin_amdgcn_perm(v[3][c >> 1], v[2][c >> 1], sel);
        o.z = __builtin_amdgcn_perm(v[5][c >> 1], v[4][c >> 1], sel);
        o.w = __builtin_amdgcn_perm(v[7][c >> 1], v[6][c >> 1], sel);
        *reinterpret_cast<uint4*>(&s_t[buf][dt_unit(cs * 8 + c, tq) * 8]) = o;
      }
#pragma unroll
      for (int h = 0; h < PPT; ++h) {
        const int u = tid + 256 * h;
        *reinterpret_cast<uint4*>(&s_p[buf][dt_unit(u >> 3, u & 7) * 8]) = q.p[h];
      }
    };
    auto mma = [&](int buf) {
      const int gq = lane >> 4, n = lane & 15;
#pragma unroll
      for (int kc = 0; kc < DT_ROWS / 32; ++kc) {
        const int gu = kc * 4 + gq;
        bf16x8 hi[NT], lo[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          hi[nt] = as_bf16x8(*reinterpret_cast<const uint4*>(&s_p[buf][dt_unit(nt * 16 + n, gu) * 8]));
          lo[nt] = as_bf16x8(
              *reinterpret_cast<const uint4*>(&s_p[buf][dt_unit((NT + nt) * 16 + n, gu) * 8]));
        }
#pragma unroll
        for (int i4 = 0; i4 < I4; ++i4) {
          const int col = w * (16 * I4) + i4 * 16 + n;
          const bf16x8 tv = as_bf16x8(*reinterpret_cast<const uint4*>(&s_t[buf][dt_unit(col, gu) * 8]));
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            if (IS_B) {
              acc[i4][nt] = mfma_16x16x32(tv, hi[nt], acc[i4][nt]);
              acc[i4][nt] = mfma_16x16x32(tv, lo[nt], acc[i4][nt]);
            } else {
              acc[i4][nt] = mfma_16x16x32(hi[nt], tv, acc[i4][nt]);
              acc[i4][nt] = mfma_16x16x32(lo[nt], tv, acc[i4][nt]);
            }
          }
        }
      }
    };
    // Steps double buffered in registers (the next step's loads are in flight
    // while a step is staged and multiplied); one exit, at the end of a pair
    // of steps, and no memory operation behind a branch, so the compiler's
    // wait counts stay exact.  LDS buffer cc & 1: a step is staged only after
    // the barrier of the step before, which every wave passes after its
    // products of the step before that.
    Step b0, b1;
    load(b0, 0);
    for (int cc = 0; cc < wch; cc += 2) {
      load(b1, cc + 1);
      __builtin_amdgcn_sched_barrier(0);       // requests stay ahead of the staging
      stage(b0, cc, 0);
      __syncthreads();
      mma(0);
      load(b0, cc + 2);
      __builtin_amdgcn_sched_barrier(0);
      stage(b1, cc + 1, 1);
      __syncthreads();
      mma(1);
    }
  }

  mfma_fence();
  if (mc == 0 && g.accumulate) return;
#pragma unroll
  for (int i4 = 0; i4 < I4; ++i4)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        int64_t oidx;
        bool valid;
        if (IS_B) {
          const int o = c0 + w * (16 * I4) + i4 * 16 + (lane >> 4) * 4 + v, j = nt * 16 + (lane & 15);
          valid = o < g.d_out && j < r;
          oidx = (int64_t)o * r + j;
        } else {
          const int j = nt * 16 + (lane >> 4) * 4 + v, k = c0 + w * (16 * I4) + i4 * 16 + (lane & 15);
          valid = j < r && k < g.d_in;
          oidx = (int64_t)j * g.d_in + k;
        }
        if (!valid) continue;
        const float val = (mc == 0) ? 0.0f : s * acc[i4][nt][v];
        out[oidx] = g.accumulate ? out[oidx] + val : val;
      }
    }
}

template <int NT>
__global__ __launch_bounds__(256) void dadb_kernel(GradArgs g) {
  constexpr int CT = dt_ct(NT);
  __shared__ __align__(16) uint16_t s_t[2][CT * DT_ROWS];
  __shared__ __align__(16) uint16_t s_p[2][2 * NT * 16 * DT_ROWS];   // [hl][j] columns
  __shared__ int s_rows[DT_WIN];
  const int nbB = (g.d_out + CT - 1) / CT, nbA = (g.d_in + CT - 1) / CT, nbt = nbB + nbA;
  const XcdRange xr = xcd_range(g.slot_count * nbt);
  for (int tile = xr.first; tile < xr.end; tile += xr.step) {
    const int sl = tile / nbt, c = tile - sl * nbt;
    const int r = uni(g.meta[g.slot_base + sl].rank);
    if (r <= 0) continue;
    if (c < nbB) {
      if (g.dB[sl] != nullptr) dadb_tile<NT, true>(g, sl, c * CT, s_t, s_p, s_rows);
    } else {
      if (g.dA[sl] != nullptr) dadb_tile<NT, false>(g, sl, (c - nbB) * CT, s_t, s_p, s_rows);
    }
  }
}

// ---------------------------------------------------------------------------
// vector-ALU path (any f32 / bf16 storage): same planes with one slice
// ---------------------------------------------------------------------------
template <bool BF16>
__device__ __forceinline__ float ldv(const void* p, int64_t i) {
  if (BF16) return bf16_to_f32(reinterpret_cast<const uint16_t*>(p)[i]);
  return reinterpret_cast<const float*>(p)[i];
}

template <bool XB, bool WB>
__global__ __launch_bounds__(256) void hg_valu_kernel(GradArgs g) {
  const int n_blocks = g.hdr[HDR_NMRB];
  for (int e = blockIdx.x; e < n_blocks; e += gridDim.x) {
    const int4 en = load_entry(g.mrb, e);
    const int a = ck_slot(g.hdr, en.x, g.num_slots), p0 = en.y, rows = en.z;
    const Slot m = load_slot(g.meta, a);
    const int r = m.rank;
    float* ph = plane(g, 0, 0);
    float* pg = plane(g, 1, 0);
    for (int q = threadIdx.x; q < MRB_ROWS * g.r_pad; q += blockDim.x) {
      const int i = q / g.r_pad, j = q - i * g.r_pad;
      float h = 0.0f, gg = 0.0f;
      if (i < rows && j < r) {
        const int t = ck_row(g.hdr, g.m_perm[p0 + i], g.n_rows);
        if (g.H_saved != nullptr) {
          h = g.H_saved[(int64_t)t * g.ldh + j];
        } else {
          for (int k = 0; k < g.d_in; ++k)
            h = fmaf(ldv<XB>(g.X, (int64_t)t * g.ldx + k), ldv<WB>(m.A, (int64_t)j * g.d_in + k), h);
        }
        for (int o = 0; o < g.d_out; ++o)
          gg = fmaf(ldv<XB>(g.dY, (int64_t)t * g.lddy + o), ldv<WB>(m.B, (int64_t)o * r + j), gg);
      }
      ph[(int64_t)j * g.p_stride + e * MRB_ROWS + i] = h;
      pg[(int64_t)j * g.p_stride + e * MRB_ROWS + i] = gg;
    }
  }
}

template <bool XB>
__global__ __launch_bounds__(256) void dadb_valu_kernel(GradArgs g) {
  // one thread per output element; elements of dB_a then dA_a, slot after slot
  const int64_t per_slot = (int64_t)LORA_MAX_RANK * (g.d_out + g.d_in);
  const int64_t total = per_slot * g.slot_count;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < total;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int sl = (int)(q / per_slot);
    const int a = g.slot_base + sl;
    const int64_t u = q - (int64_t)sl * per_slot;
    const SlotMeta m = g.meta[a];           // per-thread slot: not made uniform
    const int r = m.rank;
    if (r <= 0) continue;
    const bool isB = u < (int64_t)LORA_MAX_RANK * g.d_out;
    const int64_t v = isB ? u : u - (int64_t)LORA_MAX_RANK * g.d_out;
    int j, col;
    if (isB) {
      col = (int)(v / LORA_MAX_RANK);      // o
      j = (int)(v - (int64_t)col * LORA_MAX_RANK);
    } else {
      j = (int)(v / g.d_in);
      col = (int)(v - (int64_t)j * g.d_in);  // k
    }
    if (j >= r) continue;
    float* out = isB ? g.dB[sl] : g.dA[sl];
    if (out == nullptr) continue;
    const int moff = g.m_offsets[a], blk0 = g.m_blk[a];
    const int mc = ck_count(g.hdr, moff, g.m_counts[a], g.n_rows);
    if (mc == 0 && g.accumulate) continue;
    const float* pl = plane(g, isB ? 0 : 1, 0) + (int64_t)j * g.p_stride;
    float acc = 0.0f;
    for (int p = 0; p < mc; ++p) {
      const int t = ck_row(g.hdr, g.m_perm[moff + p], g.n_rows);
      const float hv = pl[blk0 * MRB_ROWS + p];
      const float xv = isB ? ldv<XB>(g.dY, (int64_t)t * g.lddy + col) : ldv<XB>(g.X, (int64_t)t * g.ldx + col);
      acc = fmaf(xv, hv, acc);
    }
    const int64_t oi = isB ? (int64_t)col * r + j : (int64_t)j * g.d_in + col;
    const float val = (mc == 0) ? 0.0f : m.scale * acc;
    out[oi] = g.accumulate ? out[oi] + val : val;
  }
}

GradArgs make_args(const GradLaunch& l) {
  GradArgs g{};
  g.hdr = l.o.hdr;
  g.mrb = l.o.rb;
  g.m_perm = l.m_perm;
  g.m_offsets = l.m_offsets;
  g.m_counts = l.m_counts;
  g.m_blk = l.m_blk;
  g.meta = l.o.meta;
  g.d_in = l.o.d_in;
  g.d_out = l.o.d_out;
  g.num_slots = l.o.num_slots;
  g.n_rows = l.o.n;
  g.X = l.X;
  g.ldx = l.ldx;
  g.dY = l.dY;
  g.lddy = l.lddy;
  g.H_saved = l.H_saved;
  g.ldh = l.ldh;
  g.accumulate = l.accumulate;
  g.hg = l.hg;
  g.ks = l.k_splits;
  g.p_stride = l.p_stride;
  g.r_pad = l.r_pad;
  g.fin = l.fin;
  return g;
}

int round8(long long g) { return (int)((g + 7) / 8 * 8); }

// Output pointers of slots [base, base + GRAD_SLOT_GROUP); false if none is set.
bool set_group(const GradLaunch& l, GradArgs& g, int base) {
  g.slot_base = base;
  g.slot_count = std::min(GRAD_SLOT_GROUP, l.o.num_slots - base);
  bool any = false;
  for (int i = 0; i < GRAD_SLOT_GROUP; ++i) {
    const int a = base + i;
    g.dA[i] = (i < g.slot_count && l.dA != nullptr) ? l.dA[a] : nullptr;
    g.dB[i] = (i < g.slot_count && l.dB != nullptr) ? l.dB[a] : nullptr;
    any = any || g.dA[i] != nullptr || g.dB[i] != nullptr;
  }
  return any;
}

template <int NT>
hipError_t launch_nt(const GradLaunch& l, const GradArgs& g, hipStream_t s) {
  hipError_t err;
  const int grid1 = round8(std::min<long long>((long long)l.o.rb_ub * l.k_splits, 4096));
  hipLaunchKernelGGL((hg_kernel<NT>), dim3(grid1), dim3(256), 0, s, g);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  const long long groups = 2LL * l.r_pad * l.o.rb_ub * (MRB_ROWS / 8);   // 8-column groups (upper bound)
  const int grid2 = (int)std::max<long long>(1, std::min<long long>((groups + 255) / 256, 4096));
  hipLaunchKernelGGL(hgsum_kernel, dim3(grid2), dim3(256), 0, s, g);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  for (int base = 0; base < l.o.num_slots; base += GRAD_SLOT_GROUP) {
    GradArgs gg = g;
    if (!set_group(l, gg, base)) continue;
    constexpr int CT = dt_ct(NT);
    const long long tiles = (long long)gg.slot_count *
                            ((l.o.d_out + CT - 1) / CT + (l.o.d_in + CT - 1) / CT);
    const int grid3 = round8(std::min<long long>(tiles, 8192));
    hipLaunchKernelGGL((dadb_kernel<NT>), dim3(grid3), dim3(256), 0, s, gg);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace

hipError_t launch_grad_mfma(const GradLaunch& l, hipStream_t s) {
  const GradArgs g = make_args(l);
  const int nt = (l.o.r_max + 15) / 16;
  if (nt <= 1) return launch_nt<1>(l, g, s);
  if (nt <= 2) return launch_nt<2>(l, g, s);
  if (nt <= 4) return launch_nt<4>(l, g, s);
  return launch_nt<8>(l, g, s);
}

hipError_t launch_grad_valu(const GradLaunch& l, lora_dtype x_dtype, lora_dtype w_dtype,
                            hipStream_t s) {
  const GradArgs g = make_args(l);
  const int grid1 = std::max(1, std::min(l.o.rb_ub, 4096));
  const bool xb = x_dtype == LORA_BF16, wb = w_dtype == LORA_BF16;
  if (xb && wb) hipLaunchKernelGGL((hg_valu_kernel<true, true>), dim3(grid1), dim3(256), 0, s, g);
  else if (xb) hipLaunchKernelGGL((hg_valu_kernel<true, false>), dim3(grid1), dim3(256), 0, s, g);
  else if (wb) hipLaunchKernelGGL((hg_valu_kernel<false, true>), dim3(grid1), dim3(256), 0, s, g);
  else hipLaunchKernelGGL((hg_valu_kernel<false, false>), dim3(grid1), dim3(256), 0, s, g);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  for (int base = 0; base < l.o.num_slots; base += GRAD_SLOT_GROUP) {
    GradArgs gg = g;
    if (!set_group(l, gg, base)) continue;
    const long long total = (long long)LORA_MAX_RANK * (l.o.d_out + l.o.d_in) * gg.slot_count;
    const int grid2 = (int)std::max<long long>(1, std::min<long long>((total + 255) / 256, 16384));
    if (xb) hipLaunchKernelGGL((dadb_valu_kernel<true>), dim3(grid2), dim3(256), 0, s, gg);
    else hipLaunchKernelGGL((dadb_valu_kernel<false>), dim3(grid2), dim3(256), 0, s, gg);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace lora
