// Masked, adapter-local LoRA gradients (Section 3.3 for the explicit loss mask,
// Section 3.5 for gradients kept local to the owning adapter).  The paper does
// not write the backward; it is the chain rule on the LoRA layer equation of
// Section 3.4 restricted to the trainable rows T_a^m of adapter a:
//
//   H = X_m A_a^T,  G = dY_m B_a,  dB_a = s_a dY_m^T H,  dA_a = s_a G^T X_m.
//
// Matrix-core path, four launches:
//  0. B_a^T of every live slot into the workspace, so that G reads its second
//     operand with d_out contiguous, as H reads A_a with d_in contiguous.
//  1. per trainable row block (<= 32 rows) and d-slice: partial H and G over
//     the slice, written transposed into fp32 "planes" [j][column], where row i
//     of block e sits in column 32 e + i.
//  2. the slice planes summed in slice order and split into bf16 hi + lo.
//  3. per adapter and 128-wide column tile of dB or dA: a fixed-order
//     reduction over the adapter's trainable rows, 32 rows per step; the row
//     tile is transposed through LDS and meets the hi / lo planes on the
//     matrix cores.
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
  uint16_t* bt;             // B_a^T per slot: [slot][r_pad][d_out]
};

__device__ __forceinline__ uint16_t* fin_plane(const GradArgs& g, int which, int hl) {
  return g.fin + ((int64_t)(which * 2 + hl) * g.r_pad) * g.p_stride;
}

__device__ __forceinline__ float* plane(const GradArgs& g, int which, int ks) {
  return g.hg + ((int64_t)(which * g.ks + ks) * g.r_pad) * g.p_stride;
}

// slice of a dimension for split ks, in multiples of 128
__device__ __forceinline__ void slice(int d, int nks, int ks, int& b, int& e) {
  const int w = ((d + nks - 1) / nks + 127) / 128 * 128;
  b = min(d, ks * w);
  e = min(d, b + w);
}

template <int N>
__device__ __forceinline__ void reduce_waves(f32x4 (&acc)[N], f32x4* s_red) {
  const int lane = threadIdx.x & 63, w = wave_id();
  __syncthreads();
  if (w >= 2) {
#pragma unroll
    for (int i = 0; i < N; ++i) s_red[((w - 2) * N + i) * 64 + lane] = acc[i];
  }
  __syncthreads();
  if (w < 2) {
#pragma unroll
    for (int i = 0; i < N; ++i) acc[i] += s_red[(w * N + i) * 64 + lane];
  }
  __syncthreads();
  if (w == 1) {
#pragma unroll
    for (int i = 0; i < N; ++i) s_red[i * 64 + lane] = acc[i];
  }
  __syncthreads();
  if (w == 0) {
#pragma unroll
    for (int i = 0; i < N; ++i) acc[i] += s_red[i * 64 + lane];
  }
}

// ---------------------------------------------------------------------------
// stage 0: B_a^T of every live slot, 64 rows of B per tile, through LDS
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void bt_kernel(GradArgs g) {
  __shared__ uint16_t s_b[64][LORA_MAX_RANK + 2];
  const int tid = threadIdx.x;
  const int tpo = (g.d_out + 63) / 64;
  for (int tile = blockIdx.x; tile < g.num_slots * tpo; tile += gridDim.x) {
    const int a = tile / tpo, o0 = (tile - a * tpo) * 64;
    const Slot m = load_slot(g.meta, a);
    const int r = m.rank;
    if (r <= 0) continue;
    const rsrc_t Bw = make_rsrc(m.B, (uint32_t)g.d_out * (uint32_t)r * 2u);
    const int orows = min(64, g.d_out - o0);
    __syncthreads();
    for (int i = tid; i < orows * r; i += 256) {          // B[o0 .. o0 + orows) is contiguous
      const int o = i / r, j = i - o * r;
      s_b[o][j] = (uint16_t)bload_u16(Bw, ((uint32_t)o0 * r + i) * 2u);
    }
    __syncthreads();
    uint16_t* bt = g.bt + (int64_t)a * g.r_pad * g.d_out + o0;
    for (int i = tid; i < r * 64; i += 256) {
      const int j = i >> 6, o = i & 63;
      if (o < orows) bt[(int64_t)j * g.d_out + o] = s_b[o][j];
    }
  }
}

// ---------------------------------------------------------------------------
// stage 1 (matrix cores): partial H and G for one (row block, slice).  Both are
// shrink-shaped products (rows x d-slice times rank x d-slice), streamed with
// double-buffered 16-byte loads.
// ---------------------------------------------------------------------------
template <int MT, int NT, int U>
__device__ __forceinline__ void rows_times_w(f32x4 (&acc)[MT * NT], const uint16_t* (&xr)[MT],
                                             rsrc_t W, const uint32_t (&wr)[NT], int kstart,
                                             int kstride, int kend) {
  const int kg = ((threadIdx.x & 63) >> 4) * 8;
  struct Buf {
    bf16x8 x[U][MT];
    bf16x8 w[U][NT];
    bool kv[U];
  };
  auto load = [&](Buf& b, int kb) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kb + u * kstride + kg;
      b.kv[u] = k < kend;
      const int kk = k < kend ? k : kend - 8;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) b.x[u][mt] = as_bf16x8(ldg16(xr[mt] + kk));
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) b.w[u][nt] = as_bf16x8(bload16(W, (wr[nt] + (uint32_t)kk) * 2u));
    }
  };
  // every tile is computed: no branch between a matrix-core instruction and
  // its reader (tiles past the rows or the rank are never stored)
  auto compute = [&](const Buf& b) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const bf16x8 xo = sel(b.kv[u], b.x[u][mt]);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          acc[mt * NT + nt] = mfma_16x16x32(xo, b.w[u][nt], acc[mt * NT + nt]);
      }
  };
  if (kstart < kend) {
    const int span = U * kstride;
    Buf b0, b1;
    load(b0, kstart);
    for (int kb = kstart;; kb += 2 * span) {
      const int k1 = kb + span;
      if (k1 < kend) load(b1, k1);
      compute(b0);
      if (k1 >= kend) break;
      const int k2 = k1 + span;
      if (k2 < kend) load(b0, k2);
      compute(b1);
      if (k2 >= kend) break;
    }
  }
  mfma_fence();
}

template <int NT>
__global__ __launch_bounds__(256) void hg_kernel(GradArgs g) {
  constexpr int U = NT <= 2 ? 2 : 1;
  __shared__ f32x4 s_red[2 * 4 * NT * 64];
  const int lane = threadIdx.x & 63, w = wave_id();
  const int n_blocks = g.hdr[HDR_NMRB];
  const XcdRange xr = xcd_range(n_blocks * g.ks);
  const uint16_t* X = reinterpret_cast<const uint16_t*>(g.X);
  const uint16_t* dY = reinterpret_cast<const uint16_t*>(g.dY);
  for (int tile = xr.first; tile < xr.end; tile += xr.step) {
    const int e = tile / g.ks, ks = tile - e * g.ks;
    const int4 en = load_entry(g.mrb, e);
    const int a = en.x, p0 = en.y, rows = en.z;
    const Slot m = load_slot(g.meta, a);
    const int r = m.rank;
    const rsrc_t Aw = make_rsrc(m.A, (uint32_t)r * (uint32_t)g.d_in * 2u);
    const rsrc_t Btw = make_rsrc(g.bt + (int64_t)a * g.r_pad * g.d_out,
                                 (uint32_t)r * (uint32_t)g.d_out * 2u);
    const uint16_t* xrow[2];
    const uint16_t* yrow[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const int i = mt * 16 + (lane & 15);
      const int t = g.m_perm[p0 + (i < rows ? i : rows - 1)];
      xrow[mt] = X + (int64_t)t * g.ldx;
      yrow[mt] = dY + (int64_t)t * g.lddy;
    }
    uint32_t arow[NT], brow[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int j = nt * 16 + (lane & 15);
      arow[nt] = (uint32_t)(j < r ? j : r - 1) * (uint32_t)g.d_in;
      brow[nt] = (uint32_t)(j < r ? j : r - 1) * (uint32_t)g.d_out;
    }
    // acc[0 .. 2NT) : H tiles (mt, nt); acc[2NT .. 4NT) : G tiles
    f32x4 acc[4 * NT];
#pragma unroll
    for (int i = 0; i < 4 * NT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 (&acc_h)[2 * NT] = *reinterpret_cast<f32x4(*)[2 * NT]>(&acc[0]);
    f32x4 (&acc_g)[2 * NT] = *reinterpret_cast<f32x4(*)[2 * NT]>(&acc[2 * NT]);
    if (g.H_saved == nullptr) {
      int kb, ke;
      slice(g.d_in, g.ks, ks, kb, ke);
      rows_times_w<2, NT, U>(acc_h, xrow, Aw, arow, kb + w * 32, 128, ke);
    }
    {
      int ob, oe;
      slice(g.d_out, g.ks, ks, ob, oe);
      rows_times_w<2, NT, U>(acc_g, yrow, Btw, brow, ob + w * 32, 128, oe);
    }
    vmem_drained();
    reduce_waves<4 * NT>(acc, s_red);
    if (w == 0) {
      float* ph = plane(g, 0, ks);
      float* pg = plane(g, 1, ks);
      const int col0 = e * 32;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int i = mt * 16 + (lane >> 4) * 4 + v;
            const int j = nt * 16 + (lane & 15);
            if (j >= g.r_pad) continue;
            const bool in = i < rows;
            if (g.H_saved == nullptr) ph[(int64_t)j * g.p_stride + col0 + i] = in ? acc[mt * NT + nt][v] : 0.0f;
            pg[(int64_t)j * g.p_stride + col0 + i] = in ? acc[2 * NT + mt * NT + nt][v] : 0.0f;
          }
      if (g.H_saved != nullptr) {
        for (int q = lane; q < 32 * g.r_pad; q += 64) {
          const int i = q / g.r_pad, j = q - i * g.r_pad;
          float h = 0.0f;
          if (ks == 0 && i < rows && j < r) h = g.H_saved[(int64_t)g.m_perm[p0 + i] * g.ldh + j];
          ph[(int64_t)j * g.p_stride + col0 + i] = h;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// stage 2: planes summed in slice order, split into bf16 hi / lo (8 columns per
// thread)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void hgsum_kernel(GradArgs g) {
  const int n8 = g.hdr[HDR_NMRB] * 4;                 // 8-column groups per plane row
  const int64_t per = (int64_t)g.r_pad * n8;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < 2 * per;
       q += (int64_t)gridDim.x * 256) {
    const int which = (int)(q / per);
    const int64_t u = q - which * per;
    const int j = (int)(u / n8), c = (int)(u - (int64_t)j * n8) * 8;
    float h[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int ks = 0; ks < g.ks; ++ks) {
      const float* p = plane(g, which, ks) + (int64_t)j * g.p_stride + c;
      const float4 x0 = ldg_f4(p), x1 = ldg_f4(p + 4);
      h[0] += x0.x; h[1] += x0.y; h[2] += x0.z; h[3] += x0.w;
      h[4] += x1.x; h[5] += x1.y; h[6] += x1.z; h[7] += x1.w;
    }
    bf16x8 hi, lo;
    split_hi_lo(h, hi, lo);
    stg16(fin_plane(g, which, 0) + (int64_t)j * g.p_stride + c, __builtin_bit_cast(uint4, hi));
    stg16(fin_plane(g, which, 1) + (int64_t)j * g.p_stride + c, __builtin_bit_cast(uint4, lo));
  }
}

// ---------------------------------------------------------------------------
// stage 3 (matrix cores): one workgroup per (slot, dB or dA, 128-column tile).
// Per 32-row step: the row tile of dY (for dB) or X (for dA) is loaded two
// steps ahead, transposed into LDS next to the step's hi / lo plane columns,
// and multiplied; LDS is double buffered, one barrier per step.
//   dB[o][j] = s sum_t dY[t][o] H[t][j]:  A operand = dY^T tile, B = H plane
//   dA[j][k] = s sum_t G[t][j] X[t][k]:   A operand = G plane, B = X^T tile
// ---------------------------------------------------------------------------
constexpr int DT_CT = 128;            // tile columns
constexpr int DT_TS = 32 + 8;         // LDS stride (bf16) of one transposed column
constexpr int DT_WIN = 512;           // row ids staged per window

template <int NT>
__global__ __launch_bounds__(256) void dadb_kernel(GradArgs g) {
  constexpr int CT = DT_CT, TS = DT_TS, PSEG = 2 * NT * 16 * 4;   // 16-byte plane pieces per step
  constexpr int PPT = (PSEG + 255) / 256;                           // per thread
  constexpr int R = 3;                                              // register ring (2 steps ahead)
  __shared__ __align__(16) uint16_t s_t[2][CT * TS];
  __shared__ __align__(16) uint16_t s_p[2][2 * NT * 16 * TS];     // [hl][j][t]
  __shared__ int s_rows[DT_WIN];
  const int lane = threadIdx.x & 63, w = wave_id(), tid = threadIdx.x;
  const int nbB = (g.d_out + CT - 1) / CT, nbA = (g.d_in + CT - 1) / CT, nbt = nbB + nbA;
  const XcdRange xr = xcd_range(g.slot_count * nbt);
  for (int tile = xr.first; tile < xr.end; tile += xr.step) {
    const int sl = tile / nbt, c = tile - sl * nbt;
    const int a = g.slot_base + sl;
    const Slot m = load_slot(g.meta, a);
    const int r = m.rank;
    if (r <= 0) continue;
    const bool isB = c < nbB;
    float* out = isB ? g.dB[sl] : g.dA[sl];
    if (out == nullptr) continue;
    const int c0 = (isB ? c : c - nbB) * CT;
    const int dcol = isB ? g.d_out : g.d_in;
    const int mc = uni(g.m_counts[a]), moff = uni(g.m_offsets[a]), blk0 = uni(g.m_blk[a]);
    const float s = m.scale;
    const uint16_t* src = reinterpret_cast<const uint16_t*>(isB ? g.dY : g.X);
    const int64_t ld = isB ? g.lddy : g.ldx;
    const uint16_t* fin0 = fin_plane(g, isB ? 0 : 1, 0);
    const uint16_t* fin1 = fin_plane(g, isB ? 0 : 1, 1);

    f32x4 acc[2][NT];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[i][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nch = (mc + 31) >> 5;
    for (int w0 = 0; w0 < nch; w0 += DT_WIN / 32) {
      const int wch = min(DT_WIN / 32, nch - w0);
      __syncthreads();
      for (int i = tid; i < DT_WIN; i += 256) {
        const int p = w0 * 32 + i;
        s_rows[i] = g.m_perm[moff + (p < mc ? p : mc - 1)];
      }
      __syncthreads();

      uint4 tr[R][2], pr[R][PPT];
      // raw loads of step cc into ring slot q (clamped addresses; masked at the LDS write)
      auto load = [&](int q, int cc) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int sgm = tid + 256 * h, i = sgm >> 4, cs = (sgm & 15) * 8;
          const int col = c0 + cs < dcol ? c0 + cs : dcol - 8;
          tr[q][h] = ldg16(src + (int64_t)s_rows[cc * 32 + i] * ld + col);
        }
        const int col0 = (blk0 + w0 + cc) * 32;
#pragma unroll
        for (int h = 0; h < PPT; ++h) {
          int sgm = tid + 256 * h;
          sgm = sgm < PSEG ? sgm : PSEG - 1;
          const int hl = sgm / (NT * 64), rem = sgm - hl * (NT * 64);
          const int j = rem >> 2, part = (rem & 3) * 8;
          pr[q][h] = ldg16((hl ? fin1 : fin0) + (int64_t)j * g.p_stride + col0 + part);
        }
      };
      auto stage = [&](int q, int cc, int buf) {
        const int rows_left = mc - (w0 + cc) * 32;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int sgm = tid + 256 * h, i = sgm >> 4, cs = (sgm & 15) * 8;
          const bool ok = i < rows_left && c0 + cs < dcol;
          const uint4 u = ok ? tr[q][h] : make_uint4(0u, 0u, 0u, 0u);
          const uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int k = 0; k < 8; ++k)
            s_t[buf][(cs + k) * TS + i] = (uint16_t)(wv[k >> 1] >> (16 * (k & 1)));
        }
#pragma unroll
        for (int h = 0; h < PPT; ++h) {
          const int sgm = tid + 256 * h;
          if (sgm >= PSEG) continue;
          const int hl = sgm / (NT * 64), rem = sgm - hl * (NT * 64);
          const int j = rem >> 2, part = (rem & 3) * 8;
          *reinterpret_cast<uint4*>(&s_p[buf][(hl * NT * 16 + j) * TS + part]) = pr[q][h];
        }
      };
      auto mma = [&](int buf) {
        const int tg = (lane >> 4) * 8, n = lane & 15;
#pragma unroll
        for (int i2 = 0; i2 < 2; ++i2) {
          const bf16x8 tv = as_bf16x8(
              *reinterpret_cast<const uint4*>(&s_t[buf][(w * 32 + i2 * 16 + n) * TS + tg]));
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const bf16x8 hi = as_bf16x8(
                *reinterpret_cast<const uint4*>(&s_p[buf][(nt * 16 + n) * TS + tg]));
            const bf16x8 lo = as_bf16x8(
                *reinterpret_cast<const uint4*>(&s_p[buf][((NT + nt) * 16 + n) * TS + tg]));
            if (isB) {
              acc[i2][nt] = mfma_16x16x32(tv, hi, acc[i2][nt]);
              acc[i2][nt] = mfma_16x16x32(tv, lo, acc[i2][nt]);
            } else {
              acc[i2][nt] = mfma_16x16x32(hi, tv, acc[i2][nt]);
              acc[i2][nt] = mfma_16x16x32(lo, tv, acc[i2][nt]);
            }
          }
        }
      };
      load(0, 0);
      if (wch > 1) load(1, 1);
      for (int cc0 = 0; cc0 < wch; cc0 += R) {
#pragma unroll
        for (int u = 0; u < R; ++u) {
          const int cc = cc0 + u;
          if (cc >= wch) break;
          if (cc + 2 < wch) load((u + 2) % R, cc + 2);
          stage(u, cc, cc & 1);
          __syncthreads();
          mma(cc & 1);
        }
      }
    }

    mfma_fence();
    if (mc == 0 && g.accumulate) continue;
#pragma unroll
    for (int i2 = 0; i2 < 2; ++i2)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          int64_t oidx;
          bool valid;
          if (isB) {
            const int o = c0 + w * 32 + i2 * 16 + (lane >> 4) * 4 + v, j = nt * 16 + (lane & 15);
            valid = o < g.d_out && j < r;
            oidx = (int64_t)o * r + j;
          } else {
            const int j = nt * 16 + (lane >> 4) * 4 + v, k = c0 + w * 32 + i2 * 16 + (lane & 15);
            valid = j < r && k < g.d_in;
            oidx = (int64_t)j * g.d_in + k;
          }
          if (!valid) continue;
          const float val = (mc == 0) ? 0.0f : s * acc[i2][nt][v];
          out[oidx] = g.accumulate ? out[oidx] + val : val;
        }
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
    const int a = en.x, p0 = en.y, rows = en.z;
    const Slot m = load_slot(g.meta, a);
    const int r = m.rank;
    float* ph = plane(g, 0, 0);
    float* pg = plane(g, 1, 0);
    for (int q = threadIdx.x; q < 32 * g.r_pad; q += blockDim.x) {
      const int i = q / g.r_pad, j = q - i * g.r_pad;
      float h = 0.0f, gg = 0.0f;
      if (i < rows && j < r) {
        const int t = g.m_perm[p0 + i];
        if (g.H_saved != nullptr) {
          h = g.H_saved[(int64_t)t * g.ldh + j];
        } else {
          for (int k = 0; k < g.d_in; ++k)
            h = fmaf(ldv<XB>(g.X, (int64_t)t * g.ldx + k), ldv<WB>(m.A, (int64_t)j * g.d_in + k), h);
        }
        for (int o = 0; o < g.d_out; ++o)
          gg = fmaf(ldv<XB>(g.dY, (int64_t)t * g.lddy + o), ldv<WB>(m.B, (int64_t)o * r + j), gg);
      }
      ph[(int64_t)j * g.p_stride + e * 32 + i] = h;
      pg[(int64_t)j * g.p_stride + e * 32 + i] = gg;
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
    const int mc = g.m_counts[a], moff = g.m_offsets[a], blk0 = g.m_blk[a];
    if (mc == 0 && g.accumulate) continue;
    const float* pl = plane(g, isB ? 0 : 1, 0) + (int64_t)j * g.p_stride;
    float acc = 0.0f;
    for (int p = 0; p < mc; ++p) {
      const int t = g.m_perm[moff + p];
      const float hv = pl[(blk0 + (p >> 5)) * 32 + (p & 31)];
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
  g.bt = l.bt;
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
  const int tpo = (l.o.d_out + 63) / 64;
  const int grid0 = std::min(l.o.num_slots * tpo, 8192);
  hipLaunchKernelGGL(bt_kernel, dim3(grid0), dim3(256), 0, s, g);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int grid1 = round8(std::min<long long>((long long)l.o.rb_ub * l.k_splits, 4096));
  hipLaunchKernelGGL((hg_kernel<NT>), dim3(grid1), dim3(256), 0, s, g);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  const long long groups = 2LL * l.r_pad * l.o.rb_ub * 4;       // 8-column groups (upper bound)
  const int grid2 = (int)std::max<long long>(1, std::min<long long>((groups + 255) / 256, 4096));
  hipLaunchKernelGGL(hgsum_kernel, dim3(grid2), dim3(256), 0, s, g);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  for (int base = 0; base < l.o.num_slots; base += GRAD_SLOT_GROUP) {
    GradArgs gg = g;
    if (!set_group(l, gg, base)) continue;
    const long long tiles = (long long)gg.slot_count *
                            ((l.o.d_out + DT_CT - 1) / DT_CT + (l.o.d_in + DT_CT - 1) / DT_CT);
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
