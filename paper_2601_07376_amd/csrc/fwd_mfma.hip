// Forward matrix-core kernels for bfloat16 X and weights (Section 3.4: the LoRA
// layer equation and the per-group residual Delta_a = s_a (X_a A_a^T) B_a^T).
//
//  shrink  H[t, :r_a] = X[t] A_a^T       one workgroup per row block of one
//                                        adapter; the 4 waves split d_in and are
//                                        summed in a fixed order through LDS.
//  expand  Y[t] += s_a H[t, :r_a] B_a^T   one workgroup per (row block, 256
//                                        output columns); float32 H enters the
//                                        bf16 matrix core as hi + lo terms.
//  fused   both, for small groups (decode rows): H stays in LDS; the output
//          columns are split over sibling workgroups that recompute the small
//          shrink from L2 and are placed on the same XCD.
//
// Matrix core: v_mfma_f32_16x16x32_bf16.  Lane l holds row (l % 16) of the A
// operand and column (l % 16) of the B operand, eight consecutive K values at
// K offset 8 * (l / 16); the accumulator lane l holds rows 4 * (l / 16) + v,
// v = 0..3, of column l % 16.
#include <algorithm>

#include "device_common.h"
#include "lora_internal.h"

namespace lora {

namespace {

struct FwdArgs {
  const int32_t* hdr;
  const int4* rb;
  const int32_t* perm;
  const SlotMeta* meta;
  int32_t d_in, d_out;
  int32_t count_word, first_word;
  const uint16_t* X;
  int64_t ldx;
  float* H;
  int64_t ldh;
  void* Y;
  int64_t ldy;
  int32_t n_chunks, chunk;
};

__device__ __forceinline__ void entry_range(const FwdArgs& p, int& first, int& count) {
  first = p.first_word >= 0 ? p.hdr[p.first_word] : 0;
  count = p.hdr[p.count_word] - first;
}

// Eight float32 H values H[row][j..j+8) (zero past r), split into hi / lo.
template <bool RANK8>
__device__ __forceinline__ void load_h_split(const float* hrow, int j, int r, bf16x8& hi,
                                             bf16x8& lo) {
  float h[8];
  if (RANK8 && j < r) {
    const float4 a = *reinterpret_cast<const float4*>(hrow + j);
    const float4 b = *reinterpret_cast<const float4*>(hrow + j + 4);
    h[0] = a.x; h[1] = a.y; h[2] = a.z; h[3] = a.w;
    h[4] = b.x; h[5] = b.y; h[6] = b.z; h[7] = b.w;
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = (j + i < r) ? hrow[j + i] : 0.0f;
  }
  split_hi_lo(h, hi, lo);
}

// Y[t, o .. o+16) += s * acc, where acc[q][v] holds output o + 4 q + v.
template <bool YBF16>
__device__ __forceinline__ void y_update16(void* Yv, int64_t ldy, int t, int o, int d_out,
                                           float s, const f32x4 (&acc)[4]) {
  if (YBF16) {
    uint16_t* Y = reinterpret_cast<uint16_t*>(Yv) + (int64_t)t * ldy;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int oc = o + 8 * c;
      if (oc >= d_out) continue;
      uint4 v = *reinterpret_cast<const uint4*>(Y + oc);
      uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = 2 * c + (i >> 1), e0 = (2 * i) & 3;
        const float y0 = bf16_to_f32(w[i] & 0xffffu);
        const float y1 = bf16_to_f32(w[i] >> 16);
        const uint32_t r0 = f32_to_bf16_rne(fmaf(s, acc[q][e0], y0));
        const uint32_t r1 = f32_to_bf16_rne(fmaf(s, acc[q][e0 + 1], y1));
        w[i] = r0 | (r1 << 16);
      }
      *reinterpret_cast<uint4*>(Y + oc) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  } else {
    float* Y = reinterpret_cast<float*>(Yv) + (int64_t)t * ldy;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int oq = o + 4 * q;
      if (oq >= d_out) continue;
      float4 v = *reinterpret_cast<const float4*>(Y + oq);
      v.x = fmaf(s, acc[q][0], v.x);
      v.y = fmaf(s, acc[q][1], v.y);
      v.z = fmaf(s, acc[q][2], v.z);
      v.w = fmaf(s, acc[q][3], v.w);
      *reinterpret_cast<float4*>(Y + oq) = v;
    }
  }
}

// Sum the four waves' accumulators in a fixed order, ((w0 + w2) + (w1 + w3)),
// leaving the total in wave 0.  s_red holds 2 x N x 64 f32x4.
template <int N>
__device__ __forceinline__ void reduce_waves(f32x4 (&acc)[N], f32x4* s_red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
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
// shrink: H[t, :r] = X[t] A^T over row blocks of up to 64 rows
// ---------------------------------------------------------------------------
template <int NT>
__global__ __launch_bounds__(256) void shrink_kernel(FwdArgs p) {
  __shared__ f32x4 s_red[2 * 4 * NT * 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int first, count;
  entry_range(p, first, count);
  const XcdRange xr = xcd_range(count);
  for (int e = xr.first; e < xr.end; e += xr.step) {
    const int4 en = p.rb[first + e];
    const int a = en.x, p0 = en.y, rows = en.z;
    const SlotMeta m = p.meta[a];
    const int r = m.rank;
    const uint16_t* A = reinterpret_cast<const uint16_t*>(m.A);
    const int mt_used = (rows + 15) >> 4, nt_used = (r + 15) >> 4;

    int trow[4];
    bool rv[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int i = mt * 16 + (lane & 15);
      rv[mt] = i < rows;
      trow[mt] = rv[mt] ? p.perm[p0 + i] : 0;
    }
    f32x4 acc[4 * NT];
#pragma unroll
    for (int i = 0; i < 4 * NT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int kg = (lane >> 4) * 8;
    for (int k0 = w * 32; k0 < p.d_in; k0 += 128) {
      const int k = k0 + kg;
      const bool kv = k < p.d_in;
      bf16x8 xa[4], wb[NT];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
        xa[mt] = (mt < mt_used && rv[mt] && kv)
                     ? as_bf16x8(ldg16(p.X + (int64_t)trow[mt] * p.ldx + k))
                     : zero_bf16x8();
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int j = nt * 16 + (lane & 15);
        wb[nt] = (j < r && kv) ? as_bf16x8(ldg16(A + (int64_t)j * p.d_in + k)) : zero_bf16x8();
      }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        if (mt >= mt_used) continue;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          if (nt >= nt_used) continue;
          acc[mt * NT + nt] = mfma_16x16x32(xa[mt], wb[nt], acc[mt * NT + nt]);
        }
      }
    }
    reduce_waves<4 * NT>(acc, s_red);
    if (w == 0) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        if (mt >= mt_used) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int i = mt * 16 + (lane >> 4) * 4 + v;
          if (i >= rows) continue;
          float* hrow = p.H + (int64_t)p.perm[p0 + i] * p.ldh;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const int j = nt * 16 + (lane & 15);
            if (j < r) hrow[j] = acc[mt * NT + nt][v];
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// expand: Y[t] += s H[t, :r] B^T over (row block, 256-column tile)
// The A operand is B's rows, permuted so that lane l's four 16x16 tiles cover
// 16 consecutive output columns: tile q, operand row m -> column
// o_w + 16 (m / 4) + 4 q + (m % 4).
// ---------------------------------------------------------------------------
template <bool YBF16, bool RANK8>
__global__ __launch_bounds__(256) void expand_kernel(FwdArgs p) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int first, count;
  entry_range(p, first, count);
  const int n_ot = (p.d_out + 255) >> 8;
  const XcdRange xr = xcd_range(count * n_ot);
  for (int tile = xr.first; tile < xr.end; tile += xr.step) {
    const int e = tile / n_ot, ot = tile - e * n_ot;
    const int o_w = ot * 256 + w * 64;
    if (o_w >= p.d_out) continue;
    const int4 en = p.rb[first + e];
    const int a = en.x, p0 = en.y, rows = en.z;
    const SlotMeta m = p.meta[a];
    const int r = m.rank;
    const float s = m.scale;
    const uint16_t* B = reinterpret_cast<const uint16_t*>(m.B);
    const int tt_used = (rows + 15) >> 4;

    int trow[4];
    bool rv[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
      const int i = tt * 16 + (lane & 15);
      rv[tt] = i < rows;
      trow[tt] = rv[tt] ? p.perm[p0 + i] : 0;
    }
    const int mrow = lane & 15;
    int orow[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) orow[q] = o_w + (mrow >> 2) * 16 + q * 4 + (mrow & 3);

    f32x4 acc[4][4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) acc[q][tt] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int jg = (lane >> 4) * 8;
    for (int j0 = 0; j0 < r; j0 += 32) {
      const int j = j0 + jg;
      bf16x8 bo[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        bo[q] = (orow[q] < p.d_out) ? load_row8(B + (int64_t)orow[q] * r, j, r, RANK8)
                                    : zero_bf16x8();
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        if (tt >= tt_used) continue;
        bf16x8 hh, hl;
        if (rv[tt]) {
          load_h_split<RANK8>(p.H + (int64_t)trow[tt] * p.ldh, j, r, hh, hl);
        } else {
          hh = zero_bf16x8();
          hl = zero_bf16x8();
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[q][tt] = mfma_16x16x32(bo[q], hh, acc[q][tt]);
          acc[q][tt] = mfma_16x16x32(bo[q], hl, acc[q][tt]);
        }
      }
    }
    const int o_y = o_w + (lane >> 4) * 16;
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
      if (tt >= tt_used || !rv[tt]) continue;
      const f32x4 col[4] = {acc[0][tt], acc[1][tt], acc[2][tt], acc[3][tt]};
      y_update16<YBF16>(p.Y, p.ldy, trow[tt], o_y, p.d_out, s, col);
    }
  }
}

// ---------------------------------------------------------------------------
// fused small-group kernel: entries of <= 16 rows; workgroup (entry, chunk)
// ---------------------------------------------------------------------------
template <bool YBF16, int NT, bool RANK8>
__global__ __launch_bounds__(256) void fused_small_kernel(FwdArgs p) {
  __shared__ f32x4 s_red[2 * NT * 64];
  __shared__ float s_h[16][NT * 16 + 4];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int first, count;
  entry_range(p, first, count);
  const int P = p.n_chunks;
  // siblings (same entry, different column chunk) share blockIdx % 8, i.e. one XCD
  const int slot = (int)(blockIdx.x >> 3);
  const int e = 8 * (slot / P) + (int)(blockIdx.x & 7);
  const int pc = slot % P;
  if (e >= count) return;
  const int4 en = p.rb[first + e];
  const int a = en.x, p0 = en.y, rows = en.z;
  const SlotMeta m = p.meta[a];
  const int r = m.rank;
  const float s = m.scale;
  const uint16_t* A = reinterpret_cast<const uint16_t*>(m.A);
  const uint16_t* B = reinterpret_cast<const uint16_t*>(m.B);
  const int nt_used = (r + 15) >> 4;

  const int i_l = lane & 15;
  const bool rv = i_l < rows;
  const int trow = rv ? p.perm[p0 + i_l] : 0;

  // ---- shrink: H[16 x r] = X[rows] A^T, d_in split over the waves
  f32x4 acc[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int kg = (lane >> 4) * 8;
  for (int k0 = w * 32; k0 < p.d_in; k0 += 128) {
    const int k = k0 + kg;
    const bool kv = k < p.d_in;
    const bf16x8 xa =
        (rv && kv) ? as_bf16x8(ldg16(p.X + (int64_t)trow * p.ldx + k)) : zero_bf16x8();
    bf16x8 wb[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int j = nt * 16 + (lane & 15);
      wb[nt] = (j < r && kv) ? as_bf16x8(ldg16(A + (int64_t)j * p.d_in + k)) : zero_bf16x8();
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
      if (nt < nt_used) acc[nt] = mfma_16x16x32(xa, wb[nt], acc[nt]);
  }
  reduce_waves<NT>(acc, s_red);
  if (w == 0) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int v = 0; v < 4; ++v) s_h[(lane >> 4) * 4 + v][nt * 16 + (lane & 15)] = acc[nt][v];
  }
  __syncthreads();

  // ---- H operand (hi / lo) for every 32-wide rank step, kept in registers
  constexpr int KS_MAX = (NT * 16 + 31) / 32;
  const int ks_used = (r + 31) >> 5;
  bf16x8 hh[KS_MAX], hl[KS_MAX];
#pragma unroll
  for (int ks = 0; ks < KS_MAX; ++ks) {
    float h[8];
    const int j = ks * 32 + (lane >> 4) * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = (j + i < r) ? s_h[i_l][j + i] : 0.0f;
    split_hi_lo(h, hh[ks], hl[ks]);
  }

  // ---- expand over this workgroup's column chunk
  const int c0 = pc * p.chunk;
  const int c1 = min(p.d_out, c0 + p.chunk);
  const int mrow = lane & 15;
  for (int o_w = c0 + w * 64; o_w < c1; o_w += 256) {
    f32x4 acc2[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc2[q] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS_MAX; ++ks) {
      if (ks >= ks_used) continue;
      const int j = ks * 32 + (lane >> 4) * 8;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int o = o_w + (mrow >> 2) * 16 + q * 4 + (mrow & 3);
        const bf16x8 bo =
            (o < c1) ? load_row8(B + (int64_t)o * r, j, r, RANK8) : zero_bf16x8();
        acc2[q] = mfma_16x16x32(bo, hh[ks], acc2[q]);
        acc2[q] = mfma_16x16x32(bo, hl[ks], acc2[q]);
      }
    }
    if (rv) y_update16<YBF16>(p.Y, p.ldy, trow, o_w + (lane >> 4) * 16, c1, s, acc2);
  }
}

template <typename K>
hipError_t launch(K kernel, int grid, const FwdArgs& a, hipStream_t s) {
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(kernel, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

int round8(int g) { return (g + 7) / 8 * 8; }

FwdArgs base_args(const OpLaunch& o) {
  FwdArgs a{};
  a.hdr = o.hdr;
  a.rb = o.rb;
  a.perm = o.perm;
  a.meta = o.meta;
  a.d_in = o.d_in;
  a.d_out = o.d_out;
  a.count_word = o.count_word;
  a.first_word = o.first_word;
  return a;
}

}  // namespace

hipError_t launch_shrink_mfma(const OpLaunch& o, const void* X, int64_t ldx, float* H,
                              int64_t ldh, hipStream_t s) {
  FwdArgs a = base_args(o);
  a.X = reinterpret_cast<const uint16_t*>(X);
  a.ldx = ldx;
  a.H = H;
  a.ldh = ldh;
  const int grid = round8(std::min(o.rb_ub, 2048));
  const int nt = (o.r_max + 15) / 16;
  if (nt <= 1) return launch(shrink_kernel<1>, grid, a, s);
  if (nt <= 2) return launch(shrink_kernel<2>, grid, a, s);
  if (nt <= 4) return launch(shrink_kernel<4>, grid, a, s);
  return launch(shrink_kernel<8>, grid, a, s);
}

hipError_t launch_expand_mfma(const OpLaunch& o, const float* H, int64_t ldh, void* Y,
                              lora_dtype y_dtype, int64_t ldy, hipStream_t s) {
  FwdArgs a = base_args(o);
  a.H = const_cast<float*>(H);
  a.ldh = ldh;
  a.Y = Y;
  a.ldy = ldy;
  const long long tiles = (long long)o.rb_ub * ((o.d_out + 255) / 256);
  const int grid = round8((int)std::min<long long>(tiles, 8192));
  const bool yb = y_dtype == LORA_BF16;
  if (yb && o.rank8) return launch(expand_kernel<true, true>, grid, a, s);
  if (yb) return launch(expand_kernel<true, false>, grid, a, s);
  if (o.rank8) return launch(expand_kernel<false, true>, grid, a, s);
  return launch(expand_kernel<false, false>, grid, a, s);
}

template <bool YB, bool R8>
static hipError_t launch_fused_nt(const OpLaunch& o, int grid, const FwdArgs& a, hipStream_t s) {
  const int nt = (o.r_max + 15) / 16;
  if (nt <= 1) return launch(fused_small_kernel<YB, 1, R8>, grid, a, s);
  if (nt <= 2) return launch(fused_small_kernel<YB, 2, R8>, grid, a, s);
  if (nt <= 4) return launch(fused_small_kernel<YB, 4, R8>, grid, a, s);
  return launch(fused_small_kernel<YB, 8, R8>, grid, a, s);
}

hipError_t launch_bgmv_mfma(const OpLaunch& o, const void* X, int64_t ldx, void* Y,
                            lora_dtype y_dtype, int64_t ldy, int32_t n_chunks, hipStream_t s) {
  FwdArgs a = base_args(o);
  a.X = reinterpret_cast<const uint16_t*>(X);
  a.ldx = ldx;
  a.Y = Y;
  a.ldy = ldy;
  const int P = std::max(1, n_chunks);
  a.n_chunks = P;
  a.chunk = ((o.d_out + P - 1) / P + 63) / 64 * 64;
  const int grid = 8 * P * ((o.rb_ub + 7) / 8);
  const bool yb = y_dtype == LORA_BF16;
  if (yb && o.rank8) return launch_fused_nt<true, true>(o, grid, a, s);
  if (yb) return launch_fused_nt<true, false>(o, grid, a, s);
  if (o.rank8) return launch_fused_nt<false, true>(o, grid, a, s);
  return launch_fused_nt<false, false>(o, grid, a, s);
}

}  // namespace lora
