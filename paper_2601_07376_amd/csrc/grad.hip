// Masked, adapter-local LoRA gradients (Section 3.3 for the explicit loss mask,
// Section 3.5 for gradients kept local to the owning adapter).  The paper does
// not write the backward; it is the chain rule on the LoRA layer equation of
// Section 3.4 restricted to the trainable rows T_a^m of adapter a:
//
//   H = X_m A_a^T,  G = dY_m B_a,  dB_a = s_a dY_m^T H,  dA_a = s_a G^T X_m.
//
// Stage 1 (per trainable row block of <= 32 rows and d-slice ks): partial H and
// G over the slice, written transposed into "planes" [j][column], where row i
// of block e sits in column 32 e + i (32-aligned, so stage 2 loads float4).
// Stage 2 (per adapter and 64-wide column block of dB or dA): a fixed-order
// reduction over the adapter's trainable rows, 32 rows per step; the partial
// planes are summed in slice order.  Rows outside T_a^m are never read.  No
// floating-point atomics anywhere, so the result is the same bytes run to run.
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
};

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
// stage 1 (matrix cores): partial H and G for one (row block, slice)
// ---------------------------------------------------------------------------
template <int NT, bool RANK8>
__global__ __launch_bounds__(256) void hg_kernel(GradArgs g) {
  constexpr int BT_STRIDE = 128 + 8;                   // bf16 elements per staged row
  __shared__ f32x4 s_red[2 * 4 * NT * 64];
  __shared__ __align__(16) uint16_t s_bt[NT * 16 * BT_STRIDE];       // B_a slab, transposed [j][o]
  const int lane = threadIdx.x & 63, w = wave_id(), tid = threadIdx.x;
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
    const rsrc_t Bw = make_rsrc(m.B, (uint32_t)g.d_out * (uint32_t)r * 2u);
    const int nt_used = (r + 15) >> 4;

    int trow[2];
    bool rv[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const int i = mt * 16 + (lane & 15);
      rv[mt] = i < rows;
      trow[mt] = rv[mt] ? g.m_perm[p0 + i] : 0;
    }
    // acc[0 .. 2NT) : H tiles (mt, nt); acc[2NT .. 4NT) : G tiles
    f32x4 acc[4 * NT];
#pragma unroll
    for (int i = 0; i < 4 * NT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int kg = (lane >> 4) * 8;

    if (g.H_saved == nullptr) {
      int kb, ke;
      slice(g.d_in, g.ks, ks, kb, ke);
      for (int k0 = kb + w * 32; k0 < ke; k0 += 128) {
        const int k = k0 + kg;
        const bool kv = k < ke;
        bf16x8 xa[2], wb[NT];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
          xa[mt] = (rv[mt] && kv) ? as_bf16x8(ldg16(X + (int64_t)trow[mt] * g.ldx + k))
                                  : zero_bf16x8();
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int j = nt * 16 + (lane & 15);
          wb[nt] = (j < r && kv) ? as_bf16x8(bload16(Aw, ((uint32_t)j * g.d_in + k) * 2u)) : zero_bf16x8();
        }
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
            if (nt < nt_used) acc[mt * NT + nt] = mfma_16x16x32(xa[mt], wb[nt], acc[mt * NT + nt]);
      }
    }

    {
      int ob, oe;
      slice(g.d_out, g.ks, ks, ob, oe);
      const int r8 = (r + 7) >> 3;
      for (int oc = ob; oc < oe; oc += 128) {
        __syncthreads();
        // stage B[oc .. oc+128, 0 .. r) transposed into s_bt[j][o - oc]
        for (int item = tid; item < 128 * r8; item += 256) {
          const int ol = item / r8, j8 = (item - ol * r8) * 8;
          const int o = oc + ol;
          bf16x8 v = (o < oe && j8 < r) ? wrow8<RANK8>(Bw, (uint32_t)o * r, j8, r) : zero_bf16x8();
          const uint4 u = __builtin_bit_cast(uint4, v);
          const uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int i = 0; i < 8; ++i)
            s_bt[(j8 + i) * BT_STRIDE + ol] = (uint16_t)(wv[i >> 1] >> (16 * (i & 1)));
        }
        __syncthreads();
        const int o = oc + w * 32 + kg;
        const bool ov = o < oe;
        bf16x8 ya[2], bb[NT];
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
          ya[mt] = (rv[mt] && ov) ? as_bf16x8(ldg16(dY + (int64_t)trow[mt] * g.lddy + o))
                                  : zero_bf16x8();
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int j = nt * 16 + (lane & 15);
          bb[nt] = as_bf16x8(*reinterpret_cast<const uint4*>(&s_bt[j * BT_STRIDE + w * 32 + kg]));
        }
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
            if (nt < nt_used)
              acc[2 * NT + mt * NT + nt] = mfma_16x16x32(ya[mt], bb[nt], acc[2 * NT + mt * NT + nt]);
      }
    }
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

// Sum of the slice planes for rows [c, c+8) of plane `which`, column j; split hi / lo.
__device__ __forceinline__ void plane8_split(const GradArgs& g, int which, int j, int col,
                                             bf16x8& hi, bf16x8& lo) {
  float h[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int ks = 0; ks < g.ks; ++ks) {
    const float* p = plane(g, which, ks) + (int64_t)j * g.p_stride + col;
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    h[0] += a.x; h[1] += a.y; h[2] += a.z; h[3] += a.w;
    h[4] += b.x; h[5] += b.y; h[6] += b.z; h[7] += b.w;
  }
  split_hi_lo(h, hi, lo);
}

// ---------------------------------------------------------------------------
// stage 2 (matrix cores): one workgroup per (adapter, 64-column block of dB or dA)
// ---------------------------------------------------------------------------
template <int NT>
__global__ __launch_bounds__(256) void dadb_kernel(GradArgs g) {
  constexpr int T_STRIDE = 32 + 8;                    // staged rows per column (+pad)
  __shared__ __align__(16) uint16_t s_t[64 * T_STRIDE];             // 32 rows x 64 columns, transposed
  const int lane = threadIdx.x & 63, w = wave_id(), tid = threadIdx.x;
  const int nbB = (g.d_out + 63) / 64, nbA = (g.d_in + 63) / 64, nbt = nbB + nbA;
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
    const int c0 = (isB ? c : c - nbB) * 64;
    const int dcol = isB ? g.d_out : g.d_in;        // columns of the contracted input
    const int mc = g.m_counts[a], moff = g.m_offsets[a], blk0 = g.m_blk[a];
    const float s = m.scale;
    const int nt_used = (r + 15) >> 4;
    const uint16_t* src = reinterpret_cast<const uint16_t*>(isB ? g.dY : g.X);
    const int64_t lds = isB ? g.lddy : g.ldx;

    f32x4 acc[NT];
#pragma unroll
    for (int i = 0; i < NT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int pb = 0; pb < mc; pb += 32) {
      __syncthreads();
      {
        const int pl = tid >> 3, cc = (tid & 7) * 8;
        const int p = pb + pl;
        uint4 u = make_uint4(0u, 0u, 0u, 0u);
        if (p < mc && c0 + cc < dcol) {
          const int t = g.m_perm[moff + p];
          u = ldg16(src + (int64_t)t * lds + c0 + cc);
        }
        const uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 8; ++i)
          s_t[(cc + i) * T_STRIDE + pl] = (uint16_t)(wv[i >> 1] >> (16 * (i & 1)));
      }
      __syncthreads();
      const int col = (blk0 + (pb >> 5)) * 32 + (lane >> 4) * 8;
      const bf16x8 tv =
          as_bf16x8(*reinterpret_cast<const uint4*>(&s_t[(w * 16 + (lane & 15)) * T_STRIDE + (lane >> 4) * 8]));
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        if (nt >= nt_used) continue;
        const int j = nt * 16 + (lane & 15);
        bf16x8 hi, lo;
        if (j < r) {
          plane8_split(g, isB ? 0 : 1, j, col, hi, lo);
        } else {
          hi = zero_bf16x8();
          lo = zero_bf16x8();
        }
        if (isB) {   // C[o][j]: A operand = staged dY^T (rows o), B operand = H (columns j)
          acc[nt] = mfma_16x16x32(tv, hi, acc[nt]);
          acc[nt] = mfma_16x16x32(tv, lo, acc[nt]);
        } else {     // C[j][k]: A operand = G^T (rows j), B operand = staged X (columns k)
          acc[nt] = mfma_16x16x32(hi, tv, acc[nt]);
          acc[nt] = mfma_16x16x32(lo, tv, acc[nt]);
        }
      }
    }
    if (mc == 0 && g.accumulate) continue;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      if (nt >= nt_used) continue;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        int oidx, valid;
        if (isB) {
          const int o = c0 + w * 16 + (lane >> 4) * 4 + v, j = nt * 16 + (lane & 15);
          valid = o < g.d_out && j < r;
          oidx = o * r + j;
        } else {
          const int j = nt * 16 + (lane >> 4) * 4 + v, k = c0 + w * 16 + (lane & 15);
          valid = j < r && k < g.d_in;
          oidx = j * g.d_in + k;
        }
        if (!valid) continue;
        const float val = (mc == 0) ? 0.0f : s * acc[nt][v];
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
  const int grid1 = round8(std::min<long long>((long long)l.o.rb_ub * l.k_splits, 4096));
  if (l.o.rank8)
    hipLaunchKernelGGL((hg_kernel<NT, true>), dim3(grid1), dim3(256), 0, s, g);
  else
    hipLaunchKernelGGL((hg_kernel<NT, false>), dim3(grid1), dim3(256), 0, s, g);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  for (int base = 0; base < l.o.num_slots; base += GRAD_SLOT_GROUP) {
    GradArgs gg = g;
    if (!set_group(l, gg, base)) continue;
    const long long tiles =
        (long long)gg.slot_count * ((l.o.d_out + 63) / 64 + (l.o.d_in + 63) / 64);
    const int grid2 = round8(std::min<long long>(tiles, 8192));
    hipLaunchKernelGGL((dadb_kernel<NT>), dim3(grid2), dim3(256), 0, s, gg);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
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
