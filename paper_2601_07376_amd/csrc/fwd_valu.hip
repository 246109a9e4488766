// Forward kernels on the vector ALU for any mix of float32 / bfloat16 storage
// (Section 3.4, LoRA layer equation).  Every dot product is a sequential
// float32 fused multiply-add chain in index order, one thread per output, so
// the result does not depend on the launch shape; the operands come from LDS.
#include <algorithm>

#include "device_common.h"
#include "lora_internal.h"

namespace lora {

namespace {

template <bool BF16>
__device__ __forceinline__ float ld(const void* p, int64_t i) {
  if (BF16) return bf16_to_f32(reinterpret_cast<const uint16_t*>(p)[i]);
  return reinterpret_cast<const float*>(p)[i];
}

struct ValuArgs {
  const int32_t* hdr;
  const int4* rb;
  const int32_t* perm;
  const SlotMeta* meta;
  int32_t d_in, d_out;
  int32_t count_word, first_word;
  const void* X;
  int64_t ldx;
  float* H;
  int64_t ldh;
  void* Y;
  int64_t ldy;
  int32_t num_slots;
  int32_t n_rows;           // rows of the batch: the bound of every row id read from the plan
};

// Work unit: an entry's rows in groups of VG; each group's operands are staged
// in LDS (the next chunk's loads in flight while a chunk is used), so the
// per-thread chains read LDS, not memory.
constexpr int VG = 16;                 // rows per unit
constexpr int VGROUPS = RB_ROWS / VG;  // most row groups of an entry

// H[t, j] = sum_k X[t, k] A[j, k] for ranks up to RM, k staged in chunks of
// VK (fewer, longer chunks for small ranks).  Thread pairs (row, j) = tid + 256 m.
template <bool XB, bool WB, int RM>
__global__ __launch_bounds__(256) void shrink_valu_kernel(ValuArgs p) {
  constexpr int VK = RM <= 32 ? 256 : 64;
  constexpr int PM = VG * RM / 256;                     // pairs per thread
  constexpr int XL = VG * VK / 256;                     // X values per thread and chunk
  constexpr int AL = RM * VK / 256;                     // A values per thread and chunk
  constexpr int KS = VK + 4;                            // LDS row stride (16-byte rows)
  __shared__ __align__(16) float s_x[VG][KS];
  __shared__ __align__(16) float s_a[RM][KS];
  const int tid = threadIdx.x;
  const int first = p.first_word >= 0 ? p.hdr[p.first_word] : 0;
  const int count = p.hdr[p.count_word] - first;
  for (int tile = blockIdx.x; tile < count * VGROUPS; tile += gridDim.x) {
    const int e = tile / VGROUPS, g = tile - e * VGROUPS;
    const int4 en = load_entry(p.rb, first + e);
    const int a = ck_slot(p.hdr, en.x, p.num_slots), rows = min(VG, en.z - g * VG), p0 = en.y + g * VG;
    if (rows <= 0) continue;
    const Slot m = load_slot(p.meta, a);
    const int r = m.rank;
    int xt[XL];
#pragma unroll
    for (int u = 0; u < XL; ++u) {
      const int i = (tid + 256 * u) / VK;
      xt[u] = ck_row(p.hdr, p.perm[p0 + (i < rows ? i : rows - 1)], p.n_rows);
    }
    float xv[XL], av[AL];
    auto fetch = [&](int k0) {
#pragma unroll
      for (int u = 0; u < XL; ++u) {
        const int k = k0 + (tid + 256 * u) % VK;
        xv[u] = k < p.d_in ? ld<XB>(p.X, (int64_t)xt[u] * p.ldx + k) : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < AL; ++u) {
        const int q = tid + 256 * u, j = q / VK, k = k0 + q % VK;
        av[u] = (j < r && k < p.d_in) ? ld<WB>(m.A, (int64_t)j * p.d_in + k) : 0.0f;
      }
    };
    float acc[PM];
#pragma unroll
    for (int i = 0; i < PM; ++i) acc[i] = 0.0f;
    fetch(0);
    for (int k0 = 0; k0 < p.d_in; k0 += VK) {
      __syncthreads();                 // the previous chunk's reads are done
#pragma unroll
      for (int u = 0; u < XL; ++u) s_x[(tid + 256 * u) / VK][(tid + 256 * u) % VK] = xv[u];
#pragma unroll
      for (int u = 0; u < AL; ++u) s_a[(tid + 256 * u) / VK][(tid + 256 * u) % VK] = av[u];
      __syncthreads();
      if (k0 + VK < p.d_in) fetch(k0 + VK);
      const int kn = min(VK, p.d_in - k0);
#pragma unroll
      for (int mm = 0; mm < PM; ++mm) {
        const int q = tid + 256 * mm, i = q / max(r, 1), j = q - i * max(r, 1);
        if (r == 0 || i >= rows) continue;
        // kn is a multiple of 8 (so is every dimension)
        float c = acc[mm];
#pragma unroll 8
        for (int kk = 0; kk < kn; kk += 4) {
          const float4 x4 = *reinterpret_cast<const float4*>(&s_x[i][kk]);
          const float4 a4 = *reinterpret_cast<const float4*>(&s_a[j][kk]);
          c = fmaf(x4.x, a4.x, c);
          c = fmaf(x4.y, a4.y, c);
          c = fmaf(x4.z, a4.z, c);
          c = fmaf(x4.w, a4.w, c);
        }
        acc[mm] = c;
      }
    }
#pragma unroll
    for (int mm = 0; mm < PM; ++mm) {
      const int q = tid + 256 * mm, i = q / max(r, 1), j = q - i * max(r, 1);
      if (r == 0 || i >= rows) continue;
      p.H[(int64_t)ck_row(p.hdr, p.perm[p0 + i], p.n_rows) * p.ldh + j] = acc[mm];
    }
  }
}

// Y[t, o] += s * sum_j H[t, j] B[o, j]; unit = (entry, 256 columns, row group),
// thread = column, the group's H rows staged in LDS.
template <bool WB, bool YB>
__global__ __launch_bounds__(256) void expand_valu_kernel(ValuArgs p) {
  constexpr int HL = VG * LORA_MAX_RANK / 256;          // H values per thread
  constexpr int JB = 32;                                // B values per thread in flight
  __shared__ float s_h[VG][LORA_MAX_RANK];
  const int tid = threadIdx.x;
  const int first = p.first_word >= 0 ? p.hdr[p.first_word] : 0;
  const int count = p.hdr[p.count_word] - first;
  const int n_ot = (p.d_out + 255) / 256;
  for (int tile = blockIdx.x; tile < count * n_ot * VGROUPS; tile += gridDim.x) {
    const int g = tile % VGROUPS, eo = tile / VGROUPS;
    const int e = eo / n_ot, o = (eo - e * n_ot) * 256 + tid;
    const int4 en = load_entry(p.rb, first + e);
    const int a = ck_slot(p.hdr, en.x, p.num_slots), rows = min(VG, en.z - g * VG), p0 = en.y + g * VG;
    if (rows <= 0) continue;
    const Slot m = load_slot(p.meta, a);
    const int r = m.rank;
    const float s = m.scale;
    // B (first JB ranks) and Y of this thread's column are requested together
    // with H, so the unit costs one round trip after the slot
    const bool ov = o < p.d_out;
    const int oc = ov ? o : p.d_out - 1;
    int yt[VG];
    float yv[VG];
#pragma unroll
    for (int i = 0; i < VG; ++i) {
      yt[i] = ck_row(p.hdr, p.perm[p0 + (i < rows ? i : rows - 1)], p.n_rows);
      const int64_t yo = (int64_t)yt[i] * p.ldy + oc;
      yv[i] = YB ? bf16_to_f32(reinterpret_cast<const uint16_t*>(p.Y)[yo])
                 : reinterpret_cast<const float*>(p.Y)[yo];
    }
    float b[JB];
    auto fetch_b = [&](int j0) {
#pragma unroll
      for (int jj = 0; jj < JB; ++jj)
        b[jj] = j0 + jj < r ? ld<WB>(m.B, (int64_t)oc * r + j0 + jj) : 0.0f;
    };
    fetch_b(0);
    __syncthreads();                   // the previous unit's reads of s_h are done
#pragma unroll
    for (int u = 0; u < HL; ++u) {
      const int q = tid + 256 * u, i = q / LORA_MAX_RANK, j = q % LORA_MAX_RANK;
      s_h[i][j] = (i < rows && j < r) ? p.H[(int64_t)ck_row(p.hdr, p.perm[p0 + i], p.n_rows) * p.ldh + j] : 0.0f;
    }
    __syncthreads();
    float acc[VG];
#pragma unroll
    for (int i = 0; i < VG; ++i) acc[i] = 0.0f;
    for (int j0 = 0; j0 < r; j0 += JB) {
      if (j0 > 0) fetch_b(j0);
      const int jn = min(JB, r - j0);
#pragma unroll
      for (int jj = 0; jj < JB; ++jj) {
        if (jj >= jn) break;
#pragma unroll
        for (int i = 0; i < VG; ++i) acc[i] = fmaf(s_h[i][j0 + jj], b[jj], acc[i]);
      }
    }
    if (!ov) continue;
#pragma unroll
    for (int i = 0; i < VG; ++i) {
      if (i >= rows) break;
      const int64_t yo = (int64_t)yt[i] * p.ldy + o;
      const float y = fmaf(s, acc[i], yv[i]);
      if (YB) reinterpret_cast<uint16_t*>(p.Y)[yo] = (uint16_t)f32_to_bf16_rne(y);
      else reinterpret_cast<float*>(p.Y)[yo] = y;
    }
  }
}

ValuArgs base_args(const OpLaunch& o) {
  ValuArgs a{};
  a.hdr = o.hdr;
  a.rb = o.rb;
  a.perm = o.perm;
  a.meta = o.meta;
  a.d_in = o.d_in;
  a.d_out = o.d_out;
  a.count_word = o.count_word;
  a.first_word = o.first_word;
  a.num_slots = o.num_slots;
  a.n_rows = o.n;
  return a;
}

}  // namespace

hipError_t launch_shrink_valu(const OpLaunch& o, const void* X, lora_dtype x_dtype,
                              int64_t ldx, lora_dtype w_dtype, float* H, int64_t ldh,
                              hipStream_t s) {
  ValuArgs a = base_args(o);
  a.X = X;
  a.ldx = ldx;
  a.H = H;
  a.ldh = ldh;
  const int grid = (int)std::max<long long>(1, std::min<long long>((long long)o.rb_ub * VGROUPS, 4096));
  const bool xb = x_dtype == LORA_BF16, wb = w_dtype == LORA_BF16;
  if (o.r_max <= 32) {
    if (xb && wb) hipLaunchKernelGGL((shrink_valu_kernel<true, true, 32>), dim3(grid), dim3(256), 0, s, a);
    else if (xb) hipLaunchKernelGGL((shrink_valu_kernel<true, false, 32>), dim3(grid), dim3(256), 0, s, a);
    else if (wb) hipLaunchKernelGGL((shrink_valu_kernel<false, true, 32>), dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL((shrink_valu_kernel<false, false, 32>), dim3(grid), dim3(256), 0, s, a);
  } else {
    constexpr int R = LORA_MAX_RANK;
    if (xb && wb) hipLaunchKernelGGL((shrink_valu_kernel<true, true, R>), dim3(grid), dim3(256), 0, s, a);
    else if (xb) hipLaunchKernelGGL((shrink_valu_kernel<true, false, R>), dim3(grid), dim3(256), 0, s, a);
    else if (wb) hipLaunchKernelGGL((shrink_valu_kernel<false, true, R>), dim3(grid), dim3(256), 0, s, a);
    else hipLaunchKernelGGL((shrink_valu_kernel<false, false, R>), dim3(grid), dim3(256), 0, s, a);
  }
  return hipGetLastError();
}

hipError_t launch_expand_valu(const OpLaunch& o, const float* H, int64_t ldh,
                              lora_dtype w_dtype, void* Y, lora_dtype y_dtype, int64_t ldy,
                              hipStream_t s) {
  ValuArgs a = base_args(o);
  a.H = const_cast<float*>(H);
  a.ldh = ldh;
  a.Y = Y;
  a.ldy = ldy;
  const long long tiles = (long long)o.rb_ub * ((o.d_out + 255) / 256) * VGROUPS;
  const int grid = (int)std::max<long long>(1, std::min<long long>(tiles, 8192));
  const bool wb = w_dtype == LORA_BF16, yb = y_dtype == LORA_BF16;
  if (wb && yb) hipLaunchKernelGGL((expand_valu_kernel<true, true>), dim3(grid), dim3(256), 0, s, a);
  else if (wb) hipLaunchKernelGGL((expand_valu_kernel<true, false>), dim3(grid), dim3(256), 0, s, a);
  else if (yb) hipLaunchKernelGGL((expand_valu_kernel<false, true>), dim3(grid), dim3(256), 0, s, a);
  else hipLaunchKernelGGL((expand_valu_kernel<false, false>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace lora
