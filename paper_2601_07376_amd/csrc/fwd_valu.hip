// Forward kernels on the vector ALU for any mix of float32 / bfloat16 storage
// (Section 3.4, LoRA layer equation).  Every dot product is a sequential
// float32 fused multiply-add chain in index order, one thread per output, so
// the result does not depend on the launch shape.
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
};

// H[t, j] = sum_k X[t, k] A[j, k]; one workgroup per entry, one thread per (row, j).
template <bool XB, bool WB>
__global__ __launch_bounds__(256) void shrink_valu_kernel(ValuArgs p) {
  const int first = p.first_word >= 0 ? p.hdr[p.first_word] : 0;
  const int count = p.hdr[p.count_word] - first;
  for (int e = blockIdx.x; e < count; e += gridDim.x) {
    const int4 en = load_entry(p.rb, first + e);
    const int a = en.x, p0 = en.y, rows = en.z;
    const Slot m = load_slot(p.meta, a);
    const int r = m.rank;
    for (int q = threadIdx.x; q < rows * r; q += blockDim.x) {
      const int i = q / r, j = q - i * r;
      const int t = p.perm[p0 + i];
      const int64_t xo = (int64_t)t * p.ldx, ao = (int64_t)j * p.d_in;
      float acc = 0.0f;
      for (int k = 0; k < p.d_in; ++k) acc = fmaf(ld<XB>(p.X, xo + k), ld<WB>(m.A, ao + k), acc);
      p.H[(int64_t)t * p.ldh + j] = acc;
    }
  }
}

// Y[t, o] += s * sum_j H[t, j] B[o, j]; workgroup per (entry, 256 columns).
template <bool WB, bool YB>
__global__ __launch_bounds__(256) void expand_valu_kernel(ValuArgs p) {
  const int first = p.first_word >= 0 ? p.hdr[p.first_word] : 0;
  const int count = p.hdr[p.count_word] - first;
  const int n_ot = (p.d_out + 255) / 256;
  for (int tile = blockIdx.x; tile < count * n_ot; tile += gridDim.x) {
    const int e = tile / n_ot, o = (tile - e * n_ot) * 256 + (int)threadIdx.x;
    if (o >= p.d_out) continue;
    const int4 en = load_entry(p.rb, first + e);
    const int a = en.x, p0 = en.y, rows = en.z;
    const Slot m = load_slot(p.meta, a);
    const int r = m.rank;
    const float s = m.scale;
    for (int i = 0; i < rows; ++i) {
      const int t = p.perm[p0 + i];
      const float* h = p.H + (int64_t)t * p.ldh;
      float acc = 0.0f;
      for (int j = 0; j < r; ++j) acc = fmaf(h[j], ld<WB>(m.B, (int64_t)o * r + j), acc);
      const int64_t yo = (int64_t)t * p.ldy + o;
      if (YB) {
        uint16_t* Y = reinterpret_cast<uint16_t*>(p.Y);
        Y[yo] = (uint16_t)f32_to_bf16_rne(fmaf(s, acc, bf16_to_f32(Y[yo])));
      } else {
        float* Y = reinterpret_cast<float*>(p.Y);
        Y[yo] = fmaf(s, acc, Y[yo]);
      }
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
  const int grid = std::max(1, std::min(o.rb_ub, 4096));
  const bool xb = x_dtype == LORA_BF16, wb = w_dtype == LORA_BF16;
  if (xb && wb) hipLaunchKernelGGL((shrink_valu_kernel<true, true>), dim3(grid), dim3(256), 0, s, a);
  else if (xb) hipLaunchKernelGGL((shrink_valu_kernel<true, false>), dim3(grid), dim3(256), 0, s, a);
  else if (wb) hipLaunchKernelGGL((shrink_valu_kernel<false, true>), dim3(grid), dim3(256), 0, s, a);
  else hipLaunchKernelGGL((shrink_valu_kernel<false, false>), dim3(grid), dim3(256), 0, s, a);
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
  const long long tiles = (long long)o.rb_ub * ((o.d_out + 255) / 256);
  const int grid = (int)std::max<long long>(1, std::min<long long>(tiles, 8192));
  const bool wb = w_dtype == LORA_BF16, yb = y_dtype == LORA_BF16;
  if (wb && yb) hipLaunchKernelGGL((expand_valu_kernel<true, true>), dim3(grid), dim3(256), 0, s, a);
  else if (wb) hipLaunchKernelGGL((expand_valu_kernel<true, false>), dim3(grid), dim3(256), 0, s, a);
  else if (yb) hipLaunchKernelGGL((expand_valu_kernel<false, true>), dim3(grid), dim3(256), 0, s, a);
  else hipLaunchKernelGGL((expand_valu_kernel<false, false>), dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace lora
