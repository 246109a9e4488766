// Measurement utility, not part of the layer: a register-only loop of bf16
// matrix-core products (v_mfma_f32_32x32x16_bf16 on 16 independent
// accumulators per wave, the operand pattern of the layer's GEMM), whose
// achieved rate calibrates the matrix-core peak on the box the benchmark runs on.
#include <hip/hip_runtime.h>

#include "device_common.h"
#include "lora_internal.h"

namespace lora {

namespace {

typedef __attribute__((ext_vector_type(16))) float f32x16;

__global__ __launch_bounds__(256, 1) void calib_mfma_kernel(float* out, int iters) {
  bf16x8 a[4], b[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[j][i] = (__bf16)(0.001f * (float)((threadIdx.x + i + j) & 15));
      b[j][i] = (__bf16)(0.002f * (float)((i + 3 * j) & 7));
    }
  f32x16 c[16];
#pragma unroll
  for (int j = 0; j < 16; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) c[j][v] = 0.0f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 16; ++j)
      c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[j >> 2], b[j & 3], c[j], 0, 0, 0);
    asm volatile("" : "+v"(a[0]), "+v"(b[0]));
  }
  mfma_fence();
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 16; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += c[j][v];
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

hipError_t launch_calib_mfma(int32_t workgroups, int32_t iters, float* out, hipStream_t s) {
  hipLaunchKernelGGL(calib_mfma_kernel, dim3(workgroups), dim3(256), 0, s, out, iters);
  return hipGetLastError();
}

}  // namespace lora
