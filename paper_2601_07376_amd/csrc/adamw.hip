// Adapter-local optimizer step: AdamW over the fp32 state of a group of
// adapter tensors (each dA_a / dB_a with its own moments and step count;
// Section 3.5 keeps gradients, optimizer moments and counters local to the
// owning policy).  The update is the published AdamW (Adam's bias-corrected
// moments, weight decay decoupled from the gradient):
//   m <- beta1 m + (1 - beta1) g,  v <- beta2 v + (1 - beta2) g^2,
//   p <- p (1 - lr wd) - lr mhat / (sqrt(vhat) + eps),
//   mhat = m / (1 - beta1^t),  vhat = v / (1 - beta2^t),
// with the bfloat16 copy of p (the adapter table's weights) written in the same
// pass.  HBM-bound: 16 bytes read and 12 (+2) written per element.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "device_common.h"
#include "lora_internal.h"

namespace lora {
namespace {

constexpr int AD_THREADS = 256;
constexpr int AD_VEC = 4;                               // elements per vector access
constexpr int AD_NV = 1;                                // vectors per thread and unit (1, 2 and 4 measured: 1 fastest)
constexpr int AD_CHUNK = AD_THREADS * AD_VEC * AD_NV;   // elements per unit

struct AdamRec {
  float* p;
  float* m;
  float* v;
  const float* g;
  uint16_t* pb;          // nullable bf16 copy
  int64_t n;
  float decay;           // 1 - lr wd
  float step_size;       // lr / (1 - beta1^t)
  float inv_sqrt_bc2;    // 1 / sqrt(1 - beta2^t)
  float eps;
  float beta1, omb1;     // beta1, 1 - beta1
  float beta2, omb2;
};

struct AdamArgs {
  AdamRec r[ADAMW_GROUP];
  int32_t first_chunk[ADAMW_GROUP + 1];   // prefix of the records' chunk counts
  int32_t count;
};

struct Elem4 {
  float4 p, m, v, g;
};

__device__ __forceinline__ void adam1(const AdamRec& R, float& p, float& m, float& v, float g) {
  m = fmaf(R.beta1, m, R.omb1 * g);
  v = fmaf(R.beta2, v, (R.omb2 * g) * g);
  const float denom = sqrtf(v) * R.inv_sqrt_bc2 + R.eps;
  p = fmaf(-R.step_size, m / denom, p * R.decay);
}

__device__ __forceinline__ void adam4(const AdamRec& R, Elem4& e) {
  adam1(R, e.p.x, e.m.x, e.v.x, e.g.x);
  adam1(R, e.p.y, e.m.y, e.v.y, e.g.y);
  adam1(R, e.p.z, e.m.z, e.v.z, e.g.z);
  adam1(R, e.p.w, e.m.w, e.v.w, e.g.w);
}

__global__ __launch_bounds__(AD_THREADS) void adamw_kernel(AdamArgs a) {
  const int total = a.first_chunk[a.count];
  for (int u = blockIdx.x; u < total; u += gridDim.x) {
    int k = 0;
    while (k + 1 < a.count && a.first_chunk[k + 1] <= u) ++k;   // uniform: the unit's record
    const AdamRec& R = a.r[k];
    const int64_t base = (int64_t)(u - a.first_chunk[k]) * AD_CHUNK;
    int64_t e[AD_NV];   // this thread's vectors, each AD_THREADS vectors apart
#pragma unroll
    for (int j = 0; j < AD_NV; ++j) e[j] = base + (int64_t)(j * AD_THREADS + threadIdx.x) * AD_VEC;
    if (e[AD_NV - 1] + AD_VEC <= R.n) {
      // every vector inside: all loads first, then the arithmetic and stores
      Elem4 x[AD_NV];
#pragma unroll
      for (int j = 0; j < AD_NV; ++j) {
        x[j].p = ldg_f4(R.p + e[j]);
        x[j].m = ldg_f4(R.m + e[j]);
        x[j].v = ldg_f4(R.v + e[j]);
        x[j].g = ldg_f4(R.g + e[j]);
      }
#pragma unroll
      for (int j = 0; j < AD_NV; ++j) {
        adam4(R, x[j]);
        stg_f4(R.p + e[j], x[j].p);
        stg_f4(R.m + e[j], x[j].m);
        stg_f4(R.v + e[j], x[j].v);
        if (R.pb != nullptr)
          *reinterpret_cast<uint2*>(R.pb + e[j]) =
              make_uint2(pack2_bf16(x[j].p.x, x[j].p.y), pack2_bf16(x[j].p.z, x[j].p.w));
      }
    } else {
      // the record's last unit: element by element up to n
      for (int h = 0; h < AD_NV; ++h) {
        const int64_t eb = e[h];
        for (int i = 0; i < AD_VEC; ++i) {
          const int64_t e = eb + i;
          if (e >= R.n) break;
          float p = R.p[e], m = R.m[e], v = R.v[e];
          adam1(R, p, m, v, R.g[e]);
          R.p[e] = p;
          R.m[e] = m;
          R.v[e] = v;
          if (R.pb != nullptr) R.pb[e] = (uint16_t)f32_to_bf16_rne(p);
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_adamw(const AdamwLaunch* t, int32_t count, hipStream_t s) {
  AdamArgs a{};
  a.count = count;
  int32_t chunks = 0;
  for (int k = 0; k < count; ++k) {
    AdamRec& R = a.r[k];
    R.p = t[k].p;
    R.m = t[k].m;
    R.v = t[k].v;
    R.g = t[k].g;
    R.pb = static_cast<uint16_t*>(t[k].p_bf16);
    R.n = t[k].n;
    R.decay = t[k].decay;
    R.step_size = t[k].step_size;
    R.inv_sqrt_bc2 = t[k].inv_sqrt_bc2;
    R.eps = t[k].eps;
    R.beta1 = t[k].beta1;
    R.omb1 = t[k].omb1;
    R.beta2 = t[k].beta2;
    R.omb2 = t[k].omb2;
    a.first_chunk[k] = chunks;
    chunks += (int32_t)((t[k].n + AD_CHUNK - 1) / AD_CHUNK);
  }
  a.first_chunk[count] = chunks;
  if (chunks == 0) return hipSuccess;
  const int grid = chunks < 4096 ? chunks : 4096;
  hipLaunchKernelGGL(adamw_kernel, dim3(grid), dim3(AD_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace lora
