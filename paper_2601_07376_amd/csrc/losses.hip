// Masked token-level losses and their gradient at the logits (the learning
// signals of Section 3.3 -- SFT weights w_t; the action mask m_t, rollout
// log-probabilities, advantages and correction weights of RL -- under the
// objectives of Section 3.5, "Forward/backward path"):
//   logp_t = z_t[y_t] - logsumexp(z_t)
//   CE:  L_t = -w_t logp_t
//   IS:  L_t = -m_t c_t A_t rho_t,  rho_t = exp(logp_t - l_old_t)
//   PPO: L_t = -m_t c_t min(rho_t A_t, clip(rho_t, 1 - lo, 1 + hi) A_t)
//   dL_t/dz_t = g_t (softmax(z_t) - onehot(y_t)),  g_t = -dL_t/dlogp_t
// The per-element exponentials (arguments <= 0) use the hardware exp2 path,
// __expf: its extra relative error, about |z - lse| 2^-24, is below the
// log-sum-exp's own summation error; per-row values use expf.
// One workgroup per row.  A row of up to LS_NV vectors per thread stays in
// registers between the two passes (one read of the logits); longer rows are
// read twice.  Inactive rows (w_t = 0, or m_t = 0) are not read: their loss and
// log-probability are 0 and their gradient row is written as zeros.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "device_common.h"
#include "lora_internal.h"

namespace lora {
namespace {

constexpr int LS_THREADS = 256;
constexpr int LS_NV = 16;     // 16-byte vectors per thread held in registers

struct LossArgs {
  int32_t kind, n, V;
  const void* z;
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
  void* dz;
  int64_t ldd;
};

// (max, sum of exp(x - max)) pairs; an empty side (max = -inf) adds nothing
__device__ __forceinline__ void lse_combine(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  const float a = m == -INFINITY ? 0.f : s * expf(m - mm);
  const float b = m2 == -INFINITY ? 0.f : s2 * expf(m2 - mm);
  m = mm;
  s = a + b;
}

template <bool ZB>
struct Vec {
  static constexpr int E = ZB ? 8 : 4;   // elements per 16-byte vector
  uint4 raw;
  __device__ __forceinline__ float at(int i) const {
    const uint32_t w = (&raw.x)[ZB ? i >> 1 : i];
    return ZB ? __uint_as_float((i & 1) ? (w & 0xffff0000u) : (w << 16)) : __uint_as_float(w);
  }
};

template <bool ZB, bool DB>
__global__ __launch_bounds__(LS_THREADS) void token_loss_kernel(LossArgs a) {
  constexpr int E = Vec<ZB>::E;
  constexpr int ES = ZB ? 2 : 4, DS = DB ? 2 : 4;
  __shared__ float s_m[4], s_s[4];
  const int t = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int V = a.V;
  const int nvec = (V + E - 1) / E;
  char* drow = reinterpret_cast<char*>(a.dz) + (int64_t)t * a.ldd * DS;

  // the row's signals (uniform loads)
  bool active;
  float wgt = 0.f, c = 1.f, A = 0.f, old = 0.f;
  if (a.kind == 0) {
    wgt = a.weight[t];
    active = wgt != 0.f;
  } else {
    active = a.mask == nullptr || a.mask[t] != 0;
    if (active) {
      c = a.corr != nullptr ? a.corr[t] : 1.f;
      A = a.adv[t];
      old = a.old_logp[t];
    }
  }
  if (!active) {
    for (int q = tid; q < nvec; q += LS_THREADS) {
      const int v0 = q * E;
      if (v0 + E <= V) {
        if (DB && E == 8) *reinterpret_cast<uint4*>(drow + (int64_t)v0 * DS) = make_uint4(0, 0, 0, 0);
        else if (DB) *reinterpret_cast<uint2*>(drow + (int64_t)v0 * DS) = make_uint2(0, 0);
        else {
          for (int h = 0; h < E / 4; ++h)
            *reinterpret_cast<uint4*>(drow + (int64_t)(v0 + 4 * h) * DS) = make_uint4(0, 0, 0, 0);
        }
      } else {
        for (int i = v0; i < V; ++i) {
          if (DB) reinterpret_cast<uint16_t*>(drow)[i] = 0;
          else reinterpret_cast<float*>(drow)[i] = 0.f;
        }
      }
    }
    if (tid == 0) {
      a.loss[t] = 0.f;
      if (a.logp != nullptr) a.logp[t] = 0.f;
    }
    return;
  }
  const int y = a.target[t];
  const bool y_ok = y >= 0 && y < V;
  const char* zrow = reinterpret_cast<const char*>(a.z) + (int64_t)t * a.ldz * ES;
  float zy = 0.f;
  if (tid == 0 && y_ok) zy = ZB ? bf16_to_f32(reinterpret_cast<const uint16_t*>(zrow)[y])
                               : reinterpret_cast<const float*>(zrow)[y];

  // pass 1: running (max, sum) per thread over its vectors q = tid + 256 k
  const bool resident = nvec <= LS_NV * LS_THREADS;
  Vec<ZB> reg[LS_NV];
  float m = -INFINITY, s = 0.f;
  for (int q0 = 0; q0 < nvec; q0 += LS_NV * LS_THREADS) {
#pragma unroll
    for (int k = 0; k < LS_NV; ++k) {
      const int q = q0 + tid + k * LS_THREADS;
      reg[k].raw = q < nvec ? ldg16(zrow + (int64_t)q * 16) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < LS_NV; ++k) {
      const int q = q0 + tid + k * LS_THREADS;
      if (q >= nvec) break;
      float cm = -INFINITY;
#pragma unroll
      for (int i = 0; i < E; ++i)
        if (q * E + i < V) cm = fmaxf(cm, reg[k].at(i));
      float cs = 0.f;
#pragma unroll
      for (int i = 0; i < E; ++i)
        if (q * E + i < V) cs += __expf(reg[k].at(i) - cm);
      lse_combine(m, s, cm, cs);
    }
  }
  // the workgroup's (max, sum) in a fixed order
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float m2 = __shfl_xor(m, off, 64), s2 = __shfl_xor(s, off, 64);
    lse_combine(m, s, m2, s2);
  }
  if (lane == 0) {
    s_m[w] = m;
    s_s[w] = s;
  }
  __syncthreads();
  m = s_m[0];
  s = s_s[0];
  lse_combine(m, s, s_m[1], s_s[1]);
  float m23 = s_m[2], s23 = s_s[2];
  lse_combine(m23, s23, s_m[3], s_s[3]);
  lse_combine(m, s, m23, s23);
  const float lse = m + logf(s);

  // the row's coefficient g = -dL/dlogp, its loss and log-probability
  __shared__ float s_g;
  if (tid == 0) {
    const float lp = y_ok ? zy - lse : NAN;
    float L, g;
    if (a.kind == 0) {
      L = -wgt * lp;
      g = wgt;
    } else {
      const float rho = expf(lp - old);
      const float un = rho * A;
      if (a.kind == 1) {
        L = -c * un;
        g = c * A * rho;
      } else {
        const float cl = fminf(fmaxf(rho, 1.f - a.clip_lo), 1.f + a.clip_hi) * A;
        if (un <= cl || !(un == un)) {
          L = -c * un;
          g = c * A * rho;
        } else {
          L = -c * cl;
          g = 0.f;
        }
      }
    }
    a.loss[t] = L;
    if (a.logp != nullptr) a.logp[t] = lp;
    s_g = y_ok ? g : NAN;
  }
  __syncthreads();
  const float g = s_g;

  // pass 2: g (exp(z - lse) - [v == y]) for every element
  for (int q0 = 0; q0 < nvec; q0 += LS_NV * LS_THREADS) {
    if (!resident) {
#pragma unroll
      for (int k = 0; k < LS_NV; ++k) {
        const int q = q0 + tid + k * LS_THREADS;
        reg[k].raw = q < nvec ? ldg16(zrow + (int64_t)q * 16) : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int k = 0; k < LS_NV; ++k) {
      const int q = q0 + tid + k * LS_THREADS;
      if (q >= nvec) break;
      const int v0 = q * E;
      float d[E];
#pragma unroll
      for (int i = 0; i < E; ++i) {
        const float p = __expf(reg[k].at(i) - lse);
        d[i] = v0 + i == y ? fmaf(g, p, -g) : g * p;
      }
      if (v0 + E <= V) {
        if (DB) {
          uint32_t o[E / 2];
#pragma unroll
          for (int i = 0; i < E / 2; ++i) o[i] = pack2_bf16(d[2 * i], d[2 * i + 1]);
          if (E == 8) *reinterpret_cast<uint4*>(drow + (int64_t)v0 * DS) = make_uint4(o[0], o[1], o[2], o[3]);
          else *reinterpret_cast<uint2*>(drow + (int64_t)v0 * DS) = make_uint2(o[0], o[1]);
        } else {
#pragma unroll
          for (int h = 0; h < E / 4; ++h)
            *reinterpret_cast<float4*>(drow + (int64_t)(v0 + 4 * h) * DS) =
                make_float4(d[4 * h], d[4 * h + 1], d[4 * h + 2], d[4 * h + 3]);
        }
      } else {
        for (int i = 0; i < E && v0 + i < V; ++i) {
          if (DB) reinterpret_cast<uint16_t*>(drow)[v0 + i] = (uint16_t)f32_to_bf16_rne(d[i]);
          else reinterpret_cast<float*>(drow)[v0 + i] = d[i];
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_token_loss(const LossLaunch& l, hipStream_t s) {
  if (l.n == 0) return hipSuccess;
  LossArgs a{};
  a.kind = l.kind;
  a.n = l.n;
  a.V = l.vocab;
  a.z = l.logits;
  a.ldz = l.ldz;
  a.target = l.target;
  a.weight = l.weight;
  a.mask = l.mask;
  a.old_logp = l.old_logp;
  a.adv = l.adv;
  a.corr = l.corr;
  a.clip_lo = l.clip_lo;
  a.clip_hi = l.clip_hi;
  a.loss = l.loss;
  a.logp = l.logp;
  a.dz = l.dlogits;
  a.ldd = l.ldd;
  const dim3 grid(l.n), block(LS_THREADS);
  if (l.logits_bf16 && l.dlogits_bf16) hipLaunchKernelGGL((token_loss_kernel<true, true>), grid, block, 0, s, a);
  else if (l.logits_bf16) hipLaunchKernelGGL((token_loss_kernel<true, false>), grid, block, 0, s, a);
  else if (l.dlogits_bf16) hipLaunchKernelGGL((token_loss_kernel<false, true>), grid, block, 0, s, a);
  else hipLaunchKernelGGL((token_loss_kernel<false, false>), grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace lora
