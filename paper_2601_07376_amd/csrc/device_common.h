// Device-side helpers shared by the kernels: storage conversions, vector loads,
// matrix-core operand types, XCD-aware tile ranges.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace lora {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;   // matrix-core operand
typedef __attribute__((ext_vector_type(4))) float f32x4;     // 16x16 accumulator slice

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// float -> bfloat16 bits, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ uint4 ldg16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
  return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ bf16x8 zero_bf16x8() {
  return __builtin_bit_cast(bf16x8, make_uint4(0u, 0u, 0u, 0u));
}

// Pack eight bfloat16 bit patterns (low 16 bits of each word) into an operand.
__device__ __forceinline__ bf16x8 pack_bf16x8(const uint32_t (&b)[8]) {
  uint4 v;
  v.x = b[0] | (b[1] << 16);
  v.y = b[2] | (b[3] << 16);
  v.z = b[4] | (b[5] << 16);
  v.w = b[6] | (b[7] << 16);
  return as_bf16x8(v);
}

// Split eight float32 values into hi = bf16(h) and lo = bf16(h - hi): the pair
// carries 16 significant bits, and h - hi is exact in float32.
__device__ __forceinline__ void split_hi_lo(const float (&h)[8], bf16x8& hi, bf16x8& lo) {
  uint32_t bh[8], bl[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    bh[i] = f32_to_bf16_rne(h[i]);
    bl[i] = f32_to_bf16_rne(h[i] - bf16_to_f32(bh[i]));
  }
  hi = pack_bf16x8(bh);
  lo = pack_bf16x8(bl);
}

__device__ __forceinline__ f32x4 mfma_16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Eight consecutive bf16 weights starting at column j of a row of `len`
// elements; columns >= len read as zero.  `aligned` promises 16-byte alignment
// and j + 8 <= len whenever j < len.
__device__ __forceinline__ bf16x8 load_row8(const uint16_t* row, int j, int len, bool aligned) {
  if (j >= len) return zero_bf16x8();
  if (aligned) return as_bf16x8(ldg16(row + j));
  uint32_t b[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) b[i] = (j + i < len) ? (uint32_t)row[j + i] : 0u;
  return pack_bf16x8(b);
}

// Tile range of the XCD this workgroup runs on.  Workgroups are dispatched to
// the 8 XCDs round-robin by id, so workgroup g runs on XCD g % 8.  Giving each
// XCD a contiguous slice of the tile list keeps tiles that share an adapter's
// weights in one XCD's L2.
struct XcdRange {
  int begin, end, step, first;
};
__device__ __forceinline__ XcdRange xcd_range(int total) {
  const int x = blockIdx.x & 7;
  const int per = (int)(gridDim.x >> 3);
  XcdRange r;
  r.begin = (int)(((long long)x * total) >> 3);
  r.end = (int)(((long long)(x + 1) * total) >> 3);
  r.step = per;
  r.first = r.begin + (int)(blockIdx.x >> 3);
  return r;
}

}  // namespace lora
