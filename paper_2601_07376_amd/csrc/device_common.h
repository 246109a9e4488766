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

typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;

// float -> bfloat16, round to nearest even (gfx950 converts in hardware,
// v_cvt_pk_bf16_f32, two values per instruction; NaN stays NaN).
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)f);
}

// Plain accessors for buffers passed as kernel arguments (the compiler knows
// those are global memory).
__device__ __forceinline__ uint4 ldg16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ void stg16(void* p, uint4 v) { *reinterpret_cast<uint4*>(p) = v; }
__device__ __forceinline__ float4 ldg_f4(const float* p) {
  return *reinterpret_cast<const float4*>(p);
}
__device__ __forceinline__ void stg_f4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
template <typename T>
__device__ __forceinline__ T ldg(const T* p) {
  return *p;
}
template <typename T>
__device__ __forceinline__ void stg(T* p, T v) {
  *p = v;
}

// Adapter weights are reached through pointers read from the slot table, which
// the compiler can only treat as generic (flat) pointers; flat loads also count
// against the LDS/scalar counter and force extra waits.  They are read with
// buffer loads instead: a buffer resource (base, size in bytes) plus 32-bit byte
// offsets.  Offsets at or past the size read as zero.  Word 3 is the gfx9-family
// resource format.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           (int)0x00020000);
}
__device__ __forceinline__ uint4 bload16(rsrc_t r, uint32_t byte_off) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint32_t bload_u16(rsrc_t r, uint32_t byte_off) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, byte_off, 0, 0);
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
  uint32_t ph[4], pl[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ph[i] = pack2_bf16(h[2 * i], h[2 * i + 1]);
    pl[i] = pack2_bf16(h[2 * i] - bf16_to_f32(ph[i] & 0xffffu), h[2 * i + 1] - bf16_to_f32(ph[i] >> 16));
  }
  hi = as_bf16x8(make_uint4(ph[0], ph[1], ph[2], ph[3]));
  lo = as_bf16x8(make_uint4(pl[0], pl[1], pl[2], pl[3]));
}

__device__ __forceinline__ f32x4 mfma_16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Wait states between the last matrix-core instruction of a sequence and the
// first vector instruction that reads its result.  The hardware does not
// interlock that dependency; the compiler inserts the wait states itself
// within straight-line code but has been seen to miss them when the reader
// sits behind a branch (the first accumulator register then reads stale).
// Call this after every matrix-core loop whose results are read after control
// flow: 3 x 8 wait states cover the longest (16-pass) instructions.
__device__ __forceinline__ void mfma_fence() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Eight consecutive bf16 weights of a row that starts at element `row0` of a
// weight buffer, columns [j, j + 8) of a row of len.  With RANK8 (len a multiple
// of 8) this is one 16-byte load from a clamped column and the lanes with
// j >= len hold another column's weights: the caller zeroes them where the
// operand is consumed (selecting at load time would make the load wait at
// once).  Without RANK8 the columns >= len are zero.
template <bool RANK8>
__device__ __forceinline__ bf16x8 wrow8(rsrc_t w, uint32_t row0, int j, int len) {
  if (RANK8) {
    const int jj = j < len ? j : len - 8;
    return as_bf16x8(bload16(w, (row0 + (uint32_t)jj) * 2u));
  }
  uint32_t b[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int jj = j + i < len ? j + i : len - 1;
    const uint32_t v = bload_u16(w, (row0 + (uint32_t)jj) * 2u);
    b[i] = (j + i < len) ? v : 0u;
  }
  return pack_bf16x8(b);
}

// Keep-loads-unconditional helper: the hot loops read from addresses that are
// always inside the buffer (clamped) and zero the lanes that are padding with a
// select, so no load sits behind a divergent branch and the compiler can keep
// many loads in flight (a divergent branch makes it wait for every outstanding
// load at the join).
__device__ __forceinline__ bf16x8 sel(bool keep, bf16x8 v) { return keep ? v : zero_bf16x8(); }


// Wait until every vector memory operation of this wave has completed.  Placed
// where all loads are known to be done anyway (right after the last use of a
// load batch), it costs nothing and tells the compiler's wait insertion that
// nothing is outstanding, so later code does not wait on the completion of
// stores issued in between.  gfx9 encoding: vmcnt 0, expcnt 7, lgkmcnt 15.
__device__ __forceinline__ void vmem_drained() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Wave-uniform views of per-tile metadata.  Entries and slot records are read
// with vector loads; readfirstlane tells the compiler the values are the same in
// every lane, so they live in scalar registers (a buffer resource built from a
// value the compiler thinks may differ per lane would be looped over lanes).
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Index of this wave in the workgroup, known to the compiler to be wave-uniform
// (so loops and branches that depend on it stay scalar, not exec-masked).
__device__ __forceinline__ int wave_id() { return uni((int)(threadIdx.x >> 6)); }

__device__ __forceinline__ int4 load_entry(const int4* list, int i) {
  const int4 e = list[i];
  return make_int4(uni(e.x), uni(e.y), uni(e.z), uni(e.w));
}

struct Slot {
  const void* A;
  const void* B;
  int rank;
  float scale;
};

__device__ __forceinline__ const void* uni_ptr(const void* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint64_t lo = (uint32_t)uni((int)(uint32_t)v);
  const uint64_t hi = (uint32_t)uni((int)(uint32_t)(v >> 32));
  return reinterpret_cast<const void*>(lo | (hi << 32));
}

template <typename Meta>
__device__ __forceinline__ Slot load_slot(const Meta* meta, int a) {
  const Meta m = meta[a];
  Slot s;
  s.A = uni_ptr(m.A);
  s.B = uni_ptr(m.B);
  s.rank = uni(m.rank);
  s.scale = __int_as_float(uni(__float_as_int(m.scale)));
  return s;
}

// ---- bounds checks of plan values (debug build) ------------------------------
// Built with LORA_DEBUG=1, every kernel that reads the plan checks each row id
// and adapter id it takes from a plan array before using it as an index: a
// value outside [0, n) or [0, num_slots) sets LORA_DATA_BOUNDS in the plan's
// data flag (header word 0, read by lora_plan_check) and is replaced by 0, so
// that no access leaves the caller's buffers.  In the release build both
// checks are the identity and compile to nothing.
#ifndef LORA_DEBUG
#define LORA_DEBUG 0
#endif
constexpr uint32_t DATA_BOUNDS_BIT = 8u;    // LORA_DATA_BOUNDS

__device__ __forceinline__ void flag_bounds(const int32_t* hdr) {
  atomicOr(reinterpret_cast<unsigned int*>(const_cast<int32_t*>(hdr)), DATA_BOUNDS_BIT);
}
// row id t of a batch of n rows
__device__ __forceinline__ int ck_row(const int32_t* hdr, int t, int n) {
#if LORA_DEBUG
  if ((unsigned)t >= (unsigned)n) {
    flag_bounds(hdr);
    return 0;
  }
#else
  (void)hdr;
  (void)n;
#endif
  return t;
}
// adapter id a of a table of S slots
__device__ __forceinline__ int ck_slot(const int32_t* hdr, int a, int S) {
#if LORA_DEBUG
  if ((unsigned)a >= (unsigned)S) {
    flag_bounds(hdr);
    return 0;
  }
#else
  (void)hdr;
  (void)S;
#endif
  return a;
}

// count of a run [off, off + cnt) of plan positions inside [0, n), or 0
__device__ __forceinline__ int ck_count(const int32_t* hdr, int off, int cnt, int n) {
#if LORA_DEBUG
  if (off < 0 || cnt < 0 || off > n - cnt) {
    flag_bounds(hdr);
    return 0;
  }
#else
  (void)hdr;
  (void)off;
  (void)n;
#endif
  return cnt;
}

// Lane shuffles through DPP (gfx9): a few cycles each, where ds_bpermute
// (__shfl and friends) costs an LDS round trip.
//   row_incl_scan   inclusive prefix sum inside each row of 16 lanes
//   wave_incl_scan  inclusive prefix sum over the 64 lanes (row scans, then the
//                   last lane of row 0 / row 1 broadcast into the later rows)
//   lane_prev/next  the value of lane - 1 / lane + 1 (`edge` at the wave ends)
__device__ __forceinline__ int row_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xf, 0xf, true);   // row_shr:8
  return x;
}
__device__ __forceinline__ int wave_incl_scan(int x) {
  x = row_incl_scan(x);
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}
__device__ __forceinline__ int lane_prev(int x, int edge) {
  return __builtin_amdgcn_update_dpp(edge, x, 0x138, 0xf, 0xf, false);  // wave_shr:1
}
__device__ __forceinline__ int lane_next(int x, int edge) {
  return __builtin_amdgcn_update_dpp(edge, x, 0x130, 0xf, 0xf, false);  // wave_shl:1
}
__device__ __forceinline__ int lane_value(int x, int l) { return __builtin_amdgcn_readlane(x, l); }

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

// Sum the four waves' accumulators in a fixed order, ((w0 + w2) + (w1 + w3)),
// leaving the total in wave 0; CH accumulators at a time through s_red
// (2 x CH x 64 f32x4).
template <int N, int CH>
__device__ __forceinline__ void reduce_waves(f32x4 (&acc)[N], f32x4* s_red) {
  const int lane = threadIdx.x & 63, w = wave_id();
#pragma unroll
  for (int c0 = 0; c0 < N; c0 += CH) {
    constexpr int C = CH;
    __syncthreads();
    if (w >= 2) {
#pragma unroll
      for (int i = 0; i < C; ++i)
        if (c0 + i < N) s_red[((w - 2) * C + i) * 64 + lane] = acc[c0 + i];
    }
    __syncthreads();
    if (w < 2) {
#pragma unroll
      for (int i = 0; i < C; ++i)
        if (c0 + i < N) acc[c0 + i] += s_red[(w * C + i) * 64 + lane];
    }
    __syncthreads();
    if (w == 1) {
#pragma unroll
      for (int i = 0; i < C; ++i)
        if (c0 + i < N) s_red[i * 64 + lane] = acc[c0 + i];
    }
    __syncthreads();
    if (w == 0) {
#pragma unroll
      for (int i = 0; i < C; ++i)
        if (c0 + i < N) acc[c0 + i] += s_red[i * 64 + lane];
    }
  }
}

}  // namespace lora
