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
// All three are bound by HBM bandwidth, so the loops are written for memory-
// level parallelism: the shrink streams X and A in double-buffered batches of
// k-steps, and Y and B loads are issued before the matrix-core work they wait on.
//
// Matrix core: v_mfma_f32_16x16x32_bf16.  Lane l holds row (l % 16) of the A
// operand and column (l % 16) of the B operand, eight consecutive K values at
// K offset 8 * (l / 16); the accumulator lane l holds rows 4 * (l / 16) + v,
// v = 0..3, of column l % 16.
#include <algorithm>

#include "device_common.h"
#include "lora_internal.h"

namespace lora {

// Target of the stores of padding lanes (rows past the block, columns past the
// output): never read.  128 bytes per thread of a workgroup.  External
// linkage, so that the compiler keeps stores whose only target it is.
__device__ __align__(256) uint4 g_store_sink[256 * 8];

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
  const SmallRec* srec;     // fused path: small-group records
  int32_t n_rec;            // records the array holds (host bound)
  int32_t ks_max;           // large groups: most d-slices of the shrink (partial planes)
  int64_t hp_stride;        // elements between partial H planes
  int32_t cw;               // expand column chunk (0: chosen from the block count)
  int32_t force_fine;       // run the 64-row kernels whatever the plan chose (input gradient)
  const int32_t* ids;       // plan-free small batch: per-row slot ids [n_ids]
  int32_t n_ids;
  int32_t num_slots;
  int32_t n_rows;           // rows of the batch: the bound of every row id read from the plan
};

__device__ __forceinline__ void entry_range(const FwdArgs& p, int& first, int& count) {
  first = p.first_word >= 0 ? p.hdr[p.first_word] : 0;
  count = p.hdr[p.count_word] - first;
}

// Eight float32 H values H[row][j..j+8), split into hi / lo; zero past r or
// when the row is padding.  hrow must point at a real row (clamped).
template <bool RANK8>
__device__ __forceinline__ void load_h_split(const float* hrow, int j, int r, bool valid,
                                             bf16x8& hi, bf16x8& lo) {
  float h[8];
  if (RANK8) {
    const int jj = j < r ? j : r - 8;
    const float4 a = ldg_f4(hrow + jj);
    const float4 b = ldg_f4(hrow + jj + 4);
    const bool k = valid && j < r;
    h[0] = k ? a.x : 0.f; h[1] = k ? a.y : 0.f; h[2] = k ? a.z : 0.f; h[3] = k ? a.w : 0.f;
    h[4] = k ? b.x : 0.f; h[5] = k ? b.y : 0.f; h[6] = k ? b.z : 0.f; h[7] = k ? b.w : 0.f;
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = (valid && j + i < r) ? ldg(hrow + j + i) : 0.0f;
  }
  split_hi_lo(h, hi, lo);
}

// ---------------------------------------------------------------------------
// Output-column layout of one wave's 64-column slice.  Tile q (0..3) of the
// expand product, operand row m, covers column
//     o_w + 32 (q / 2) + 8 (m / 4) + 4 (q % 2) + (m % 4),
// so lane l (og = l / 16) holds, for one row, the 8 consecutive columns
// o_w + 32 c + 8 og + [0, 8) of tiles q = 2c, 2c + 1 (c = 0, 1), and one load
// instruction of the wave covers 64 contiguous bytes of 16 rows.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int out_col(int o_w, int q, int m) {
  return o_w + 32 * (q >> 1) + 8 * (m >> 2) + 4 * (q & 1) + (m & 3);
}

template <bool YBF16>
struct YFrag {
  uint4 v[YBF16 ? 2 : 4];
};

template <bool YBF16>
__device__ __forceinline__ void y_load(YFrag<YBF16>& f, const void* Yv, int64_t ldy, int t,
                                       int o_w, int og, int d_out) {
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    int o = o_w + 32 * c + 8 * og;
    o = o < d_out ? o : d_out - 8;          // clamped; such lanes are never stored
    if (YBF16) {
      const uint16_t* Y = reinterpret_cast<const uint16_t*>(Yv) + (int64_t)t * ldy;
      f.v[c] = ldg16(Y + o);
    } else {
      const float* Y = reinterpret_cast<const float*>(Yv) + (int64_t)t * ldy;
      f.v[2 * c] = ldg16(Y + o);
      f.v[2 * c + 1] = ldg16(Y + o + 4);
    }
  }
}

// y = y + s * acc (float32), rounded once to the storage type, and stored.
template <bool YBF16>
__device__ __forceinline__ void y_store(const YFrag<YBF16>& f, void* Yv, int64_t ldy, int t,
                                        int o_w, int og, int d_out, float s,
                                        const f32x4 (&acc)[4]) {
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int o = o_w + 32 * c + 8 * og;
    if (o >= d_out) continue;
    if (YBF16) {
      uint16_t* Y = reinterpret_cast<uint16_t*>(Yv) + (int64_t)t * ldy;
      const uint32_t w[4] = {f.v[c].x, f.v[c].y, f.v[c].z, f.v[c].w};
      uint32_t o4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = 2 * c + (i >> 1), e0 = (2 * i) & 3;
        o4[i] = pack2_bf16(fmaf(s, acc[q][e0], bf16_to_f32(w[i] & 0xffffu)),
                           fmaf(s, acc[q][e0 + 1], bf16_to_f32(w[i] >> 16)));
      }
      stg16(Y + o, make_uint4(o4[0], o4[1], o4[2], o4[3]));
    } else {
      float* Y = reinterpret_cast<float*>(Yv) + (int64_t)t * ldy;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint4 u = f.v[2 * c + h];
        const f32x4 a = acc[2 * c + h];
        float4 v;
        v.x = fmaf(s, a[0], __uint_as_float(u.x));
        v.y = fmaf(s, a[1], __uint_as_float(u.y));
        v.z = fmaf(s, a[2], __uint_as_float(u.z));
        v.w = fmaf(s, a[3], __uint_as_float(u.w));
        stg_f4(Y + o + 4 * h, v);
      }
    }
  }
}

// acc[mt * NT + nt] += X[rows of mt] A[rows of nt]^T over this wave's k-steps
// k0 = kstart + i * kstride (k0 < kend).  xr[mt] points at a real X row and
// ar[nt] is the element offset of a real A row; padding lanes use a clamped row,
// and the caller discards the output rows / columns they produce.  Loads
// come in batches of U k-steps, double buffered so one batch is in flight while
// the previous one feeds the matrix cores.
template <int MT, int NT, int U>
__device__ __forceinline__ void shrink_steps(f32x4 (&acc)[MT * NT], const uint16_t* (&xr)[MT],
                                             rsrc_t A, const uint32_t (&ar)[NT], int kstart,
                                             int kstride, int kend) {
  const int kg = ((threadIdx.x & 63) >> 4) * 8;
  struct Buf {
    bf16x8 x[U][MT];
    bf16x8 w[U][NT];
    bool kv[U];
  };
  // raw loads from clamped addresses; nothing here consumes the loaded data
  auto load = [&](Buf& b, int kb) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = kb + u * kstride + kg;
      b.kv[u] = k < kend;
      const int kk = k < kend ? k : kend - 8;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) b.x[u][mt] = as_bf16x8(ldg16(xr[mt] + kk));
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        b.w[u][nt] = as_bf16x8(bload16(A, (ar[nt] + (uint32_t)kk) * 2u));
    }
  };
  // the K tail (k >= kend) is zeroed on the X operand where it is consumed.
  // Every tile is computed (tiles past the rows or the rank hold values that
  // are never stored): no branch separates a matrix-core instruction from its
  // reader.
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
    // the next batch is requested unconditionally (past the end every lane
    // reads a clamped address and the batch is never consumed): a load behind a
    // branch would make the compiler wait for every outstanding load at the join
    for (int kb = kstart;; kb += 2 * span) {
      const int k1 = kb + span;
      load(b1, k1);
      compute(b0);
      if (k1 >= kend) break;
      const int k2 = k1 + span;
      load(b0, k2);
      compute(b1);
      if (k2 >= kend) break;
    }
  }
  mfma_fence();
}

// ---------------------------------------------------------------------------
// Large groups: row blocks of up to 256 rows.  In both kernels wave w owns
// rows 64 w .. 64 w + 63 of the block (four 16-row tiles) and the workgroup
// stages the weight columns of each 32-wide step in LDS once for all four
// waves, so a block reads its adapter's weights once (not once per wave, and
// a 256-row block amortises them over four times the rows of a 64-row one).
// Loads run several steps ahead through register rings; LDS is double
// buffered with one barrier per step.
// ---------------------------------------------------------------------------

__device__ __forceinline__ int shrink_splits(const FwdArgs& p, int count) {
  return shrink_slices(p.ks_max, count);
}

// slice ks of [0, d) in multiples of 32
__device__ __forceinline__ void kslice(int d, int nks, int ks, int& b, int& e) {
  const int w = ((d + nks - 1) / nks + 31) / 32 * 32;
  b = min(d, ks * w);
  e = min(d, b + w);
}

// Pipeline shape shared by both kernels: the k- (or column-) steps of a unit
// are taken in batches of U steps, double buffered in registers (the loads of
// batch b + 1 are in flight while batch b feeds the matrix cores) and in LDS
// (one barrier per batch).  Every load of a batch is issued unconditionally
// (batches past the end repeat the last one and are never consumed), weight
// pieces first, and every store is unconditional too (padding lanes write to
// a sink): memory operations behind branches would make the compiler's wait
// counts conservative and drain the pipeline.
//
// LDS reuse: a wave stages batch b + 2 into a buffer only after the barrier of
// batch b + 1, which every wave reaches after its reads of batch b.


// ---------------------------------------------------------------------------
// shrink: Hp[ks][t, :r] = X[t, slice ks] A[:, slice ks]^T; with one slice this
// is H itself.  Work unit = (row block, d-slice).
// ---------------------------------------------------------------------------
template <int NT, int U>
__global__ __launch_bounds__(256) void shrink_kernel(FwdArgs p) {
  constexpr int AS = NT * 16;                  // staged A rows (rank padded to 16)
  constexpr int AP = AS * 4;                   // 16-byte A pieces per step
  constexpr int APT = (AP + 255) / 256;        // ... per thread
  constexpr int TS = 32 + 8;                   // LDS stride (bf16) of one staged row
  __shared__ __align__(16) uint16_t s_a[2][U][AS * TS];
  const int lane = threadIdx.x & 63, w = wave_id(), tid = threadIdx.x;
  const int mrow = lane & 15, kg = (lane >> 4) * 8;
  if (p.hdr[HDR_RB_ROWS] == RB_FINE) return;     // the fine kernel's batch
  int first, count;
  entry_range(p, first, count);
  const int nks = shrink_splits(p, count);
  const XcdRange xr = xcd_range(count * nks);
  for (int unit = xr.first; unit < xr.end; unit += xr.step) {
    const int e = unit / nks, ks = unit - e * nks;
    const int4 en = load_entry(p.rb, first + e);
    const int a = ck_slot(p.hdr, en.x, p.num_slots), p0 = en.y, rows = en.z;
    const Slot m = load_slot(p.meta, a);
    const int r = m.rank;
    const rsrc_t A = make_rsrc(m.A, (uint32_t)r * (uint32_t)p.d_in * 2u);
    int kb, ke;
    kslice(p.d_in, nks, ks, kb, ke);
    const int nst = max(1, (ke - kb + 31) / 32);
    const int nb = (nst + U - 1) / U;
    const int kend = max(ke, 8);

    const uint16_t* xrow[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int i = 64 * w + 16 * mt + mrow;
      xrow[mt] = p.X + (int64_t)ck_row(p.hdr, ldg(p.perm + p0 + (i < rows ? i : rows - 1)), p.n_rows) * p.ldx;
    }
    // row ids of the accumulator layout (rows 4 (l / 16) + v of each tile),
    // requested now so that the stores at the end do not wait on them
    int orow[4][4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = 64 * w + 16 * mt + (lane >> 4) * 4 + v;
        orow[mt][v] = ck_row(p.hdr, ldg(p.perm + p0 + (i < rows ? i : rows - 1)), p.n_rows);
      }
    // this thread's A pieces: row j (clamped to the rank), columns 8 c .. 8 c + 7
    // of a step.  With fewer pieces than threads (rank <= 32) several threads
    // load the same piece and store the same bytes.
    uint32_t arow[APT];
    int acol[APT], apos[APT];
#pragma unroll
    for (int h = 0; h < APT; ++h) {
      const int pc = (tid + 256 * h) & (AP - 1);   // (AP is a power of two)
      const int j = pc >> 2;
      arow[h] = (uint32_t)(j < r ? j : r - 1) * (uint32_t)p.d_in;
      acol[h] = (pc & 3) * 8;
      apos[h] = j * TS + acol[h];
    }

    f32x4 acc[4][NT];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    struct Buf {
      uint4 a[U][APT];
      uint4 x[U][4];
    };
    auto load = [&](Buf& b, int bt) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k0 = kb + 32 * (bt * U + u);
#pragma unroll
        for (int h = 0; h < APT; ++h) {
          const int ka = k0 + acol[h];
          b.a[u][h] = bload16(A, (arow[h] + (uint32_t)(ka < kend ? ka : kend - 8)) * 2u);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k = kb + 32 * (bt * U + u) + kg;
        const int kk = k < kend ? k : kend - 8;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) b.x[u][mt] = ldg16(xrow[mt] + kk);
      }
    };
    auto stage = [&](const Buf& b, int buf) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int h = 0; h < APT; ++h)
          *reinterpret_cast<uint4*>(&s_a[buf][u][apos[h]]) = b.a[u][h];
    };
    // steps past the slice (k >= ke) are zeroed on the X operand
    auto compute = [&](const Buf& b, int bt, int buf) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool kv = kb + 32 * (bt * U + u) + kg < ke;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const bf16x8 wv =
              as_bf16x8(*reinterpret_cast<const uint4*>(&s_a[buf][u][(nt * 16 + mrow) * TS + kg]));
#pragma unroll
          for (int mt = 0; mt < 4; ++mt)
            acc[mt][nt] = mfma_16x16x32(sel(kv, as_bf16x8(b.x[u][mt])), wv, acc[mt][nt]);
        }
      }
    };
    Buf b0, b1;
    load(b0, 0);
    __syncthreads();                 // the previous unit's reads of s_a are done
    // one exit, at the end of a pair of batches (a break between the halves
    // would give the compiler a path on which b1's loads are still pending
    // at the top, and a wait for all of them there)
    for (int bt = 0; bt < nb; bt += 2) {
      load(b1, min(bt + 1, nb - 1));
      __builtin_amdgcn_sched_barrier(0);
      stage(b0, 0);
      __syncthreads();
      compute(b0, bt, 0);
      load(b0, min(bt + 2, nb - 1));
      __builtin_amdgcn_sched_barrier(0);
      stage(b1, 1);
      __syncthreads();
      if (bt + 1 < nb) compute(b1, bt + 1, 1);
    }
    mfma_fence();
    float* H = p.H + (int64_t)ks * p.hp_stride;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = 64 * w + 16 * mt + (lane >> 4) * 4 + v;
        if (i >= rows) continue;
        float* hrow = H + (int64_t)orow[mt][v] * p.ldh;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          const int j = nt * 16 + mrow;
          if (j < r) stg(hrow + j, acc[mt][nt][v]);
        }
      }
  }
}

// ---------------------------------------------------------------------------
// expand: Y[t] += s (sum_ks Hp[ks][t, :r]) B^T.  Work unit = (row block, 1024
// output columns).  Each wave's H operands (hi / lo) are formed once per unit;
// the B rows of each 32-column step are staged in LDS for all waves.
//
// Step layout: tile q (0, 1), operand row m, covers column
// o_w + 8 (m / 4) + 4 q + (m % 4), so lane l (og = l / 16) holds the 8
// consecutive columns o_w + 8 og + [0, 8) of one row: one 16-byte load for a
// bf16 Y, and the wave's load covers 64 contiguous bytes of 16 rows.
// ---------------------------------------------------------------------------
template <bool YBF16>
struct Y8 {
  uint4 v[YBF16 ? 1 : 2];
};

template <bool YBF16>
__device__ __forceinline__ void y8_load(Y8<YBF16>& f, const void* Yv, int64_t ldy, int t, int o,
                                        int d_out) {
  o = o < d_out ? o : d_out - 8;            // clamped; such lanes store to the sink
  if (YBF16) {
    f.v[0] = ldg16(reinterpret_cast<const uint16_t*>(Yv) + (int64_t)t * ldy + o);
  } else {
    const float* Y = reinterpret_cast<const float*>(Yv) + (int64_t)t * ldy + o;
    f.v[0] = ldg16(Y);
    f.v[1] = ldg16(Y + 4);
  }
}

// y + s * acc, rounded once to the storage type, stored to dst (the row's 8
// columns, or the sink)
// y + s * acc for the 8 columns of a lane, rounded once to the storage type:
// 16 bytes (bf16) or 32 bytes (f32) in out[0..1]
template <bool YBF16>
__device__ __forceinline__ void y8_combine(const Y8<YBF16>& f, float s, const f32x4& a0,
                                           const f32x4& a1, uint4 (&out)[2]) {
  if (YBF16) {
    const uint32_t w[4] = {f.v[0].x, f.v[0].y, f.v[0].z, f.v[0].w};
    uint32_t o4[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4& a = (i < 2) ? a0 : a1;
      const int e0 = (2 * i) & 3;
      o4[i] = pack2_bf16(fmaf(s, a[e0], bf16_to_f32(w[i] & 0xffffu)),
                         fmaf(s, a[e0 + 1], bf16_to_f32(w[i] >> 16)));
    }
    out[0] = make_uint4(o4[0], o4[1], o4[2], o4[3]);
  } else {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint4 u = f.v[h];
      const f32x4& a = h ? a1 : a0;
      out[h] = make_uint4(__float_as_uint(fmaf(s, a[0], __uint_as_float(u.x))),
                          __float_as_uint(fmaf(s, a[1], __uint_as_float(u.y))),
                          __float_as_uint(fmaf(s, a[2], __uint_as_float(u.z))),
                          __float_as_uint(fmaf(s, a[3], __uint_as_float(u.w))));
    }
  }
}

// Results leave through LDS.  A store instruction in the matrix-core layout
// covers 64 bytes of each of 16 rows (half cache lines); one that covers whole
// 128-byte lines of 8 rows moves read-modify-write traffic markedly faster.
// So each wave writes its results for 128 bytes of every row (two steps of a
// bf16 Y, one of an f32 Y) into its own LDS area, then stores them with 8
// lanes per row.
template <bool YBF16, bool RANK8, int KSM, int U>
__global__ __launch_bounds__(256, (KSM == 1 || (YBF16 && KSM == 2 && U == 1)) ? 2 : 1) void expand_kernel(FwdArgs p) {
  constexpr int BS = KSM * 32, TS = BS + 8;    // staged ranks per column; LDS stride
  constexpr int BP = 32 * BS / 8;              // 16-byte B pieces per step (rank padded)
  constexpr int BPT = (BP + 255) / 256;        // ... per thread
  constexpr int ES = YBF16 ? 2 : 4;            // bytes per Y element
  constexpr int SP = YBF16 ? 2 : 1;            // steps per 128 bytes of a row
  constexpr int OS = 128 + 16;                 // bytes per row of a wave's output area
  __shared__ __align__(16) uint16_t s_b[2][U][32 * TS];
  __shared__ __align__(16) unsigned char s_o[4][64 * OS];
  const int lane = threadIdx.x & 63, w = wave_id(), tid = threadIdx.x;
  const int og = lane >> 4, mrow = lane & 15, jg = og * 8;
  unsigned char* const so = s_o[w];
  uint4* const sink = g_store_sink + 8 * tid;
  if (p.hdr[HDR_RB_ROWS] == RB_FINE) return;     // the fine kernel's batch
  int first, count;
  entry_range(p, first, count);
  const int nks = shrink_splits(p, count);
  // column chunk of a unit (finer chunks, tried for batches with few row
  // blocks, measured slower: each unit repeats the H prologue)
  const int CW = p.cw > 0 ? p.cw : 1024;
  const int n_ch = (p.d_out + CW - 1) / CW;
  const XcdRange xr = xcd_range(count * n_ch);
  for (int unit = xr.first; unit < xr.end; unit += xr.step) {
    const int e = unit / n_ch, ch = unit - e * n_ch;
    const int c0 = ch * CW, c1 = min(p.d_out, c0 + CW);
    const int nst = (c1 - c0 + 31) / 32;
    const int4 en = load_entry(p.rb, first + e);
    const int a = ck_slot(p.hdr, en.x, p.num_slots), p0 = en.y, rows = en.z;
    const Slot m = load_slot(p.meta, a);
    const int r = m.rank;
    const float s = m.scale;
    const rsrc_t Bw = make_rsrc(m.B, (uint32_t)p.d_out * (uint32_t)r * 2u);

    // rows of the matrix-core layout: tile tt, lane row mrow
    int trow[4];
    bool rv[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
      const int i = 64 * w + 16 * tt + mrow;
      rv[tt] = i < rows;
      trow[tt] = ck_row(p.hdr, ldg(p.perm + p0 + (i < rows ? i : rows - 1)), p.n_rows);
    }
    // rows of the store layout: instruction i, lane row lane / 8 (padding rows
    // store to the sink)
    int srow[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int ri = 64 * w + 8 * i + (lane >> 3);
      srow[i] = ri < rows ? ck_row(p.hdr, ldg(p.perm + p0 + ri), p.n_rows) : -1;
    }

    // H operands (hi / lo) of the wave's rows: the slices' partial sums added
    // in slice order, loaded once per unit (one round trip per plane: every
    // rank step and row tile of a plane requested together).
    float4 h[KSM][4][2];
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks)
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        h[ks][tt][0] = make_float4(0.f, 0.f, 0.f, 0.f);
        h[ks][tt][1] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    if constexpr (RANK8) {
      for (int sl = 0; sl < nks; ++sl) {
        const float* Hs = p.H + (int64_t)sl * p.hp_stride;
        float4 q[KSM][4][2];
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks) {
          const int j = ks * 32 + jg;
          const int jj = j < r ? j : r - 8;
#pragma unroll
          for (int tt = 0; tt < 4; ++tt) {
            const float* hrow = Hs + (int64_t)trow[tt] * p.ldh;
            q[ks][tt][0] = ldg_f4(hrow + jj);
            q[ks][tt][1] = ldg_f4(hrow + jj + 4);
          }
        }
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks)
#pragma unroll
          for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int c = 0; c < 2; ++c) {
              float4& d = h[ks][tt][c];
              const float4 x = q[ks][tt][c];
              d.x += x.x; d.y += x.y; d.z += x.z; d.w += x.w;
            }
      }
    } else {
      // ranks not a multiple of 8: element loads, one rank step at a time
      // (fewer registers in flight)
#pragma unroll
      for (int ks = 0; ks < KSM; ++ks) {
        const int j = ks * 32 + jg;
        for (int sl = 0; sl < nks; ++sl) {
          const float* Hs = p.H + (int64_t)sl * p.hp_stride;
#pragma unroll
          for (int tt = 0; tt < 4; ++tt) {
            const float* hrow = Hs + (int64_t)trow[tt] * p.ldh;
            float e[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) e[i] = ldg(hrow + (j + i < r ? j + i : r - 1));
            float4& d0 = h[ks][tt][0];
            float4& d1 = h[ks][tt][1];
            d0.x += e[0]; d0.y += e[1]; d0.z += e[2]; d0.w += e[3];
            d1.x += e[4]; d1.y += e[5]; d1.z += e[6]; d1.w += e[7];
          }
        }
      }
    }
    bf16x8 hh[KSM][4], hl[KSM][4];
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks) {
      const int j = ks * 32 + jg;
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        float hv[8] = {h[ks][tt][0].x, h[ks][tt][0].y, h[ks][tt][0].z, h[ks][tt][0].w,
                       h[ks][tt][1].x, h[ks][tt][1].y, h[ks][tt][1].z, h[ks][tt][1].w};
#pragma unroll
        for (int i = 0; i < 8; ++i) hv[i] = (rv[tt] && j + i < r) ? hv[i] : 0.0f;
        split_hi_lo(hv, hh[ks][tt], hl[ks][tt]);
      }
    }
    vmem_drained();

    // this thread's B pieces: column col of a step, ranks 8 jq .. 8 jq + 7
    int bcol[BPT], bj[BPT];
#pragma unroll
    for (int h = 0; h < BPT; ++h) {
      const int pc = (tid + 256 * h) & (BP - 1);   // (BP is a power of two)
      bcol[h] = pc / (BS / 8);
      bj[h] = (pc - bcol[h] * (BS / 8)) * 8;
    }

    // bf16 Y, one step per batch: Y comes in through the wave's output area
    // as whole 128-byte lines of 8 rows (the 2-step group of the first step's
    // batch), the way the results leave; else in the matrix-core layout
    constexpr bool YL = YBF16 && U == 1;
    int lrow[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) lrow[i] = srow[i] >= 0 ? srow[i] : trow[0];
    struct Buf {
      uint4 b[U][BPT];
      Y8<YBF16> y[YL ? 1 : U][YL ? 1 : 4];
      uint4 yl[YL ? 8 : 1];
    };
    // group: the batch starts a 128-byte group of columns (YL: it brings the
    // group's Y lines)
    auto load = [&](Buf& q, int st0, bool group) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ob = c0 + 32 * min(st0 + u, nst - 1);
#pragma unroll
        for (int h = 0; h < BPT; ++h) {
          int oc = ob + bcol[h];
          oc = oc < p.d_out ? oc : p.d_out - 1;
          q.b[u][h] = __builtin_bit_cast(uint4, wrow8<RANK8>(Bw, (uint32_t)oc * r, bj[h], r));
        }
      }
      if constexpr (YL) {
        if (group) {
          int o = c0 + 32 * min(st0, nst - 1) + (lane & 7) * 8;
          o = o < p.d_out ? o : p.d_out - 8;
#pragma unroll
          for (int i = 0; i < 8; ++i)
            q.yl[i] = ldg16(reinterpret_cast<const uint16_t*>(p.Y) + (int64_t)lrow[i] * p.ldy + o);
        }
      } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int ob = c0 + 32 * min(st0 + u, nst - 1);
#pragma unroll
          for (int tt = 0; tt < 4; ++tt)
            y8_load<YBF16>(q.y[u][tt], p.Y, p.ldy, trow[tt], ob + 8 * og, p.d_out);
        }
      }
    };
    auto stage = [&](const Buf& q, int buf) {
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int h = 0; h < BPT; ++h)
          *reinterpret_cast<uint4*>(&s_b[buf][u][bcol[h] * TS + bj[h]]) = q.b[u][h];
    };
    // product of step st (batch slot u), added to Y, into the wave's output area
    auto run = [&](const Buf& q, int u, int st, int buf, bool group) {
      if constexpr (YL) {
        if (group) {                   // the group's Y lines into the area
          asm volatile("" ::: "memory");
#pragma unroll
          for (int i = 0; i < 8; ++i)
            *reinterpret_cast<uint4*>(so + (8 * i + (lane >> 3)) * OS + (lane & 7) * 16) = q.yl[i];
          asm volatile("" ::: "memory");
        }
      }
      f32x4 acc[2][4];
#pragma unroll
      for (int qq = 0; qq < 2; ++qq)
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) acc[qq][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KSM; ++ks) {
        const bool jv = ks * 32 + jg < r;
#pragma unroll
        for (int qq = 0; qq < 2; ++qq) {
          const int oc = 8 * (mrow >> 2) + 4 * qq + (mrow & 3);
          const bf16x8 b = sel(jv, as_bf16x8(*reinterpret_cast<const uint4*>(
                                       &s_b[buf][u][oc * TS + ks * 32 + jg])));
#pragma unroll
          for (int tt = 0; tt < 4; ++tt) {
            acc[qq][tt] = mfma_16x16x32(b, hh[ks][tt], acc[qq][tt]);
            acc[qq][tt] = mfma_16x16x32(b, hl[ks][tt], acc[qq][tt]);
          }
        }
      }
      mfma_fence();
      const int cb = ((st % SP) * 32 + 8 * og) * ES;    // byte column in the area
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        uint4 out[2];
        Y8<YBF16> yv;
        if constexpr (YL) yv.v[0] = *reinterpret_cast<const uint4*>(so + (16 * tt + mrow) * OS + cb);
        else yv = q.y[YL ? 0 : u][YL ? 0 : tt];
        y8_combine<YBF16>(yv, s, acc[0][tt], acc[1][tt], out);
        unsigned char* d = so + (16 * tt + mrow) * OS + cb;
        *reinterpret_cast<uint4*>(d) = out[0];
        if (!YBF16) *reinterpret_cast<uint4*>(d + 16) = out[1];
      }
    };
    // the output area's 128 bytes per row, from step st0 on, to Y
    auto flush = [&](int st0) {
      asm volatile("" ::: "memory");   // the area's writes above come first
      const int o = c0 + 32 * st0 + (lane & 7) * (16 / ES);
      const bool ov = o < c1;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint4 v = *reinterpret_cast<const uint4*>(so + (8 * i + (lane >> 3)) * OS + (lane & 7) * 16);
        uint4* dst = (ov && srow[i] >= 0)
                         ? reinterpret_cast<uint4*>(reinterpret_cast<char*>(p.Y) +
                                                    ((int64_t)srow[i] * p.ldy + o) * ES)
                         : sink + i;
        stg16(dst, v);
      }
      asm volatile("" ::: "memory");   // ... and the next writes come after the reads
    };
    // a batch of U steps from st0: products, and a flush after every SP-th step
    auto batch = [&](const Buf& q, int st0, int buf, bool group) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        run(q, u, st0 + u, buf, group && u == 0);
        if ((st0 + u) % SP == SP - 1) flush(st0 + u - (SP - 1));
      }
    };
    // Batches in pairs, double buffered in registers and LDS: the loads of the
    // next batch are in flight while a batch feeds the matrix cores.  Loads are
    // unconditional (past the last step they repeat it) and so are stores;
    // steps past the chunk store to the sink.  One exit, at the end of a pair.
    Buf b0, b1;
    load(b0, 0, true);
    // as many stores (to the sink) as a pair ends with after its last loads,
    // so that the loop is entered with the same sequence of memory operations
    // outstanding as it loops back with, and the compiler's wait counts stay
    // exact
    constexpr int TAIL = 8 * (U >= SP ? U / SP : 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < TAIL; ++i) stg16(sink + (i & 7), make_uint4(0u, 0u, 0u, (uint32_t)i));
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();                 // the previous unit's reads of s_b are done
    // (U = 1 with SP = 2: b0 always holds an even step, which starts a group)
    for (int st = 0; st < nst; st += 2 * U) {
      load(b1, st + U, U >= SP);
      __builtin_amdgcn_sched_barrier(0);
      stage(b0, 0);
      __syncthreads();
      batch(b0, st, 0, true);
      load(b0, st + 2 * U, true);
      __builtin_amdgcn_sched_barrier(0);
      stage(b1, 1);
      __syncthreads();
      batch(b1, st + U, 1, U >= SP);
    }
  }
}

// ---------------------------------------------------------------------------
// Large groups in 64-row blocks.  Batches whose large groups are few or short
// give too few 256-row blocks to fill the chip, and a 256-row block that holds
// a short group spends most of its work on padding rows.  Here the four waves
// of a workgroup share the block's 64 rows: the shrink splits the d-slice's
// k-steps over the waves (partial sums meet in LDS in a fixed order), the
// expand splits the unit's columns over the waves (H formed once per unit in
// LDS, each wave loading the B rows of its own columns, no barrier in the
// column loop).
// ---------------------------------------------------------------------------
// WT (input gradient): the weight is B_a as stored, [K][r] with K = p.d_in,
// gathered (eight 2-byte loads per lane and k-step, packed when multiplied).
template <int NT, bool WT>
__global__ __launch_bounds__(256) void shrink_fine_kernel(FwdArgs p) {
  constexpr int N = 4 * NT, CH = N < 16 ? N : 16;
  __shared__ f32x4 s_red[2 * CH * 64];
  const int lane = threadIdx.x & 63, w = wave_id();
  const int mrow = lane & 15, kg = (lane >> 4) * 8;
  if (!p.force_fine && p.hdr[HDR_RB_ROWS] != RB_FINE) return;   // the coarse kernel's batch
  int first, count;
  entry_range(p, first, count);
  const int nks = shrink_splits(p, count);
  const XcdRange xr = xcd_range(count * nks);
  for (int unit = xr.first; unit < xr.end; unit += xr.step) {
    const int e = unit / nks, ks = unit - e * nks;
    const int4 en = load_entry(p.rb, first + e);
    const int a = ck_slot(p.hdr, en.x, p.num_slots), p0 = en.y, rows = en.z;
    const Slot m = load_slot(p.meta, a);
    const int r = m.rank;
    const rsrc_t A = make_rsrc(WT ? m.B : m.A, (uint32_t)r * (uint32_t)p.d_in * 2u);
    int kb, ke;
    kslice(p.d_in, nks, ks, kb, ke);
    const int kend = max(ke, 8);
    const int nst = max(1, (ke - kb + 31) / 32);
    const int rounds = (nst + 3) / 4;            // k-steps per wave: w, w + 4, ...

    const uint16_t* xrow[4];
    int orow[4][4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      const int i = 16 * mt + mrow;
      xrow[mt] = p.X + (int64_t)ck_row(p.hdr, ldg(p.perm + p0 + (i < rows ? i : rows - 1)), p.n_rows) * p.ldx;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int io = 16 * mt + (lane >> 4) * 4 + v;
        orow[mt][v] = ck_row(p.hdr, ldg(p.perm + p0 + (io < rows ? io : rows - 1)), p.n_rows);
      }
    }
    uint32_t arow[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int j = nt * 16 + mrow;
      arow[nt] = WT ? (uint32_t)(j < r ? j : r - 1) : (uint32_t)(j < r ? j : r - 1) * (uint32_t)p.d_in;
    }
    f32x4 acc[N];
#pragma unroll
    for (int i = 0; i < N; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    struct Buf {
      bf16x8 x[4];
      bf16x8 a[WT ? 1 : NT];
      uint32_t e[WT ? NT : 1][8];
      bool kv;
    };
    auto load = [&](Buf& b, int i) {
      const int k = kb + 32 * (w + 4 * i) + kg;
      b.kv = k < ke;
      const int kk = k < kend ? k : kend - 8;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        if (!WT) {
          b.a[WT ? 0 : nt] = as_bf16x8(bload16(A, (arow[nt] + (uint32_t)kk) * 2u));
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q)
            b.e[WT ? nt : 0][q] = bload_u16(A, ((uint32_t)(kk + q) * (uint32_t)r + arow[nt]) * 2u);
        }
      }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) b.x[mt] = as_bf16x8(ldg16(xrow[mt] + kk));
    };
    auto compute = [&](const Buf& b) {
      bf16x8 av[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) av[nt] = WT ? pack_bf16x8(b.e[WT ? nt : 0]) : b.a[WT ? 0 : nt];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const bf16x8 xo = sel(b.kv, b.x[mt]);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt * NT + nt] = mfma_16x16x32(xo, av[nt], acc[mt * NT + nt]);
      }
    };
    // rounds double buffered in registers; one exit, at the end of a pair
    // (rounds past the end read clamped addresses and add zeros)
    Buf b0, b1;
    load(b0, 0);
    for (int i = 0; i < rounds; i += 2) {
      load(b1, i + 1);
      __builtin_amdgcn_sched_barrier(0);
      compute(b0);
      load(b0, i + 2);
      __builtin_amdgcn_sched_barrier(0);
      compute(b1);
      // wait states on the back edge between the last product and the loop
      // head, where the compiler may read an accumulator register
      __builtin_amdgcn_sched_barrier(0);
      asm volatile("s_nop 7");
      __builtin_amdgcn_sched_barrier(0);
    }
    mfma_fence();
    vmem_drained();
    reduce_waves<N, CH>(acc, s_red);
    if (w == 0) {
      float* H = p.H + (int64_t)ks * p.hp_stride;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int i = 16 * mt + (lane >> 4) * 4 + v;
          if (i >= rows) continue;
          float* hrow = H + (int64_t)orow[mt][v] * p.ldh;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const int j = nt * 16 + mrow;
            if (j < r) stg(hrow + j, acc[mt * NT + nt][v]);
          }
        }
    }
  }
}

// WT (input gradient): the weight is A_a as stored, [r][p.d_out], gathered
// (eight 2-byte loads per operand, packed when multiplied).
template <bool YBF16, bool RANK8, int KSM, int U, bool WT>
__global__ __launch_bounds__(256, KSM == 1 ? 2 : 1) void expand_fine_kernel(FwdArgs p) {
  constexpr int HS = KSM * 32, HT = HS + 4;    // H columns (rank padded); LDS stride
  constexpr int ES = YBF16 ? 2 : 4;            // bytes per Y element
  constexpr int SP = YBF16 ? 2 : 1;            // steps per 128 bytes of a row
  constexpr int OS = 128 + 16;                 // bytes per row of a wave's output area
  constexpr int HQ = 2 * KSM;                  // float4 of a row per thread and plane
  __shared__ __align__(16) float s_h[64 * HT];
  __shared__ __align__(16) unsigned char s_o[4][64 * OS];
  const int lane = threadIdx.x & 63, w = wave_id(), tid = threadIdx.x;
  const int og = lane >> 4, mrow = lane & 15, jg = og * 8;
  unsigned char* const so = s_o[w];
  uint4* const sink = g_store_sink + 8 * tid;
  if (!p.force_fine && p.hdr[HDR_RB_ROWS] != RB_FINE) return;   // the coarse kernel's batch
  int first, count;
  entry_range(p, first, count);
  const int nks = shrink_splits(p, count);
  // column chunk: the input gradient's (force_fine) is p.cw; a forward
  // batch's comes from the block count, so that the (block, chunk) units about
  // fill the workgroups the chip holds at once (two per CU up to rank 32, else
  // one), in whole 128-byte groups, four waves' worth at a time
  const int ngr_all = (p.d_out + 32 * SP - 1) / (32 * SP);
  const int n_want = max(1, min((KSM == 1 ? 512 : 256) / max(count, 1), ngr_all / 4));
  const int CW = p.force_fine ? (p.cw > 0 ? p.cw : 1024)
                              : (ngr_all + 4 * n_want - 1) / (4 * n_want) * 4 * (32 * SP);
  const int QW = CW / 4;                       // columns per wave
  const int n_ch = (p.d_out + CW - 1) / CW;
  const XcdRange xr = xcd_range(count * n_ch);
  for (int unit = xr.first; unit < xr.end; unit += xr.step) {
    const int e = unit / n_ch, ch = unit - e * n_ch;
    const int c0 = ch * CW, c1 = min(p.d_out, c0 + CW);
    const int4 en = load_entry(p.rb, first + e);
    const int a = ck_slot(p.hdr, en.x, p.num_slots), p0 = en.y, rows = en.z;
    const Slot m = load_slot(p.meta, a);
    const int r = m.rank;
    const float s = m.scale;
    const rsrc_t Bw = make_rsrc(WT ? m.A : m.B, (uint32_t)p.d_out * (uint32_t)r * 2u);
    // this wave's columns
    const int cw0 = min(c0 + w * QW, c1), cw1 = min(c1, cw0 + QW);
    const int nst = (cw1 - cw0 + 31) / 32;

    int trow[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
      const int i = 16 * tt + mrow;
      trow[tt] = ck_row(p.hdr, ldg(p.perm + p0 + (i < rows ? i : rows - 1)), p.n_rows);
    }
    int srow[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int ri = 8 * i + (lane >> 3);
      srow[i] = ri < rows ? ck_row(p.hdr, ldg(p.perm + p0 + ri), p.n_rows) : -1;
    }

    // H of the block's rows: thread -> row tid / 4, float4 quarter tid % 4 of
    // the rank columns; the slices' planes requested in one round trip and
    // added in slice order (rows past the block and ranks past r are zero)
    {
      const int hr = tid >> 2, hq = tid & 3;
      const int hrow = ck_row(p.hdr, ldg(p.perm + p0 + (hr < rows ? hr : rows - 1)), p.n_rows);
      float4 q[SHRINK_KS_MAX][HQ];
#pragma unroll
      for (int sl = 0; sl < SHRINK_KS_MAX; ++sl) {
        const float* Hs = p.H + (int64_t)min(sl, nks - 1) * p.hp_stride + (int64_t)hrow * p.ldh;
#pragma unroll
        for (int c = 0; c < HQ; ++c) {
          const int j = 4 * (hq + 4 * c);
          if (RANK8) {
            q[sl][c] = ldg_f4(Hs + (j < r ? j : r - 4));
          } else {
            q[sl][c] = make_float4(ldg(Hs + min(j, r - 1)), ldg(Hs + min(j + 1, r - 1)),
                                   ldg(Hs + min(j + 2, r - 1)), ldg(Hs + min(j + 3, r - 1)));
          }
        }
      }
      __syncthreads();                 // the previous unit's reads of s_h are done
#pragma unroll
      for (int c = 0; c < HQ; ++c) {
        const int j = 4 * (hq + 4 * c);
        float4 h = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int sl = 0; sl < SHRINK_KS_MAX; ++sl) {
          if (sl >= nks) break;
          h.x += q[sl][c].x; h.y += q[sl][c].y; h.z += q[sl][c].z; h.w += q[sl][c].w;
        }
        const bool ok = hr < rows;
        h.x = (ok && j < r) ? h.x : 0.f;
        h.y = (ok && j + 1 < r) ? h.y : 0.f;
        h.z = (ok && j + 2 < r) ? h.z : 0.f;
        h.w = (ok && j + 3 < r) ? h.w : 0.f;
        *reinterpret_cast<float4*>(&s_h[hr * HT + j]) = h;
      }
      __syncthreads();
    }
    bf16x8 hh[KSM][4], hl[KSM][4];
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks)
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        const float* hp = &s_h[(16 * tt + mrow) * HT + ks * 32 + jg];
        const float4 x0 = *reinterpret_cast<const float4*>(hp);
        const float4 x1 = *reinterpret_cast<const float4*>(hp + 4);
        const float hv[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
        split_hi_lo(hv, hh[ks][tt], hl[ks][tt]);
      }
    vmem_drained();

    struct Buf {
      bf16x8 b[WT ? 1 : U][KSM][2];
      uint32_t e[WT ? U : 1][KSM][2][8];     // gathered weights (WT)
      Y8<YBF16> y[U][4];
    };
    auto load = [&](Buf& q, int st0) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ob = cw0 + 32 * max(0, min(st0 + u, nst - 1));
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks)
#pragma unroll
          for (int qq = 0; qq < 2; ++qq) {
            int oc = ob + 8 * (mrow >> 2) + 4 * qq + (mrow & 3);
            oc = oc < p.d_out ? oc : p.d_out - 1;
            if (!WT) {
              q.b[WT ? 0 : u][ks][qq] = wrow8<RANK8>(Bw, (uint32_t)oc * r, ks * 32 + jg, r);
            } else {
#pragma unroll
              for (int i = 0; i < 8; ++i) {
                const int j = ks * 32 + jg + i;
                q.e[WT ? u : 0][ks][qq][i] =
                    bload_u16(Bw, ((uint32_t)(j < r ? j : r - 1) * (uint32_t)p.d_out + (uint32_t)oc) * 2u);
              }
            }
          }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ob = cw0 + 32 * max(0, min(st0 + u, nst - 1));
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
          y8_load<YBF16>(q.y[u][tt], p.Y, p.ldy, trow[tt], ob + 8 * og, p.d_out);
      }
    };
    auto run = [&](const Buf& q, int u, int st) {
      f32x4 acc[2][4];
#pragma unroll
      for (int qq = 0; qq < 2; ++qq)
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) acc[qq][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KSM; ++ks) {
        const bool jv = ks * 32 + jg < r;
#pragma unroll
        for (int qq = 0; qq < 2; ++qq) {
          bf16x8 b;
          if (!WT) {
            b = q.b[WT ? 0 : u][ks][qq];
          } else {
            uint32_t ev[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) ev[i] = ks * 32 + jg + i < r ? q.e[WT ? u : 0][ks][qq][i] : 0u;
            b = pack_bf16x8(ev);
          }
          b = sel(jv, b);
#pragma unroll
          for (int tt = 0; tt < 4; ++tt) {
            acc[qq][tt] = mfma_16x16x32(b, hh[ks][tt], acc[qq][tt]);
            acc[qq][tt] = mfma_16x16x32(b, hl[ks][tt], acc[qq][tt]);
          }
        }
      }
      mfma_fence();
      const int cb = ((st % SP) * 32 + 8 * og) * ES;
#pragma unroll
      for (int tt = 0; tt < 4; ++tt) {
        uint4 out[2];
        y8_combine<YBF16>(q.y[u][tt], s, acc[0][tt], acc[1][tt], out);
        unsigned char* d = so + (16 * tt + mrow) * OS + cb;
        *reinterpret_cast<uint4*>(d) = out[0];
        if (!YBF16) *reinterpret_cast<uint4*>(d + 16) = out[1];
      }
    };
    auto flush = [&](int st0) {
      asm volatile("" ::: "memory");
      const int o = cw0 + 32 * st0 + (lane & 7) * (16 / ES);
      const bool ov = o < cw1;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint4 v = *reinterpret_cast<const uint4*>(so + (8 * i + (lane >> 3)) * OS + (lane & 7) * 16);
        uint4* dst = (ov && srow[i] >= 0)
                         ? reinterpret_cast<uint4*>(reinterpret_cast<char*>(p.Y) +
                                                    ((int64_t)srow[i] * p.ldy + o) * ES)
                         : sink + i;
        stg16(dst, v);
      }
      asm volatile("" ::: "memory");
    };
    auto batch = [&](const Buf& q, int st0) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        run(q, u, st0 + u);
        if ((st0 + u) % SP == SP - 1) flush(st0 + u - (SP - 1));
      }
    };
    Buf b0, b1;
    load(b0, 0);
    constexpr int TAIL = 8 * (U >= SP ? U / SP : 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < TAIL; ++i) stg16(sink + (i & 7), make_uint4(0u, 0u, 0u, (uint32_t)i));
    __builtin_amdgcn_sched_barrier(0);
    for (int st = 0; st < nst; st += 2 * U) {
      load(b1, st + U);
      __builtin_amdgcn_sched_barrier(0);
      batch(b0, st);
      load(b0, st + 2 * U);
      __builtin_amdgcn_sched_barrier(0);
      batch(b1, st + U);
    }
  }
}

// ---------------------------------------------------------------------------
// fused small-group kernel: one small-group record (<= 16 rows of one adapter)
// per workgroup, and a chunk of at most 64 * FW * FSL output columns.
//
// The record (128 bytes, written by the plan) holds the weight pointers, rank,
// scale and row ids, so one round trip yields everything; the chunk's B (small
// ranks) and Y are then requested before the shrink streams X and A, whose k-
// steps are spread over all FW waves.  The waves' partial H are summed in a
// fixed order through LDS; H (hi / lo) feeds the expand of each wave's column
// slices.  Sibling workgroups (same record, other column chunks) share
// blockIdx % 8, so they run on one XCD and read A from its L2.
// ---------------------------------------------------------------------------
constexpr int FW = 8;     // waves per fused workgroup
constexpr int FSL = 2;    // 64-column slices per wave

template <bool YBF16, int NT, bool RANK8>
__global__ __launch_bounds__(FW * 64) void fused_small_kernel(FwdArgs p) {
  // k-steps per load batch (two batches in flight)
  constexpr int U = NT == 1 ? 8 : (NT == 2 ? 4 : (NT == 4 ? 2 : 1));
  constexpr int KSM = (NT * 16 + 31) / 32;
  constexpr bool B_AHEAD = KSM == 1;          // B of every slice requested up front
  __shared__ f32x4 s_red[FW * NT * 64];
  __shared__ float s_h[16][NT * 16 + 4];
  const int lane = threadIdx.x & 63, w = wave_id();
  const int og = lane >> 4, mrow = lane & 15;
  const int P = p.n_chunks;
  // siblings (same record, different column chunk) share blockIdx % 8, i.e. one XCD
  const int slot = (int)(blockIdx.x >> 3);
  const int e = 8 * (slot / P) + (int)(blockIdx.x & 7);
  const int pc = slot % P;

  // ---- the record and the entry count, in one round trip (the record index is
  // clamped to the array; records at or past the count are never used)
  const int er = min(e, p.n_rec - 1);
  const int4* rec = reinterpret_cast<const int4*>(p.srec + er);
  const int4 h0 = rec[0], h1 = rec[1];
  const int trow_rec = ldg(&p.srec[er].row[mrow]);
  const int count = p.hdr[p.count_word];
  if (e >= count) return;
  const int trow = ck_row(p.hdr, trow_rec, p.n_rows);
  const void* Ap = uni_ptr(reinterpret_cast<const void*>(
      (uint64_t)(uint32_t)h0.x | ((uint64_t)(uint32_t)h0.y << 32)));
  const void* Bp = uni_ptr(reinterpret_cast<const void*>(
      (uint64_t)(uint32_t)h0.z | ((uint64_t)(uint32_t)h0.w << 32)));
  const int rows = uni(h1.x), r = uni(h1.y);
  const float s = __int_as_float(uni(h1.z));
  const rsrc_t A = make_rsrc(Ap, (uint32_t)r * (uint32_t)p.d_in * 2u);
  const rsrc_t Bw = make_rsrc(Bp, (uint32_t)p.d_out * (uint32_t)r * 2u);
  const bool rv = mrow < rows;
  const int c0 = pc * p.chunk;
  const int c1 = min(p.d_out, c0 + p.chunk);

  // ---- B (small ranks) and Y of this wave's column slices, requested first
  bf16x8 bo_ahead[B_AHEAD ? FSL : 1][4];
  if (B_AHEAD) {
#pragma unroll
    for (int sl = 0; sl < FSL; ++sl) {
      const int o_w = c0 + 64 * (w + FW * sl);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int o = out_col(o_w, q, mrow);
        bo_ahead[B_AHEAD ? sl : 0][q] =
            wrow8<RANK8>(Bw, (uint32_t)(o < c1 ? o : c1 - 1) * r, og * 8, r);
      }
    }
  }
  YFrag<YBF16> yf[FSL];
#pragma unroll
  for (int sl = 0; sl < FSL; ++sl)
    y_load<YBF16>(yf[sl], p.Y, p.ldy, trow, c0 + 64 * (w + FW * sl), og, c1);

  // ---- shrink: H[16 x r] = X[rows] A^T, the k-steps spread over the waves
  f32x4 acc[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  {
    const uint16_t* xrow[1] = {p.X + (int64_t)trow * p.ldx};
    uint32_t arow[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int j = nt * 16 + mrow;
      arow[nt] = (uint32_t)(j < r ? j : r - 1) * (uint32_t)p.d_in;
    }
    shrink_steps<1, NT, U>(acc, xrow, A, arow, w * 32, 32 * FW, p.d_in);
  }
  vmem_drained();           // B and Y were requested before the shrink loads

  // ---- sum the waves' partial H in a fixed order (wave 0, 1, ..., FW - 1)
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) s_red[(w * NT + nt) * 64 + lane] = acc[nt];
  __syncthreads();
  {
    const float* red = reinterpret_cast<const float*>(s_red);
    for (int i = threadIdx.x; i < NT * 256; i += FW * 64) {
      const int nt = i >> 8, l = (i >> 2) & 63, v = i & 3;
      float sum = red[((0 * NT + nt) * 64 + l) * 4 + v];
#pragma unroll
      for (int ww = 1; ww < FW; ++ww) sum += red[((ww * NT + nt) * 64 + l) * 4 + v];
      s_h[(l >> 4) * 4 + v][nt * 16 + (l & 15)] = sum;
    }
  }
  __syncthreads();

  // ---- H operand (hi / lo) for every 32-wide rank step
  bf16x8 hh[KSM], hl[KSM];
#pragma unroll
  for (int ks = 0; ks < KSM; ++ks) {
    float h[8];
    const int j = ks * 32 + og * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = (j + i < r) ? s_h[mrow][j + i] : 0.0f;
    split_hi_lo(h, hh[ks], hl[ks]);
  }

  // ---- expand over this wave's column slices
#pragma unroll
  for (int sl = 0; sl < FSL; ++sl) {
    const int o_w = c0 + 64 * (w + FW * sl);
    if (o_w >= c1) continue;
    f32x4 acc2[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc2[q] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        bf16x8 bo;
        if (B_AHEAD) {
          bo = bo_ahead[B_AHEAD ? sl : 0][q];
        } else {
          const int o = out_col(o_w, q, mrow);
          bo = wrow8<RANK8>(Bw, (uint32_t)(o < c1 ? o : c1 - 1) * r, ks * 32 + og * 8, r);
        }
        bo = sel(ks * 32 + og * 8 < r, bo);
        acc2[q] = mfma_16x16x32(bo, hh[ks], acc2[q]);
        acc2[q] = mfma_16x16x32(bo, hl[ks], acc2[q]);
      }
    }
    mfma_fence();
    if (rv) y_store<YBF16>(yf[sl], p.Y, p.ldy, trow, o_w, og, c1, s, acc2);
  }
}

// ---------------------------------------------------------------------------
// Split small-group path, for small groups whose weights are large: the fused
// kernel's sibling workgroups each re-read the whole of A, which then
// dominates.  Here the shrink runs per (record, d-slice) and reads A once,
// writing partial H planes to the workspace; the expand runs per (record,
// column chunk), sums the planes in slice order and applies B as the fused
// kernel does.
//
// Partial planes: plane sl at p.H + sl * p.hp_stride, record e's 16 x p.ldh
// floats at e * 16 * p.ldh (rows and rank columns past the record's are
// don't-care values, never used).
// ---------------------------------------------------------------------------
constexpr int SPLIT_SMAX = 8;     // most d-slices of the split shrink

template <int NT, int U>
__global__ __launch_bounds__(256) void small_shrink_kernel(FwdArgs p) {
  __shared__ f32x4 s_red[2 * NT * 64];
  const int lane = threadIdx.x & 63, w = wave_id();
  const int mrow = lane & 15;
  const int S = p.ks_max;
  const int e = (int)blockIdx.x / S, sl = (int)blockIdx.x - e * S;
  const int er = min(e, p.n_rec - 1);
  const int4 h0 = *reinterpret_cast<const int4*>(p.srec + er);
  const int4 h1 = *(reinterpret_cast<const int4*>(p.srec + er) + 1);
  const int trow_rec = ldg(&p.srec[er].row[mrow]);
  const int count = p.hdr[p.count_word];
  if (e >= count) return;
  const int trow = ck_row(p.hdr, trow_rec, p.n_rows);
  const void* Ap = uni_ptr(reinterpret_cast<const void*>(
      (uint64_t)(uint32_t)h0.x | ((uint64_t)(uint32_t)h0.y << 32)));
  const int r = uni(h1.y);
  const rsrc_t A = make_rsrc(Ap, (uint32_t)r * (uint32_t)p.d_in * 2u);
  int kb, ke;
  kslice(p.d_in, S, sl, kb, ke);

  f32x4 acc[NT];
#pragma unroll
  for (int i = 0; i < NT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  const uint16_t* xrow[1] = {p.X + (int64_t)trow * p.ldx};
  uint32_t arow[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int j = nt * 16 + mrow;
    arow[nt] = (uint32_t)(j < r ? j : r - 1) * (uint32_t)p.d_in;
  }
  shrink_steps<1, NT, U>(acc, xrow, A, arow, kb + w * 32, 128, ke);
  reduce_waves<NT, NT>(acc, s_red);
  if (w == 0) {
    float* Hp = p.H + (int64_t)sl * p.hp_stride + (int64_t)e * 16 * p.ldh;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int v = 0; v < 4; ++v) stg(Hp + ((lane >> 4) * 4 + v) * p.ldh + nt * 16 + mrow, acc[nt][v]);
  }
}

template <bool YBF16, int NT, bool RANK8>
__global__ __launch_bounds__(FW * 64) void small_expand_kernel(FwdArgs p) {
  constexpr int KSM = (NT * 16 + 31) / 32;
  constexpr int LDH = NT * 16;                // row stride of the partial planes
  constexpr bool B_AHEAD = KSM <= 2;          // B of every slice requested up front
  __shared__ __align__(16) float s_p[SPLIT_SMAX * 16 * LDH];
  const int lane = threadIdx.x & 63, w = wave_id();
  const int og = lane >> 4, mrow = lane & 15;
  const int P = p.n_chunks, S = p.ks_max;
  // siblings (same record, different column chunk) share blockIdx % 8, i.e. one XCD
  const int slot = (int)(blockIdx.x >> 3);
  const int e = 8 * (slot / P) + (int)(blockIdx.x & 7);
  const int pc = slot % P;
  const int er = min(e, p.n_rec - 1);
  const int4 h0 = *reinterpret_cast<const int4*>(p.srec + er);
  const int4 h1 = *(reinterpret_cast<const int4*>(p.srec + er) + 1);
  const int trow_rec = ldg(&p.srec[er].row[mrow]);
  const int count = p.hdr[p.count_word];
  // the record's partial planes depend on e alone: requested in the same
  // round trip as the record (clamped, unconditional; stored to LDS below)
  constexpr int PQ = (SPLIT_SMAX * 16 * LDH / 4 + FW * 64 - 1) / (FW * 64);
  const int n4 = S * 16 * LDH / 4;
  float4 pv[PQ];
#pragma unroll
  for (int u = 0; u < PQ; ++u) {
    int i = (int)threadIdx.x + u * FW * 64;
    i = i < n4 ? i : n4 - 1;
    const int pl = i / (16 * LDH / 4), q = i - pl * (16 * LDH / 4);
    pv[u] = ldg_f4(p.H + (int64_t)pl * p.hp_stride + (int64_t)er * 16 * LDH + 4 * q);
  }
  if (e >= count) return;
  const int trow = ck_row(p.hdr, trow_rec, p.n_rows);
  const void* Bp = uni_ptr(reinterpret_cast<const void*>(
      (uint64_t)(uint32_t)h0.z | ((uint64_t)(uint32_t)h0.w << 32)));
  const int rows = uni(h1.x), r = uni(h1.y);
  const float s = __int_as_float(uni(h1.z));
  const rsrc_t Bw = make_rsrc(Bp, (uint32_t)p.d_out * (uint32_t)r * 2u);
  const bool rv = mrow < rows;
  const int c0 = pc * p.chunk;
  const int c1 = min(p.d_out, c0 + p.chunk);

  // ---- the partial planes into LDS
#pragma unroll
  for (int u = 0; u < PQ; ++u) {
    const int i = (int)threadIdx.x + u * FW * 64;
    if (i < n4) reinterpret_cast<float4*>(s_p)[i] = pv[u];
  }
  // ---- B (ranks up to 64) and Y of this wave's column slices
  bf16x8 bo_ahead[B_AHEAD ? FSL : 1][B_AHEAD ? KSM : 1][4];
  if (B_AHEAD) {
#pragma unroll
    for (int sl = 0; sl < FSL; ++sl) {
      const int o_w = c0 + 64 * (w + FW * sl);
#pragma unroll
      for (int ks = 0; ks < KSM; ++ks)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int o = out_col(o_w, q, mrow);
          bo_ahead[B_AHEAD ? sl : 0][B_AHEAD ? ks : 0][q] =
              wrow8<RANK8>(Bw, (uint32_t)(o < c1 ? o : c1 - 1) * r, ks * 32 + og * 8, r);
        }
    }
  }
  YFrag<YBF16> yf[FSL];
#pragma unroll
  for (int sl = 0; sl < FSL; ++sl)
    y_load<YBF16>(yf[sl], p.Y, p.ldy, trow, c0 + 64 * (w + FW * sl), og, c1);
  __syncthreads();

  // ---- H = sum of the planes in slice order, as hi / lo operands
  bf16x8 hh[KSM], hl[KSM];
#pragma unroll
  for (int ks = 0; ks < KSM; ++ks) {
    float h[8];
    const int j = ks * 32 + og * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = 0.0f;
    if (j < LDH) {
      for (int pl = 0; pl < S; ++pl) {
        const float* row = s_p + (pl * 16 + mrow) * LDH + j;
#pragma unroll
        for (int i = 0; i < 8; ++i) h[i] += row[i];
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = (rv && j + i < r) ? h[i] : 0.0f;
    split_hi_lo(h, hh[ks], hl[ks]);
  }

  // ---- expand over this wave's column slices
#pragma unroll
  for (int sl = 0; sl < FSL; ++sl) {
    const int o_w = c0 + 64 * (w + FW * sl);
    f32x4 acc2[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) acc2[q] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        bf16x8 bo;
        if (B_AHEAD) {
          bo = bo_ahead[B_AHEAD ? sl : 0][B_AHEAD ? ks : 0][q];
        } else {
          const int o = out_col(o_w, q, mrow);
          bo = wrow8<RANK8>(Bw, (uint32_t)(o < c1 ? o : c1 - 1) * r, ks * 32 + og * 8, r);
        }
        bo = sel(ks * 32 + og * 8 < r, bo);
        acc2[q] = mfma_16x16x32(bo, hh[ks], acc2[q]);
        acc2[q] = mfma_16x16x32(bo, hl[ks], acc2[q]);
      }
    }
    mfma_fence();
    if (rv && o_w < c1) y_store<YBF16>(yf[sl], p.Y, p.ldy, trow, o_w, og, c1, s, acc2);
  }
}

// ---------------------------------------------------------------------------
// Plan-free small batches (decode).  Each workgroup finds the rows of its own
// slot a, T_a = {t : ids[t] = a} (Section 3.4's grouping of rows by adapter),
// by scanning the id array, so no plan is built and nothing else runs first.
// Shrink unit = (slot, d-slice): the slot's rows in 16-row tiles times A's
// slice, written to partial planes Hp[slice][t][0, LDH).  Expand unit = (slot,
// column chunk): H = the planes summed in slice order, Y[t] += s H B^T.
// Ids outside [0, S) and ids of empty slots match no workgroup: those rows are
// left as they are, as with a plan.
// ---------------------------------------------------------------------------
// Rows t < n with ids[t] == a, ascending, into s_rows; the count (the same in
// every thread).  ids_request issues the loads of the ids (n <= IDS_MAX_ROWS,
// all at once), ids_rows_of compacts them.
template <int NTHR>
struct IdsRegs {
  int v[IDS_MAX_ROWS / NTHR];
};
template <int NTHR>
__device__ __forceinline__ void ids_request(const int32_t* ids, int n, IdsRegs<NTHR>& q) {
#pragma unroll
  for (int c = 0; c < IDS_MAX_ROWS / NTHR; ++c) {
    const int i = c * NTHR + (int)threadIdx.x;
    q.v[c] = i < n ? ldg(ids + i) : -1;
  }
}
template <int NTHR>
__device__ __forceinline__ int ids_rows_of(const IdsRegs<NTHR>& q, int n, int a, int* s_rows, int* s_wc) {
  constexpr int NW = NTHR / 64, PER = IDS_MAX_ROWS / NTHR;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int base = 0;
#pragma unroll
  for (int c = 0; c < PER; ++c) {
    if (c * NTHR >= n) break;
    const bool f = q.v[c] == a;
    const uint64_t msk = __ballot(f);
    const int pre = __popcll(msk & ((1ull << lane) - 1ull));
    if (lane == 0) s_wc[w] = __popcll(msk);
    __syncthreads();
    int off = base, tot = 0;
#pragma unroll
    for (int qq = 0; qq < NW; ++qq) {
      const int cq = s_wc[qq];
      off += qq < w ? cq : 0;
      tot += cq;
    }
    if (f) s_rows[off + pre] = c * NTHR + tid;
    base += tot;
    __syncthreads();
  }
  return base;
}

template <int NT, int U>
__global__ __launch_bounds__(256) void ids_shrink_kernel(FwdArgs p) {
  __shared__ f32x4 s_red[2 * NT * 64];
  __shared__ int s_rows[IDS_MAX_ROWS];
  __shared__ int s_wc[4];
  const int lane = threadIdx.x & 63, w = wave_id();
  const int mrow = lane & 15;
  const int S = p.ks_max;
  const int a = (int)blockIdx.x / S, sl = (int)blockIdx.x - a * S;
  if (a >= p.num_slots) return;
  // the slot record and the ids are requested together (neither waits for
  // the other)
  const Slot m = load_slot(p.meta, a);
  IdsRegs<256> iq;
  ids_request<256>(p.ids, p.n_ids, iq);
  const int r = m.rank;
  if (r <= 0) return;
  const int cnt = ids_rows_of<256>(iq, p.n_ids, a, s_rows, s_wc);
  if (cnt == 0) return;
  const rsrc_t A = make_rsrc(m.A, (uint32_t)r * (uint32_t)p.d_in * 2u);
  int kb, ke;
  kslice(p.d_in, S, sl, kb, ke);
  uint32_t arow[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int j = nt * 16 + mrow;
    arow[nt] = (uint32_t)(j < r ? j : r - 1) * (uint32_t)p.d_in;
  }
  float* Hp = p.H + (int64_t)sl * p.hp_stride;
  for (int t0 = 0; t0 < cnt; t0 += 16) {
    const int i = t0 + mrow;
    const uint16_t* xrow[1] = {p.X + (int64_t)s_rows[i < cnt ? i : cnt - 1] * p.ldx};
    f32x4 acc[NT];
#pragma unroll
    for (int q = 0; q < NT; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
    shrink_steps<1, NT, U>(acc, xrow, A, arow, kb + w * 32, 128, ke);
    reduce_waves<NT, NT>(acc, s_red);
    if (w == 0) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int ii = t0 + (lane >> 4) * 4 + v;
        if (ii >= cnt) continue;
        float* hrow = Hp + (int64_t)s_rows[ii] * p.ldh;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) stg(hrow + nt * 16 + mrow, acc[nt][v]);
      }
    }
  }
}

template <bool YBF16, int NT, bool RANK8>
__global__ __launch_bounds__(FW * 64) void ids_expand_kernel(FwdArgs p) {
  constexpr int KSM = (NT * 16 + 31) / 32;
  constexpr int LDH = NT * 16;                // row stride of the partial planes
  constexpr bool B_AHEAD = KSM <= 2;          // B of every slice requested up front
  __shared__ int s_rows[IDS_MAX_ROWS];
  __shared__ int s_wc[FW];
  const int lane = threadIdx.x & 63, w = wave_id();
  const int og = lane >> 4, mrow = lane & 15;
  const int P = p.n_chunks, S = p.ks_max;
  // siblings (same slot, different column chunk) share blockIdx % 8, i.e. one XCD
  const int slot = (int)(blockIdx.x >> 3);
  const int a = 8 * (slot / P) + (int)(blockIdx.x & 7);
  const int pc = slot % P;
  if (a >= p.num_slots) return;
  // the slot record and the ids are requested together; B (which needs only
  // the record) before the ids are compacted
  const Slot m = load_slot(p.meta, a);
  IdsRegs<FW * 64> iq;
  ids_request<FW * 64>(p.ids, p.n_ids, iq);
  const int r = m.rank;
  if (r <= 0) return;
  const float s = m.scale;
  const rsrc_t Bw = make_rsrc(m.B, (uint32_t)p.d_out * (uint32_t)r * 2u);
  const int c0 = pc * p.chunk;
  const int c1 = min(p.d_out, c0 + p.chunk);
  // B of this wave's column slices does not depend on the rows: requested
  // before the id scan
  bf16x8 bo_ahead[B_AHEAD ? FSL : 1][B_AHEAD ? KSM : 1][4];
  if (B_AHEAD) {
#pragma unroll
    for (int sl = 0; sl < FSL; ++sl) {
      const int o_w = c0 + 64 * (w + FW * sl);
#pragma unroll
      for (int ks = 0; ks < KSM; ++ks)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int o = out_col(o_w, q, mrow);
          bo_ahead[B_AHEAD ? sl : 0][B_AHEAD ? ks : 0][q] =
              wrow8<RANK8>(Bw, (uint32_t)(o < c1 ? o : c1 - 1) * r, ks * 32 + og * 8, r);
        }
    }
  }
  const int cnt = ids_rows_of<FW * 64>(iq, p.n_ids, a, s_rows, s_wc);
  for (int t0 = 0; t0 < cnt; t0 += 16) {
    const int i = t0 + mrow;
    const bool rv = i < cnt;
    const int trow = s_rows[rv ? i : cnt - 1];
    YFrag<YBF16> yf[FSL];
#pragma unroll
    for (int sl = 0; sl < FSL; ++sl)
      y_load<YBF16>(yf[sl], p.Y, p.ldy, trow, c0 + 64 * (w + FW * sl), og, c1);
    // ---- H = sum of the planes in slice order, as hi / lo operands.  Up to
    // rank 64 every plane of the lane's row is requested together; above, one
    // plane at a time (register budget).
    float h[KSM][8];
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e) h[ks][e] = 0.0f;
    if constexpr (KSM <= 2) {
#pragma unroll
      for (int ks = 0; ks < KSM; ++ks) {
        const int j = ks * 32 + og * 8;
        const int jj = j < LDH ? j : LDH - 8;
        float4 q0[SPLIT_SMAX], q1[SPLIT_SMAX];
#pragma unroll
        for (int pl = 0; pl < SPLIT_SMAX; ++pl) {
          const float* row = p.H + (int64_t)min(pl, S - 1) * p.hp_stride + (int64_t)trow * p.ldh + jj;
          q0[pl] = ldg_f4(row);
          q1[pl] = ldg_f4(row + 4);
        }
#pragma unroll
        for (int pl = 0; pl < SPLIT_SMAX; ++pl) {
          if (pl >= S) break;
          h[ks][0] += q0[pl].x; h[ks][1] += q0[pl].y; h[ks][2] += q0[pl].z; h[ks][3] += q0[pl].w;
          h[ks][4] += q1[pl].x; h[ks][5] += q1[pl].y; h[ks][6] += q1[pl].z; h[ks][7] += q1[pl].w;
        }
      }
    } else {
      for (int pl = 0; pl < S; ++pl) {
        float4 q0[KSM], q1[KSM];
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks) {
          const int j = ks * 32 + og * 8;
          const float* row = p.H + (int64_t)pl * p.hp_stride + (int64_t)trow * p.ldh + (j < LDH ? j : LDH - 8);
          q0[ks] = ldg_f4(row);
          q1[ks] = ldg_f4(row + 4);
        }
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks) {
          h[ks][0] += q0[ks].x; h[ks][1] += q0[ks].y; h[ks][2] += q0[ks].z; h[ks][3] += q0[ks].w;
          h[ks][4] += q1[ks].x; h[ks][5] += q1[ks].y; h[ks][6] += q1[ks].z; h[ks][7] += q1[ks].w;
        }
      }
    }
    bf16x8 hh[KSM], hl[KSM];
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks) {
      const int j = ks * 32 + og * 8;
#pragma unroll
      for (int e = 0; e < 8; ++e) h[ks][e] = (rv && j < LDH && j + e < r) ? h[ks][e] : 0.0f;
      split_hi_lo(h[ks], hh[ks], hl[ks]);
    }
    // ---- expand over this wave's column slices
#pragma unroll
    for (int sl = 0; sl < FSL; ++sl) {
      const int o_w = c0 + 64 * (w + FW * sl);
      f32x4 acc2[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) acc2[q] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KSM; ++ks) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          bf16x8 bo;
          if (B_AHEAD) {
            bo = bo_ahead[B_AHEAD ? sl : 0][B_AHEAD ? ks : 0][q];
          } else {
            const int o = out_col(o_w, q, mrow);
            bo = wrow8<RANK8>(Bw, (uint32_t)(o < c1 ? o : c1 - 1) * r, ks * 32 + og * 8, r);
          }
          bo = sel(ks * 32 + og * 8 < r, bo);
          acc2[q] = mfma_16x16x32(bo, hh[ks], acc2[q]);
          acc2[q] = mfma_16x16x32(bo, hl[ks], acc2[q]);
        }
      }
      mfma_fence();
      if (rv && o_w < c1) y_store<YBF16>(yf[sl], p.Y, p.ldy, trow, o_w, og, c1, s, acc2);
    }
  }
}

template <typename K>
hipError_t launch(K kernel, int grid, const FwdArgs& a, hipStream_t s, int threads = 256) {
  if (grid <= 0) return hipSuccess;
  hipLaunchKernelGGL(kernel, dim3(grid), dim3(threads), 0, s, a);
  return hipGetLastError();
}

int round8(long long g) { return (int)((g + 7) / 8 * 8); }

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
  a.num_slots = o.num_slots;
  a.n_rows = o.n;
  return a;
}

// One 32-column step per batch (two measured no faster).
template <bool YB, bool R8, int KSM>
hipError_t launch_expand_u(int grid, const FwdArgs& a, hipStream_t s) {
  return launch(expand_kernel<YB, R8, KSM, 1>, grid, a, s);
}

template <bool YB, bool R8>
hipError_t launch_expand_ks(const OpLaunch& o, int grid, int gridf, const FwdArgs& a, hipStream_t s) {
  const int ks = (o.r_max + 31) / 32;
  // both block sizes, as in the shrink
  hipError_t err = ks <= 1   ? launch(expand_fine_kernel<YB, R8, 1, YB ? 2 : 1, false>, gridf, a, s)
                   : ks <= 2 ? launch(expand_fine_kernel<YB, R8, 2, YB ? 2 : 1, false>, gridf, a, s)
                             : launch(expand_fine_kernel<YB, R8, 4, 1, false>, gridf, a, s);
  if (err != hipSuccess) return err;
  if (ks <= 1) return launch_expand_u<YB, R8, 1>(grid, a, s);
  if (ks <= 2) return launch_expand_u<YB, R8, 2>(grid, a, s);
  return launch_expand_u<YB, R8, 4>(grid, a, s);
}

template <bool YB, bool R8>
hipError_t launch_fused_nt(const OpLaunch& o, int grid, const FwdArgs& a, hipStream_t s) {
  const int nt = (o.r_max + 15) / 16;
  constexpr int T = FW * 64;
  if (nt <= 1) return launch(fused_small_kernel<YB, 1, R8>, grid, a, s, T);
  if (nt <= 2) return launch(fused_small_kernel<YB, 2, R8>, grid, a, s, T);
  if (nt <= 4) return launch(fused_small_kernel<YB, 4, R8>, grid, a, s, T);
  return launch(fused_small_kernel<YB, 8, R8>, grid, a, s, T);
}

}  // namespace

hipError_t launch_shrink_mfma(const OpLaunch& o, const void* X, int64_t ldx, float* H,
                              int64_t ldh, int32_t ks_max, int64_t hp_stride, hipStream_t s) {
  FwdArgs a = base_args(o);
  a.X = reinterpret_cast<const uint16_t*>(X);
  a.ldx = ldx;
  a.H = H;
  a.ldh = ldh;
  a.ks_max = std::min(std::max(ks_max, 1), SHRINK_KS_MAX);   // the expand sums at most this many planes
  a.hp_stride = hp_stride;
  // (row block, d-slice) units: blocks x min(ks_max, 256 / blocks) <= max(blocks, 256)
  const int grid = round8(std::min<long long>((long long)o.coarse_ub * a.ks_max, 2048));
  const int gridf = round8(std::min<long long>((long long)o.fine_ub * a.ks_max, 2048));
  const int nt = (o.r_max + 15) / 16;
  // the plan picks the block size on the device: both kernels are launched and
  // the one for the other size returns at once
  hipError_t err = nt <= 1   ? launch(shrink_fine_kernel<1, false>, gridf, a, s)
                   : nt <= 2 ? launch(shrink_fine_kernel<2, false>, gridf, a, s)
                   : nt <= 4 ? launch(shrink_fine_kernel<4, false>, gridf, a, s)
                             : launch(shrink_fine_kernel<8, false>, gridf, a, s);
  if (err != hipSuccess) return err;
  // one 32-wide k-step per batch: the 4096 x 256-row prefill shrink measured
  // 41 us at one step, 42 at two and 46 at four (fewer requests in flight per
  // wave keep the HBM streams more orderly; the matrix cores are idle anyway)
  if (nt <= 1) return launch(shrink_kernel<1, 1>, grid, a, s);
  if (nt <= 2) return launch(shrink_kernel<2, 1>, grid, a, s);
  if (nt <= 4) return launch(shrink_kernel<4, 1>, grid, a, s);
  return launch(shrink_kernel<8, 1>, grid, a, s);
}

// Input gradient over the plan's masked 64-row blocks (o.rb, o.perm and
// o.count_word describe them; o.d_in is the width of dY, o.d_out that of dX):
// G = dY B_a into d-sliced planes, then dX += s_a G A_a, both weights read as
// stored through gathers.
hipError_t launch_grad_x_mfma(const OpLaunch& o, const void* dY, int64_t lddy, float* H, int64_t ldh,
                              int64_t hp_stride, void* dX, lora_dtype dx_dtype, int64_t lddx,
                              hipStream_t s) {
  FwdArgs a = base_args(o);
  a.X = reinterpret_cast<const uint16_t*>(dY);
  a.ldx = lddy;
  a.H = H;
  a.ldh = ldh;
  a.ks_max = SHRINK_KS_MAX;
  a.hp_stride = hp_stride;
  a.force_fine = 1;
  const int nt = (o.r_max + 15) / 16;
  const int grid1 = round8(std::min<long long>((long long)o.fine_ub * a.ks_max, 2048));
  hipError_t err = nt <= 1   ? launch(shrink_fine_kernel<1, true>, grid1, a, s)
                   : nt <= 2 ? launch(shrink_fine_kernel<2, true>, grid1, a, s)
                   : nt <= 4 ? launch(shrink_fine_kernel<4, true>, grid1, a, s)
                             : launch(shrink_fine_kernel<8, true>, grid1, a, s);
  if (err != hipSuccess) return err;
  a.Y = dX;
  a.ldy = lddx;
  a.cw = 1024;
  const int grid2 = round8(std::min<long long>((long long)o.fine_ub * ((o.d_out + 1023) / 1024), 4096));
  const int ks = (o.r_max + 31) / 32;
  const bool yb = dx_dtype == LORA_BF16;
#define GX(YB, R8)                                                                           \
  (ks <= 1   ? launch(expand_fine_kernel<YB, R8, 1, 1, true>, grid2, a, s)                  \
   : ks <= 2 ? launch(expand_fine_kernel<YB, R8, 2, 1, true>, grid2, a, s)                  \
             : launch(expand_fine_kernel<YB, R8, 4, 1, true>, grid2, a, s))
  if (yb) return o.rank8 ? GX(true, true) : GX(true, false);
  return o.rank8 ? GX(false, true) : GX(false, false);
#undef GX
}

hipError_t launch_expand_mfma(const OpLaunch& o, const float* H, int64_t ldh, int32_t ks_max,
                              int64_t hp_stride, void* Y, lora_dtype y_dtype, int64_t ldy,
                              hipStream_t s) {
  FwdArgs a = base_args(o);
  a.H = const_cast<float*>(H);
  a.ldh = ldh;
  a.ks_max = std::min(std::max(ks_max, 1), SHRINK_KS_MAX);   // the expand sums at most this many planes
  a.hp_stride = hp_stride;
  a.Y = Y;
  a.ldy = ldy;
  // (row block, 1024-column chunk) units of the 256-row kernel (the 64-row
  // kernel picks its own chunk from the block count and loops over its units)
  a.cw = 1024;
  const long long n_ch = (o.d_out + a.cw - 1) / a.cw;
  const int grid = round8(std::min<long long>((long long)o.coarse_ub * n_ch, 4096));
  const int gridf = round8(std::min<long long>((long long)o.fine_ub * n_ch, 4096));
  const bool yb = y_dtype == LORA_BF16;
  if (yb && o.rank8) return launch_expand_ks<true, true>(o, grid, gridf, a, s);
  if (yb) return launch_expand_ks<true, false>(o, grid, gridf, a, s);
  if (o.rank8) return launch_expand_ks<false, true>(o, grid, gridf, a, s);
  return launch_expand_ks<false, false>(o, grid, gridf, a, s);
}

template <bool YB, bool R8>
hipError_t launch_small_expand_nt(const OpLaunch& o, int grid, const FwdArgs& a, hipStream_t s) {
  const int nt = (o.r_max + 15) / 16;
  constexpr int T = FW * 64;
  if (nt <= 1) return launch(small_expand_kernel<YB, 1, R8>, grid, a, s, T);
  if (nt <= 2) return launch(small_expand_kernel<YB, 2, R8>, grid, a, s, T);
  if (nt <= 4) return launch(small_expand_kernel<YB, 4, R8>, grid, a, s, T);
  return launch(small_expand_kernel<YB, 8, R8>, grid, a, s, T);
}

hipError_t launch_small_split_mfma(const OpLaunch& o, const void* X, int64_t ldx, void* Y,
                                   lora_dtype y_dtype, int64_t ldy, int32_t n_chunks,
                                   int32_t slices, float* part, hipStream_t s) {
  FwdArgs a = base_args(o);
  a.X = reinterpret_cast<const uint16_t*>(X);
  a.ldx = ldx;
  a.Y = Y;
  a.ldy = ldy;
  a.srec = o.srec;
  a.n_rec = std::max(o.rb_ub, 1);
  const int nt = (o.r_max + 15) / 16;
  const int tiles = nt <= 1 ? 1 : nt <= 2 ? 2 : nt <= 4 ? 4 : 8;
  a.H = part;
  a.ldh = tiles * 16;
  a.ks_max = std::min(std::max(slices, 1), SPLIT_SMAX);
  a.hp_stride = (int64_t)a.n_rec * 16 * a.ldh;
  const int g1 = a.n_rec * a.ks_max;
  hipError_t e;
  if (tiles == 1) e = launch(small_shrink_kernel<1, 4>, g1, a, s);
  else if (tiles == 2) e = launch(small_shrink_kernel<2, 4>, g1, a, s);
  else if (tiles == 4) e = launch(small_shrink_kernel<4, 2>, g1, a, s);
  else e = launch(small_shrink_kernel<8, 1>, g1, a, s);
  if (e != hipSuccess) return e;
  constexpr int CW = 64 * FW * FSL;
  const int P = std::max({1, n_chunks, (o.d_out + CW - 1) / CW});
  a.n_chunks = P;
  a.chunk = ((o.d_out + P - 1) / P + 63) / 64 * 64;
  const int grid = 8 * P * ((o.rb_ub + 7) / 8);
  const bool yb = y_dtype == LORA_BF16;
  if (yb && o.rank8) return launch_small_expand_nt<true, true>(o, grid, a, s);
  if (yb) return launch_small_expand_nt<true, false>(o, grid, a, s);
  if (o.rank8) return launch_small_expand_nt<false, true>(o, grid, a, s);
  return launch_small_expand_nt<false, false>(o, grid, a, s);
}

template <bool YB, bool R8>
hipError_t launch_ids_expand_nt(int nt, int grid, const FwdArgs& a, hipStream_t s) {
  constexpr int T = FW * 64;
  if (nt <= 1) return launch(ids_expand_kernel<YB, 1, R8>, grid, a, s, T);
  if (nt <= 2) return launch(ids_expand_kernel<YB, 2, R8>, grid, a, s, T);
  if (nt <= 4) return launch(ids_expand_kernel<YB, 4, R8>, grid, a, s, T);
  return launch(ids_expand_kernel<YB, 8, R8>, grid, a, s, T);
}

hipError_t launch_ids_mfma(const IdsLaunch& l, hipStream_t s) {
  FwdArgs a{};
  a.meta = l.meta;
  a.d_in = l.d_in;
  a.d_out = l.d_out;
  a.num_slots = l.num_slots;
  a.ids = l.ids;
  a.n_ids = l.n;
  a.X = reinterpret_cast<const uint16_t*>(l.X);
  a.ldx = l.ldx;
  a.Y = l.Y;
  a.ldy = l.ldy;
  const int nt = (l.r_max + 15) / 16;
  const int tiles = nt <= 1 ? 1 : nt <= 2 ? 2 : nt <= 4 ? 4 : 8;
  a.H = l.H;
  a.ldh = tiles * 16;
  a.ks_max = std::min(std::max(l.slices, 1), SPLIT_SMAX);
  a.hp_stride = (int64_t)std::max(l.n, 1) * a.ldh;
  const int g1 = l.num_slots * a.ks_max;
  hipError_t e;
  if (tiles == 1) e = launch(ids_shrink_kernel<1, 8>, g1, a, s);
  else if (tiles == 2) e = launch(ids_shrink_kernel<2, 8>, g1, a, s);
  else if (tiles == 4) e = launch(ids_shrink_kernel<4, 2>, g1, a, s);
  else e = launch(ids_shrink_kernel<8, 1>, g1, a, s);
  if (e != hipSuccess) return e;
  constexpr int CW = 64 * FW * FSL;
  const int P = std::max({1, l.n_chunks, (l.d_out + CW - 1) / CW});
  a.n_chunks = P;
  a.chunk = ((l.d_out + P - 1) / P + 63) / 64 * 64;
  const int grid = 8 * P * ((l.num_slots + 7) / 8);
  if (l.y_bf16 && l.rank8) return launch_ids_expand_nt<true, true>(nt, grid, a, s);
  if (l.y_bf16) return launch_ids_expand_nt<true, false>(nt, grid, a, s);
  if (l.rank8) return launch_ids_expand_nt<false, true>(nt, grid, a, s);
  return launch_ids_expand_nt<false, false>(nt, grid, a, s);
}

hipError_t launch_bgmv_mfma(const OpLaunch& o, const void* X, int64_t ldx, void* Y,
                            lora_dtype y_dtype, int64_t ldy, int32_t n_chunks, hipStream_t s) {
  FwdArgs a = base_args(o);
  a.X = reinterpret_cast<const uint16_t*>(X);
  a.ldx = ldx;
  a.Y = Y;
  a.ldy = ldy;
  // each workgroup covers at most CW columns (FSL slices of 64 per wave)
  constexpr int CW = 64 * FW * FSL;
  const int P = std::max({1, n_chunks, (o.d_out + CW - 1) / CW});
  a.n_chunks = P;
  a.chunk = ((o.d_out + P - 1) / P + 63) / 64 * 64;
  a.srec = o.srec;
  a.n_rec = std::max(o.rb_ub, 1);
  const int grid = 8 * P * ((o.rb_ub + 7) / 8);
  const bool yb = y_dtype == LORA_BF16;
  if (yb && o.rank8) return launch_fused_nt<true, true>(o, grid, a, s);
  if (yb) return launch_fused_nt<true, false>(o, grid, a, s);
  if (o.rank8) return launch_fused_nt<false, true>(o, grid, a, s);
  return launch_fused_nt<false, false>(o, grid, a, s);
}

}  // namespace lora
