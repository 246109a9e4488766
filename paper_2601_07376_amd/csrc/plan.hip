// Row grouping by adapter id on the device: the gather step of the paper's
// gather-group-compute-scatter structure (Section 3.4, Figure 2) and the
// routing of trainable rows by adapter identity (Section 3.5).
//
// One workgroup of 1024 threads (16 waves).  Phase 0 reads every row's id once
// (batched loads), validates it and keeps the pair (id, id under the mask) in
// LDS (or, for very long batches, in the plan workspace).  Wave w then owns a
// contiguous slice of the rows, and a stable counting sort takes two passes
// over the slice: pass A builds per-wave histograms in LDS, a prefix over
// (adapter, wave) turns them into write cursors, and pass B re-walks the slice
// in row order and scatters each row to its cursor.  Rows of one adapter inside
// a 64-row chunk are found with ballots over the bits of the id, so a chunk
// needs no atomics: the lowest lane of each id group owns that group's cursor.
#include "device_common.h"
#include "lora_internal.h"

namespace lora {

namespace {

constexpr int LDS_ROWS = 20480;        // rows whose ids fit in LDS
constexpr int LDS_SEG_WORDS = PLAN_WAVES * LORA_MAX_SLOTS;   // segment table staging

__device__ __forceinline__ uint64_t lanemask_lt() {
  return (1ull << __lane_id()) - 1ull;
}

// Lanes of this wave holding the same key (all 64 lanes must call).
__device__ __forceinline__ uint64_t match_peers(int key, int nbits) {
  uint64_t peers = ~0ull;
  for (int b = 0; b < nbits; ++b) {
    const bool bit = (key >> b) & 1;
    const uint64_t bal = __ballot(bit);
    peers &= bit ? bal : ~bal;
  }
  return peers;
}

// Exclusive prefix sum over the 1024 threads of the block (all must call).
__device__ int block_excl_scan(int v, int* s_wsum, int& total) {
  const int lane = threadIdx.x & 63, w = wave_id();
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_wsum[w] = x;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < PLAN_WAVES; ++i) {
    const int s = s_wsum[i];
    base += (i < w) ? s : 0;
    tot += s;
  }
  __syncthreads();
  total = tot;
  return base + x - v;
}

// Packed row ids: low half = id + 1, high half = id under the mask + 1.
struct Rows {
  const int32_t* pk;
  int n;
  __device__ __forceinline__ int eff(int t) const { return (pk[t] & 0xffff) - 1; }
  __device__ __forceinline__ int eff_m(int t) const { return (pk[t] >> 16) - 1; }
};

struct Out {
  int32_t* counts;
  int32_t* offsets;
  int32_t* perm;
  int32_t* dup_counts;    // when the mask is absent the trainable grouping is the same
  int32_t* dup_offsets;
  int32_t* dup_perm;
  int32_t* run_start;
  int32_t* run_len;
  int32_t* run_adapter;
};

// One stable grouping pass.  Returns, for thread a < S, the count and offset of
// adapter a, and (in every thread) the number of grouped rows and of runs.
template <bool MASKED, bool RUNS, bool DUP>
__device__ void group_pass(const Rows& R, int S, int (*s_hist)[LORA_MAX_SLOTS], int* s_wsum,
                           int (*s_runs)[PLAN_WAVES], int* s_scalar, const Out& out,
                           int& my_count, int& my_offset, int& n_act, int& n_runs) {
  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int n = R.n;
  const int nbits = 32 - __clz(S);
  const int L = (((n + PLAN_WAVES - 1) / PLAN_WAVES) + 63) / 64 * 64;
  const int beg = min(n, w * L), end = min(n, beg + L);

  for (int i = tid; i < PLAN_WAVES * LORA_MAX_SLOTS; i += PLAN_THREADS) {
    if ((i % LORA_MAX_SLOTS) < S) s_hist[i / LORA_MAX_SLOTS][i % LORA_MAX_SLOTS] = 0;
  }
  __syncthreads();

  // ---- pass A: per-wave histograms and run counts
  int n_st = 0, n_ed = 0;
  for (int base = beg; base < end; base += 64) {
    const int t = base + lane;
    const bool valid = t < end;
    const int e = valid ? (MASKED ? R.eff_m(t) : R.eff(t)) : -1;
    const uint64_t peers = match_peers(e + 1, nbits);
    if (e >= 0 && lane == __ffsll((unsigned long long)peers) - 1)
      s_hist[w][e] += __popcll(peers);
    if (RUNS) {
      bool st = false, ed = false;
      if (valid && e >= 0) {
        st = (t == 0) || R.eff(t - 1) != e;
        ed = (t == n - 1) || R.eff(t + 1) != e;
      }
      n_st += __popcll(__ballot(st));
      n_ed += __popcll(__ballot(ed));
    }
  }
  if (RUNS && lane == 0) {
    s_runs[0][w] = n_st;
    s_runs[1][w] = n_ed;
  }
  __syncthreads();

  // ---- cursors: per adapter, the prefix over waves; then the prefix over adapters
  int cnt = 0;
  if (tid < S) {
    for (int ww = 0; ww < PLAN_WAVES; ++ww) {
      const int v = s_hist[ww][tid];
      s_hist[ww][tid] = cnt;
      cnt += v;
    }
  }
  int total;
  const int off = block_excl_scan(tid < S ? cnt : 0, s_wsum, total);
  if (tid < S) {
    out.counts[tid] = cnt;
    out.offsets[tid] = off;
    if (DUP) {
      out.dup_counts[tid] = cnt;
      out.dup_offsets[tid] = off;
    }
    for (int ww = 0; ww < PLAN_WAVES; ++ww) s_hist[ww][tid] += off;
  }
  if (tid == 0) {
    out.offsets[S] = total;
    if (DUP) out.dup_offsets[S] = total;
    if (RUNS) {
      int a0 = 0, a1 = 0;
      for (int ww = 0; ww < PLAN_WAVES; ++ww) {
        const int v0 = s_runs[0][ww], v1 = s_runs[1][ww];
        s_runs[0][ww] = a0;
        s_runs[1][ww] = a1;
        a0 += v0;
        a1 += v1;
      }
      s_scalar[0] = a0;
    }
  }
  my_count = cnt;
  my_offset = off;
  n_act = total;
  __syncthreads();

  // ---- pass B: scatter rows to their cursors, in row order
  int rsb = RUNS ? s_runs[0][w] : 0, reb = RUNS ? s_runs[1][w] : 0;
  for (int base = beg; base < end; base += 64) {
    const int t = base + lane;
    const bool valid = t < end;
    const int e = valid ? (MASKED ? R.eff_m(t) : R.eff(t)) : -1;
    const uint64_t peers = match_peers(e + 1, nbits);
    const bool leader = e >= 0 && lane == __ffsll((unsigned long long)peers) - 1;
    int cur = 0;
    if (e >= 0) cur = s_hist[w][e];
    if (e >= 0) {
      const int pos = cur + __popcll(peers & lanemask_lt());
      out.perm[pos] = t;
      if (DUP) out.dup_perm[pos] = t;
    }
    if (leader) s_hist[w][e] = cur + __popcll(peers);
    if (RUNS) {
      bool st = false, ed = false;
      if (valid && e >= 0) {
        st = (t == 0) || R.eff(t - 1) != e;
        ed = (t == n - 1) || R.eff(t + 1) != e;
      }
      const uint64_t sb = __ballot(st), eb = __ballot(ed);
      if (st) {
        const int k = rsb + __popcll(sb & lanemask_lt());
        out.run_start[k] = t;
        out.run_adapter[k] = e;
      }
      if (ed) out.run_len[reb + __popcll(eb & lanemask_lt())] = t;  // last row; length below
      rsb += __popcll(sb);
      reb += __popcll(eb);
    }
  }
  __syncthreads();
  n_runs = 0;
  if (RUNS) {
    n_runs = s_scalar[0];
    for (int k = tid; k < n_runs; k += PLAN_THREADS)
      out.run_len[k] = out.run_len[k] - out.run_start[k] + 1;
    __syncthreads();
  }
}

// PK_LDS: the packed ids live in LDS (n <= LDS_ROWS), else in the workspace.
// SEG_LDS: the segment table is staged in LDS.  Both are template parameters so
// that every access has one known address space (a pointer that may be either
// compiles to generic loads that wait on both memory counters).
template <bool PK_LDS, bool SEG_LDS>
__global__ __launch_bounds__(PLAN_THREADS) void plan_kernel(PlanLaunch a) {
  __shared__ int s_hist[PLAN_WAVES][LORA_MAX_SLOTS];
  __shared__ int s_rank[LORA_MAX_SLOTS];
  __shared__ int32_t s_pk[LDS_ROWS];
  __shared__ int s_wsum[PLAN_WAVES];
  __shared__ int s_runs[2][PLAN_WAVES];
  __shared__ int s_scalar[4];
  __shared__ unsigned s_flags;

  const int tid = threadIdx.x;
  const int n = a.n, S = a.num_slots;
  if (tid == 0) s_flags = 0u;
  for (int i = tid; i < S; i += PLAN_THREADS) s_rank[i] = a.meta[i].rank;
  uint32_t flags = 0u;

  // ---- segment table: staged in LDS (in the histogram area) when it fits
  const bool seg = a.seg_offsets != nullptr;
  const int ns = a.num_segs;
  int* s_seg = &s_hist[0][0];
  const int32_t* seg_off = SEG_LDS ? s_seg : a.seg_offsets;
  const int32_t* seg_ad = SEG_LDS ? s_seg + ns + 1 : a.seg_adapter;
  int any_bad = 0;
  if (seg) {
    if (SEG_LDS) {
      for (int i = tid; i <= ns; i += PLAN_THREADS) s_seg[i] = a.seg_offsets[i];
      for (int i = tid; i < ns; i += PLAN_THREADS) s_seg[ns + 1 + i] = a.seg_adapter[i];
      __syncthreads();
    }
    bool bad = false;
    for (int s = tid; s <= ns; s += PLAN_THREADS) {
      const int o = seg_off[s];
      if (s == 0 && o != 0) bad = true;
      if (s == ns && o != n) bad = true;
      if (s < ns && seg_off[s + 1] < o) bad = true;
    }
    any_bad = __syncthreads_or(bad ? 1 : 0);
    if (any_bad) flags |= LORA_DATA_BAD_SEGMENTS;
  }
  __syncthreads();

  // ---- phase 0: validated ids, packed with the ids under the mask
  int32_t* pk = PK_LDS ? s_pk : a.d.seg_ids;
  constexpr int UNR = 8;
  for (int base = 0; base < n; base += PLAN_THREADS * UNR) {
    int raw[UNR];
    int mk[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int t = base + u * PLAN_THREADS + tid;
      raw[u] = -1;
      mk[u] = 1;
      if (t < n) {
        if (!seg) {
          raw[u] = a.idx[t];
        } else if (!any_bad) {
          int lo = 0, hi = ns;         // seg_off[lo] <= t < seg_off[hi]
          while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (seg_off[mid] <= t) lo = mid;
            else hi = mid;
          }
          raw[u] = seg_ad[lo];
        }
        if (a.mask != nullptr) mk[u] = a.mask[t];
      }
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int t = base + u * PLAN_THREADS + tid;
      if (t >= n) continue;
      int e = raw[u];
      if (e < -1 || e >= S) {
        flags |= LORA_DATA_BAD_ID;
        e = -1;
      } else if (e >= 0 && s_rank[e] <= 0) {
        flags |= LORA_DATA_EMPTY_SLOT;
        e = -1;
      }
      const int em = mk[u] ? e : -1;
      pk[t] = (e + 1) | ((em + 1) << 16);
    }
  }
  __syncthreads();

  const Rows R{pk, n};
  int cnt, off, n_act, n_runs;
  int mcnt, moff, m_n_act, unused;
  const Out out{a.d.counts, a.d.offsets, a.d.perm, a.d.m_counts, a.d.m_offsets, a.d.m_perm,
                a.d.run_start, a.d.run_len, a.d.run_adapter};
  if (a.mask == nullptr) {
    group_pass<false, true, true>(R, S, s_hist, s_wsum, s_runs, s_scalar, out, cnt, off, n_act,
                                  n_runs);
    mcnt = cnt;
    moff = off;
    m_n_act = n_act;
  } else {
    group_pass<false, true, false>(R, S, s_hist, s_wsum, s_runs, s_scalar, out, cnt, off, n_act,
                                   n_runs);
    const Out mout{a.d.m_counts, a.d.m_offsets, a.d.m_perm, nullptr, nullptr, nullptr,
                   nullptr, nullptr, nullptr};
    group_pass<true, false, false>(R, S, s_hist, s_wsum, s_runs, s_scalar, mout, mcnt, moff,
                                   m_n_act, unused);
  }

  // ---- entry lists.  Large groups: blocks of RB_ROWS rows; small groups:
  // entries of at most SMALL_ROWS rows, placed after every large-group block.
  const bool live = tid < S;
  const bool small = live && cnt > 0 && cnt <= a.small_max;
  const int nbl = (live && cnt > a.small_max) ? (cnt + RB_ROWS - 1) / RB_ROWS : 0;
  const int nbs = small ? (cnt + SMALL_ROWS - 1) / SMALL_ROWS : 0;
  const int nbm = live ? (mcnt + MRB_ROWS - 1) / MRB_ROWS : 0;
  int tot_l, tot_s, tot_m;
  const int pl = block_excl_scan(nbl, s_wsum, tot_l);
  const int ps = block_excl_scan(nbs, s_wsum, tot_s);
  const int pm = block_excl_scan(nbm, s_wsum, tot_m);
  for (int i = 0; i < nbl; ++i)
    a.d.rb[pl + i] = make_int4(tid, off + i * RB_ROWS, min(RB_ROWS, cnt - i * RB_ROWS), 0);
  for (int i = 0; i < nbs; ++i)
    a.d.rb[tot_l + ps + i] =
        make_int4(tid, off + i * SMALL_ROWS, min(SMALL_ROWS, cnt - i * SMALL_ROWS), 1);
  if (live) a.d.m_blk[tid] = pm;
  for (int i = 0; i < nbm; ++i)
    a.d.mrb[pm + i] = make_int4(tid, moff + i * MRB_ROWS, min(MRB_ROWS, mcnt - i * MRB_ROWS), 0);

  if (flags) atomicOr(&s_flags, flags);
  __syncthreads();
  if (tid == 0) {
    int32_t* h = a.d.hdr;
    h[HDR_FLAGS] = (int32_t)s_flags;
    h[HDR_NACT] = n_act;
    h[HDR_NRUNS] = n_runs;
    h[HDR_MNACT] = m_n_act;
    h[HDR_NRB_LARGE] = tot_l;
    h[HDR_NRB_TOTAL] = tot_l + tot_s;
    h[HDR_NMRB] = tot_m;
  }
}

}  // namespace

hipError_t launch_plan(const PlanLaunch& a, hipStream_t s) {
  const bool pk_lds = a.n <= LDS_ROWS;
  const bool seg_lds = a.seg_offsets != nullptr && 2 * a.num_segs + 1 <= LDS_SEG_WORDS;
  if (pk_lds && seg_lds)
    hipLaunchKernelGGL((plan_kernel<true, true>), dim3(1), dim3(PLAN_THREADS), 0, s, a);
  else if (pk_lds)
    hipLaunchKernelGGL((plan_kernel<true, false>), dim3(1), dim3(PLAN_THREADS), 0, s, a);
  else if (seg_lds)
    hipLaunchKernelGGL((plan_kernel<false, true>), dim3(1), dim3(PLAN_THREADS), 0, s, a);
  else
    hipLaunchKernelGGL((plan_kernel<false, false>), dim3(1), dim3(PLAN_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace lora
