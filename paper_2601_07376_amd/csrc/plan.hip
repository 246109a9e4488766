// Row grouping by adapter id on the device: the gather step of the paper's
// gather-group-compute-scatter structure (Section 3.4, Figure 2) and the
// routing of trainable rows by adapter identity (Section 3.5).
//
// One workgroup of 1024 threads (16 waves).  Wave w owns a contiguous slice of
// the rows.  A stable counting sort takes two passes over the slice: pass A
// builds per-wave histograms in LDS, a prefix over (adapter, wave) turns them
// into write cursors, and pass B re-walks the slice in row order and scatters
// each row to its cursor.  Rows of one adapter inside a 64-row chunk are found
// with ballots over the bits of the id, so a chunk needs no atomics: the lowest
// lane of each id group owns that group's cursor.
#include "device_common.h"
#include "lora_internal.h"

namespace lora {

namespace {

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
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
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

struct Ctx {
  const int32_t* ids;
  const uint8_t* mask;
  const int* s_rank;
  int n, S;
  uint32_t flags;

  // Id after validation (-1 for invalid ids and empty slots, which set flags).
  __device__ __forceinline__ int eff(int t) {
    const int e = ids[t];
    if (e < -1 || e >= S) {
      flags |= LORA_DATA_BAD_ID;
      return -1;
    }
    if (e >= 0 && s_rank[e] <= 0) {
      flags |= LORA_DATA_EMPTY_SLOT;
      return -1;
    }
    return e;
  }
  __device__ __forceinline__ int eff_m(int t) {
    const int e = eff(t);
    return (mask == nullptr || mask[t] != 0) ? e : -1;
  }
};

// One stable grouping pass.  Writes counts[S], offsets[S+1], perm[n_act] and,
// when RUNS, the maximal runs.  Returns (per thread a < S) the count and
// offset of adapter a.
template <bool MASKED, bool RUNS>
__device__ void group_pass(Ctx& c, int (*s_hist)[LORA_MAX_SLOTS], int* s_wsum,
                           int (*s_runs)[PLAN_WAVES], int* s_scalar, int32_t* counts,
                           int32_t* offsets, int32_t* perm, int32_t* run_start,
                           int32_t* run_len, int32_t* run_adapter, int& my_count,
                           int& my_offset, int& n_act, int& n_runs) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int n = c.n, S = c.S;
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
    const int e = valid ? (MASKED ? c.eff_m(t) : c.eff(t)) : -1;
    const uint64_t peers = match_peers(e + 1, nbits);
    if (e >= 0 && lane == __ffsll((unsigned long long)peers) - 1)
      s_hist[w][e] += __popcll(peers);
    if (RUNS) {
      const int up = __shfl_up(e, 1);
      const int dn = __shfl_down(e, 1);
      bool st = false, ed = false;
      if (valid && e >= 0) {
        const int ep = (t == 0) ? -2 : (lane > 0 ? up : c.eff(t - 1));
        const int en = (t == n - 1) ? -2 : ((lane < 63 && t + 1 < end) ? dn : c.eff(t + 1));
        st = ep != e;
        ed = en != e;
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
    counts[tid] = cnt;
    offsets[tid] = off;
    for (int ww = 0; ww < PLAN_WAVES; ++ww) s_hist[ww][tid] += off;
  }
  if (tid == 0) {
    offsets[S] = total;
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
    const int e = valid ? (MASKED ? c.eff_m(t) : c.eff(t)) : -1;
    const uint64_t peers = match_peers(e + 1, nbits);
    const bool leader = e >= 0 && lane == __ffsll((unsigned long long)peers) - 1;
    int cur = 0;
    if (e >= 0) cur = s_hist[w][e];
    if (e >= 0) perm[cur + __popcll(peers & lanemask_lt())] = t;
    if (leader) s_hist[w][e] = cur + __popcll(peers);
    if (RUNS) {
      const int up = __shfl_up(e, 1);
      const int dn = __shfl_down(e, 1);
      bool st = false, ed = false;
      if (valid && e >= 0) {
        const int ep = (t == 0) ? -2 : (lane > 0 ? up : c.eff(t - 1));
        const int en = (t == n - 1) ? -2 : ((lane < 63 && t + 1 < end) ? dn : c.eff(t + 1));
        st = ep != e;
        ed = en != e;
      }
      const uint64_t sb = __ballot(st), eb = __ballot(ed);
      if (st) {
        const int k = rsb + __popcll(sb & lanemask_lt());
        run_start[k] = t;
        run_adapter[k] = e;
      }
      if (ed) run_len[reb + __popcll(eb & lanemask_lt())] = t;  // last row; length below
      rsb += __popcll(sb);
      reb += __popcll(eb);
    }
  }
  __syncthreads();
  if (RUNS) {
    n_runs = s_scalar[0];
    for (int k = tid; k < n_runs; k += PLAN_THREADS) run_len[k] = run_len[k] - run_start[k] + 1;
    __syncthreads();
  }
}

__global__ __launch_bounds__(PLAN_THREADS) void plan_kernel(PlanLaunch a) {
  __shared__ int s_hist[PLAN_WAVES][LORA_MAX_SLOTS];
  __shared__ int s_rank[LORA_MAX_SLOTS];
  __shared__ int s_wsum[PLAN_WAVES];
  __shared__ int s_runs[2][PLAN_WAVES];
  __shared__ int s_scalar[4];
  __shared__ unsigned s_flags;

  const int tid = threadIdx.x;
  const int n = a.n, S = a.num_slots;
  if (tid == 0) s_flags = 0u;
  for (int i = tid; i < S; i += PLAN_THREADS) s_rank[i] = a.meta[i].rank;

  Ctx c;
  c.ids = a.idx;
  c.mask = a.mask;
  c.s_rank = s_rank;
  c.n = n;
  c.S = S;
  c.flags = 0u;

  // ---- segment mode: expand the segment table into per-row ids
  if (a.seg_offsets != nullptr) {
    bool bad = false;
    for (int s = tid; s <= a.num_segs; s += PLAN_THREADS) {
      const int o = a.seg_offsets[s];
      if (s == 0 && o != 0) bad = true;
      if (s == a.num_segs && o != n) bad = true;
      if (s < a.num_segs && a.seg_offsets[s + 1] < o) bad = true;
    }
    const int any_bad = __syncthreads_or(bad ? 1 : 0);
    if (any_bad) c.flags |= LORA_DATA_BAD_SEGMENTS;
    for (int t = tid; t < n; t += PLAN_THREADS) {
      int id = -1;
      if (!any_bad) {
        int lo = 0, hi = a.num_segs;       // seg_offsets[lo] <= t < seg_offsets[hi]
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (a.seg_offsets[mid] <= t) lo = mid;
          else hi = mid;
        }
        id = a.seg_adapter[lo];
      }
      a.d.seg_ids[t] = id;
    }
    c.ids = a.d.seg_ids;
  }
  __syncthreads();

  int cnt, off, n_act, n_runs = 0;
  group_pass<false, true>(c, s_hist, s_wsum, s_runs, s_scalar, a.d.counts, a.d.offsets,
                          a.d.perm, a.d.run_start, a.d.run_len, a.d.run_adapter, cnt, off,
                          n_act, n_runs);
  int mcnt, moff, m_n_act, unused = 0;
  group_pass<true, false>(c, s_hist, s_wsum, s_runs, s_scalar, a.d.m_counts, a.d.m_offsets,
                          a.d.m_perm, nullptr, nullptr, nullptr, mcnt, moff, m_n_act, unused);

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

  if (c.flags) atomicOr(&s_flags, c.flags);
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
  hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(PLAN_THREADS), 0, s, a);
  return hipGetLastError();
}

}  // namespace lora
