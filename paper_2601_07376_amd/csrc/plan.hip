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
  const int x = wave_incl_scan(v);
  if (lane == 63) s_wsum[w] = x;
  __syncthreads();
  const int c = row_incl_scan(lane < PLAN_WAVES ? s_wsum[lane] : 0);   // lanes 0..15
  const int base = lane_value(c, w) - lane_value(x, 63);
  total = lane_value(c, PLAN_WAVES - 1);
  __syncthreads();
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
  int32_t* run_end;
  int32_t* run_adapter;
};

// One stable grouping pass.  Returns, for thread a < S, the count and offset of
// adapter a, and (in every thread) the number of grouped rows and of runs.
// s_hist holds one counter per (adapter, wave), adapter-major: [a * 16 + w].
template <bool MASKED, bool RUNS, bool DUP>
__device__ void group_pass(const Rows& R, int S, int* s_hist, int* s_cnt, int* s_wsum,
                           int (*s_runs)[PLAN_WAVES], int* s_scalar, const Out& out,
                           int& my_count, int& my_offset, int& n_act, int& n_runs) {
  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int n = R.n;
  const int nbits = 32 - __clz(S);
  const int L = (((n + PLAN_WAVES - 1) / PLAN_WAVES) + 63) / 64 * 64;
  const int beg = min(n, w * L), end = min(n, beg + L);

  for (int i = tid; i < S * PLAN_WAVES; i += PLAN_THREADS) s_hist[i] = 0;
  __syncthreads();

  // ---- pass A: per-wave histograms and run counts
  int n_st = 0, n_ed = 0;
  for (int base = beg; base < end; base += 64) {
    const int t = base + lane;
    const bool valid = t < end;
    const int e = valid ? (MASKED ? R.eff_m(t) : R.eff(t)) : -1;
    const uint64_t peers = match_peers(e + 1, nbits);
    if (e >= 0 && lane == __ffsll((unsigned long long)peers) - 1)
      s_hist[e * PLAN_WAVES + w] += __popcll(peers);
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

  // ---- cursors: per adapter, the prefix over its 16 wave counters (one row of
  // 16 lanes per adapter); then the prefix over adapters
  for (int k0 = 0; k0 < S * PLAN_WAVES; k0 += PLAN_THREADS) {
    const int k = k0 + tid;
    const bool act = k < S * PLAN_WAVES;
    const int v = act ? s_hist[k] : 0;
    const int incl = row_incl_scan(v);
    if (act) {
      s_hist[k] = incl - v;
      if ((k & 15) == 15) s_cnt[k >> 4] = incl;
    }
  }
  __syncthreads();
  const int cnt = tid < S ? s_cnt[tid] : 0;
  int total;
  const int off = block_excl_scan(cnt, s_wsum, total);
  if (tid < S) {
    out.counts[tid] = cnt;
    out.offsets[tid] = off;
    if (DUP) {
      out.dup_counts[tid] = cnt;
      out.dup_offsets[tid] = off;
    }
    s_cnt[tid] = off;
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
    if (e >= 0) cur = s_cnt[e] + s_hist[e * PLAN_WAVES + w];
    if (e >= 0) {
      const int pos = cur + __popcll(peers & lanemask_lt());
      out.perm[pos] = t;
      if (DUP) out.dup_perm[pos] = t;
    }
    if (leader) s_hist[e * PLAN_WAVES + w] += __popcll(peers);
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
      if (ed) out.run_end[reb + __popcll(eb & lanemask_lt())] = t;
      rsb += __popcll(sb);
      reb += __popcll(eb);
    }
  }
  __syncthreads();
  n_runs = RUNS ? s_scalar[0] : 0;
}

// PK_LDS: the packed ids live in LDS (n <= LDS_ROWS), else in the workspace.
// SEG_LDS: the segment table is staged in LDS.  Both are template parameters so
// that every access has one known address space (a pointer that may be either
// compiles to generic loads that wait on both memory counters).
template <bool PK_LDS, bool SEG_LDS>
__global__ __launch_bounds__(PLAN_THREADS) void plan_kernel(PlanLaunch a) {
  __shared__ int s_hist[PLAN_WAVES * LORA_MAX_SLOTS];
  __shared__ int s_rank[LORA_MAX_SLOTS];
  __shared__ int s_cnt[LORA_MAX_SLOTS];
  __shared__ int32_t s_pk[LDS_ROWS];
  __shared__ int s_wsum[PLAN_WAVES];
  __shared__ int s_runs[2][PLAN_WAVES];
  __shared__ int s_scalar[4];
  __shared__ unsigned s_flags;

  const int tid = threadIdx.x;
  const int n = a.n, S = a.num_slots;
  if (tid == 0) s_flags = 0u;
  for (int i = tid; i < S; i += PLAN_THREADS) s_rank[i] = a.meta[i].rank;
  SlotMeta my_meta{};
  if (tid < S) my_meta = a.meta[tid];
  uint32_t flags = 0u;

  // ---- segment table: staged in LDS (in the histogram area) when it fits
  const bool seg = a.seg_offsets != nullptr;
  const int ns = a.num_segs;
  int* s_seg = s_hist;
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
                a.d.run_start, a.d.run_end, a.d.run_adapter};
  if (a.mask == nullptr) {
    group_pass<false, true, true>(R, S, s_hist, s_cnt, s_wsum, s_runs, s_scalar, out, cnt, off, n_act,
                                  n_runs);
    mcnt = cnt;
    moff = off;
    m_n_act = n_act;
  } else {
    group_pass<false, true, false>(R, S, s_hist, s_cnt, s_wsum, s_runs, s_scalar, out, cnt, off, n_act,
                                   n_runs);
    const Out mout{a.d.m_counts, a.d.m_offsets, a.d.m_perm, nullptr, nullptr, nullptr,
                   nullptr, nullptr, nullptr};
    group_pass<true, false, false>(R, S, s_hist, s_cnt, s_wsum, s_runs, s_scalar, mout, mcnt, moff,
                                   m_n_act, unused);
  }

  // ---- entry lists.  Large groups: blocks of RB_ROWS rows (RB_FINE rows when
  // the batch has fewer than FINE_BELOW coarse blocks); small groups: entries
  // of at most SMALL_ROWS rows, placed after every large-group block.
  const bool live = tid < S;
  const bool small = live && cnt > 0 && cnt <= a.small_max;
  const bool large = live && cnt > a.small_max;
  const int nbc = large ? (cnt + RB_ROWS - 1) / RB_ROWS : 0;
  const int nbf = large ? (cnt + RB_FINE - 1) / RB_FINE : 0;
  const int nbs = small ? (cnt + SMALL_ROWS - 1) / SMALL_ROWS : 0;
  const int nbm = live ? (mcnt + MRB_ROWS - 1) / MRB_ROWS : 0;
  int tot_c, tot_f, tot_s, tot_m;
  const int pc = block_excl_scan(nbc, s_wsum, tot_c);
  const int pf = block_excl_scan(nbf, s_wsum, tot_f);
  const int ps = block_excl_scan(nbs, s_wsum, tot_s);
  const int pm = block_excl_scan(nbm, s_wsum, tot_m);
  // block size of the whole batch, chosen on the host (the launches follow it)
  const bool fine = a.fine != 0;
  const int rbr = fine ? RB_FINE : RB_ROWS, nbl = fine ? nbf : nbc, pl = fine ? pf : pc;
  const int tot_l = fine ? tot_f : tot_c;
  for (int i = 0; i < nbl; ++i)
    a.d.rb[pl + i] = make_int4(tid, off + i * rbr, min(rbr, cnt - i * rbr), 0);
  for (int i = 0; i < nbs; ++i) {
    const int rows = min(SMALL_ROWS, cnt - i * SMALL_ROWS);
    a.d.rb[tot_l + ps + i] = make_int4(tid, off + i * SMALL_ROWS, rows, 1);
    SmallRec* r = a.d.srec + ps + i;
    r->A = my_meta.A;
    r->B = my_meta.B;
    r->rows = rows;
    r->rank = my_meta.rank;
    r->scale = my_meta.scale;
    r->adapter = tid;
  }
  if (live) a.d.m_blk[tid] = pm;
  for (int i = 0; i < nbm; ++i)
    a.d.mrb[pm + i] = make_int4(tid, moff + i * MRB_ROWS, min(MRB_ROWS, mcnt - i * MRB_ROWS), 0);

  if (flags) atomicOr(&s_flags, flags);
  __syncthreads();
  // record rows, from the entries and perm just written (visible to the whole
  // workgroup after the barrier); padding slots repeat the entry's last row
  for (int k = tid; k < tot_s * SMALL_ROWS; k += PLAN_THREADS) {
    const int q = k / SMALL_ROWS, j = k % SMALL_ROWS;
    const int4 en = a.d.rb[tot_l + q];
    a.d.srec[q].row[j] = a.d.perm[en.y + min(j, en.z - 1)];
  }
  if (tid == 0) {
    int32_t* h = a.d.hdr;
    h[HDR_FLAGS] = (int32_t)s_flags;
    h[HDR_NACT] = n_act;
    h[HDR_NRUNS] = n_runs;
    h[HDR_MNACT] = m_n_act;
    h[HDR_NRB_LARGE] = tot_l;
    h[HDR_NRB_TOTAL] = tot_l + tot_s;
    h[HDR_RB_ROWS] = rbr;
    h[HDR_NMRB] = tot_m;
    h[HDR_NSMALL] = tot_s;
  }
}

// ---------------------------------------------------------------------------
// Batches of at most PLAN_THREADS rows (decode steps).  Thread t owns row t, so
// every step is a single parallel pass and nothing is read from memory twice:
//   1. ids, mask, slot ranks and (adapter threads) slot records are loaded at
//      once, and the per-(adapter, wave) counters are cleared;
//   2. ids are validated; ballots group each wave's rows by id and the lowest
//      lane of each group stores the group's size;
//   3. a 16-wide scan per adapter turns the per-wave sizes into cursors, and
//      rows find the starts and ends of maximal runs;
//   4. one block-wide scan gives adapter offsets, entry positions and run
//      indices together; adapter threads write counts, offsets and entries;
//   5. rows scatter themselves to perm (and m_perm), to their record slot and
//      to their run (start, adapter and last row).
// ---------------------------------------------------------------------------
constexpr int SEG_STAGE = 4096;   // LDS words for the segment table

// Exclusive scan of N values per thread over the block; total[i] = sum.
template <int N, int WV = PLAN_WAVES>
__device__ __forceinline__ void block_scan_n(int (&v)[N], int (&total)[N],
                                             int (*s_w)[PLAN_WAVES]) {
  const int lane = threadIdx.x & 63, w = wave_id();
  int x[N];
#pragma unroll
  for (int i = 0; i < N; ++i) {
    x[i] = wave_incl_scan(v[i]);
    if (lane == 63) s_w[i][w] = x[i];
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int c = row_incl_scan(lane < WV ? s_w[i][lane] : 0);   // lanes 0..WV-1
    total[i] = lane_value(c, WV - 1);
    v[i] = lane_value(c, w) - lane_value(x[i], 63) + x[i] - v[i];
  }
  __syncthreads();
}

// T threads (T / 64 waves, at most 16); n <= T and num_slots <= T.  The
// per-(adapter, wave) counters keep a stride of 16 waves.
template <bool MASKED, bool SEG, int T>
__global__ __launch_bounds__(T) void plan_small_kernel(PlanLaunch a) {
  constexpr int WV = T / 64;
  __shared__ int s_rank[LORA_MAX_SLOTS];
  __shared__ unsigned short s_wc[LORA_MAX_SLOTS * PLAN_WAVES];    // [adapter][wave]
  __shared__ unsigned short s_wcm[MASKED ? LORA_MAX_SLOTS * PLAN_WAVES : 1];
  __shared__ int s_cnt[LORA_MAX_SLOTS];
  __shared__ int s_mcnt[MASKED ? LORA_MAX_SLOTS : 1];
  __shared__ int s_off[LORA_MAX_SLOTS];
  __shared__ int s_moff[MASKED ? LORA_MAX_SLOTS : 1];
  __shared__ int s_sbase[LORA_MAX_SLOTS];
  __shared__ int s_last[LORA_MAX_SLOTS];      // each group's last row
  __shared__ int s_seg[SEG ? SEG_STAGE : 1];
  __shared__ int s_efirst[WV], s_elast[WV];
  __shared__ int s_w[8][PLAN_WAVES];
  __shared__ unsigned s_flags;

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int n = a.n, S = a.num_slots, ns = a.num_segs;
  const PlanDev& d = a.d;

  // ---- 1. loads
  if (tid == 0) s_flags = 0u;
  int raw = -1, mk = 1;
  SlotMeta my{};
  if (tid < S) my = a.meta[tid];
  if (!SEG) {
    if (tid < n) raw = a.idx[tid];
  } else {
    for (int i = tid; i <= ns; i += T) s_seg[i] = a.seg_offsets[i];
    for (int i = tid; i < ns; i += T) s_seg[ns + 1 + i] = a.seg_adapter[i];
  }
  if (MASKED && tid < n) mk = a.mask[tid];
  for (int i = tid; i < S * PLAN_WAVES; i += T) {
    s_wc[i] = 0;
    if (MASKED) s_wcm[i] = 0;
  }
  if (tid < S) {
    s_rank[tid] = my.rank;
    s_last[tid] = -1;
  }
  __syncthreads();

  uint32_t flags = 0u;
  if (SEG) {
    bool bad = false;
    for (int i = tid; i <= ns; i += T) {
      const int o = s_seg[i];
      if (i == 0 && o != 0) bad = true;
      if (i == ns && o != n) bad = true;
      if (i < ns && s_seg[i + 1] < o) bad = true;
    }
    if (__syncthreads_or(bad ? 1 : 0)) {
      flags |= LORA_DATA_BAD_SEGMENTS;
    } else if (tid < n) {
      int lo = 0, hi = ns;             // s_seg[lo] <= tid < s_seg[hi]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (s_seg[mid] <= tid) lo = mid;
        else hi = mid;
      }
      raw = s_seg[ns + 1 + lo];
    }
  }

  // ---- 2. validation and per-wave group sizes
  int e = -1;
  if (tid < n) {
    int v = raw;
    if (v < -1 || v >= S) {
      flags |= LORA_DATA_BAD_ID;
      v = -1;
    } else if (v >= 0 && s_rank[v] <= 0) {
      flags |= LORA_DATA_EMPTY_SLOT;
      v = -1;
    }
    e = v;
  }
  const int em = (MASKED && !mk) ? -1 : e;
  const int nbits = 32 - __clz(S);
  const uint64_t lt = lanemask_lt();
  const uint64_t peers = match_peers(e + 1, nbits);
  const int rank_in = __popcll(peers & lt);
  if (e >= 0 && rank_in == 0) s_wc[e * PLAN_WAVES + w] = (unsigned short)__popcll(peers);
  if (e >= 0 && rank_in == __popcll(peers) - 1) atomicMax(&s_last[e], tid);
  int mrank_in = 0;
  if (MASKED) {
    const uint64_t mpeers = match_peers(em + 1, nbits);
    mrank_in = __popcll(mpeers & lt);
    if (em >= 0 && mrank_in == 0) s_wcm[em * PLAN_WAVES + w] = (unsigned short)__popcll(mpeers);
  }
  if (lane == 0) s_efirst[w] = e;
  if (lane == 63) s_elast[w] = e;
  __syncthreads();

  // ---- 3. cursors (exclusive prefix over waves) and run boundaries
  if constexpr (WV <= 4) {
    // few waves: one thread per adapter walks its WV counters
    if (tid < S) {
      int c = 0, cm = 0;
#pragma unroll
      for (int ww = 0; ww < WV; ++ww) {
        const int x = s_wc[tid * PLAN_WAVES + ww];
        s_wc[tid * PLAN_WAVES + ww] = (unsigned short)c;
        c += x;
        if (MASKED) {
          const int xm = s_wcm[tid * PLAN_WAVES + ww];
          s_wcm[tid * PLAN_WAVES + ww] = (unsigned short)cm;
          cm += xm;
        }
      }
      s_cnt[tid] = c;
      if (MASKED) s_mcnt[tid] = cm;
    }
  } else for (int k0 = 0; k0 < S * PLAN_WAVES; k0 += T) {
    const int k = k0 + tid;
    const bool act = k < S * PLAN_WAVES;
    const int v = act ? (int)s_wc[k] : 0;
    const int incl = row_incl_scan(v);
    if (act) {
      s_wc[k] = (unsigned short)(incl - v);
      if ((k & 15) == 15) s_cnt[k >> 4] = incl;
    }
    if (MASKED) {
      const int vm = act ? (int)s_wcm[k] : 0;
      const int im = row_incl_scan(vm);
      if (act) {
        s_wcm[k] = (unsigned short)(im - vm);
        if ((k & 15) == 15) s_mcnt[k >> 4] = im;
      }
    }
  }
  const int ep = lane_prev(e, w > 0 ? s_elast[w - 1] : -1);
  const int en = lane_next(e, w + 1 < WV ? s_efirst[w + 1] : -1);
  const bool st = e >= 0 && ep != e;
  const bool ed = e >= 0 && en != e;
  __syncthreads();

  // ---- 4. offsets, entry positions and run indices in one scan
  const bool live = tid < S;
  const int cnt = live ? s_cnt[tid] : 0;
  const int mcnt = MASKED ? (live ? s_mcnt[tid] : 0) : cnt;
  const bool small = live && cnt > 0 && cnt <= a.small_max;
  const bool large = live && cnt > a.small_max;
  const int nbc = large ? (cnt + RB_ROWS - 1) / RB_ROWS : 0;
  const int nbf = large ? (cnt + RB_FINE - 1) / RB_FINE : 0;
  const int nbs = small ? (cnt + SMALL_ROWS - 1) / SMALL_ROWS : 0;
  const int nbm = live ? (mcnt + MRB_ROWS - 1) / MRB_ROWS : 0;
  // eight scans as four: pairs packed in 16-bit halves (every total is at
  // most n <= 1024, so nothing carries into the upper half)
  int pv[4] = {cnt | (mcnt << 16), nbc | (nbs << 16), nbm | (nbf << 16),
               (st ? 1 : 0) | ((ed ? 1 : 0) << 16)};
  int ptot[4];
  block_scan_n<4, WV>(pv, ptot, s_w);
  int v[8], tot[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int lo = i == 0 ? 0 : i == 1 ? 2 : i == 2 ? 4 : 5;
    const int hi = i == 0 ? 1 : i == 1 ? 3 : i == 2 ? 7 : 6;
    v[lo] = pv[i] & 0xffff;
    v[hi] = (int)((unsigned)pv[i] >> 16);
    tot[lo] = ptot[i] & 0xffff;
    tot[hi] = (int)((unsigned)ptot[i] >> 16);
  }
  const int off = v[0], moff = v[1], ps = v[3], pm = v[4];
  // block size of the whole batch, chosen on the host (the launches follow it)
  const bool fine = a.fine != 0;
  const int rbr = fine ? RB_FINE : RB_ROWS, nbl = fine ? nbf : nbc, pl = fine ? v[7] : v[2];
  const int tot_l = fine ? tot[7] : tot[2];
  if (live) {
    d.counts[tid] = cnt;
    d.offsets[tid] = off;
    d.m_counts[tid] = mcnt;
    d.m_offsets[tid] = moff;
    d.m_blk[tid] = pm;
    s_off[tid] = off;
    if (MASKED) s_moff[tid] = moff;
    s_sbase[tid] = small ? ps : -1;
    for (int i = 0; i < nbl; ++i)
      d.rb[pl + i] = make_int4(tid, off + i * rbr, min(rbr, cnt - i * rbr), 0);
    for (int i = 0; i < nbs; ++i) {
      const int rows = min(SMALL_ROWS, cnt - i * SMALL_ROWS);
      d.rb[tot_l + ps + i] = make_int4(tid, off + i * SMALL_ROWS, rows, 1);
      // the record's first 32 bytes as two 16-byte stores
      int4* r4 = reinterpret_cast<int4*>(d.srec + ps + i);
      const uint64_t pa = reinterpret_cast<uint64_t>(my.A), pb = reinterpret_cast<uint64_t>(my.B);
      r4[0] = make_int4((int)(uint32_t)pa, (int)(uint32_t)(pa >> 32), (int)(uint32_t)pb,
                        (int)(uint32_t)(pb >> 32));
      r4[1] = make_int4(rows, my.rank, __float_as_int(my.scale), tid);
    }
    if (nbs > 0) {
      // padding slots of the group's last record repeat its last row (the
      // scatter below writes the real slots)
      const int lr = s_last[tid];
      int* rr = d.srec[ps + nbs - 1].row;
      int j = cnt - (nbs - 1) * SMALL_ROWS;
      for (; j < SMALL_ROWS && (j & 3) != 0; ++j) rr[j] = lr;
      for (; j < SMALL_ROWS; j += 4) *reinterpret_cast<int4*>(rr + j) = make_int4(lr, lr, lr, lr);
    }
    for (int i = 0; i < nbm; ++i)
      d.mrb[pm + i] = make_int4(tid, moff + i * MRB_ROWS, min(MRB_ROWS, mcnt - i * MRB_ROWS), 0);
  }
  if (tid == 0) {
    d.offsets[S] = tot[0];
    d.m_offsets[S] = tot[1];
  }
  if (flags) atomicOr(&s_flags, flags);
  __syncthreads();

  // ---- 5. scatter
  // (every index below is < n or < the record count by construction; the
  // guards only keep a broken invariant from writing outside the arrays)
  if (e >= 0) {
    const int o = s_off[e];
    const int pos = o + (int)s_wc[e * PLAN_WAVES + w] + rank_in;
    if ((unsigned)pos < (unsigned)n) {
      d.perm[pos] = tid;
      if (!MASKED) d.m_perm[pos] = tid;
    }
    const int sb = s_sbase[e];
    const int rel = pos - o;
    const int q = sb + rel / SMALL_ROWS;
    if (sb >= 0 && rel >= 0 && q < tot[3]) {
      SmallRec* r = d.srec + q;
      const int j = rel % SMALL_ROWS;
      r->row[j] = tid;
    }
  }
  if (MASKED && em >= 0) {
    const int pos = s_moff[em] + (int)s_wcm[em * PLAN_WAVES + w] + mrank_in;
    if ((unsigned)pos < (unsigned)n) d.m_perm[pos] = tid;
  }
  if (st && (unsigned)v[5] < (unsigned)n) {
    d.run_start[v[5]] = tid;
    d.run_adapter[v[5]] = e;
  }
  if (ed && (unsigned)v[6] < (unsigned)n) d.run_end[v[6]] = tid;
  if (tid == 0) {
    int32_t* h = d.hdr;
    h[HDR_FLAGS] = (int32_t)s_flags;
    h[HDR_NACT] = tot[0];
    h[HDR_NRUNS] = tot[5];
    h[HDR_MNACT] = tot[1];
    h[HDR_NRB_LARGE] = tot_l;
    h[HDR_NRB_TOTAL] = tot_l + tot[3];
    h[HDR_RB_ROWS] = rbr;
    h[HDR_NMRB] = tot[4];
    h[HDR_NSMALL] = tot[3];
  }
}


// ---------------------------------------------------------------------------
// Batches of (PLAN_THREADS, PLAN_MULTI_MAX] rows: two launches over chunks of
// PLAN_THREADS rows, one workgroup per chunk.
//   count:   ids validated; each row's rank among its chunk's rows of the same
//            adapter (and under the mask); per-chunk adapter histograms, run
//            starts and data flags.
//   scatter: each chunk adds the histograms of the chunks before it (and of
//            all chunks, for the adapter offsets), then its rows scatter to
//            perm, m_perm, their record slot and their run; the first chunk
//            writes counts, offsets, entry lists and the header.
// ---------------------------------------------------------------------------
template <bool MASKED, bool SEG>
__global__ __launch_bounds__(PLAN_THREADS) void plan_count_kernel(PlanLaunch a) {
  __shared__ int s_rank[LORA_MAX_SLOTS];
  __shared__ unsigned short s_wc[LORA_MAX_SLOTS * PLAN_WAVES];    // [adapter][wave]
  __shared__ unsigned short s_wcm[MASKED ? LORA_MAX_SLOTS * PLAN_WAVES : 1];
  __shared__ int s_seg[SEG ? SEG_STAGE : 1];
  __shared__ int s_elast[PLAN_WAVES];
  __shared__ int s_nst;
  __shared__ unsigned s_flags;

  const int tid = threadIdx.x, lane = tid & 63, w = wave_id();
  const int n = a.n, S = a.num_slots, ns = a.num_segs;
  const int c = blockIdx.x, t = c * PLAN_THREADS + tid;
  const PlanDev& d = a.d;

  if (tid == 0) {
    s_flags = 0u;
    s_nst = 0;
  }
  int raw = -1, rawp = -1, mk = 1;
  if (!SEG) {
    if (t < n) raw = a.idx[t];
    if (tid == 0 && t > 0) rawp = a.idx[t - 1];
  } else {
    for (int i = tid; i <= ns; i += PLAN_THREADS) s_seg[i] = a.seg_offsets[i];
    for (int i = tid; i < ns; i += PLAN_THREADS) s_seg[ns + 1 + i] = a.seg_adapter[i];
  }
  if (MASKED && t < n) mk = a.mask[t];
  for (int i = tid; i < S * PLAN_WAVES; i += PLAN_THREADS) {
    s_wc[i] = 0;
    if (MASKED) s_wcm[i] = 0;
  }
  if (tid < S) s_rank[tid] = a.meta[tid].rank;
  __syncthreads();

  uint32_t flags = 0u;
  if (SEG) {
    bool bad = false;
    for (int i = tid; i <= ns; i += PLAN_THREADS) {
      const int o = s_seg[i];
      if (i == 0 && o != 0) bad = true;
      if (i == ns && o != n) bad = true;
      if (i < ns && s_seg[i + 1] < o) bad = true;
    }
    if (__syncthreads_or(bad ? 1 : 0)) {
      flags |= LORA_DATA_BAD_SEGMENTS;
    } else {
      auto seg_of = [&](int row) {
        int lo = 0, hi = ns;             // s_seg[lo] <= row < s_seg[hi]
        while (hi - lo > 1) {
          const int mid = (lo + hi) >> 1;
          if (s_seg[mid] <= row) lo = mid;
          else hi = mid;
        }
        return s_seg[ns + 1 + lo];
      };
      if (t < n) raw = seg_of(t);
      if (tid == 0 && t > 0) rawp = seg_of(t - 1);
    }
  }
  auto validate = [&](int v, bool report) {
    if (v < -1 || v >= S) {
      if (report) flags |= LORA_DATA_BAD_ID;
      return -1;
    }
    if (v >= 0 && s_rank[v] <= 0) {
      if (report) flags |= LORA_DATA_EMPTY_SLOT;
      return -1;
    }
    return v;
  };
  const int e = t < n ? validate(raw, true) : -1;
  const int ep0 = (tid == 0 && t > 0) ? validate(rawp, false) : -1;   // previous chunk's last row
  const int em = (MASKED && !mk) ? -1 : e;
  const int nbits = 32 - __clz(S);
  const uint64_t lt = lanemask_lt();
  const uint64_t peers = match_peers(e + 1, nbits);
  const int rank_in = __popcll(peers & lt);
  if (e >= 0 && rank_in == 0) s_wc[e * PLAN_WAVES + w] = (unsigned short)__popcll(peers);
  int mrank_in = 0;
  if (MASKED) {
    const uint64_t mpeers = match_peers(em + 1, nbits);
    mrank_in = __popcll(mpeers & lt);
    if (em >= 0 && mrank_in == 0) s_wcm[em * PLAN_WAVES + w] = (unsigned short)__popcll(mpeers);
  }
  if (lane == 63) s_elast[w] = e;
  __syncthreads();

  // per adapter: exclusive prefix over waves, chunk total to the histogram
  for (int k0 = 0; k0 < S * PLAN_WAVES; k0 += PLAN_THREADS) {
    const int k = k0 + tid;
    const bool act = k < S * PLAN_WAVES;
    const int v = act ? (int)s_wc[k] : 0;
    const int incl = row_incl_scan(v);
    if (act) {
      s_wc[k] = (unsigned short)(incl - v);
      if ((k & 15) == 15) d.ch_hist[c * S + (k >> 4)] = incl;
    }
    if (MASKED) {
      const int vm = act ? (int)s_wcm[k] : 0;
      const int im = row_incl_scan(vm);
      if (act) {
        s_wcm[k] = (unsigned short)(im - vm);
        if ((k & 15) == 15) d.ch_mhist[c * S + (k >> 4)] = im;
      }
    }
  }
  const int ep = lane_prev(e, w > 0 ? s_elast[w - 1] : ep0);
  const uint64_t stb = __ballot(e >= 0 && ep != e);
  if (lane == 0 && stb) atomicAdd(&s_nst, __popcll(stb));
  __syncthreads();

  if (t < n) {
    d.seg_ids[t] = e >= 0 ? (e + 1) | (((int)s_wc[e * PLAN_WAVES + w] + rank_in) << 16) : 0;
    if (MASKED)
      d.minfo[t] = em >= 0 ? (em + 1) | (((int)s_wcm[em * PLAN_WAVES + w] + mrank_in) << 16) : 0;
  }
  if (flags) atomicOr(&s_flags, flags);
  __syncthreads();
  if (tid == 0) {
    d.ch_runs[c] = s_nst;
    d.ch_flags[c] = (int32_t)s_flags;
  }
}

template <bool MASKED>
__global__ __launch_bounds__(PLAN_THREADS) void plan_scatter_kernel(PlanLaunch a) {
  __shared__ int s_base[LORA_MAX_SLOTS];      // adapter offset + its rows in earlier chunks
  __shared__ int s_mbase[MASKED ? LORA_MAX_SLOTS : 1];
  __shared__ int s_off[LORA_MAX_SLOTS];
  __shared__ int s_cnt[LORA_MAX_SLOTS];
  __shared__ int s_sbase[LORA_MAX_SLOTS];
  __shared__ int s_w[8][PLAN_WAVES];
  __shared__ int s_misc[4];

  const int tid = threadIdx.x;
  const int n = a.n, S = a.num_slots;
  const PlanDev& d = a.d;
  const int C = d.chunks, c = blockIdx.x, t = c * PLAN_THREADS + tid;
  const int t0 = c * PLAN_THREADS;

  // this chunk's rows (and their neighbours, for the run boundaries)
  const int info = t < n ? d.seg_ids[t] : 0;
  const int infop = (t > 0 && t - 1 < n) ? d.seg_ids[t - 1] : 0;
  const int infon = t + 1 < n ? d.seg_ids[t + 1] : 0;
  const int minf = (MASKED && t < n) ? d.minfo[t] : 0;

  // per adapter: rows in all chunks and in the chunks before this one
  int cnt = 0, pre = 0, mcnt = 0, mpre = 0;
  if (tid < S) {
    for (int cc = 0; cc < C; ++cc) {
      const int v = d.ch_hist[cc * S + tid];
      cnt += v;
      pre += cc < c ? v : 0;
      if (MASKED) {
        const int vm = d.ch_mhist[cc * S + tid];
        mcnt += vm;
        mpre += cc < c ? vm : 0;
      }
    }
  }
  if (!MASKED) {
    mcnt = cnt;
    mpre = pre;
  }
  if (tid == 0) {
    int rpre = 0, rtot = 0;
    uint32_t fl = 0u;
    for (int cc = 0; cc < C; ++cc) {
      const int r = d.ch_runs[cc];
      rtot += r;
      rpre += cc < c ? r : 0;
      fl |= (uint32_t)d.ch_flags[cc];
    }
    // a run that crosses into this chunk ends here, not before it
    const int eb = t0 > 0 ? (d.seg_ids[t0 - 1] & 0xffff) - 1 : -1;
    const int ef = (d.seg_ids[t0] & 0xffff) - 1;
    s_misc[0] = rpre;
    s_misc[1] = rtot;
    s_misc[2] = (int)fl;
    s_misc[3] = rpre - ((eb >= 0 && eb == ef) ? 1 : 0);
  }

  const int e = (info & 0xffff) - 1;
  const int ep = t > 0 ? (infop & 0xffff) - 1 : -1;
  const int en = t + 1 < n ? (infon & 0xffff) - 1 : -1;
  const bool st = e >= 0 && ep != e;
  const bool ed = e >= 0 && en != e;

  const bool live = tid < S;
  const bool small = live && cnt > 0 && cnt <= a.small_max;
  const bool large = live && cnt > a.small_max;
  const int nbc = large ? (cnt + RB_ROWS - 1) / RB_ROWS : 0;
  const int nbf = large ? (cnt + RB_FINE - 1) / RB_FINE : 0;
  const int nbs = small ? (cnt + SMALL_ROWS - 1) / SMALL_ROWS : 0;
  const int nbm = live ? (mcnt + MRB_ROWS - 1) / MRB_ROWS : 0;
  int v[8] = {cnt, mcnt, nbc, nbs, nbm, st ? 1 : 0, ed ? 1 : 0, nbf};
  int tot[8];
  block_scan_n<8>(v, tot, s_w);            // (barriers inside: s_misc is visible after it)
  const int off = v[0], moff = v[1], ps = v[3], pm = v[4];
  // block size of the whole batch, chosen on the host (the launches follow it)
  const bool fine = a.fine != 0;
  const int rbr = fine ? RB_FINE : RB_ROWS, nbl = fine ? nbf : nbc, pl = fine ? v[7] : v[2];
  const int tot_l = fine ? tot[7] : tot[2];
  if (live) {
    s_base[tid] = off + pre;
    if (MASKED) s_mbase[tid] = moff + mpre;
    s_off[tid] = off;
    s_cnt[tid] = cnt;
    s_sbase[tid] = small ? ps : -1;
  }
  if (c == 0) {
    if (live) {
      const SlotMeta my = a.meta[tid];
      d.counts[tid] = cnt;
      d.offsets[tid] = off;
      d.m_counts[tid] = mcnt;
      d.m_offsets[tid] = moff;
      d.m_blk[tid] = pm;
      for (int i = 0; i < nbl; ++i)
        d.rb[pl + i] = make_int4(tid, off + i * rbr, min(rbr, cnt - i * rbr), 0);
      for (int i = 0; i < nbs; ++i) {
        const int rows = min(SMALL_ROWS, cnt - i * SMALL_ROWS);
        d.rb[tot_l + ps + i] = make_int4(tid, off + i * SMALL_ROWS, rows, 1);
        SmallRec* r = d.srec + ps + i;
        r->A = my.A;
        r->B = my.B;
        r->rows = rows;
        r->rank = my.rank;
        r->scale = my.scale;
        r->adapter = tid;
      }
      for (int i = 0; i < nbm; ++i)
        d.mrb[pm + i] = make_int4(tid, moff + i * MRB_ROWS, min(MRB_ROWS, mcnt - i * MRB_ROWS), 0);
    }
    if (tid == 0) {
      d.offsets[S] = tot[0];
      d.m_offsets[S] = tot[1];
      int32_t* h = d.hdr;
      h[HDR_FLAGS] = s_misc[2];
      h[HDR_NACT] = tot[0];
      h[HDR_NRUNS] = s_misc[1];
      h[HDR_MNACT] = tot[1];
      h[HDR_NRB_LARGE] = tot_l;
      h[HDR_NRB_TOTAL] = tot_l + tot[3];
      h[HDR_RB_ROWS] = rbr;
      h[HDR_NMRB] = tot[4];
      h[HDR_NSMALL] = tot[3];
    }
  }
  __syncthreads();

  // (every index below is < n or < the record count by construction; the
  // guards only keep a broken invariant from writing outside the arrays)
  if (e >= 0) {
    const int pos = s_base[e] + (info >> 16);
    if ((unsigned)pos < (unsigned)n) {
      d.perm[pos] = t;
      if (!MASKED) d.m_perm[pos] = t;
    }
    const int sb = s_sbase[e];
    const int rel = pos - s_off[e];
    const int q = sb + rel / SMALL_ROWS;
    if (sb >= 0 && rel >= 0 && q < tot[3]) {
      SmallRec* r = d.srec + q;
      const int j = rel % SMALL_ROWS;
      r->row[j] = t;
      if (rel == s_cnt[e] - 1)
        for (int jj = j + 1; jj < SMALL_ROWS; ++jj) r->row[jj] = t;
    }
  }
  if (MASKED) {
    const int em = (minf & 0xffff) - 1;
    if (em >= 0) {
      const int pos = s_mbase[em] + (minf >> 16);
      if ((unsigned)pos < (unsigned)n) d.m_perm[pos] = t;
    }
  }
  const int ks = s_misc[0] + v[5], ke = s_misc[3] + v[6];
  if (st && (unsigned)ks < (unsigned)n) {
    d.run_start[ks] = t;
    d.run_adapter[ks] = e;
  }
  if (ed && (unsigned)ke < (unsigned)n) d.run_end[ke] = t;
}

}  // namespace

hipError_t launch_plan(const PlanLaunch& a, hipStream_t s) {
  const bool seg = a.seg_offsets != nullptr;
  if (a.n <= PLAN_THREADS && (!seg || 2 * a.num_segs + 1 <= SEG_STAGE)) {
    const bool m = a.mask != nullptr;
    // a quarter of the threads (fewer waves at every barrier and scan) when
    // the rows and the slots fit
    if (a.n <= 256 && a.num_slots <= 256) {
      if (m && seg) hipLaunchKernelGGL((plan_small_kernel<true, true, 256>), dim3(1), dim3(256), 0, s, a);
      else if (m) hipLaunchKernelGGL((plan_small_kernel<true, false, 256>), dim3(1), dim3(256), 0, s, a);
      else if (seg) hipLaunchKernelGGL((plan_small_kernel<false, true, 256>), dim3(1), dim3(256), 0, s, a);
      else hipLaunchKernelGGL((plan_small_kernel<false, false, 256>), dim3(1), dim3(256), 0, s, a);
      return hipGetLastError();
    }
    constexpr int T = PLAN_THREADS;
    if (m && seg) hipLaunchKernelGGL((plan_small_kernel<true, true, T>), dim3(1), dim3(T), 0, s, a);
    else if (m) hipLaunchKernelGGL((plan_small_kernel<true, false, T>), dim3(1), dim3(T), 0, s, a);
    else if (seg) hipLaunchKernelGGL((plan_small_kernel<false, true, T>), dim3(1), dim3(T), 0, s, a);
    else hipLaunchKernelGGL((plan_small_kernel<false, false, T>), dim3(1), dim3(T), 0, s, a);
    return hipGetLastError();
  }
  if (a.d.chunks > 0 && (!seg || 2 * a.num_segs + 1 <= SEG_STAGE)) {
    const dim3 g(a.d.chunks), b(PLAN_THREADS);
    const bool m = a.mask != nullptr;
    if (m && seg) hipLaunchKernelGGL((plan_count_kernel<true, true>), g, b, 0, s, a);
    else if (m) hipLaunchKernelGGL((plan_count_kernel<true, false>), g, b, 0, s, a);
    else if (seg) hipLaunchKernelGGL((plan_count_kernel<false, true>), g, b, 0, s, a);
    else hipLaunchKernelGGL((plan_count_kernel<false, false>), g, b, 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (m) hipLaunchKernelGGL((plan_scatter_kernel<true>), g, b, 0, s, a);
    else hipLaunchKernelGGL((plan_scatter_kernel<false>), g, b, 0, s, a);
    return hipGetLastError();
  }
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
