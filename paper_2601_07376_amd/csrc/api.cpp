// Host side of the C ABI: argument validation, the adapter table, plan objects,
// workspace carving and kernel dispatch.  Nothing here allocates device memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstddef>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "lora_internal.h"

struct lora_table {
  int32_t num_slots, d_in, d_out;
  lora_dtype w_dtype;
  void* dev_meta;
  std::vector<lora::SlotMeta> host;
};

struct lora_plan {
  const lora_table* table;
  int32_t n;
  void* ws;
  lora::PlanLayout L;
  lora::PlanDev d;
  int32_t r_max;        // largest live rank when the plan was built
  bool rank8;           // every live rank is a multiple of 8
  int32_t small_max;    // groups of <= small_max rows use the fused small-group kernel
  bool fine;            // large groups in blocks of RB_FINE rows (else RB_ROWS)
  lora_policy pol;      // path selection of the ops on this plan (-1 fields: library choice)
};

namespace {

thread_local std::string g_err;

lora_status fail(lora_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

lora_status ok() {
  g_err.clear();
  return LORA_OK;
}

lora_status hip_fail(hipError_t e, const char* what) {
  return fail(LORA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t al256(size_t x) { return (x + 255) & ~size_t(255); }

bool valid_dtype(lora_dtype d) { return d == LORA_F32 || d == LORA_BF16; }

size_t dsize(lora_dtype d) { return d == LORA_BF16 ? 2 : 4; }

// Output-column chunks per small-group entry (sibling workgroups).
int32_t small_chunks_policy(const lora_plan* p) {
  if (p->pol.small_chunks > 0) return p->pol.small_chunks;
  return std::max(1, std::min(16, (p->table->d_out + 1023) / 1024));
}

// Most d-slices of the gradient's first stage (the kernel uses fewer when
// there are enough row blocks to fill the chip).
int32_t grad_splits_policy(const lora_plan* p) {
  if (p->pol.grad_splits > 0) return std::min(p->pol.grad_splits, lora::GRAD_SPLITS_MAX);
  const int32_t d = std::min(p->table->d_in, p->table->d_out);
  return std::max(1, std::min(lora::GRAD_SPLITS_MAX, (d + 511) / 512));   // slices of >= 512
}

// Each field is -1 (the library's choice) or inside its documented range.
lora_status check_policy(const lora_policy& q) {
  const bool ok = q.small_max >= -1 && q.small_split >= -1 && q.small_split <= 1 &&
                  (q.split_slices == -1 || (q.split_slices >= 1 && q.split_slices <= lora::SPLIT_SLICES_MAX)) &&
                  (q.small_chunks == -1 || (q.small_chunks >= 1 && q.small_chunks <= 16)) &&
                  q.fork >= -1 && q.fork <= 1 &&
                  (q.grad_splits == -1 || (q.grad_splits >= 1 && q.grad_splits <= lora::GRAD_SPLITS_MAX)) &&
                  (q.block_rows == -1 || q.block_rows == lora::RB_FINE || q.block_rows == lora::RB_ROWS);
  if (!ok)
    return fail(LORA_ERR_VALUE, "policy field out of range (small_max %d, small_split %d, split_slices %d, "
                "small_chunks %d, fork %d, grad_splits %d, block_rows %d)", q.small_max, q.small_split,
                q.split_slices, q.small_chunks, q.fork, q.grad_splits, q.block_rows);
  return LORA_OK;
}

lora_policy default_policy() {
  lora_policy q;
  q.small_max = q.small_split = q.split_slices = q.small_chunks = q.fork = q.grad_splits = -1;
  q.block_rows = -1;
  return q;
}

// host upper bounds of the entry lists
int32_t ub_large(const lora_plan* p) {
  if (p->small_max == INT32_MAX) return 0;
  const int32_t S = p->table->num_slots, n = p->n;
  return n / lora::RB_FINE + std::min(S, n / (p->small_max + 1)) + 1;   // either block size
}
// ... in the block size the plan uses, and 0 for the other one: the grouped
// launches of that size are skipped
int32_t ub_coarse(const lora_plan* p) {
  if (p->small_max == INT32_MAX || p->fine) return 0;
  const int32_t S = p->table->num_slots, n = p->n;
  return n / lora::RB_ROWS + std::min(S, n / (p->small_max + 1)) + 1;
}
int32_t ub_fine(const lora_plan* p) { return p->fine ? ub_large(p) : 0; }
int32_t ub_small(const lora_plan* p) {
  const int32_t S = p->table->num_slots, n = p->n;
  const int64_t all = n / lora::SMALL_ROWS + std::min(S, n) + 1;
  if (p->small_max == INT32_MAX) return (int32_t)all;
  const int64_t per = ((int64_t)p->small_max + lora::SMALL_ROWS - 1) / lora::SMALL_ROWS;
  return (int32_t)std::min<int64_t>(all, (int64_t)std::min(S, n) * per + 1);
}
int32_t ub_mrb(const lora_plan* p) {
  return p->n / lora::MRB_ROWS + std::min(p->table->num_slots, p->n) + 1;
}

lora::OpLaunch op_base(const lora_plan* p) {
  lora::OpLaunch o{};
  o.hdr = p->d.hdr;
  o.rb = p->d.rb;
  o.srec = p->d.srec;
  o.perm = p->d.perm;
  o.meta = static_cast<const lora::SlotMeta*>(p->table->dev_meta);
  o.n = p->n;
  o.d_in = p->table->d_in;
  o.d_out = p->table->d_out;
  o.num_slots = p->table->num_slots;
  o.r_max = p->r_max;
  o.rank8 = p->rank8;
  return o;
}

// rows == 0: the matrix is never touched and may be NULL
lora_status check_matrix(const void* ptr, lora_dtype dt, int64_t ld, int32_t cols,
                         const char* name, int32_t rows = 1) {
  if (ptr == nullptr && rows == 0) return valid_dtype(dt) ? LORA_OK : fail(LORA_ERR_DTYPE, "%s: unknown dtype %d", name, (int)dt);
  if (ptr == nullptr) return fail(LORA_ERR_NULL, "%s is NULL", name);
  if (!valid_dtype(dt)) return fail(LORA_ERR_DTYPE, "%s: unknown dtype %d", name, (int)dt);
  if (ld < cols) return fail(LORA_ERR_SHAPE, "%s: leading dim %lld < %d", name, (long long)ld, cols);
  if (ld % 8 != 0) return fail(LORA_ERR_ALIGN, "%s: leading dim %lld not a multiple of 8", name, (long long)ld);
  if (!aligned(ptr, 16)) return fail(LORA_ERR_ALIGN, "%s not 16-byte aligned", name);
  return LORA_OK;
}

lora_status check_plan(const lora_plan* p) {
  if (p == nullptr) return fail(LORA_ERR_NULL, "plan is NULL");
  return LORA_OK;
}

// ---- debug build: outputs disjoint from inputs and from each other ------------
#ifndef LORA_DEBUG
#define LORA_DEBUG 0
#endif
constexpr bool kDebug = LORA_DEBUG != 0;

// Bytes [lo, hi) of one buffer of an op (empty when lo == hi).
struct Span {
  uintptr_t lo, hi;
  const char* what;
  int32_t slot;        // adapter weights and gradients: their slot, else -1
};

// rows x cols elements of es bytes, rows ld elements apart
Span rows_span(const void* ptr, int64_t rows, int64_t cols, int64_t ld, size_t es, const char* what,
               int32_t slot = -1) {
  if (ptr == nullptr || rows <= 0 || cols <= 0) return Span{0, 0, what, slot};
  const uintptr_t lo = reinterpret_cast<uintptr_t>(ptr);
  return Span{lo, lo + (uintptr_t)(((rows - 1) * ld + cols) * (int64_t)es), what, slot};
}
Span bytes_span(const void* ptr, size_t bytes, const char* what) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(ptr);
  return ptr == nullptr ? Span{0, 0, what, -1} : Span{lo, lo + bytes, what, -1};
}

// The buffers one call reads (inputs) and writes (outputs).  check() fails
// with LORA_ERR_ALIAS when an output overlaps an input or another output.
class Disjoint {
 public:
  explicit Disjoint(const char* op) : op_(op) {}
  void in(const Span& s) {
    if (s.lo < s.hi) ins_.push_back(s);
  }
  void out(const Span& s) {
    if (s.lo < s.hi) outs_.push_back(s);
  }
  // the device copy of the slot table and every live slot's A and B
  void weights(const lora_table* t) {
    in(bytes_span(t->dev_meta, (size_t)t->num_slots * sizeof(lora::SlotMeta), "the slot table"));
    const size_t es = dsize(t->w_dtype);
    for (int32_t a = 0; a < t->num_slots; ++a) {
      const lora::SlotMeta& m = t->host[a];
      if (m.rank <= 0) continue;
      in(rows_span(m.A, m.rank, t->d_in, t->d_in, es, "A", a));
      in(rows_span(m.B, t->d_out, m.rank, m.rank, es, "B", a));
    }
  }
  void plan(const lora_plan* p) { in(bytes_span(p->ws, p->L.total, "the plan workspace")); }
  lora_status check() {
    auto by_lo = [](const Span& a, const Span& b) { return a.lo < b.lo; };
    std::sort(outs_.begin(), outs_.end(), by_lo);
    for (size_t i = 0; i + 1 < outs_.size(); ++i)      // sorted: an overlap shows between neighbours
      if (outs_[i + 1].lo < outs_[i].hi) return report(outs_[i], outs_[i + 1]);
    std::sort(ins_.begin(), ins_.end(), by_lo);
    std::vector<uintptr_t> hi_max(ins_.size());
    for (size_t i = 0; i < ins_.size(); ++i) hi_max[i] = std::max(ins_[i].hi, i ? hi_max[i - 1] : 0);
    for (const Span& o : outs_) {
      // inputs starting before o ends; one of them reaches past o's start?
      const size_t k = std::lower_bound(ins_.begin(), ins_.end(), Span{o.hi, o.hi, "", -1}, by_lo) -
                       ins_.begin();
      if (k == 0 || hi_max[k - 1] <= o.lo) continue;
      for (size_t i = k; i-- > 0;)
        if (ins_[i].hi > o.lo) return report(o, ins_[i]);
    }
    return LORA_OK;
  }

 private:
  lora_status report(const Span& a, const Span& b) {
    char sa[48] = "", sb[48] = "";
    if (a.slot >= 0) snprintf(sa, sizeof(sa), " of slot %d", a.slot);
    if (b.slot >= 0) snprintf(sb, sizeof(sb), " of slot %d", b.slot);
    return fail(LORA_ERR_ALIAS, "%s: %s%s overlaps %s%s", op_, a.what, sa, b.what, sb);
  }
  const char* op_;
  std::vector<Span> ins_, outs_;
};

lora_status make_plan(const lora_table* t, int32_t n, const int32_t* idx,
                      const int32_t* seg_offsets, const int32_t* seg_adapter, int32_t num_segs,
                      const uint8_t* mask, const lora_policy* policy, void* ws, size_t ws_bytes,
                      hipStream_t stream, lora_plan** out) {
  if (out == nullptr) return fail(LORA_ERR_NULL, "out is NULL");
  *out = nullptr;
  if (t == nullptr) return fail(LORA_ERR_NULL, "table is NULL");
  const lora_policy pol = policy != nullptr ? *policy : default_policy();
  {
    const lora_status st = check_policy(pol);
    if (st != LORA_OK) return st;
  }
  if (n < 0 || n > LORA_MAX_ROWS) return fail(LORA_ERR_SHAPE, "n = %d outside [0, %d]", n, LORA_MAX_ROWS);
  if (ws == nullptr) return fail(LORA_ERR_NULL, "plan workspace is NULL");
  if (!aligned(ws, 16)) return fail(LORA_ERR_ALIGN, "plan workspace not 16-byte aligned");
  const lora::PlanLayout L = lora::plan_layout(n, t->num_slots);
  if (ws_bytes < L.total)
    return fail(LORA_ERR_WORKSPACE, "plan workspace %zu bytes < %zu", ws_bytes, L.total);
  if (seg_offsets == nullptr && n > 0 && idx == nullptr) return fail(LORA_ERR_NULL, "idx is NULL");
  if (idx != nullptr && !aligned(idx, 4)) return fail(LORA_ERR_ALIGN, "idx not 4-byte aligned");

  lora_plan* p = new (std::nothrow) lora_plan();
  if (p == nullptr) return fail(LORA_ERR_SHAPE, "host allocation failed");
  p->table = t;
  p->n = n;
  p->ws = ws;
  p->L = L;
  char* b = static_cast<char*>(ws);
  p->d.hdr = reinterpret_cast<int32_t*>(b + L.hdr);
  p->d.counts = reinterpret_cast<int32_t*>(b + L.counts);
  p->d.offsets = reinterpret_cast<int32_t*>(b + L.offsets);
  p->d.perm = reinterpret_cast<int32_t*>(b + L.perm);
  p->d.run_start = reinterpret_cast<int32_t*>(b + L.run_start);
  p->d.run_end = reinterpret_cast<int32_t*>(b + L.run_end);
  p->d.run_adapter = reinterpret_cast<int32_t*>(b + L.run_adapter);
  p->d.m_counts = reinterpret_cast<int32_t*>(b + L.m_counts);
  p->d.m_offsets = reinterpret_cast<int32_t*>(b + L.m_offsets);
  p->d.m_perm = reinterpret_cast<int32_t*>(b + L.m_perm);
  p->d.m_blk = reinterpret_cast<int32_t*>(b + L.m_blk);
  p->d.rb = reinterpret_cast<int4*>(b + L.rb);
  p->d.mrb = reinterpret_cast<int4*>(b + L.mrb);
  p->d.srec = reinterpret_cast<lora::SmallRec*>(b + L.srec);
  p->d.seg_ids = reinterpret_cast<int32_t*>(b + L.seg_ids);
  p->d.ch_hist = reinterpret_cast<int32_t*>(b + L.ch_hist);
  p->d.ch_mhist = reinterpret_cast<int32_t*>(b + L.ch_mhist);
  p->d.ch_runs = reinterpret_cast<int32_t*>(b + L.ch_runs);
  p->d.ch_flags = reinterpret_cast<int32_t*>(b + L.ch_flags);
  p->d.minfo = reinterpret_cast<int32_t*>(b + L.minfo);
  p->d.chunks = L.chunks;
  p->r_max = 0;
  p->rank8 = true;
  for (const auto& s : t->host) {
    if (s.rank <= 0) continue;
    p->r_max = std::max(p->r_max, s.rank);
    p->rank8 = p->rank8 && (s.rank % 8 == 0);
  }
  p->pol = pol;
  p->small_max = pol.small_max >= 0 ? pol.small_max : lora::small_max_policy(n, t->num_slots);
  p->fine = pol.block_rows >= 0 ? pol.block_rows == lora::RB_FINE : lora::fine_policy(n);

  lora::PlanLaunch a{};
  a.d = p->d;
  a.idx = seg_offsets ? nullptr : idx;
  a.seg_offsets = seg_offsets;
  a.seg_adapter = seg_adapter;
  a.num_segs = num_segs;
  a.mask = mask;
  a.meta = static_cast<const lora::SlotMeta*>(t->dev_meta);
  a.n = n;
  a.num_slots = t->num_slots;
  a.small_max = p->small_max;
  a.fine = p->fine ? 1 : 0;
  hipError_t e = lora::launch_plan(a, stream);
  if (e != hipSuccess) {
    delete p;
    return hip_fail(e, "plan kernel launch");
  }
  *out = p;
  return ok();
}

}  // namespace

namespace lora {

// Small-group policy.  Batches of up to 1024 rows (decode steps) send every
// adapter group through the small-group kernels.  Larger batches with fewer
// than 4 SMALL_ROWS rows per slot send groups of up to 2 SMALL_ROWS rows there
// (two records each at most; many small groups are then likely, and they run
// beside the large ones on the second stream: the skewed mixed batch measured
// 92.4 against 95.8 us per apply with a limit of SMALL_ROWS), and the larger
// groups through the grouped shrink + expand.  Other batches send none: a few
// small groups cost less as blocks of the grouped kernels than two more
// launches.
int32_t small_max_policy(int32_t n, int32_t S) {
  if (n <= 1024) return INT32_MAX;
  return (int64_t)n < (int64_t)4 * SMALL_ROWS * S ? 2 * SMALL_ROWS : 0;
}
// Large-group blocks of RB_FINE rows below FINE_BELOW coarse blocks' worth of
// rows (RB_ROWS blocks could not cover the chip), else RB_ROWS.  Chosen on the
// host, so only the grouped kernels of that block size are launched.
bool fine_policy(int32_t n) { return (int64_t)n < (int64_t)FINE_BELOW * RB_ROWS; }

// Gradient workspace: fp32 partial planes (two per d-slice) and the summed bf16
// hi / lo planes.
GradLayout grad_layout(int32_t mrb_ub, int32_t r_max) {
  GradLayout G{};
  const size_t r_pad = (size_t)(std::max(r_max, 1) + 15) / 16 * 16;
  const size_t p_stride = (size_t)mrb_ub * MRB_ROWS;
  size_t o = 0;
  G.partial = o; o += al256(2 * GRAD_SPLITS_MAX * r_pad * p_stride * 4);
  G.fin = o;     o += al256(2 * 2 * r_pad * p_stride * 2);
  G.total = o;
  return G;
}

PlanLayout plan_layout(int32_t n, int32_t S) {
  PlanLayout L{};
  const size_t nn = (size_t)std::max(n, 1);
  size_t o = 0;
  L.hdr = o;         o += al256(HDR_WORDS * 4);
  L.counts = o;      o += al256((size_t)S * 4);
  L.offsets = o;     o += al256((size_t)(S + 1) * 4);
  L.perm = o;        o += al256(nn * 4);
  L.run_start = o;   o += al256(nn * 4);
  L.run_end = o;     o += al256(nn * 4);
  L.run_adapter = o; o += al256(nn * 4);
  L.m_counts = o;    o += al256((size_t)S * 4);
  L.m_offsets = o;   o += al256((size_t)(S + 1) * 4);
  L.m_perm = o;      o += al256(nn * 4);
  L.m_blk = o;       o += al256((size_t)S * 4);
  L.rb_max = n / SMALL_ROWS + std::min(S, n) + 1;
  L.mrb_max = n / MRB_ROWS + std::min(S, n) + 1;
  L.rb = o;          o += al256((size_t)L.rb_max * 16);
  L.mrb = o;         o += al256((size_t)L.mrb_max * 16);
  // small-group records: every group may be small (whatever the plan's
  // small-group bound, so the size depends on n and S alone)
  L.srec_max = std::max(L.rb_max, 1);
  L.srec = o;        o += al256((size_t)L.srec_max * sizeof(SmallRec));
  L.seg_ids = o;     o += al256(nn * 4);
  L.chunks = (n > PLAN_THREADS && n <= PLAN_MULTI_MAX) ? (n + PLAN_THREADS - 1) / PLAN_THREADS : 0;
  const size_t ch = (size_t)L.chunks;
  L.ch_hist = o;     o += al256(ch * S * 4);
  L.ch_mhist = o;    o += al256(ch * S * 4);
  L.ch_runs = o;     o += al256(ch * 4);
  L.ch_flags = o;    o += al256(ch * 4);
  L.minfo = o;       o += al256(ch ? nn * 4 : 0);
  L.total = o;
  return L;
}

}  // namespace lora

namespace {

// A second stream per device (default priority) for the small-group path of
// a mixed batch, which runs beside the grouped path: the two write disjoint
// rows of Y and disjoint parts of the workspace.  Created at the first call
// that can use it outside stream capture; the fork and join are events, so a
// captured call records both streams into the caller's graph.  One mutex
// orders the host-side fork sequences of concurrent callers.
struct AuxStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
constexpr int AUX_DEVICES = 64;
std::mutex g_aux_mutex;
AuxStream g_aux[AUX_DEVICES];

// Whether the second stream can join `caller` now.  A stream that joined a
// capture stays part of it until that capture ends, so the fork is taken only
// when the second stream is outside every capture (the caller may be capturing:
// the fork then brings the second stream into the caller's capture), or when
// both are in the same capture sequence (a later call of the same capture).
// Otherwise (an eager call while another stream's capture holds the second
// stream, or two different captures) the call runs on the caller's stream
// alone.  The host mutex orders these checks with the forks that follow them.
bool can_fork(hipStream_t caller, hipStream_t aux) {
  hipStreamCaptureStatus cc = hipStreamCaptureStatusNone, ca = hipStreamCaptureStatusNone;
  unsigned long long ic = 0, ia = 0;
  if (hipStreamGetCaptureInfo(caller, &cc, &ic) != hipSuccess) return false;
  if (hipStreamGetCaptureInfo(aux, &ca, &ia) != hipSuccess) return false;
  if (cc == hipStreamCaptureStatusInvalidated || ca == hipStreamCaptureStatusInvalidated) return false;
  if (ca == hipStreamCaptureStatusNone) return true;
  return cc == hipStreamCaptureStatusActive && ca == hipStreamCaptureStatusActive && ic == ia;
}

// the device's second stream, or nullptr (forking off, creation refused
// during capture, the second stream held by another capture, or a creation
// failure: the caller then runs one stream)
AuxStream* aux_stream(hipStream_t caller) {
  // the caller's stream decides the device (the null stream: the current one)
  int cur = 0, dev = 0;
  if (hipGetDevice(&cur) != hipSuccess) return nullptr;
  dev = cur;
  if (caller != nullptr && hipStreamGetDevice(caller, &dev) != hipSuccess) return nullptr;
  if (dev < 0 || dev >= AUX_DEVICES) return nullptr;
  AuxStream& a = g_aux[dev];
  if (a.s != nullptr) return can_fork(caller, a.s) ? &a : nullptr;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(caller, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return nullptr;
  if (dev != cur && hipSetDevice(dev) != hipSuccess) return nullptr;
  hipStream_t s = nullptr;
  hipEvent_t f = nullptr, j = nullptr;
  bool made = hipStreamCreateWithFlags(&s, hipStreamNonBlocking) == hipSuccess;
  // the fork and join order work of this one device: no system-scope fence
  // (measured 81.3 against 85.7 us per skewed-batch apply)
  const unsigned ef = hipEventDisableTiming | hipEventDisableSystemFence;
  made = made && hipEventCreateWithFlags(&f, ef) == hipSuccess;
  made = made && hipEventCreateWithFlags(&j, ef) == hipSuccess;
  if (!made) {
    if (j != nullptr) (void)hipEventDestroy(j);
    if (f != nullptr) (void)hipEventDestroy(f);
    if (s != nullptr) (void)hipStreamDestroy(s);
  } else {
    a.s = s;
    a.fork = f;
    a.join = j;
  }
  if (dev != cur) (void)hipSetDevice(cur);
  return made ? &a : nullptr;
}

// Whether a grouped batch forks its small-group path.  The fork and join cost
// about 10 us of queue latency, so they pay only when both paths have work;
// the host cannot see the grouping (it is built on the device), so it expects
// small groups when the batch has fewer than 4 x SMALL_ROWS rows per table
// slot.
bool fork_policy(const lora_plan* p) {
  if (p->pol.fork >= 0) return p->pol.fork == 1;
  return (int64_t)p->n < (int64_t)4 * lora::SMALL_ROWS * p->table->num_slots;
}

}  // namespace

extern "C" {

int32_t lora_abi_version(void) { return LORA_ABI_VERSION; }

const char* lora_status_string(lora_status s) {
  switch (s) {
    case LORA_OK: return "ok";
    case LORA_ERR_NULL: return "null pointer";
    case LORA_ERR_SHAPE: return "bad shape";
    case LORA_ERR_DTYPE: return "unsupported dtype";
    case LORA_ERR_ALIGN: return "misaligned pointer or leading dimension";
    case LORA_ERR_RANK: return "rank out of range";
    case LORA_ERR_SLOT: return "slot out of range";
    case LORA_ERR_DATA: return "device data error (bad ids or segments)";
    case LORA_ERR_WORKSPACE: return "workspace too small";
    case LORA_ERR_HIP: return "HIP runtime error";
    case LORA_ERR_VALUE: return "hyperparameter or step number out of range";
    case LORA_ERR_ALIAS: return "an output overlaps an input or another output";
  }
  return "unknown status";
}

const char* lora_last_error(void) { return g_err.c_str(); }

int32_t lora_build_flags(void) { return kDebug ? LORA_BUILD_DEBUG : 0; }

lora_status lora_debug_plan_poke(lora_plan* p, int32_t array, int32_t index, int32_t value,
                                 void* stream) {
  if (!kDebug) return fail(LORA_ERR_VALUE, "lora_debug_plan_poke: debug build only");
  if (p == nullptr) return fail(LORA_ERR_NULL, "plan is NULL");
  int32_t* base = nullptr;
  int64_t len = 0, word = index;
  switch (array) {
    case LORA_PLAN_PERM: base = p->d.perm; len = p->n; break;
    case LORA_PLAN_M_PERM: base = p->d.m_perm; len = p->n; break;
    case LORA_PLAN_SMALL_ROW:          // row index % 16 of record index / 16
      base = reinterpret_cast<int32_t*>(p->d.srec);
      len = (int64_t)p->L.srec_max * lora::SMALL_ROWS;
      word = (int64_t)(index / lora::SMALL_ROWS) * (sizeof(lora::SmallRec) / 4) +
             offsetof(lora::SmallRec, row) / 4 + index % lora::SMALL_ROWS;
      break;
    default: return fail(LORA_ERR_VALUE, "lora_debug_plan_poke: unknown array %d", array);
  }
  if (index < 0 || index >= len)
    return fail(LORA_ERR_VALUE, "lora_debug_plan_poke: index %d outside [0, %lld)", index, (long long)len);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(base + word, &value, 4, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);     // `value` lives on this stack
  if (e != hipSuccess) return hip_fail(e, "plan poke");
  return ok();
}

// ---- table -----------------------------------------------------------------

size_t lora_table_device_bytes(int32_t num_slots) {
  if (num_slots <= 0) return 0;
  return (size_t)num_slots * sizeof(lora::SlotMeta);
}

lora_status lora_table_create(int32_t num_slots, int32_t d_in, int32_t d_out, lora_dtype w_dtype,
                              void* dev_meta, size_t dev_meta_bytes, lora_table** out) {
  if (out == nullptr) return fail(LORA_ERR_NULL, "out is NULL");
  *out = nullptr;
  if (num_slots < 1 || num_slots > LORA_MAX_SLOTS)
    return fail(LORA_ERR_SHAPE, "num_slots = %d outside [1, %d]", num_slots, LORA_MAX_SLOTS);
  for (int32_t d : {d_in, d_out}) {
    if (d < 8 || d > LORA_MAX_DIM) return fail(LORA_ERR_SHAPE, "dim %d outside [8, %d]", d, LORA_MAX_DIM);
    if (d % 8 != 0) return fail(LORA_ERR_SHAPE, "dim %d not a multiple of 8", d);
  }
  if (!valid_dtype(w_dtype)) return fail(LORA_ERR_DTYPE, "unknown weight dtype %d", (int)w_dtype);
  if (dev_meta == nullptr) return fail(LORA_ERR_NULL, "dev_meta is NULL");
  if (!aligned(dev_meta, 16)) return fail(LORA_ERR_ALIGN, "dev_meta not 16-byte aligned");
  if (dev_meta_bytes < lora_table_device_bytes(num_slots))
    return fail(LORA_ERR_WORKSPACE, "dev_meta %zu bytes < %zu", dev_meta_bytes,
                lora_table_device_bytes(num_slots));
  lora_table* t = new (std::nothrow) lora_table();
  if (t == nullptr) return fail(LORA_ERR_SHAPE, "host allocation failed");
  t->num_slots = num_slots;
  t->d_in = d_in;
  t->d_out = d_out;
  t->w_dtype = w_dtype;
  t->dev_meta = dev_meta;
  t->host.assign(num_slots, lora::SlotMeta{nullptr, nullptr, 0, 0.0f, {0, 0}});
  *out = t;
  return ok();
}

lora_status lora_table_set(lora_table* t, int32_t slot, int32_t rank, float scale, const void* A,
                           const void* B) {
  if (t == nullptr) return fail(LORA_ERR_NULL, "table is NULL");
  if (slot < 0 || slot >= t->num_slots)
    return fail(LORA_ERR_SLOT, "slot %d outside [0, %d)", slot, t->num_slots);
  if (rank < 1 || rank > LORA_MAX_RANK)
    return fail(LORA_ERR_RANK, "rank %d outside [1, %d]", rank, LORA_MAX_RANK);
  if (A == nullptr || B == nullptr) return fail(LORA_ERR_NULL, "A or B is NULL");
  if (!aligned(A, 16) || !aligned(B, 16)) return fail(LORA_ERR_ALIGN, "A or B not 16-byte aligned");
  t->host[slot] = lora::SlotMeta{A, B, rank, scale, {0, 0}};
  return ok();
}

lora_status lora_table_clear(lora_table* t, int32_t slot) {
  if (t == nullptr) return fail(LORA_ERR_NULL, "table is NULL");
  if (slot < 0 || slot >= t->num_slots)
    return fail(LORA_ERR_SLOT, "slot %d outside [0, %d)", slot, t->num_slots);
  t->host[slot] = lora::SlotMeta{nullptr, nullptr, 0, 0.0f, {0, 0}};
  return ok();
}

lora_status lora_table_upload(lora_table* t, void* stream) {
  if (t == nullptr) return fail(LORA_ERR_NULL, "table is NULL");
  hipError_t e = hipMemcpyAsync(t->dev_meta, t->host.data(), t->host.size() * sizeof(lora::SlotMeta),
                                hipMemcpyHostToDevice, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "table upload");
  return ok();
}

void lora_table_destroy(lora_table* t) { delete t; }

// ---- plan ------------------------------------------------------------------

size_t lora_plan_workspace_bytes(int32_t n, int32_t num_slots) {
  if (n < 0 || num_slots < 1) return 0;
  return lora::plan_layout(n, num_slots).total;
}

lora_status lora_plan_build(const lora_table* t, int32_t n, const int32_t* idx, const uint8_t* mask,
                            void* ws, size_t ws_bytes, void* stream, lora_plan** out) {
  return make_plan(t, n, idx, nullptr, nullptr, 0, mask, nullptr, ws, ws_bytes,
                   static_cast<hipStream_t>(stream), out);
}

void lora_policy_init(lora_policy* q) {
  if (q != nullptr) *q = default_policy();
}

lora_status lora_plan_build_policy(const lora_table* t, int32_t n, const int32_t* idx,
                                   const uint8_t* mask, const lora_policy* policy, void* ws,
                                   size_t ws_bytes, void* stream, lora_plan** out) {
  return make_plan(t, n, idx, nullptr, nullptr, 0, mask, policy, ws, ws_bytes,
                   static_cast<hipStream_t>(stream), out);
}

lora_status lora_plan_build_segments(const lora_table* t, int32_t n, int32_t num_segs,
                                     const int32_t* seg_offsets, const int32_t* seg_adapter,
                                     const uint8_t* mask, void* ws, size_t ws_bytes, void* stream,
                                     lora_plan** out) {
  if (out != nullptr) *out = nullptr;
  if (num_segs < 0 || num_segs > LORA_MAX_ROWS)
    return fail(LORA_ERR_SHAPE, "num_segs = %d out of range", num_segs);
  if (seg_offsets == nullptr) return fail(LORA_ERR_NULL, "seg_offsets is NULL");
  if (num_segs > 0 && seg_adapter == nullptr) return fail(LORA_ERR_NULL, "seg_adapter is NULL");
  if (!aligned(seg_offsets, 4) || (seg_adapter != nullptr && !aligned(seg_adapter, 4)))
    return fail(LORA_ERR_ALIGN, "segment arrays not 4-byte aligned");
  return make_plan(t, n, nullptr, seg_offsets, seg_adapter, num_segs, mask, nullptr, ws, ws_bytes,
                   static_cast<hipStream_t>(stream), out);
}

lora_status lora_plan_export(const lora_plan* p, int32_t* counts, int32_t* offsets, int32_t* perm,
                             int32_t* n_runs, int32_t* run_start, int32_t* run_len,
                             int32_t* run_adapter, int32_t* m_counts, int32_t* m_offsets,
                             int32_t* m_perm, uint32_t* data_flags, void* stream) {
  lora_status st = check_plan(p);
  if (st != LORA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t S = p->table->num_slots, n = p->n;
  // the device keeps the last row of each run; the length needs the start too
  std::vector<int32_t> start_tmp;
  int32_t* run_start_h = run_start;
  if (run_len != nullptr && run_start_h == nullptr) {
    start_tmp.resize(std::max<size_t>(n, 1));
    run_start_h = start_tmp.data();
  }
  struct Item {
    void* dst;
    const void* src;
    size_t bytes;
  };
  int32_t hdr[lora::HDR_WORDS];
  const Item items[] = {
      {hdr, p->d.hdr, sizeof(hdr)},
      {counts, p->d.counts, S * 4},
      {offsets, p->d.offsets, (S + 1) * 4},
      {perm, p->d.perm, n * 4},
      {run_start_h, p->d.run_start, n * 4},
      {run_len, p->d.run_end, n * 4},
      {run_adapter, p->d.run_adapter, n * 4},
      {m_counts, p->d.m_counts, S * 4},
      {m_offsets, p->d.m_offsets, (S + 1) * 4},
      {m_perm, p->d.m_perm, n * 4},
  };
  for (const Item& it : items) {
    if (it.dst == nullptr || it.bytes == 0) continue;
    hipError_t e = hipMemcpyAsync(it.dst, it.src, it.bytes, hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) return hip_fail(e, "plan export copy");
  }
  hipError_t e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "plan export sync");
  const int32_t nr = hdr[lora::HDR_NRUNS];
  if (run_len != nullptr)
    for (int32_t k = 0; k < nr; ++k) run_len[k] = run_len[k] - run_start_h[k] + 1;
  if (n_runs != nullptr) *n_runs = nr;
  if (data_flags != nullptr) *data_flags = (uint32_t)hdr[lora::HDR_FLAGS];
  return ok();
}

lora_status lora_plan_check(const lora_plan* p, uint32_t* data_flags, void* stream) {
  lora_status st = check_plan(p);
  if (st != LORA_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t flags = 0;
  hipError_t e = hipMemcpyAsync(&flags, p->d.hdr + lora::HDR_FLAGS, 4, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "plan check");
  if (data_flags != nullptr) *data_flags = (uint32_t)flags;
  if (flags != 0) return fail(LORA_ERR_DATA, "device data flags 0x%x", (unsigned)flags);
  return ok();
}

void lora_plan_destroy(lora_plan* p) { delete p; }

// ---- forward ---------------------------------------------------------------

lora_status lora_shrink(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx, float* H,
                        int64_t ldh, void* stream) {
  lora_status st = check_plan(p);
  if (st != LORA_OK) return st;
  const lora_table* t = p->table;
  if ((st = check_matrix(X, x_dtype, ldx, t->d_in, "X", p->n)) != LORA_OK) return st;
  if ((st = check_matrix(H, LORA_F32, ldh, std::max(p->r_max, 1), "H", p->n)) != LORA_OK) return st;
  if (kDebug) {
    Disjoint d("lora_shrink");
    d.out(rows_span(H, p->n, std::max(p->r_max, 1), ldh, 4, "H"));
    d.in(rows_span(X, p->n, t->d_in, ldx, dsize(x_dtype), "X"));
    d.weights(t);
    d.plan(p);
    if ((st = d.check()) != LORA_OK) return st;
  }
  if (p->n == 0) return ok();
  lora::OpLaunch o = op_base(p);
  o.count_word = lora::HDR_NRB_TOTAL;
  o.first_word = -1;
  o.rb_ub = ub_large(p) + ub_small(p);
  o.coarse_ub = p->fine ? 0 : ub_coarse(p) + ub_small(p);
  o.fine_ub = p->fine ? ub_fine(p) + ub_small(p) : 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (x_dtype == LORA_BF16 && t->w_dtype == LORA_BF16)
    e = lora::launch_shrink_mfma(o, X, ldx, H, ldh, 1, 0, s);
  else
    e = lora::launch_shrink_valu(o, X, x_dtype, ldx, t->w_dtype, H, ldh, s);
  if (e != hipSuccess) return hip_fail(e, "shrink launch");
  return ok();
}

lora_status lora_expand(const lora_plan* p, const float* H, int64_t ldh, void* Y, lora_dtype y_dtype,
                        int64_t ldy, void* stream) {
  lora_status st = check_plan(p);
  if (st != LORA_OK) return st;
  const lora_table* t = p->table;
  if ((st = check_matrix(H, LORA_F32, ldh, std::max(p->r_max, 1), "H", p->n)) != LORA_OK) return st;
  if ((st = check_matrix(Y, y_dtype, ldy, t->d_out, "Y", p->n)) != LORA_OK) return st;
  if (kDebug) {
    Disjoint d("lora_expand");
    d.out(rows_span(Y, p->n, t->d_out, ldy, dsize(y_dtype), "Y"));
    d.in(rows_span(H, p->n, std::max(p->r_max, 1), ldh, 4, "H"));
    d.weights(t);
    d.plan(p);
    if ((st = d.check()) != LORA_OK) return st;
  }
  if (p->n == 0) return ok();
  lora::OpLaunch o = op_base(p);
  o.count_word = lora::HDR_NRB_TOTAL;
  o.first_word = -1;
  o.rb_ub = ub_large(p) + ub_small(p);
  o.coarse_ub = p->fine ? 0 : ub_coarse(p) + ub_small(p);
  o.fine_ub = p->fine ? ub_fine(p) + ub_small(p) : 0;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (t->w_dtype == LORA_BF16)
    e = lora::launch_expand_mfma(o, H, ldh, 1, 0, Y, y_dtype, ldy, s);
  else
    e = lora::launch_expand_valu(o, H, ldh, t->w_dtype, Y, y_dtype, ldy, s);
  if (e != hipSuccess) return hip_fail(e, "expand launch");
  return ok();
}

// Apply workspace: the float32 H of every row, once per d-slice of the grouped
// shrink (the vector path uses one plane), then the partial planes of the split
// small-group path.
size_t apply_h_bytes(const lora_plan* p) {
  const int64_t ldh = (std::max(p->r_max, 1) + 7) / 8 * 8;
  return al256((size_t)std::max(p->n, 1) * ldh * 4) * lora::SHRINK_KS_MAX;
}
size_t apply_split_bytes(const lora_plan* p) {
  // rank padding of the planes: the kernels' 16-column tile count, 1, 2, 4 or 8
  const int nt = (std::max(p->r_max, 1) + 15) / 16;
  const int64_t ldp = 16 * (nt <= 1 ? 1 : nt <= 2 ? 2 : nt <= 4 ? 4 : 8);
  return al256((size_t)lora::SPLIT_SLICES_MAX * std::max(ub_small(p), 1) * 16 * ldp * 4);
}
size_t lora_apply_workspace_bytes(const lora_plan* p) {
  if (p == nullptr) return 0;
  return apply_h_bytes(p) + apply_split_bytes(p);
}

// Small groups take the split path (shrink per d-slice, then expand) unless
// d_in is short: the fused kernel saves a launch, but each of its P sibling
// workgroups (column chunks) reads all of A, which dominates once A is large.
// The split path measured faster on the 4096-wide decode batch and on the
// skewed mixed batch.  Four d-slices (of at least 256 columns) measured best
// on both.
bool small_split_policy(const lora_plan* p) {
  if (p->pol.small_split >= 0) return p->pol.small_split != 0;
  return p->table->d_in >= 1024;
}
int32_t small_split_slices(const lora_plan* p) {
  const int sl = p->pol.split_slices > 0 ? p->pol.split_slices : std::min(4, p->table->d_in / 256);
  return std::max(1, std::min(lora::SPLIT_SLICES_MAX, sl));
}


}  // extern "C"

namespace {

// lora_apply with the workspace given; `allow_fork` = false keeps the whole
// call on the caller's stream (no second stream is created or used).
lora_status apply_impl(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx, void* Y,
                       lora_dtype y_dtype, int64_t ldy, void* ws, size_t ws_bytes, void* stream,
                       bool allow_fork) {
  lora_status st = check_plan(p);
  if (st != LORA_OK) return st;
  const lora_table* t = p->table;
  if ((st = check_matrix(X, x_dtype, ldx, t->d_in, "X", p->n)) != LORA_OK) return st;
  if ((st = check_matrix(Y, y_dtype, ldy, t->d_out, "Y", p->n)) != LORA_OK) return st;
  const size_t need = lora_apply_workspace_bytes(p);
  const bool mfma = x_dtype == LORA_BF16 && t->w_dtype == LORA_BF16;
  const bool needs_ws = !mfma || ub_large(p) > 0;
  if (needs_ws) {
    if (ws == nullptr) return fail(LORA_ERR_NULL, "apply workspace is NULL");
    if (!aligned(ws, 16)) return fail(LORA_ERR_ALIGN, "apply workspace not 16-byte aligned");
    if (ws_bytes < need) return fail(LORA_ERR_WORKSPACE, "apply workspace %zu bytes < %zu", ws_bytes, need);
  }
  if (kDebug) {
    Disjoint d(allow_fork ? "lora_apply" : "lora_apply_noalloc");
    d.out(rows_span(Y, p->n, t->d_out, ldy, dsize(y_dtype), "Y"));
    if (needs_ws) d.out(bytes_span(ws, need, "the workspace"));
    d.in(rows_span(X, p->n, t->d_in, ldx, dsize(x_dtype), "X"));
    d.weights(t);
    d.plan(p);
    if ((st = d.check()) != LORA_OK) return st;
  }
  if (p->n == 0) return ok();
  hipStream_t s = static_cast<hipStream_t>(stream);
  float* H = static_cast<float*>(ws);
  const int64_t ldh = (std::max(p->r_max, 1) + 7) / 8 * 8;
  lora::OpLaunch o = op_base(p);
  hipError_t e = hipSuccess;
  if (mfma) {
    // a mixed batch: the small-group path on the second stream, forked from
    // and joined back into the caller's
    std::unique_lock<std::mutex> lk(g_aux_mutex, std::defer_lock);
    AuxStream* aux = nullptr;
    hipStream_t s_small = s;
    const bool has_small = p->small_max > 0;     // else the plan has no small group
    if (allow_fork && has_small && ub_large(p) > 0 && fork_policy(p)) {
      lk.lock();
      aux = aux_stream(s);
      if (aux != nullptr) {
        if ((e = hipEventRecord(aux->fork, s)) != hipSuccess) return hip_fail(e, "fork record");
        if ((e = hipStreamWaitEvent(aux->s, aux->fork, 0)) != hipSuccess) return hip_fail(e, "fork wait");
        s_small = aux->s;
      } else {
        lk.unlock();
      }
    }
    if (has_small) {
      lora::OpLaunch os = o;
      os.count_word = lora::HDR_NSMALL;
      os.first_word = -1;
      os.rb_ub = ub_small(p);
      // (the split path needs the workspace; without a usable one the fused
      // kernel runs)
      if (ws != nullptr && ws_bytes >= need && aligned(ws, 16) && small_split_policy(p)) {
        float* part = reinterpret_cast<float*>(static_cast<char*>(ws) + apply_h_bytes(p));
        e = lora::launch_small_split_mfma(os, X, ldx, Y, y_dtype, ldy, small_chunks_policy(p),
                                          small_split_slices(p), part, s_small);
        if (e != hipSuccess) return hip_fail(e, "split small-group launch");
      } else {
        e = lora::launch_bgmv_mfma(os, X, ldx, Y, y_dtype, ldy, small_chunks_policy(p), s_small);
        if (e != hipSuccess) return hip_fail(e, "fused small-group launch");
      }
    }
    if (aux != nullptr && (e = hipEventRecord(aux->join, aux->s)) != hipSuccess)
      return hip_fail(e, "join record");
    if (ub_large(p) > 0) {
      o.count_word = lora::HDR_NRB_LARGE;
      o.first_word = -1;
      o.rb_ub = ub_large(p);
      o.coarse_ub = ub_coarse(p);
      o.fine_ub = ub_fine(p);
      const int64_t plane = (int64_t)(al256((size_t)std::max(p->n, 1) * ldh * 4) / 4);
      e = lora::launch_shrink_mfma(o, X, ldx, H, ldh, lora::SHRINK_KS_MAX, plane, s);
      if (e == hipSuccess)
        e = lora::launch_expand_mfma(o, H, ldh, lora::SHRINK_KS_MAX, plane, Y, y_dtype, ldy, s);
      if (e != hipSuccess) return hip_fail(e, "grouped shrink/expand launch");
    }
    if (aux != nullptr && (e = hipStreamWaitEvent(s, aux->join, 0)) != hipSuccess)
      return hip_fail(e, "join wait");
  } else {
    o.count_word = lora::HDR_NRB_TOTAL;
    o.first_word = -1;
    o.rb_ub = ub_large(p) + ub_small(p);
    e = lora::launch_shrink_valu(o, X, x_dtype, ldx, t->w_dtype, H, ldh, s);
    if (e == hipSuccess) e = lora::launch_expand_valu(o, H, ldh, t->w_dtype, Y, y_dtype, ldy, s);
    if (e != hipSuccess) return hip_fail(e, "vector-path launch");
  }
  return ok();
}

}  // namespace

extern "C" {

lora_status lora_apply(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx, void* Y,
                       lora_dtype y_dtype, int64_t ldy, void* ws, size_t ws_bytes, void* stream) {
  return apply_impl(p, X, x_dtype, ldx, Y, y_dtype, ldy, ws, ws_bytes, stream, true);
}

// ---- plan-free small batch -------------------------------------------------

namespace {
// live rank bound and d-slices of lora_apply_ids (from the table's host copy of
// the slot metadata, as lora_plan_build takes them)
struct IdsShape {
  int32_t r_max;
  bool rank8;
  int32_t slices;
  int64_t ldp;          // row stride of the partial planes: 16 x rank tiles
};
IdsShape ids_shape(const lora_table* t) {
  IdsShape q{0, true, 1, 16};
  for (const auto& s : t->host) {
    if (s.rank <= 0) continue;
    q.r_max = std::max(q.r_max, s.rank);
    q.rank8 = q.rank8 && (s.rank % 8 == 0);
  }
  const int nt = (std::max(q.r_max, 1) + 15) / 16;
  q.ldp = 16 * (nt <= 1 ? 1 : nt <= 2 ? 2 : nt <= 4 ? 4 : 8);
  q.slices = std::max(1, std::min(lora::SPLIT_SLICES_MAX, std::min(4, t->d_in / 256)));
  return q;
}
}  // namespace

size_t lora_apply_ids_workspace_bytes(const lora_table* t, int32_t n) {
  if (t == nullptr || n <= 0 || n > LORA_APPLY_IDS_MAX_ROWS) return 0;
  const IdsShape q = ids_shape(t);
  if (q.r_max == 0) return 0;
  return al256((size_t)q.slices * (size_t)n * (size_t)q.ldp * 4);
}

lora_status lora_apply_ids(const lora_table* t, int32_t n, const int32_t* idx, const void* X,
                           lora_dtype x_dtype, int64_t ldx, void* Y, lora_dtype y_dtype,
                           int64_t ldy, void* ws, size_t ws_bytes, void* stream) {
  if (t == nullptr) return fail(LORA_ERR_NULL, "table is NULL");
  if (n < 0 || n > LORA_APPLY_IDS_MAX_ROWS)
    return fail(LORA_ERR_SHAPE, "lora_apply_ids: n = %d outside [0, %d]", n, LORA_APPLY_IDS_MAX_ROWS);
  lora_status st;
  if ((st = check_matrix(X, x_dtype, ldx, t->d_in, "X", n)) != LORA_OK) return st;
  if ((st = check_matrix(Y, y_dtype, ldy, t->d_out, "Y", n)) != LORA_OK) return st;
  if (x_dtype != LORA_BF16 || t->w_dtype != LORA_BF16)
    return fail(LORA_ERR_DTYPE, "lora_apply_ids needs bfloat16 X and adapter weights");
  if (n > 0 && idx == nullptr) return fail(LORA_ERR_NULL, "idx is NULL");
  if (idx != nullptr && !aligned(idx, 4)) return fail(LORA_ERR_ALIGN, "idx not 4-byte aligned");
  const size_t need = lora_apply_ids_workspace_bytes(t, n);
  if (need > 0) {
    if (ws == nullptr) return fail(LORA_ERR_NULL, "apply_ids workspace is NULL");
    if (!aligned(ws, 16)) return fail(LORA_ERR_ALIGN, "apply_ids workspace not 16-byte aligned");
    if (ws_bytes < need) return fail(LORA_ERR_WORKSPACE, "apply_ids workspace %zu bytes < %zu", ws_bytes, need);
  }
  if (kDebug) {
    Disjoint d("lora_apply_ids");
    d.out(rows_span(Y, n, t->d_out, ldy, dsize(y_dtype), "Y"));
    if (need > 0) d.out(bytes_span(ws, need, "the workspace"));
    d.in(rows_span(X, n, t->d_in, ldx, dsize(x_dtype), "X"));
    d.in(bytes_span(idx, (size_t)n * 4, "idx"));
    d.weights(t);
    if ((st = d.check()) != LORA_OK) return st;
  }
  const IdsShape q = ids_shape(t);
  if (n == 0 || q.r_max == 0) return ok();
  lora::IdsLaunch l{};
  l.meta = static_cast<const lora::SlotMeta*>(t->dev_meta);
  l.num_slots = t->num_slots;
  l.d_in = t->d_in;
  l.d_out = t->d_out;
  l.r_max = q.r_max;
  l.rank8 = q.rank8;
  l.y_bf16 = y_dtype == LORA_BF16;
  l.ids = idx;
  l.n = n;
  l.X = X;
  l.ldx = ldx;
  l.Y = Y;
  l.ldy = ldy;
  l.H = static_cast<float*>(ws);
  l.slices = q.slices;
  l.n_chunks = std::max(1, std::min(16, (t->d_out + 1023) / 1024));
  const hipError_t e = lora::launch_ids_mfma(l, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "apply_ids launch");
  return ok();
}

lora_status lora_apply_noalloc(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                               void* Y, lora_dtype y_dtype, int64_t ldy, void* stream) {
  lora_status st = check_plan(p);
  if (st != LORA_OK) return st;
  const size_t need = lora_apply_workspace_bytes(p);
  if (need > (size_t)LORA_NOALLOC_SCRATCH_BYTES)
    return fail(LORA_ERR_WORKSPACE,
                "lora_apply_noalloc: this plan needs %zu bytes of scratch, more than the %zu bytes "
                "the library holds per GPU (use lora_apply with a caller workspace)",
                need, (size_t)LORA_NOALLOC_SCRATCH_BYTES);
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* ws = nullptr;
  const hipError_t e = lora::noalloc_scratch(s, &ws);
  if (e != hipSuccess) return hip_fail(e, "scratch address");
  return apply_impl(p, X, x_dtype, ldx, Y, y_dtype, ldy, ws, LORA_NOALLOC_SCRATCH_BYTES, stream, false);
}

// ---- measurement utility ------------------------------------------------------

lora_status lora_calibrate_mfma(int32_t workgroups, int32_t iters, float* out, void* stream) {
  if (workgroups < 1 || workgroups > (1 << 16) || iters < 1)
    return fail(LORA_ERR_SHAPE, "workgroups %d / iters %d out of range", workgroups, iters);
  if (out == nullptr) return fail(LORA_ERR_NULL, "out is NULL");
  const hipError_t e = lora::launch_calib_mfma(workgroups, iters, out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "calibration launch");
  return ok();
}

// ---- the whole adapted layer ---------------------------------------------------

// SHRINK_KS_MAX fp32 planes [n, pad8(r_max)], then the packed bf16 s_a H
// [n, 2 linear_rank_cols(r_max)]
size_t lora_linear_workspace_bytes(const lora_plan* p) {
  if (p == nullptr) return 0;
  return apply_h_bytes(p) +
         al256((size_t)std::max(p->n, 1) * 2 * lora::linear_rank_cols(p->r_max) * 2);
}

lora_status lora_linear(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                        const void* W, lora_dtype w_dtype, int64_t ldw, void* Y, lora_dtype y_dtype,
                        int64_t ldy, void* ws, size_t ws_bytes, void* stream) {
  lora_status st = check_plan(p);
  if (st != LORA_OK) return st;
  const lora_table* t = p->table;
  if ((st = check_matrix(X, x_dtype, ldx, t->d_in, "X", p->n)) != LORA_OK) return st;
  if ((st = check_matrix(Y, y_dtype, ldy, t->d_out, "Y", p->n)) != LORA_OK) return st;
  if (W == nullptr) return fail(LORA_ERR_NULL, "W is NULL");
  if ((st = check_matrix(W, w_dtype, ldw, t->d_in, "W")) != LORA_OK) return st;
  if (x_dtype != LORA_BF16 || w_dtype != LORA_BF16 || t->w_dtype != LORA_BF16)
    return fail(LORA_ERR_DTYPE, "lora_linear needs bfloat16 X, W and adapter weights");
  // a 256-row tile of any operand must span less than 2^31 bytes (32-bit offsets)
  constexpr int64_t LD_MAX = int64_t(1) << 21;
  if (ldx > LD_MAX || ldw > LD_MAX || ldy > LD_MAX)
    return fail(LORA_ERR_SHAPE, "lora_linear: leading dimensions above %lld elements", (long long)LD_MAX);
  {
    // Y must not overlap X or W (it is written while they are read)
    const uintptr_t yb = (uintptr_t)Y, ye = yb + (uintptr_t)std::max(p->n, 1) * (uintptr_t)ldy * dsize(y_dtype);
    const uintptr_t xb = (uintptr_t)X, xe = xb + (uintptr_t)std::max(p->n, 1) * (uintptr_t)ldx * 2u;
    const uintptr_t wb = (uintptr_t)W, we = wb + (uintptr_t)t->d_out * (uintptr_t)ldw * 2u;
    if (p->n > 0 && ((yb < xe && xb < ye) || (yb < we && wb < ye)))
      return fail(LORA_ERR_SHAPE, "Y overlaps X or W");
  }
  const size_t need = lora_linear_workspace_bytes(p);
  if (ws == nullptr) return fail(LORA_ERR_NULL, "linear workspace is NULL");
  if (!aligned(ws, 16)) return fail(LORA_ERR_ALIGN, "linear workspace not 16-byte aligned");
  if (ws_bytes < need) return fail(LORA_ERR_WORKSPACE, "linear workspace %zu bytes < %zu", ws_bytes, need);
  if (kDebug) {
    Disjoint d("lora_linear");
    d.out(rows_span(Y, p->n, t->d_out, ldy, dsize(y_dtype), "Y"));
    d.out(bytes_span(ws, need, "the workspace"));
    d.in(rows_span(X, p->n, t->d_in, ldx, 2, "X"));
    d.in(rows_span(W, t->d_out, t->d_in, ldw, 2, "W"));
    d.weights(t);
    d.plan(p);
    if ((st = d.check()) != LORA_OK) return st;
  }
  if (p->n == 0) return ok();
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t ldh = (std::max(p->r_max, 1) + 7) / 8 * 8;
  const int64_t plane = (int64_t)(al256((size_t)std::max(p->n, 1) * ldh * 4) / 4);
  float* H = static_cast<float*>(ws);
  lora::OpLaunch o = op_base(p);
  hipError_t e = hipSuccess;
  if (p->r_max > 0) {
    // H of every row with an adapter (all entries: large-group blocks and
    // small-group entries), in SHRINK_KS_MAX partial planes
    lora::OpLaunch os = o;
    os.count_word = lora::HDR_NRB_TOTAL;
    os.first_word = -1;
    os.rb_ub = ub_large(p) + ub_small(p);
    os.coarse_ub = p->fine ? 0 : ub_coarse(p) + ub_small(p);
    os.fine_ub = p->fine ? ub_fine(p) + ub_small(p) : 0;
    e = lora::launch_shrink_mfma(os, X, ldx, H, ldh, lora::SHRINK_KS_MAX, plane, s);
    if (e != hipSuccess) return hip_fail(e, "linear shrink launch");
  }
  lora::LinearLaunch l{};
  l.X = X;
  l.ldx = ldx;
  l.W = W;
  l.ldw = ldw;
  l.Y = Y;
  l.ldy = ldy;
  l.y_bf16 = y_dtype == LORA_BF16;
  l.run_start = p->d.run_start;
  l.run_end = p->d.run_end;
  l.run_adapter = p->d.run_adapter;
  l.H = H;
  l.ldh = ldh;
  l.hp_stride = plane;
  l.ks_max = lora::SHRINK_KS_MAX;
  l.Hs = reinterpret_cast<uint16_t*>(static_cast<char*>(ws) + apply_h_bytes(p));
  o.rb_ub = ub_large(p) + ub_small(p);
  e = lora::launch_linear_mfma(o, l, s);
  if (e != hipSuccess) return hip_fail(e, "linear launch");
  return ok();
}

// ---- backward --------------------------------------------------------------

namespace {
// buffers of the adapter gradients (debug build): dA_a and dB_a written;
// X, dY, H_saved, the weights and the plan read
void grad_spans(Disjoint& d, const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                const void* dY, lora_dtype dy_dtype, int64_t lddy, const float* H_saved, int64_t ldh,
                float* const* dA, float* const* dB) {
  const lora_table* t = p->table;
  for (int32_t a = 0; a < t->num_slots; ++a) {
    const int32_t r = t->host[a].rank;
    if (dA != nullptr) d.out(rows_span(dA[a], r, t->d_in, t->d_in, 4, "dA", a));
    if (dB != nullptr) d.out(rows_span(dB[a], t->d_out, r, r, 4, "dB", a));
  }
  d.in(rows_span(X, p->n, t->d_in, ldx, dsize(x_dtype), "X"));
  d.in(rows_span(dY, p->n, t->d_out, lddy, dsize(dy_dtype), "dY"));
  d.in(rows_span(H_saved, p->n, std::max(p->r_max, 1), ldh, 4, "H_saved"));
  d.weights(t);
  d.plan(p);
}
}  // namespace

size_t lora_grad_workspace_bytes(const lora_plan* p) {
  if (p == nullptr) return 0;
  return lora::grad_layout(ub_mrb(p), p->r_max).total;
}

lora_status lora_grad(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                      const void* dY, lora_dtype dy_dtype, int64_t lddy, const float* H_saved,
                      int64_t ldh, float* const* dA, float* const* dB, int32_t accumulate,
                      void* ws, size_t ws_bytes, void* stream) {
  lora_status st = check_plan(p);
  if (st != LORA_OK) return st;
  const lora_table* t = p->table;
  if ((st = check_matrix(X, x_dtype, ldx, t->d_in, "X", p->n)) != LORA_OK) return st;
  if ((st = check_matrix(dY, dy_dtype, lddy, t->d_out, "dY", p->n)) != LORA_OK) return st;
  if (x_dtype != dy_dtype) return fail(LORA_ERR_DTYPE, "X and dY dtypes differ");
  if (H_saved != nullptr &&
      (st = check_matrix(H_saved, LORA_F32, ldh, std::max(p->r_max, 1), "H_saved", p->n)) != LORA_OK)
    return st;
  for (int32_t a = 0; a < t->num_slots; ++a) {
    const float* pa = dA ? dA[a] : nullptr;
    const float* pb = dB ? dB[a] : nullptr;
    if ((pa || pb) && t->host[a].rank <= 0)
      return fail(LORA_ERR_SLOT, "gradient requested for empty slot %d", a);
    if ((pa && !aligned(pa, 16)) || (pb && !aligned(pb, 16)))
      return fail(LORA_ERR_ALIGN, "gradient buffer of slot %d not 16-byte aligned", a);
  }
  const size_t need = lora_grad_workspace_bytes(p);
  if (ws == nullptr) return fail(LORA_ERR_NULL, "grad workspace is NULL");
  if (!aligned(ws, 16)) return fail(LORA_ERR_ALIGN, "grad workspace not 16-byte aligned");
  if (ws_bytes < need) return fail(LORA_ERR_WORKSPACE, "grad workspace %zu bytes < %zu", ws_bytes, need);
  if (kDebug) {
    Disjoint d("lora_grad");
    grad_spans(d, p, X, x_dtype, ldx, dY, dy_dtype, lddy, H_saved, ldh, dA, dB);
    d.out(bytes_span(ws, need, "the workspace"));
    if ((st = d.check()) != LORA_OK) return st;
  }

  const bool mfma = x_dtype == LORA_BF16 && t->w_dtype == LORA_BF16;
  lora::GradLaunch g{};
  g.o = op_base(p);
  g.o.rb = p->d.mrb;
  g.o.rb_ub = ub_mrb(p);
  g.o.count_word = lora::HDR_NMRB;
  g.o.first_word = -1;
  g.m_perm = p->d.m_perm;
  g.m_offsets = p->d.m_offsets;
  g.m_counts = p->d.m_counts;
  g.m_blk = p->d.m_blk;
  g.X = X;
  g.ldx = ldx;
  g.dY = dY;
  g.lddy = lddy;
  g.H_saved = H_saved;
  g.ldh = ldh;
  g.dA = dA;
  g.dB = dB;
  g.accumulate = accumulate;
  const lora::GradLayout GL = lora::grad_layout(ub_mrb(p), p->r_max);
  char* wsb = static_cast<char*>(ws);
  g.hg = reinterpret_cast<float*>(wsb + GL.partial);
  g.fin = reinterpret_cast<uint16_t*>(wsb + GL.fin);
  g.k_splits = mfma ? grad_splits_policy(p) : 1;
  g.p_stride = ub_mrb(p) * lora::MRB_ROWS;
  g.r_pad = (std::max(p->r_max, 1) + 15) / 16 * 16;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // n = 0 still runs: slots with no trainable row must receive zeros.
  hipError_t e = mfma ? lora::launch_grad_mfma(g, s)
                      : lora::launch_grad_valu(g, x_dtype, t->w_dtype, s);
  if (e != hipSuccess) return hip_fail(e, "gradient launch");
  return ok();
}

// ---- input gradient ----------------------------------------------------------

size_t lora_grad_x_workspace_bytes(const lora_plan* p) {
  if (p == nullptr) return 0;
  return apply_h_bytes(p);   // SHRINK_KS_MAX fp32 planes [n, pad8(r_max)]
}

lora_status lora_grad_x(const lora_plan* p, const void* dY, lora_dtype dy_dtype, int64_t lddy,
                        void* dX, lora_dtype dx_dtype, int64_t lddx, void* ws, size_t ws_bytes,
                        void* stream) {
  lora_status st = check_plan(p);
  if (st != LORA_OK) return st;
  const lora_table* t = p->table;
  if ((st = check_matrix(dY, dy_dtype, lddy, t->d_out, "dY", p->n)) != LORA_OK) return st;
  if ((st = check_matrix(dX, dx_dtype, lddx, t->d_in, "dX", p->n)) != LORA_OK) return st;
  if (dy_dtype != LORA_BF16 || t->w_dtype != LORA_BF16)
    return fail(LORA_ERR_DTYPE, "input gradient needs bfloat16 dY and weights");
  const size_t need = lora_grad_x_workspace_bytes(p);
  if (ws == nullptr) return fail(LORA_ERR_NULL, "input-gradient workspace is NULL");
  if (!aligned(ws, 16)) return fail(LORA_ERR_ALIGN, "input-gradient workspace not 16-byte aligned");
  if (ws_bytes < need)
    return fail(LORA_ERR_WORKSPACE, "input-gradient workspace %zu bytes < %zu", ws_bytes, need);
  if (kDebug) {
    Disjoint d("lora_grad_x");
    d.out(rows_span(dX, p->n, t->d_in, lddx, dsize(dx_dtype), "dX"));
    d.out(bytes_span(ws, need, "the workspace"));
    d.in(rows_span(dY, p->n, t->d_out, lddy, dsize(dy_dtype), "dY"));
    d.weights(t);
    d.plan(p);
    if ((st = d.check()) != LORA_OK) return st;
  }
  if (p->n == 0) return ok();
  lora::OpLaunch o = op_base(p);
  o.d_in = t->d_out;                 // the shrink reads dY rows
  o.d_out = t->d_in;                 // the expand writes dX rows
  o.rb = p->d.mrb;
  o.perm = p->d.m_perm;
  o.count_word = lora::HDR_NMRB;
  o.first_word = -1;
  o.rb_ub = ub_mrb(p);
  o.fine_ub = ub_mrb(p);
  const int64_t ldh = (std::max(p->r_max, 1) + 7) / 8 * 8;
  const int64_t plane = (int64_t)(al256((size_t)std::max(p->n, 1) * ldh * 4) / 4);
  hipError_t e = lora::launch_grad_x_mfma(o, dY, lddy, static_cast<float*>(ws), ldh, plane, dX,
                                          dx_dtype, lddx, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "input-gradient launch");
  return ok();
}

// ---- combined backward -----------------------------------------------------------

size_t lora_backward_workspace_bytes(const lora_plan* p) {
  if (p == nullptr) return 0;
  return al256(lora_grad_workspace_bytes(p)) + lora_grad_x_workspace_bytes(p);
}

lora_status lora_backward(const lora_plan* p, const void* X, lora_dtype x_dtype, int64_t ldx,
                          const void* dY, lora_dtype dy_dtype, int64_t lddy, const float* H_saved,
                          int64_t ldh, float* const* dA, float* const* dB, int32_t accumulate,
                          void* dX, lora_dtype dx_dtype, int64_t lddx, void* ws, size_t ws_bytes,
                          void* stream) {
  lora_status st = check_plan(p);
  if (st != LORA_OK) return st;
  const lora_table* t = p->table;
  // the input gradient's own checks first: once the adapter gradients are
  // enqueued, nothing may fail before the input gradient is
  if ((st = check_matrix(dY, dy_dtype, lddy, t->d_out, "dY", p->n)) != LORA_OK) return st;
  if ((st = check_matrix(dX, dx_dtype, lddx, t->d_in, "dX", p->n)) != LORA_OK) return st;
  if (dy_dtype != LORA_BF16 || t->w_dtype != LORA_BF16)
    return fail(LORA_ERR_DTYPE, "the input gradient needs bfloat16 dY and weights");
  const size_t need = lora_backward_workspace_bytes(p);
  if (ws == nullptr) return fail(LORA_ERR_NULL, "backward workspace is NULL");
  if (!aligned(ws, 16)) return fail(LORA_ERR_ALIGN, "backward workspace not 16-byte aligned");
  if (ws_bytes < need) return fail(LORA_ERR_WORKSPACE, "backward workspace %zu bytes < %zu", ws_bytes, need);
  if (kDebug) {
    Disjoint d("lora_backward");
    grad_spans(d, p, X, x_dtype, ldx, dY, dy_dtype, lddy, H_saved, ldh, dA, dB);
    d.out(rows_span(dX, p->n, t->d_in, lddx, dsize(dx_dtype), "dX"));
    d.out(bytes_span(ws, need, "the workspace"));
    if ((st = d.check()) != LORA_OK) return st;
  }
  const size_t off = al256(lora_grad_workspace_bytes(p));
  char* wsb = static_cast<char*>(ws);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the input gradient on the second stream beside the adapter gradients:
  // both read the plan and dY as they are when the call is made, and write
  // disjoint outputs and workspace parts
  std::unique_lock<std::mutex> lk(g_aux_mutex);
  AuxStream* aux = p->n > 0 ? aux_stream(s) : nullptr;
  hipError_t e;
  if (aux != nullptr && (e = hipEventRecord(aux->fork, s)) != hipSuccess) return hip_fail(e, "fork record");
  st = lora_grad(p, X, x_dtype, ldx, dY, dy_dtype, lddy, H_saved, ldh, dA, dB, accumulate, wsb, off,
                 stream);
  if (st != LORA_OK) return st;
  if (aux == nullptr) {
    lk.unlock();
    return lora_grad_x(p, dY, dy_dtype, lddy, dX, dx_dtype, lddx, wsb + off, ws_bytes - off, stream);
  }
  if ((e = hipStreamWaitEvent(aux->s, aux->fork, 0)) != hipSuccess) return hip_fail(e, "fork wait");
  st = lora_grad_x(p, dY, dy_dtype, lddy, dX, dx_dtype, lddx, wsb + off, ws_bytes - off, aux->s);
  if ((e = hipEventRecord(aux->join, aux->s)) != hipSuccess) return hip_fail(e, "join record");
  if ((e = hipStreamWaitEvent(s, aux->join, 0)) != hipSuccess) return hip_fail(e, "join wait");
  return st;
}

// ---- adapter-local optimizer step ---------------------------------------------

static_assert(sizeof(lora_adamw_tensor) == 72 && offsetof(lora_adamw_tensor, n) == 40 &&
                  offsetof(lora_adamw_tensor, step) == 48 &&
                  offsetof(lora_adamw_tensor, weight_decay) == 68,
              "lora_adamw_tensor layout");

lora_status lora_adamw_step(const lora_adamw_tensor* tensors, int32_t count, void* stream) {
  if (count < 0) return fail(LORA_ERR_SHAPE, "tensor count %d < 0", count);
  if (count == 0) return ok();
  if (tensors == nullptr) return fail(LORA_ERR_NULL, "tensors is NULL");
  struct Span {
    uintptr_t b, e;
    bool written;
  };
  std::vector<Span> spans;
  std::vector<lora::AdamwLaunch> recs;
  recs.reserve(count);
  for (int32_t k = 0; k < count; ++k) {
    const lora_adamw_tensor& t = tensors[k];
    if (t.n < 0) return fail(LORA_ERR_SHAPE, "tensor %d: n = %lld < 0", k, (long long)t.n);
    if (t.step < 1) return fail(LORA_ERR_VALUE, "tensor %d: step %d < 1", k, t.step);
    const bool hyper_ok = std::isfinite(t.lr) && t.lr >= 0.f && std::isfinite(t.beta1) &&
                          t.beta1 >= 0.f && t.beta1 < 1.f && std::isfinite(t.beta2) &&
                          t.beta2 >= 0.f && t.beta2 < 1.f && std::isfinite(t.eps) && t.eps > 0.f &&
                          std::isfinite(t.weight_decay) && t.weight_decay >= 0.f;
    if (!hyper_ok)
      return fail(LORA_ERR_VALUE, "tensor %d: lr %g, betas (%g, %g), eps %g, weight decay %g out of range",
                  k, t.lr, t.beta1, t.beta2, t.eps, t.weight_decay);
    if (t.n == 0) continue;
    if (t.p == nullptr || t.m == nullptr || t.v == nullptr || t.g == nullptr)
      return fail(LORA_ERR_NULL, "tensor %d: p, m, v or g is NULL", k);
    if (!aligned(t.p, 16) || !aligned(t.m, 16) || !aligned(t.v, 16) || !aligned(t.g, 16) ||
        !aligned(t.p_bf16, 16))
      return fail(LORA_ERR_ALIGN, "tensor %d: an array is not 16-byte aligned", k);
    const uintptr_t f = (uintptr_t)t.n * 4u;
    spans.push_back({(uintptr_t)t.p, (uintptr_t)t.p + f, true});
    spans.push_back({(uintptr_t)t.m, (uintptr_t)t.m + f, true});
    spans.push_back({(uintptr_t)t.v, (uintptr_t)t.v + f, true});
    spans.push_back({(uintptr_t)t.g, (uintptr_t)t.g + f, false});
    if (t.p_bf16 != nullptr)
      spans.push_back({(uintptr_t)t.p_bf16, (uintptr_t)t.p_bf16 + (uintptr_t)t.n * 2u, true});
    lora::AdamwLaunch r{};
    r.p = t.p;
    r.m = t.m;
    r.v = t.v;
    r.g = t.g;
    r.p_bf16 = t.p_bf16;
    r.n = t.n;
    const double lr = t.lr, b1 = t.beta1, b2 = t.beta2;
    r.decay = (float)(1.0 - lr * (double)t.weight_decay);
    r.step_size = (float)(lr / (1.0 - std::pow(b1, (double)t.step)));
    r.inv_sqrt_bc2 = (float)(1.0 / std::sqrt(1.0 - std::pow(b2, (double)t.step)));
    r.eps = t.eps;
    r.beta1 = t.beta1;
    r.omb1 = (float)(1.0 - b1);
    r.beta2 = t.beta2;
    r.omb2 = (float)(1.0 - b2);
    recs.push_back(r);
  }
  // a written array may overlap nothing; read-only gradients may be shared
  std::sort(spans.begin(), spans.end(), [](const Span& x, const Span& y) { return x.b < y.b; });
  uintptr_t end_all = 0, end_w = 0;
  for (const Span& sp : spans) {
    if (sp.b < (sp.written ? end_all : end_w))
      return fail(LORA_ERR_SHAPE, "optimizer arrays overlap");
    end_all = std::max(end_all, sp.e);
    if (sp.written) end_w = std::max(end_w, sp.e);
  }
  for (size_t k0 = 0; k0 < recs.size(); k0 += lora::ADAMW_GROUP) {
    const int32_t c = (int32_t)std::min<size_t>(lora::ADAMW_GROUP, recs.size() - k0);
    hipError_t e = lora::launch_adamw(recs.data() + k0, c, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "optimizer launch");
  }
  return ok();
}

// ---- masked token-level losses ------------------------------------------------

lora_status lora_token_loss(lora_loss_kind kind, int32_t n, int32_t vocab, const void* logits,
                            lora_dtype logits_dtype, int64_t ldz, const int32_t* target,
                            const float* weight, const uint8_t* mask, const float* old_logp,
                            const float* adv, const float* corr, float clip_lo, float clip_hi,
                            float* loss, float* logp, void* dlogits, lora_dtype dlogits_dtype,
                            int64_t ldd, void* stream) {
  if (kind != LORA_LOSS_CE && kind != LORA_LOSS_IS && kind != LORA_LOSS_PPO)
    return fail(LORA_ERR_VALUE, "unknown loss kind %d", (int)kind);
  if (n < 0 || n > LORA_MAX_ROWS) return fail(LORA_ERR_SHAPE, "n = %d out of range", n);
  if (vocab < 1 || vocab > LORA_MAX_VOCAB) return fail(LORA_ERR_SHAPE, "vocab = %d out of range", vocab);
  if (!(std::isfinite(clip_lo) && clip_lo >= 0.f && std::isfinite(clip_hi) && clip_hi >= 0.f))
    return fail(LORA_ERR_VALUE, "clip range (%g, %g) out of range", clip_lo, clip_hi);
  lora_status st;
  if ((st = check_matrix(logits, logits_dtype, ldz, vocab, "logits", n)) != LORA_OK) return st;
  if ((st = check_matrix(dlogits, dlogits_dtype, ldd, vocab, "dlogits", n)) != LORA_OK) return st;
  if (n == 0) return ok();
  if (target == nullptr || loss == nullptr) return fail(LORA_ERR_NULL, "target or loss is NULL");
  if (kind == LORA_LOSS_CE && weight == nullptr) return fail(LORA_ERR_NULL, "cross-entropy needs weight");
  if (kind != LORA_LOSS_CE && (old_logp == nullptr || adv == nullptr))
    return fail(LORA_ERR_NULL, "policy-gradient losses need old_logp and adv");
  const uintptr_t zb = (uintptr_t)logits, ze = zb + (uintptr_t)n * (uintptr_t)ldz * dsize(logits_dtype);
  const uintptr_t db = (uintptr_t)dlogits, de = db + (uintptr_t)n * (uintptr_t)ldd * dsize(dlogits_dtype);
  if (zb < de && db < ze) return fail(LORA_ERR_SHAPE, "dlogits overlaps logits");
  lora::LossLaunch l{};
  l.kind = (int32_t)kind;
  l.n = n;
  l.vocab = vocab;
  l.logits = logits;
  l.logits_bf16 = logits_dtype == LORA_BF16;
  l.ldz = ldz;
  l.target = target;
  l.weight = weight;
  l.mask = mask;
  l.old_logp = old_logp;
  l.adv = adv;
  l.corr = corr;
  l.clip_lo = clip_lo;
  l.clip_hi = clip_hi;
  l.loss = loss;
  l.logp = logp;
  l.dlogits = dlogits;
  l.dlogits_bf16 = dlogits_dtype == LORA_BF16;
  l.ldd = ldd;
  hipError_t e = lora::launch_token_loss(l, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "token-loss launch");
  return ok();
}

}  // extern "C"
