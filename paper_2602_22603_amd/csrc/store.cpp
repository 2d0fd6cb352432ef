// store.cpp - host side of libsq: the paged KV store's metadata (page
// allocator, refcounts, per-sequence page lists, positions and cursor spans),
// planning of every device operation, and the extern "C" ABI of include/sq.h.
//
// The model follows SideQuest's statement of the problem (arXiv 2602.22603):
// a context that grows by appends (Algorithm 1, Phase 3), a forked auxiliary
// branch that shares the context's storage (Phase 2; §3.4 "Storage Costs"),
// and clear_kv over cursor ids applied between main-thread turns (Phase 1;
// §3.1 steps 3-4).  Conventions the paper leaves open:
//   * pages are taken lowest free id first, one at a time in page-list order;
//   * eviction is out of place: the kept tail from page floor(f/P) on is
//     gathered into fresh pages taken before any old page is released;
//   * positions are carried through eviction, never recomputed;
//   * every call validates everything before it changes anything.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <functional>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/sq.h"
#include "sq_kernels.hpp"

namespace {

thread_local std::string g_err;
thread_local uint64_t g_fails = 0; // failures on this thread (the call trace reads it)

sq_status fail(sq_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  ++g_fails;
  return st;
}

// ---- host call trace -------------------------------------------------------
// One line per state-changing or compute call while a trace is open: the
// call, its arguments, its host time and its outcome.  Off by default; the
// cost when off is one relaxed atomic load per call.
std::mutex g_trace_mu;
FILE *g_trace = nullptr;
bool g_trace_owned = false;
std::atomic<bool> g_trace_on{false};

struct CallTrace {
  const char *name;
  bool on;
  uint64_t fails0 = 0;
  std::chrono::steady_clock::time_point t0;
  char args[224];
  CallTrace(const char *n, const char *fmt, ...) __attribute__((format(printf, 3, 4)))
      : name(n), on(g_trace_on.load(std::memory_order_relaxed)) {
    if (!on) return;
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(args, sizeof(args), fmt, ap);
    va_end(ap);
    fails0 = g_fails;
    t0 = std::chrono::steady_clock::now();
  }
  ~CallTrace() {
    if (!on) return;
    const double us =
        std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count();
    std::lock_guard<std::mutex> lk(g_trace_mu);
    if (!g_trace) return;
    if (g_fails != fails0) std::fprintf(g_trace, "sq %s(%s) host_us=%.1f error: %s\n", name, args, us, g_err.c_str());
    else std::fprintf(g_trace, "sq %s(%s) host_us=%.1f ok\n", name, args, us);
    std::fflush(g_trace);
  }
};
#define SQ_TRACE_CALL(name, ...) CallTrace sq_call_trace_(name, __VA_ARGS__)

sq_status trace_open(const char *path) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  FILE *f = nullptr;
  bool owned = false;
  if (path && std::strcmp(path, "-") == 0) {
    f = stderr;
  } else if (path) {
    f = std::fopen(path, "a");
    if (!f) return fail(SQ_ERR_INVALID, "cannot open trace file %s", path);
    owned = true;
  }
  if (g_trace_owned && g_trace) std::fclose(g_trace);
  g_trace = f;
  g_trace_owned = owned;
  g_trace_on.store(f != nullptr, std::memory_order_relaxed);
  return SQ_OK;
}

// SQ_TRACE in the environment when the library loads: "1" or "-" logs to
// stderr, any other value is a file to append to.
struct TraceFromEnv {
  TraceFromEnv() {
    const char *e = std::getenv("SQ_TRACE");
    if (!e || !*e || std::strcmp(e, "0") == 0) return;
    (void)trace_open(std::strcmp(e, "1") == 0 ? "-" : e);
  }
} g_trace_from_env;

sq_status hip_fail(hipError_t e, const char *what) {
  return fail(SQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr uint64_t kAlign = 256;
uint64_t align_up(uint64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
  uint64_t pt, mask, keep, dst, src, upload, part_m, part_l, part_acc, step, scales, total;
  uint64_t upload_elems;
};

Layout layout_of(const sq_store_config &c) {
  Layout L{};
  const uint64_t max_tok = (uint64_t)c.max_pages_per_seq * c.page_size;
  uint64_t off = 0;
  auto take = [&](uint64_t bytes) {
    const uint64_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L.pt = take((uint64_t)c.max_seqs * c.max_pages_per_seq * 4);
  L.mask = take((uint64_t)c.max_seqs * c.max_pages_per_seq * 4);
  L.keep = take(max_tok);
  L.dst = take(max_tok * 4);
  L.src = take(max_tok * 4);
  // spans of an eviction: its own and the masked runs, at most
  // SQ_MAX_EVICT_SPANS each; then the fresh ids (or a keep-mask row)
  L.upload_elems = 6ull * SQ_MAX_EVICT_SPANS + (uint64_t)c.max_pages_per_seq;
  L.upload = take(L.upload_elems * 4);
  L.part_m = take((uint64_t)sq::kMaxItems * sq::kRows * 4);
  L.part_l = take((uint64_t)sq::kMaxItems * sq::kRows * 4);
  L.part_acc = take((uint64_t)sq::kMaxItems * sq::kRows * c.head_dim * 4);
  L.step = take(sizeof(sq::StepPlan));
  L.scales = take((uint64_t)c.num_layers * 4 * 4);
  L.total = off;
  return L;
}

bool shape_ok(const sq_store_config *c, bool device, std::string *why) {
  auto bad = [&](const char *m) {
    if (why) *why = m;
    return false;
  };
  if (!c) return bad("null configuration");
  if (c->num_layers < 1 || c->num_kv_heads < 1 || c->num_q_heads < 1 || c->head_dim < 1 ||
      c->page_size < 1 || c->num_pages < 1 || c->max_seqs < 1 || c->max_pages_per_seq < 1)
    return bad("every size must be positive");
  if (c->num_q_heads % c->num_kv_heads) return bad("num_q_heads must be a multiple of num_kv_heads");
  if ((int64_t)c->max_pages_per_seq * c->page_size > (int64_t)INT32_MAX / 2)
    return bad("max_pages_per_seq * page_size too large");
  if (c->evict_chunk_pages < 0) return bad("evict_chunk_pages must be >= 0");
  if (c->flags & ~(SQ_STORE_METADATA_ONLY | SQ_STORE_EVICT_REMAP | SQ_STORE_KV_FP8 |
                   SQ_STORE_EVICT_INPLACE))
    return bad("unknown flags");
  if ((c->flags & SQ_STORE_EVICT_INPLACE) &&
      ((c->flags & SQ_STORE_EVICT_REMAP) || c->evict_chunk_pages > 0))
    return bad("in-place eviction excludes remap and evict_chunk_pages");
  if (c->flags & SQ_STORE_KV_FP8) {
    if (!c->kv_scales) return bad("an 8-bit store needs kv_scales");
    for (int i = 0; i < 2 * c->num_layers; ++i)
      if (!std::isfinite(c->kv_scales[i]) || !(c->kv_scales[i] > 0.f))
        return bad("kv_scales must be finite and positive");
  }
  if (device) {
    const int grp = c->num_q_heads / c->num_kv_heads;
    if (c->page_size != sq::kPage) return bad("device mode needs page_size 16");
    if (c->head_dim != 64 && c->head_dim != 128) return bad("device mode needs head_dim 64 or 128");
    if (grp != 1 && grp != 2 && grp != 4 && grp != 8) return bad("num_q_heads / num_kv_heads must be 1, 2, 4 or 8");
    if (c->max_seqs > 255) return bad("device mode supports at most 255 sequences");
  }
  return true;
}

struct PosRun {
  int64_t idx0; // first logical index
  int64_t pos0; // its position
  int64_t n;
};

struct Seq {
  bool live = false;
  std::vector<int32_t> pages;
  int64_t length = 0;
  int64_t next_pos = 0;
  std::vector<PosRun> runs;                             // positions of tokens
  std::map<int32_t, std::pair<int64_t, int64_t>> spans; // cursor -> [start, end)
  std::map<int64_t, int64_t> nonempty;                  // start -> end of non-empty spans
  int32_t parent = -1;
  // Keep masks of deferred evictions, one 16-bit word per page (bit s = slot
  // s attended); empty while no slot is masked.
  std::vector<uint16_t> kmask;
  int64_t n_masked = 0;
};

bool slot_kept(const Seq &q, int64_t i, int P) {
  return q.kmask.empty() || ((q.kmask[i / P] >> (i % P)) & 1);
}

// Maximal runs [s, e) of masked slots, in order (whole kept pages skipped).
std::vector<std::pair<int64_t, int64_t>> masked_runs(const Seq &q, int P) {
  std::vector<std::pair<int64_t, int64_t>> runs;
  if (q.kmask.empty()) return runs;
  int64_t i = 0;
  while (i < q.length) {
    if (i % P == 0 && q.kmask[i / P] == 0xffff) {
      i += P;
      continue;
    }
    if (slot_kept(q, i, P)) {
      ++i;
      continue;
    }
    int64_t j = i;
    while (j < q.length && !slot_kept(q, j, P)) ++j;
    runs.push_back({i, j});
    i = j;
  }
  return runs;
}

// Number of maximal masked runs in the keep words km (P <= 16 slots a word).
int64_t count_runs(const std::vector<uint16_t> &km, int P) {
  int64_t n = 0;
  uint32_t prev_masked = 0; // the last slot of the previous page is masked
  for (uint16_t w : km) {
    const uint32_t z = ~(uint32_t)w & ((1u << P) - 1u);   // masked slots
    const uint32_t starts = z & ~((z << 1) | prev_masked); // a run starts where the slot before is kept
    n += __builtin_popcount(starts);
    prev_masked = (z >> (P - 1)) & 1u;
  }
  return n;
}

// New pages of a masked sequence start with every slot kept.
void grow_kmask(Seq &q) {
  if (!q.kmask.empty()) q.kmask.resize(q.pages.size(), 0xffff);
}

enum ProfKind { kProfValu, kProfMfma, kProfMerge, kProfScan, kProfGather, kProfAppend, kProfExtend,
                kProfKinds };

struct ProfPair {
  hipEvent_t a, b;
  int kind;
};

int64_t pos_at(const Seq &s, int64_t i) {
  // runs are ordered by idx0 and cover [0, length)
  size_t lo = 0, hi = s.runs.size();
  while (hi - lo > 1) {
    const size_t mid = (lo + hi) / 2;
    if (s.runs[mid].idx0 <= i) lo = mid;
    else hi = mid;
  }
  return s.runs[lo].pos0 + (i - s.runs[lo].idx0);
}

void runs_append(Seq &s, int64_t n) {
  if (n <= 0) return;
  if (!s.runs.empty()) {
    PosRun &r = s.runs.back();
    if (r.idx0 + r.n == s.length && r.pos0 + r.n == s.next_pos) {
      r.n += n;
      return;
    }
  }
  s.runs.push_back({s.length, s.next_pos, n});
}

std::vector<PosRun> runs_truncate(const std::vector<PosRun> &runs, int64_t f) {
  std::vector<PosRun> out;
  for (const PosRun &r : runs) {
    if (r.idx0 >= f) break;
    PosRun c = r;
    if (c.idx0 + c.n > f) c.n = f - c.idx0;
    out.push_back(c);
  }
  return out;
}

// Tokens evicted before index x, for sorted disjoint spans with prefix sums.
int64_t evicted_before(const std::vector<std::pair<int64_t, int64_t>> &sp,
                       const std::vector<int64_t> &prefix, int64_t x) {
  // number of spans with start < x
  size_t lo = 0, hi = sp.size();
  while (lo < hi) {
    const size_t mid = (lo + hi) / 2;
    if (sp[mid].first < x) lo = mid + 1;
    else hi = mid;
  }
  if (lo == 0) return 0;
  const size_t k = lo - 1; // last span starting before x
  return prefix[k] + (std::min(sp[k].second, x) - sp[k].first);
}

} // namespace

struct sq_store {
  sq_store_config cfg{};
  bool device = false;
  bool kv8 = false;              // the pools hold E4M3 codes
  std::vector<float> kv_scales;  // [NL][2] (8-bit store)
  float k_scale(int l) const { return kv8 ? kv_scales[2 * l] : 1.f; }
  float v_scale(int l) const { return kv8 ? kv_scales[2 * l + 1] : 1.f; }
  float inv(float x) const { return (float)(1.0 / (double)x); }
  int64_t elem_bytes() const { return kv8 ? 1 : 2; } // bytes per K or V element
  int P = 16, G = 1, D = 128;
  std::vector<int32_t> refcount;
  std::vector<uint64_t> freebits;
  int32_t free_hint = 0;
  int64_t n_free = 0;
  std::vector<Seq> seqs;
  sq_stats st{};
  int64_t peak_pages = 0;

  // device
  sq::Pools pools{};
  Layout lay{};
  int32_t *pt_dev = nullptr;
  // keep-mask mirror, the page table's shape.  A masked sequence's row is
  // uploaded whole; other rows are read only by plans that include a masked
  // sequence, which first set them to all-kept if mask_dirty says they may
  // hold old masks (of a released or compacted sequence, or never written).
  int32_t *mask_dev = nullptr;
  std::vector<char> mask_dirty;
  uint8_t *ev_keep = nullptr;
  int32_t *ev_dst = nullptr, *ev_src = nullptr, *ev_upload = nullptr;
  float *part_m = nullptr, *part_l = nullptr, *part_acc = nullptr;
  // the device array of the allocation-free decode entry point on this
  // store's GPU (looked up at creation; spart_err if that failed)
  sq::StaticPartials spart{};
  hipError_t spart_err = hipErrorNotInitialized;
  int32_t *staging = nullptr;
  hipEvent_t staging_ev = nullptr;
  bool staging_pending = false;
  hipStream_t last_stream = nullptr;
  sq::StepPlan *step_dev = nullptr;     // the step plan in the workspace
  // two pinned host copies of the plan, used in turn: a step waits only for
  // the upload of the step before the last, so the host runs a step ahead
  sq::StepPlan *step_staging[2] = {nullptr, nullptr};
  hipEvent_t step_ev[2] = {nullptr, nullptr};
  bool step_pending[2] = {false, false};
  int step_buf = 0;
  bool have_last_evict = false;
  int64_t last_evict_L = 0, last_evict_Lp = 0;

  // tuning
  int cus = 256;              // compute units (device query in device mode)
  int wg_per_cu[2] = {8, 3};  // resident workgroups per CU (VALU, MFMA), from occupancy
  int wg_per_cu_rb2 = 2;      // the same for the two-row-block MFMA kernel
  int min_wg_pages_valu = 8;
  int min_wg_pages_mfma = 8; // small launches still fill a round of resident workgroups
  // flattened pages appended to every row of a launch (VALU, MFMA): a
  // piece's start-up cost in page equivalents, so the even split evens time
  int row_pad[2] = {2, 16};

  // every call that changes sequence metadata bumps gen; a begun decode
  // step is valid while gen is what sq_step_begin left
  uint64_t gen = 0;
  struct Step {
    bool active = false;
    uint64_t gen = 0;
    int32_t batch = 0, mode = 0;
    bool launch[2] = {false, false}; // VALU, MFMA
    int32_t grid[2] = {0, 0};
    int32_t window = 0; // the windowed plan's window (0: no windowed plan)
    int64_t kv_bytes = 0, kv_bytes_logical = 0;
    int64_t kv_bytes_w = 0, kv_bytes_logical_w = 0;
  } step;

  // profiling
  bool prof_on = false;
  std::vector<ProfPair> prof_pending;
  std::vector<hipEvent_t> ev_pool;
  double prof_ms[kProfKinds] = {};
  int64_t prof_n[kProfKinds] = {};

  // ---- allocator ----
  int64_t live_pages() const { return (int64_t)cfg.num_pages - n_free; }

  int32_t alloc_page() {
    const int32_t nw = (int32_t)freebits.size();
    for (int32_t w = free_hint / 64; w < nw; ++w) {
      if (freebits[w]) {
        const int bit = __builtin_ctzll(freebits[w]);
        const int32_t id = w * 64 + bit;
        freebits[w] &= ~(1ull << bit);
        free_hint = id + 1;
        --n_free;
        refcount[id] = 1;
        peak_pages = std::max(peak_pages, live_pages());
        return id;
      }
    }
    return -1; // callers check n_free first
  }

  // n pages, lowest free ids first, in order (callers check n_free first)
  void alloc_pages(int64_t n, int32_t *out) {
    const int32_t nw = (int32_t)freebits.size();
    int64_t got = 0;
    for (int32_t w = free_hint / 64; w < nw && got < n; ++w) {
      uint64_t bits = freebits[w];
      while (bits && got < n) {
        const int bit = __builtin_ctzll(bits);
        const int32_t id = w * 64 + bit;
        bits &= bits - 1;
        refcount[id] = 1;
        out[got++] = id;
        free_hint = id + 1;
      }
      freebits[w] = bits;
    }
    n_free -= got;
    peak_pages = std::max(peak_pages, live_pages());
  }

  void unref(int32_t id, int64_t *freed) {
    if (--refcount[id] == 0) {
      freebits[id / 64] |= 1ull << (id % 64);
      if (id < free_hint) free_hint = id;
      ++n_free;
      if (freed) ++*freed;
    }
  }

  Seq *get(sq_seq h) {
    if (h < 0 || h >= (int32_t)seqs.size() || !seqs[h].live) return nullptr;
    return &seqs[h];
  }

  int32_t *pt_row(sq_seq h) { return pt_dev + (int64_t)h * cfg.max_pages_per_seq; }
  int32_t *mask_row(sq_seq h) { return mask_dev + (int64_t)h * cfg.max_pages_per_seq; }

  // ---- profiling ----
  hipEvent_t take_event() {
    if (!ev_pool.empty()) {
      hipEvent_t e = ev_pool.back();
      ev_pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
  bool prof_begin(hipStream_t s, ProfPair *pp, int kind) {
    if (!prof_on) return false;
    pp->a = take_event();
    pp->b = take_event();
    pp->kind = kind;
    if (!pp->a || !pp->b) return false;
    (void)hipEventRecord(pp->a, s);
    return true;
  }
  void prof_end(hipStream_t s, ProfPair *pp, bool active) {
    if (!active) return;
    (void)hipEventRecord(pp->b, s);
    prof_pending.push_back(*pp);
  }
};

namespace {

sq_status check_stream_store(sq_store *s) {
  if (!s) return fail(SQ_ERR_INVALID, "null store");
  return SQ_OK;
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

// Upload host int32 data to the workspace through the pinned staging buffer,
// in stream order.  The staging buffer is reused only after the copy that
// last read it has completed.
sq_status upload(sq_store *s, int32_t *dev_dst, const int32_t *src, size_t n, hipStream_t strm) {
  if (n == 0) return SQ_OK;
  if (s->staging_pending) {
    hipError_t e = hipEventSynchronize(s->staging_ev);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(staging)");
    s->staging_pending = false;
  }
  std::memcpy(s->staging, src, n * 4);
  hipError_t e = hipMemcpyAsync(dev_dst, s->staging, n * 4, hipMemcpyHostToDevice, strm);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(upload)");
  e = hipEventRecord(s->staging_ev, strm);
  if (e != hipSuccess) return hip_fail(e, "hipEventRecord(staging)");
  s->staging_pending = true;
  return SQ_OK;
}

// The whole keep-mask row of sequence h (all-kept past its pages).
sq_status upload_mask_row(sq_store *s, sq_seq h, hipStream_t strm) {
  const Seq &q = s->seqs[h];
  std::vector<int32_t> row(s->cfg.max_pages_per_seq, 0xffff);
  for (size_t i = 0; i < q.kmask.size(); ++i) row[i] = q.kmask[i];
  s->mask_dirty[h] = 1;
  return upload(s, s->mask_row(h), row.data(), row.size(), strm);
}

// Before a plan that reads keep masks: rows of unmasked sequences in it
// that may hold old masks become all-kept.
sq_status clean_mask_rows(sq_store *s, const sq_seq *seqs, int32_t batch, hipStream_t strm) {
  for (int b = 0; b < batch; ++b) {
    const sq_seq h = seqs[b];
    if (s->seqs[h].n_masked > 0 || !s->mask_dirty[h]) continue;
    hipError_t e = sq::launch_fill_i32(s->mask_row(h), 0xffff, s->cfg.max_pages_per_seq, strm);
    if (e != hipSuccess) return hip_fail(e, "keep-mask row");
    s->mask_dirty[h] = 0;
  }
  return SQ_OK;
}

// ---------------------------------------------------------------------------
// Decode planning.
struct PlanSeg {
  sq::Seg seg;
  bool mfma;
  int32_t members[sq::kMaxMembers];
};

struct Plan {
  std::vector<PlanSeg> segs;
  int n_groups = 0;
  int64_t total[2] = {0, 0}; // flattened pages per launch (0: VALU, 1: MFMA)
  int32_t n_wg[2] = {0, 0};  // workgroups per launch
  int32_t rb[2] = {1, 1};    // row blocks of 16 query rows per tile (MFMA launch: 1 or 2)
  int32_t slot_base[2] = {0, 0};
  int32_t seg_index[sq::kMaxSegs]; // index of each segment inside its launch
  bool pages_reread = false; // some page is read by more than one segment
  bool masked = false;       // some entry has slots masked by deferred evictions
  int32_t n_slots = 0;       // partial slots the launches write
  int64_t kv_bytes = 0, kv_bytes_logical = 0, io_bytes = 0;
  int64_t kv_bytes_valu = 0, kv_bytes_mfma = 0;
};

// Index of the first i < n with a[i] != b[i] (n if none): memcmp over blocks,
// then the block that differs element by element.
template <class T> int64_t first_diff(const T *a, const T *b, int64_t n) {
  constexpr int64_t B = 256;
  int64_t i = 0;
  while (i + B <= n && std::memcmp(a + i, b + i, B * sizeof(T)) == 0) i += B;
  while (i < n && a[i] == b[i]) ++i;
  return i;
}

// keep_last >= 0: each entry attends only to its last keep_last cached
// tokens (a window), read on its own; < 0: every token.  max_rb: row blocks
// of 16 query rows a tile may take (2 for a plain decode call on a bf16
// store, whose wide tiles then run on the two-block kernel; 1 for the
// fused step, whose launches are fixed per batch and mode, and for an
// 8-bit store).
sq_status build_plan(sq_store *s, const sq_seq *seqs, int32_t batch, int32_t mode, Plan *plan,
                     int64_t keep_last = -1, int max_rb = 1) {
  const int64_t tok_bytes = (int64_t)s->cfg.num_kv_heads * s->cfg.head_dim * 2 * s->elem_bytes();
  if (s->kv8) max_rb = 1;
  const int max_mem = std::min(sq::kMaxMembers, max_rb * sq::kRows / s->G);
  const bool grouping = mode == SQ_ATTN_AUTO || mode == SQ_ATTN_SHARED_PREFIX;
  // AUTO reads a sequence on its own on the MFMA tile too
  const bool single_mfma = mode == SQ_ATTN_MFMA || mode == SQ_ATTN_AUTO;

  auto add_seg = [&](int32_t row, int32_t page0, int64_t ntok, bool mfma,
                     const std::vector<int> &members, int32_t tok0 = 0) {
    PlanSeg ps{};
    ps.seg.page0 = page0;
    ps.seg.ntok = (int32_t)ntok;
    ps.seg.rmt = (uint32_t)row | (uint32_t)members.size() << 8 | (uint32_t)tok0 << 16;
    ps.seg.mem[0] = ps.seg.mem[1] = 0;
    for (size_t j = 0; j < members.size(); ++j) {
      ps.seg.mem[j >> 2] |= (uint32_t)members[j] << (8 * (j & 3));
      ps.members[j] = members[j];
    }
    ps.mfma = mfma;
    plan->segs.push_back(ps);
  };
  // per entry: page list, keep masks (null: none) and full pages
  const int32_t *pages_of[sq::kMaxBatch];
  const uint16_t *kmask_of[sq::kMaxBatch];
  int64_t full_of[sq::kMaxBatch];
  for (int b = 0; b < batch; ++b) {
    const Seq &q = s->seqs[seqs[b]];
    pages_of[b] = q.pages.data();
    kmask_of[b] = q.kmask.empty() ? nullptr : q.kmask.data();
    full_of[b] = q.length / s->P;
    plan->masked = plan->masked || q.n_masked > 0;
  }
  auto full_pages = [&](int b) { return full_of[b]; };
  auto page_at = [&](int b, int64_t i) { return pages_of[b][i]; };
  // entries share a page only when they also mask the same slots of it
  auto key_at = [&](int b, int64_t i) -> int64_t {
    return (int64_t)pages_of[b][i] | (int64_t)(kmask_of[b] ? kmask_of[b][i] : 0xffff) << 32;
  };
  auto add_private = [&](int b, int64_t p0) {
    const int64_t rest = s->seqs[seqs[b]].length - p0 * s->P;
    if (rest > 0) add_seg(seqs[b], (int32_t)p0, rest, single_mfma, {b});
  };

  // Sequences whose page lists agree on a run of physical pages share that
  // run (an auxiliary branch aliases its parent's pages, a branch of a
  // branch aliases both).  The entries reaching page p0 together split by
  // the id of their page p0; each part of two or more reads the run they
  // all share once, on the multi-query tile (at most max_mem entries per
  // tile, so a wider part is read once per tile), then splits again after
  // it: a tree of shared runs, at most kMaxSrc - 1 deep, each entry's own
  // suffix at the leaf.
  std::function<void(const std::vector<int> &, int64_t, int)> node =
      [&](const std::vector<int> &mem, int64_t p0, int depth) {
        std::vector<std::pair<int64_t, std::vector<int>>> parts; // first-seen order
        for (int b : mem) {
          const int64_t key = full_pages(b) > p0 ? key_at(b, p0) : -1;
          auto it = std::find_if(parts.begin(), parts.end(),
                                 [&](const auto &pt) { return key >= 0 && pt.first == key; });
          if (it == parts.end()) parts.push_back({key, {b}});
          else it->second.push_back(b);
        }
        for (auto &pt : parts) {
          const std::vector<int> &part = pt.second;
          if (pt.first < 0 || part.size() < 2 || depth >= sq::kMaxSrc - 1) {
            if (pt.first >= 0 && part.size() >= 2) plan->pages_reread = true; // too deep
            for (int b : part) add_private(b, p0);
            continue;
          }
          if ((int)part.size() > max_mem) plan->pages_reread = true;
          for (size_t c0 = 0; c0 < part.size(); c0 += max_mem) {
            const std::vector<int> tile(part.begin() + c0,
                                        part.begin() + std::min(part.size(), c0 + max_mem));
            if (tile.size() < 2) {
              add_private(tile[0], p0);
              continue;
            }
            // they share page p0, and every later full page both the page
            // ids and the keep masks of the tile agree on
            int64_t p1 = full_pages(tile[0]);
            for (int b : tile) p1 = std::min(p1, full_pages(b));
            for (size_t m = 1; m < tile.size(); ++m) {
              const int b = tile[m], b0 = tile[0];
              const int64_t n = p1 - p0 - 1;
              int64_t d = first_diff(pages_of[b] + p0 + 1, pages_of[b0] + p0 + 1, n);
              if (kmask_of[b] || kmask_of[b0]) {
                for (int64_t i = 0; i < d; ++i)
                  if (key_at(b, p0 + 1 + i) != key_at(b0, p0 + 1 + i)) {
                    d = i;
                    break;
                  }
              }
              p1 = p0 + 1 + d;
            }
            ++plan->n_groups;
            add_seg(seqs[tile[0]], (int32_t)p0, (p1 - p0) * s->P, true, tile);
            node(tile, p1, depth + 1);
          }
        }
      };

  if (keep_last >= 0) {
    // windows: [lo, L) from page lo / P, masked below lo % P on that page
    for (int b = 0; b < batch; ++b) {
      const int64_t L = s->seqs[seqs[b]].length, lo = std::max<int64_t>(0, L - keep_last);
      plan->kv_bytes_logical += (L - lo) * tok_bytes;
      const int64_t p0 = lo / s->P;
      if (L > lo) add_seg(seqs[b], (int32_t)p0, L - p0 * s->P, single_mfma, {b}, (int32_t)(lo - p0 * s->P));
    }
    plan->pages_reread = batch > 1; // branches' windows often meet on shared pages
  } else if (grouping) {
    for (int b = 0; b < batch; ++b) plan->kv_bytes_logical += s->seqs[seqs[b]].length * tok_bytes;
    std::vector<int> all(batch);
    for (int b = 0; b < batch; ++b) all[b] = b;
    node(all, 0, 0);
  } else {
    for (int b = 0; b < batch; ++b) plan->kv_bytes_logical += s->seqs[seqs[b]].length * tok_bytes;
    // per-sequence tiles; pages two entries share are read twice
    for (int b = 0; b < batch && !plan->pages_reread; ++b)
      for (int c = b + 1; c < batch; ++c)
        if (full_pages(b) > 0 && full_pages(c) > 0 && page_at(b, 0) == page_at(c, 0)) {
          plan->pages_reread = true;
          break;
        }
    for (int b = 0; b < batch; ++b) add_private(b, 0);
  }

  if ((int)plan->segs.size() > sq::kMaxSegs)
    return fail(SQ_ERR_INVALID, "decode batch needs %d segments (max %d)", (int)plan->segs.size(),
                sq::kMaxSegs);
  // Each launch lays its segments' rows (segment, KV head) end to end in one
  // flattened page range and splits it evenly over its workgroups: at most
  // one round of the GPU's resident workgroups, at least `min_wg_pages`
  // pages each, never more workgroups than pages.
  const int hkv = s->cfg.num_kv_heads;
  for (const PlanSeg &ps : plan->segs)
    if (ps.mfma && ps.seg.nmem() * s->G > sq::kRows) plan->rb[1] = 2;
  int count[2] = {0, 0};
  for (size_t i = 0; i < plan->segs.size(); ++i) {
    PlanSeg &ps = plan->segs[i];
    const int L = ps.mfma ? 1 : 0;
    const int64_t np = (ps.seg.ntok + s->P - 1) / s->P;
    ps.seg.start = (int32_t)plan->total[L];
    plan->seg_index[i] = count[L]++;
    plan->total[L] += (np + s->row_pad[L]) * hkv;
    const int64_t seg_bytes = (int64_t)(ps.seg.ntok - ps.seg.tok0()) * tok_bytes;
    plan->kv_bytes += seg_bytes;
    (L == 0 ? plan->kv_bytes_valu : plan->kv_bytes_mfma) += seg_bytes;
    plan->io_bytes += np * 4;
  }
  int32_t slots = 0;
  for (int L = 0; L < 2; ++L) {
    if (plan->total[L] == 0) continue;
    if (plan->total[L] > INT32_MAX) return fail(SQ_ERR_INVALID, "decode batch too large");
    const int64_t fill = (int64_t)s->cus * (plan->rb[L] == 2 ? s->wg_per_cu_rb2 : s->wg_per_cu[L]);
    const int64_t min_pages = L == 1 ? s->min_wg_pages_mfma : s->min_wg_pages_valu;
    int64_t n = std::min<int64_t>(fill, (plan->total[L] + min_pages - 1) / min_pages);
    n = std::max<int64_t>(1, std::min<int64_t>(n, plan->total[L]));
    // each workgroup's piece of each row owns rb consecutive slots
    const int64_t room = (sq::kMaxItems - slots) / plan->rb[L] - (int64_t)count[L] * hkv;
    if (room < 1) return fail(SQ_ERR_INVALID, "decode batch needs too many partial slots");
    n = std::min<int64_t>(n, room);
    plan->n_wg[L] = (int32_t)n;
    plan->slot_base[L] = slots;
    slots += ((int32_t)n + count[L] * hkv) * plan->rb[L];
  }
  plan->n_slots = slots;
  plan->io_bytes += (int64_t)batch * s->cfg.num_q_heads * s->cfg.head_dim * (2 + 4);
  return SQ_OK;
}

// A layer's region of a pool (element strides; E4M3 elements are bytes).
uint16_t *layer_pool(sq_store *s, uint16_t *pool, int32_t layer) {
  return reinterpret_cast<uint16_t *>(reinterpret_cast<char *>(pool) +
                                      layer * s->pools.layer_stride * (s->kv8 ? 1 : 2));
}

// The arguments of a layer's decode launches that no plan changes (the
// partials in the workspace, or in `pp`).
sq::DecodeStatic decode_static(sq_store *s, int32_t layer, const void *q, float scale, bool nt,
                               const sq::StaticPartials *pp = nullptr) {
  sq::DecodeStatic st{};
  st.q = static_cast<const uint16_t *>(q);
  st.k = layer_pool(s, s->pools.k, layer);
  st.v = layer_pool(s, s->pools.v, layer);
  st.pt = s->pt_dev;
  st.mask = s->mask_dev;
  st.part_m = pp ? pp->m : s->part_m;
  st.part_l = pp ? pp->l : s->part_l;
  st.part_acc = pp ? pp->acc : s->part_acc;
  st.page_stride = s->pools.page_stride;
  st.head_stride = s->pools.head_stride;
  st.max_pages = s->cfg.max_pages_per_seq;
  st.hq = s->cfg.num_q_heads;
  st.hkv = s->cfg.num_kv_heads;
  // an 8-bit store's K scale joins the score scale
  st.scale_log2 = (float)((double)scale * 1.4426950408889634 * (double)s->k_scale(layer));
  st.nontemporal = nt ? 1 : 0;
  st.kv8 = s->kv8 ? 1 : 0;
  return st;
}

sq::MergeStatic merge_static(sq_store *s, int32_t layer, float *out, const float *sinks,
                             const sq::StaticPartials *pp = nullptr) {
  sq::MergeStatic st{};
  st.out = out;
  st.sinks = sinks;
  st.sink_scale = 1.4426950408889634f;
  st.out_scale = s->v_scale(layer); // 1 unless the store is 8-bit
  st.part_m = pp ? pp->m : s->part_m;
  st.part_l = pp ? pp->l : s->part_l;
  st.part_acc = pp ? pp->acc : s->part_acc;
  st.hq = s->cfg.num_q_heads;
  st.group = s->G;
  st.hkv = s->cfg.num_kv_heads;
  return st;
}

// The two launches' plans and every entry's merge sources.
void fill_dyn(sq_store *s, const Plan &plan, sq::DecodeDyn dyn[2], sq::MergeDyn *md) {
  for (int L = 0; L < 2; ++L) {
    sq::DecodeDyn &d = dyn[L];
    d.n_segs = 0;
    for (const PlanSeg &ps : plan.segs)
      if (ps.mfma == (L == 1)) d.segs[d.n_segs++] = ps.seg;
    d.total = (int32_t)plan.total[L];
    d.row_pad = s->row_pad[L];
    d.masked = plan.masked ? 1 : 0;
    d.rb = plan.rb[L];
    d.n_wg = plan.n_wg[L];
    d.slot_base = plan.slot_base[L];
    md->total[L] = d.total;
    md->row_pad[L] = d.row_pad;
    md->n_wg[L] = d.n_wg;
    md->slot_base[L] = d.slot_base;
    md->rb[L] = d.rb;
  }
  for (size_t i = 0; i < plan.segs.size(); ++i) {
    const PlanSeg &ps = plan.segs[i];
    md->seg_start[i] = ps.seg.start;
    md->seg_npages[i] = (ps.seg.ntok + s->P - 1) / s->P;
    md->seg_meta[i] = (ps.mfma ? 1 : 0) | plan.seg_index[i] << 1;
    for (int j = 0; j < ps.seg.nmem(); ++j) {
      const int b = ps.members[j];
      const int e = md->n_src[b]++;
      md->src[b][e >> 1] |= (uint32_t)(i | j << 8) << (16 * (e & 1));
    }
  }
}

// A small call's merge row lists in the arguments (MergeRows): the same
// arithmetic the merge kernel does from the plan's tables, done here once.
void fill_inline_rows(const sq_store *s, int batch, sq::MergeArgs *ma) {
  const sq::MergeDyn &md = ma->dyn;
  const int hkv = s->cfg.num_kv_heads;
  ma->n_inline = 0;
  if (hkv > sq::kInlineG || (int64_t)batch * sq::kInlineG > sq::kInlineRows) return;
  for (int b = 0; b < batch; ++b)
    for (int g = 0; g < hkv; ++g) {
      sq::MergeRows &r = ma->rows[b * sq::kInlineG + g];
      for (int e = 0; e < sq::kMaxSrc; ++e) {
        r.base[e] = 0;
        r.cnt_step[e] = 0;
        if (e >= md.n_src[b]) continue;
        const int sr = (int)((md.src[b][e >> 1] >> (16 * (e & 1))) & 0xffff);
        const int si = sr & 0xff, member = (sr >> 8) & 0xf;
        const int L = md.seg_meta[si] & 1, seg = md.seg_meta[si] >> 1;
        const int np = md.seg_npages[si];
        const int64_t R = (int64_t)md.seg_start[si] + (int64_t)g * (np + md.row_pad[L]);
        const int w_lo = sq::wg_of(R, md.total[L], md.n_wg[L]);
        const int w_hi = sq::wg_of(R + np - 1, md.total[L], md.n_wg[L]);
        const int rb = md.rb[L];
        r.base[e] = (md.slot_base[L] + rb * (w_lo + seg * hkv + g)) * sq::kRows + member * s->G;
        r.cnt_step[e] = (w_hi - w_lo + 1) | (rb * sq::kRows) << 16;
      }
    }
  ma->n_inline = 1;
}

} // namespace

// ===========================================================================
extern "C" {

int32_t sq_abi_version(void) { return SQ_ABI_VERSION; }

sq_status sq_trace_open(const char *path) { return trace_open(path); }

const char *sq_last_error(void) { return g_err.c_str(); }

uint64_t sq_workspace_bytes(const sq_store_config *cfg) {
  if (!shape_ok(cfg, !(cfg && (cfg->flags & SQ_STORE_METADATA_ONLY)), nullptr)) return 0;
  if (cfg->flags & SQ_STORE_METADATA_ONLY) return 0;
  return layout_of(*cfg).total;
}

uint64_t sq_pool_bytes(const sq_store_config *cfg, int32_t which) {
  if (!shape_ok(cfg, false, nullptr)) return 0;
  const uint64_t kv = (uint64_t)cfg->num_layers * cfg->num_pages * cfg->num_kv_heads *
                      cfg->page_size * cfg->head_dim * ((cfg->flags & SQ_STORE_KV_FP8) ? 1 : 2);
  if (which == 0 || which == 1) return kv;
  if (which == 2) return (uint64_t)cfg->num_pages * cfg->page_size * 4;
  return 0;
}

sq_status sq_store_create(const sq_store_config *cfg, sq_store **out) {
  SQ_TRACE_CALL("sq_store_create", "layers=%d q_heads=%d kv_heads=%d head_dim=%d pages=%d flags=%u", cfg ? cfg->num_layers : -1, cfg ? cfg->num_q_heads : -1, cfg ? cfg->num_kv_heads : -1, cfg ? cfg->head_dim : -1, cfg ? cfg->num_pages : -1, cfg ? cfg->flags : 0u);
  if (!out) return fail(SQ_ERR_INVALID, "null output pointer");
  const bool device = cfg && !(cfg->flags & SQ_STORE_METADATA_ONLY);
  std::string why;
  if (!shape_ok(cfg, device, &why)) return fail(SQ_ERR_INVALID, "bad configuration: %s", why.c_str());
  Layout lay{};
  if (device) {
    if (!cfg->k_pool || !cfg->v_pool || !cfg->pos_pool || !cfg->workspace)
      return fail(SQ_ERR_INVALID, "device mode needs k_pool, v_pool, pos_pool and workspace");
    if (((uintptr_t)cfg->k_pool | (uintptr_t)cfg->v_pool | (uintptr_t)cfg->pos_pool |
         (uintptr_t)cfg->workspace) & 255u)
      return fail(SQ_ERR_INVALID, "pools and workspace must be 256-byte aligned");
    lay = layout_of(*cfg);
    if (cfg->workspace_bytes < lay.total)
      return fail(SQ_ERR_INVALID, "workspace too small: %llu < %llu bytes",
                  (unsigned long long)cfg->workspace_bytes, (unsigned long long)lay.total);
  }
  sq_store *s = new sq_store();
  s->cfg = *cfg;
  s->device = device;
  s->kv8 = (cfg->flags & SQ_STORE_KV_FP8) != 0;
  if (s->kv8) s->kv_scales.assign(cfg->kv_scales, cfg->kv_scales + 2 * cfg->num_layers);
  s->cfg.kv_scales = s->kv8 ? s->kv_scales.data() : nullptr;
  s->P = cfg->page_size;
  s->G = cfg->num_q_heads / cfg->num_kv_heads;
  s->D = cfg->head_dim;
  s->refcount.assign(cfg->num_pages, 0);
  s->freebits.assign((cfg->num_pages + 63) / 64, 0);
  for (int32_t i = 0; i < cfg->num_pages; ++i) s->freebits[i / 64] |= 1ull << (i % 64);
  s->n_free = cfg->num_pages;
  s->seqs.resize(cfg->max_seqs);
  if (device) {
    s->lay = lay;
    char *ws = static_cast<char *>(cfg->workspace);
    s->pt_dev = reinterpret_cast<int32_t *>(ws + lay.pt);
    s->mask_dev = reinterpret_cast<int32_t *>(ws + lay.mask);
    s->mask_dirty.assign(cfg->max_seqs, 1);
    s->ev_keep = reinterpret_cast<uint8_t *>(ws + lay.keep);
    s->ev_dst = reinterpret_cast<int32_t *>(ws + lay.dst);
    s->ev_src = reinterpret_cast<int32_t *>(ws + lay.src);
    s->ev_upload = reinterpret_cast<int32_t *>(ws + lay.upload);
    s->part_m = reinterpret_cast<float *>(ws + lay.part_m);
    s->part_l = reinterpret_cast<float *>(ws + lay.part_l);
    s->part_acc = reinterpret_cast<float *>(ws + lay.part_acc);
    s->step_dev = reinterpret_cast<sq::StepPlan *>(ws + lay.step);
    sq::Pools &p = s->pools;
    p.k = static_cast<uint16_t *>(cfg->k_pool);
    p.v = static_cast<uint16_t *>(cfg->v_pool);
    p.pos = cfg->pos_pool;
    p.nl = cfg->num_layers;
    p.hkv = cfg->num_kv_heads;
    p.d = cfg->head_dim;
    p.np = cfg->num_pages;
    p.page_stride = (int64_t)s->P * s->D;
    p.head_stride = p.page_stride * cfg->num_pages;
    p.layer_stride = p.head_stride * cfg->num_kv_heads;
    p.kv8 = s->kv8 ? 1 : 0;
    if (s->kv8) { // K scale, V scale and their inverses per layer, on the device
      std::vector<float> sc(4 * cfg->num_layers);
      for (int l = 0; l < cfg->num_layers; ++l) {
        sc[4 * l] = s->k_scale(l);
        sc[4 * l + 1] = s->v_scale(l);
        sc[4 * l + 2] = s->inv(s->k_scale(l));
        sc[4 * l + 3] = s->inv(s->v_scale(l));
      }
      float *dev = reinterpret_cast<float *>(ws + lay.scales);
      hipError_t e = hipMemcpy(dev, sc.data(), sc.size() * 4, hipMemcpyHostToDevice);
      if (e != hipSuccess) {
        delete s;
        return hip_fail(e, "hipMemcpy(kv scales)");
      }
      p.scales = dev;
    }
    {
      int dev = 0, cus = 0, nb = 0;
      if (hipGetDevice(&dev) == hipSuccess &&
          hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
          cus > 0)
        s->cus = cus;
      if (sq::decode_blocks_per_cu(s->kv8 ? 3 : 0, s->D, s->G, &nb) == hipSuccess && nb > 0)
        s->wg_per_cu[0] = nb;
      nb = 0;
      if (sq::decode_blocks_per_cu(s->kv8 ? 2 : 1, s->D, s->G, &nb) == hipSuccess && nb > 0)
        s->wg_per_cu[1] = nb;
      nb = 0;
      if (s->G > 1 && sq::decode_blocks_per_cu(4, s->D, s->G, &nb) == hipSuccess && nb > 0)
        s->wg_per_cu_rb2 = nb;
    }
    // set-up of the allocation-free entry point: its device array's address
    // on this GPU (a failure only disables that entry point)
    s->spart_err = sq::static_partials(&s->spart);
    void *host = nullptr;
    hipError_t e = hipHostMalloc(&host, lay.upload_elems * 4, hipHostMallocDefault);
    if (e != hipSuccess) {
      delete s;
      return hip_fail(e, "hipHostMalloc(staging)");
    }
    s->staging = static_cast<int32_t *>(host);
    e = hipEventCreateWithFlags(&s->staging_ev, hipEventDisableTiming);
    if (e != hipSuccess) {
      (void)hipHostFree(host);
      delete s;
      return hip_fail(e, "hipEventCreate");
    }
    for (int i = 0; i < 2 && e == hipSuccess; ++i) {
      void *sh = nullptr;
      e = hipHostMalloc(&sh, sizeof(sq::StepPlan), hipHostMallocDefault);
      if (e == hipSuccess) {
        s->step_staging[i] = static_cast<sq::StepPlan *>(sh);
        e = hipEventCreateWithFlags(&s->step_ev[i], hipEventDisableTiming);
      }
    }
    if (e != hipSuccess) {
      (void)hipEventDestroy(s->staging_ev);
      (void)hipHostFree(host);
      for (int i = 0; i < 2; ++i) {
        if (s->step_staging[i]) (void)hipHostFree(s->step_staging[i]);
        if (s->step_ev[i]) (void)hipEventDestroy(s->step_ev[i]);
      }
      delete s;
      return hip_fail(e, "step plan staging");
    }
  }
  *out = s;
  return SQ_OK;
}

sq_status sq_store_destroy(sq_store *s) {
  SQ_TRACE_CALL("sq_store_destroy", "store=%p", (void *)s);
  if (!s) return fail(SQ_ERR_INVALID, "null store");
  if (s->device) {
    if (s->staging_pending) (void)hipEventSynchronize(s->staging_ev);
    for (auto &pp : s->prof_pending) {
      (void)hipEventSynchronize(pp.b);
      (void)hipEventDestroy(pp.a);
      (void)hipEventDestroy(pp.b);
    }
    for (hipEvent_t e : s->ev_pool) (void)hipEventDestroy(e);
    if (s->staging_ev) (void)hipEventDestroy(s->staging_ev);
    if (s->staging) (void)hipHostFree(s->staging);
    for (int i = 0; i < 2; ++i) {
      if (s->step_pending[i]) (void)hipEventSynchronize(s->step_ev[i]);
      if (s->step_ev[i]) (void)hipEventDestroy(s->step_ev[i]);
      if (s->step_staging[i]) (void)hipHostFree(s->step_staging[i]);
    }
  }
  delete s;
  return SQ_OK;
}

sq_status sq_seq_create(sq_store *s, sq_seq *out) {
  SQ_TRACE_CALL("sq_seq_create", "store=%p", (void *)s);
  if (!s || !out) return fail(SQ_ERR_INVALID, "null argument");
  for (int32_t h = 0; h < s->cfg.max_seqs; ++h) {
    if (!s->seqs[h].live) {
      s->seqs[h] = Seq();
      s->seqs[h].live = true;
      ++s->st.live_seqs;
      *out = h;
      return SQ_OK;
    }
  }
  return fail(SQ_ERR_INVALID, "all %d sequence handles are live", s->cfg.max_seqs);
}

sq_status sq_append(sq_store *s, sq_seq h, int32_t n, const void *k_new, const void *v_new,
                    void *stream) {
  SQ_TRACE_CALL("sq_append", "store=%p seq=%d n=%d", (void *)s, h, n);
  if (!s) return fail(SQ_ERR_INVALID, "null store");
  Seq *q = s->get(h);
  if (!q) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", h);
  if (n < 0) return fail(SQ_ERR_INVALID, "negative token count");
  if (n == 0) return SQ_OK;
  const int64_t new_len = q->length + n;
  const int64_t want = (new_len + s->P - 1) / s->P;
  if (want > s->cfg.max_pages_per_seq)
    return fail(SQ_ERR_INVALID, "sequence %d would need %lld pages (max %d)", h, (long long)want,
                s->cfg.max_pages_per_seq);
  if (want - (int64_t)q->pages.size() > s->n_free)
    return fail(SQ_ERR_NO_PAGES, "append needs %lld pages, %lld free",
                (long long)(want - (int64_t)q->pages.size()), (long long)s->n_free);
  if (s->device) {
    if (!k_new || !v_new) return fail(SQ_ERR_INVALID, "null K/V");
    if (!aligned16(k_new) || !aligned16(v_new)) return fail(SQ_ERR_INVALID, "K/V must be 16-byte aligned");
    if (q->next_pos + n > INT32_MAX) return fail(SQ_ERR_INVALID, "positions exceed int32");
  }
  ++s->gen;
  const int64_t old_len = q->length;
  const int32_t old_np = (int32_t)q->pages.size();
  while ((int64_t)q->pages.size() < want) q->pages.push_back(s->alloc_page());
  grow_kmask(*q);
  runs_append(*q, n);
  const int64_t pos0 = q->next_pos;
  q->length = new_len;
  q->next_pos += n;
  s->st.append_tokens += n;
  if (!s->device) return SQ_OK;

  hipStream_t strm = static_cast<hipStream_t>(stream);
  s->last_stream = strm;
  // launches of at most kMaxAppendPages pages each
  int64_t t = 0;
  while (t < n) {
    const int64_t gidx = old_len + t; // global token index
    const int32_t first_page = (int32_t)(gidx / s->P);
    const int32_t slot0 = (int32_t)(gidx % s->P);
    const int64_t room = (int64_t)sq::kMaxAppendPages * s->P - slot0;
    const int64_t cnt = std::min<int64_t>(room, n - t);
    sq::AppendArgs a{};
    a.n_tok = (int32_t)cnt;
    a.n_total = n;
    a.tok0 = (int32_t)t;
    a.slot0 = slot0;
    a.pos0 = (int32_t)(pos0 + t);
    a.n_pages = (int32_t)((slot0 + cnt + s->P - 1) / s->P);
    a.pt_first = first_page;
    a.new_from = std::max(0, old_np - first_page);
    a.pt_row = s->pt_row(h);
    for (int i = 0; i < a.n_pages; ++i) a.page_ids[i] = q->pages[first_page + i];
    ProfPair pp;
    const bool on = s->prof_begin(strm, &pp, kProfAppend);
    hipError_t e = sq::launch_append(s->pools, a, k_new, v_new, strm);
    s->prof_end(strm, &pp, on);
    if (e != hipSuccess) return hip_fail(e, "append kernel");
    t += cnt;
  }
  return SQ_OK;
}

namespace {

// One token for each of `batch` distinct sequences (sq_append_batch and
// sq_step_begin): the checks, made before anything changes.
// Attention options, checked; null = none.
sq_status take_opts(const sq_attn_opts *opts, sq_attn_opts *o) {
  *o = sq_attn_opts{};
  if (!opts) return SQ_OK;
  if (opts->window < 0) return fail(SQ_ERR_INVALID, "window %d < 0", opts->window);
  if (opts->reserved != 0) return fail(SQ_ERR_INVALID, "sq_attn_opts.reserved must be 0");
  if (((uintptr_t)opts->sinks & 3u) != 0) return fail(SQ_ERR_INVALID, "sinks must be 4-byte aligned");
  *o = *opts;
  return SQ_OK;
}

sq_status check_one_token_each(sq_store *s, const sq_seq *seqs, int32_t batch) {
  if (!s || !seqs) return fail(SQ_ERR_INVALID, "null argument");
  if (batch < 1 || batch > SQ_MAX_BATCH) return fail(SQ_ERR_INVALID, "batch must be in [1, %d]", SQ_MAX_BATCH);
  int64_t need = 0;
  for (int b = 0; b < batch; ++b) {
    Seq *q = s->get(seqs[b]);
    if (!q) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", seqs[b]);
    for (int c = 0; c < b; ++c)
      if (seqs[c] == seqs[b]) return fail(SQ_ERR_INVALID, "sequence %d repeated in the batch", seqs[b]);
    if (q->length % s->P == 0) {
      if (q->length / s->P + 1 > s->cfg.max_pages_per_seq)
        return fail(SQ_ERR_INVALID, "sequence %d is at its page-list capacity", seqs[b]);
      ++need;
    }
    if (s->device && q->next_pos + 1 > INT32_MAX) return fail(SQ_ERR_INVALID, "positions exceed int32");
  }
  if (need > s->n_free) return fail(SQ_ERR_NO_PAGES, "append needs %lld pages, %lld free",
                                    (long long)need, (long long)s->n_free);
  return SQ_OK;
}

// ... and the change: each sequence gets its next slot (a new page when its
// last one is full, lowest id first, in batch order) and position.  Returns
// where each token goes: page, slot, position and the page-table index to
// set (or -1).
struct TokenSlots {
  int32_t page[sq::kMaxBatch], slot[sq::kMaxBatch], pos[sq::kMaxBatch], pt_index[sq::kMaxBatch];
};
void take_one_token_each(sq_store *s, const sq_seq *seqs, int32_t batch, TokenSlots *t) {
  ++s->gen;
  for (int b = 0; b < batch; ++b) {
    Seq &q = s->seqs[seqs[b]];
    t->pt_index[b] = -1;
    if (q.length % s->P == 0) {
      q.pages.push_back(s->alloc_page());
      grow_kmask(q);
      t->pt_index[b] = seqs[b] * s->cfg.max_pages_per_seq + (int32_t)q.pages.size() - 1;
    }
    t->page[b] = q.pages[q.length / s->P];
    t->slot[b] = (int32_t)(q.length % s->P);
    t->pos[b] = (int32_t)q.next_pos;
    runs_append(q, 1);
    q.length += 1;
    q.next_pos += 1;
  }
  s->st.append_tokens += batch;
}

// One decode call: the partials in the store's workspace (pp null), or in
// pp's buffers - the allocation-free entry point, which also records no
// profiling events (creating one may allocate).
sq_status decode_call(sq_store *s, int32_t layer, const sq_seq *seqs, int32_t batch, const void *q,
                      float *out, float scale, int32_t mode, const sq_attn_opts *opts,
                      void *stream, const sq::StaticPartials *pp) {
  sq_attn_opts o{};
  sq_status r = take_opts(opts, &o);
  if (r != SQ_OK) return r;
  if (!s || !seqs) return fail(SQ_ERR_INVALID, "null argument");
  if (!s->device) return fail(SQ_ERR_INVALID, "metadata-only store cannot run attention");
  if (batch < 1 || batch > SQ_MAX_BATCH) return fail(SQ_ERR_INVALID, "batch must be in [1, %d]", SQ_MAX_BATCH);
  if (layer < 0 || layer >= s->cfg.num_layers) return fail(SQ_ERR_INVALID, "layer %d out of range", layer);
  if (mode < SQ_ATTN_AUTO || mode > SQ_ATTN_MFMA) return fail(SQ_ERR_INVALID, "unknown mode %d", mode);
  if (!q || !out || !aligned16(q) || !aligned16(out))
    return fail(SQ_ERR_INVALID, "q and out must be non-null and 16-byte aligned");
  if (!std::isfinite(scale)) return fail(SQ_ERR_INVALID, "scale must be finite");
  for (int b = 0; b < batch; ++b)
    if (!s->get(seqs[b])) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", seqs[b]);
  Plan plan;
  r = build_plan(s, seqs, batch, mode, &plan, o.window > 0 ? o.window : -1, 2);
  if (r != SQ_OK) return r;
  if (plan.masked && o.window > 0)
    return fail(SQ_ERR_INVALID, "a window over a sequence with masked slots (compact it first)");
  if (pp && plan.n_slots > pp->slots)
    return fail(SQ_ERR_INVALID,
                "this call needs %d partial slots; the allocation-free entry point holds %d",
                plan.n_slots, pp->slots);

  hipStream_t strm = static_cast<hipStream_t>(stream);
  s->last_stream = strm;
  if (plan.masked) {
    r = clean_mask_rows(s, seqs, batch, strm);
    if (r != SQ_OK) return r;
  }
  sq::DecodeArgs da[2]{};
  sq::MergeArgs ma{};
  da[0].st = decode_static(s, layer, q, scale, !plan.pages_reread, pp);
  da[1].st = da[0].st;
  ma.st = merge_static(s, layer, out, o.sinks, pp);
  sq::DecodeDyn dyn[2]{};
  fill_dyn(s, plan, dyn, &ma.dyn);
  fill_inline_rows(s, batch, &ma);
  for (int pass = 0; pass < 2; ++pass) {
    da[pass].dyn = dyn[pass];
    if (da[pass].dyn.n_wg == 0) continue;
    ProfPair pe;
    const bool on = !pp && s->prof_begin(strm, &pe, pass == 0 ? kProfValu : kProfMfma);
    hipError_t e = pass == 0 ? sq::launch_decode_valu(s->D, s->G, da[pass], strm)
                             : sq::launch_decode_mfma(s->D, s->G, da[pass], strm);
    s->prof_end(strm, &pe, on);
    if (e != hipSuccess) return hip_fail(e, "decode kernel");
  }
  ProfPair pe;
  const bool on = !pp && s->prof_begin(strm, &pe, kProfMerge);
  hipError_t e = sq::launch_decode_merge(s->D, batch, ma, strm);
  s->prof_end(strm, &pe, on);
  if (e != hipSuccess) return hip_fail(e, "decode merge");
  ++s->st.decode_calls;
  s->st.decode_kv_bytes += plan.kv_bytes;
  s->st.decode_kv_bytes_logical += plan.kv_bytes_logical;
  return SQ_OK;
}

} // namespace

sq_status sq_append_batch(sq_store *s, const sq_seq *seqs, int32_t batch, const void *k_new,
                          const void *v_new, void *stream) {
  SQ_TRACE_CALL("sq_append_batch", "store=%p batch=%d", (void *)s, batch);
  sq_status r = check_one_token_each(s, seqs, batch);
  if (r != SQ_OK) return r;
  if (s->device) {
    if (!k_new || !v_new) return fail(SQ_ERR_INVALID, "null K/V");
    if (!aligned16(k_new) || !aligned16(v_new)) return fail(SQ_ERR_INVALID, "K/V must be 16-byte aligned");
  }
  TokenSlots t;
  take_one_token_each(s, seqs, batch, &t);
  sq::AppendBatchArgs a{};
  a.n = batch;
  a.pt = s->pt_dev;
  for (int b = 0; b < batch; ++b) {
    a.page[b] = t.page[b];
    a.slot[b] = t.slot[b];
    a.pos[b] = t.pos[b];
    a.pt_index[b] = t.pt_index[b];
  }
  if (!s->device) return SQ_OK;
  hipStream_t strm = static_cast<hipStream_t>(stream);
  s->last_stream = strm;
  ProfPair pp;
  const bool on = s->prof_begin(strm, &pp, kProfAppend);
  hipError_t e = sq::launch_append_batch(s->pools, a, k_new, v_new, strm);
  s->prof_end(strm, &pp, on);
  if (e != hipSuccess) return hip_fail(e, "append_batch kernel");
  return SQ_OK;
}

sq_status sq_span_mark(sq_store *s, sq_seq h, int32_t cursor, int64_t start, int64_t end) {
  SQ_TRACE_CALL("sq_span_mark", "store=%p seq=%d cursor=%d start=%lld end=%lld", (void *)s, h, cursor, (long long)start, (long long)end);
  if (!s) return fail(SQ_ERR_INVALID, "null store");
  Seq *q = s->get(h);
  if (!q) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", h);
  if (cursor < 0 || q->spans.count(cursor))
    return fail(SQ_ERR_INVALID, "cursor %d negative or already registered", cursor);
  if (!(0 <= start && start <= end && end <= q->length))
    return fail(SQ_ERR_SPAN, "span [%lld, %lld) outside [0, %lld]", (long long)start,
                (long long)end, (long long)q->length);
  if (end > start) {
    auto it = q->nonempty.lower_bound(start);
    if (it != q->nonempty.end() && it->first < end)
      return fail(SQ_ERR_SPAN, "span overlaps [%lld, %lld)", (long long)it->first, (long long)it->second);
    if (it != q->nonempty.begin()) {
      --it;
      if (it->second > start)
        return fail(SQ_ERR_SPAN, "span overlaps [%lld, %lld)", (long long)it->first, (long long)it->second);
    }
    q->nonempty[start] = end;
  }
  q->spans[cursor] = {start, end};
  return SQ_OK;
}

sq_status sq_fork(sq_store *s, sq_seq parent, int64_t fork_len, sq_seq *child, void *stream) {
  SQ_TRACE_CALL("sq_fork", "store=%p parent=%d fork_len=%lld", (void *)s, parent, (long long)fork_len);
  if (!s || !child) return fail(SQ_ERR_INVALID, "null argument");
  Seq *par = s->get(parent);
  if (!par) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", parent);
  if (!(0 <= fork_len && fork_len <= par->length))
    return fail(SQ_ERR_INVALID, "fork point %lld outside [0, %lld]", (long long)fork_len,
                (long long)par->length);
  int32_t h = -1;
  for (int32_t i = 0; i < s->cfg.max_seqs; ++i)
    if (!s->seqs[i].live) {
      h = i;
      break;
    }
  if (h < 0) return fail(SQ_ERR_INVALID, "all %d sequence handles are live", s->cfg.max_seqs);
  const int64_t full = fork_len / s->P;
  const int64_t tail = fork_len % s->P;
  if (tail && s->n_free < 1) return fail(SQ_ERR_NO_PAGES, "no page for the fork's tail copy");

  ++s->gen;
  Seq c;
  c.live = true;
  c.pages.assign(par->pages.begin(), par->pages.begin() + full);
  for (int32_t p : c.pages) ++s->refcount[p];
  int32_t tail_page = -1;
  if (tail) {
    tail_page = s->alloc_page();
    c.pages.push_back(tail_page);
  }
  c.length = fork_len;
  c.runs = runs_truncate(par->runs, fork_len);
  c.next_pos = fork_len == par->length ? par->next_pos : pos_at(*par, fork_len);
  for (auto &kv : par->spans)
    if (kv.second.second <= fork_len) {
      c.spans[kv.first] = kv.second;
      if (kv.second.second > kv.second.first) c.nonempty[kv.second.first] = kv.second.second;
    }
  c.parent = parent;
  if (par->n_masked > 0) { // the child's slots keep their masks
    c.kmask.assign(par->kmask.begin(), par->kmask.begin() + full);
    if (tail) c.kmask.push_back((uint16_t)(par->kmask[full] | (0xffffu << tail)));
    for (int64_t i = 0; i < fork_len; ++i) c.n_masked += !slot_kept(c, i, s->P);
    if (c.n_masked == 0) c.kmask.clear();
  }
  const int32_t src_tail_page = tail ? par->pages[full] : -1;
  s->seqs[h] = std::move(c);
  ++s->st.live_seqs;
  ++s->st.fork_calls;
  if (tail) ++s->st.fork_tail_copies;
  *child = h;
  if (!s->device) return SQ_OK;

  hipStream_t strm = static_cast<hipStream_t>(stream);
  s->last_stream = strm;
  hipError_t e = sq::launch_copy_i32(s->pt_row(h), s->pt_row(parent), (int32_t)full, -1,
                                     tail_page, strm);
  if (e != hipSuccess) return hip_fail(e, "fork page-table copy");
  if (tail) {
    e = sq::launch_copy_page(s->pools, src_tail_page, tail_page, strm);
    if (e != hipSuccess) return hip_fail(e, "fork tail copy");
  }
  if (s->seqs[h].n_masked > 0) {
    sq_status r = upload_mask_row(s, h, strm);
    if (r != SQ_OK) return r;
  }
  return SQ_OK;
}

sq_status sq_release(sq_store *s, sq_seq h) {
  SQ_TRACE_CALL("sq_release", "store=%p seq=%d", (void *)s, h);
  if (!s) return fail(SQ_ERR_INVALID, "null store");
  Seq *q = s->get(h);
  if (!q) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", h);
  ++s->gen;
  for (int32_t p : q->pages) s->unref(p, nullptr);
  *q = Seq();
  --s->st.live_seqs;
  return SQ_OK;
}

sq_status sq_evict_spans(sq_store *s, sq_seq h, const int32_t *cursor_ids, int32_t n,
                         void *stream, sq_evict_stats *stats) {
  return sq_evict_spans_ex(s, h, cursor_ids, n, 0, stream, stats);
}

sq_status sq_compact(sq_store *s, sq_seq h, void *stream, sq_evict_stats *stats) {
  SQ_TRACE_CALL("sq_compact", "store=%p seq=%d", (void *)s, h);
  return sq_evict_spans_ex(s, h, nullptr, 0, 0, stream, stats);
}

namespace {
// Deferred eviction: the spans' slots are masked, nothing moves.
sq_status evict_deferred(sq_store *s, sq_seq h, const std::vector<int32_t> &ids,
                         const std::vector<std::pair<int64_t, int64_t>> &sp, void *stream,
                         sq_evict_stats *stats) {
  if (s->P > 16) return fail(SQ_ERR_INVALID, "deferred eviction needs page_size <= 16");
  Seq *q = s->get(h);
  std::vector<uint16_t> km = q->kmask;
  if (km.empty()) km.assign(q->pages.size(), 0xffff);
  int64_t newly = 0;
  for (const auto &se : sp) // clear the span's bits page by page
    for (int64_t pg = se.first / s->P; pg * s->P < se.second; ++pg) {
      const int64_t lo = std::max<int64_t>(se.first - pg * s->P, 0);
      const int64_t hi = std::min<int64_t>(se.second - pg * s->P, s->P);
      const uint32_t bits = ((1u << hi) - 1u) & ~((1u << lo) - 1u);
      newly += __builtin_popcount(km[pg] & bits);
      km[pg] = (uint16_t)(km[pg] & ~bits);
    }
  const int64_t n_runs = count_runs(km, s->P);
  if (n_runs > SQ_MAX_EVICT_SPANS)
    return fail(SQ_ERR_INVALID, "sequence %d would hold %lld masked runs (max %d): compact it first",
                h, (long long)n_runs, SQ_MAX_EVICT_SPANS);
  sq_evict_stats es{};
  es.first_evicted = q->length;
  for (size_t pg = 0; pg < km.size(); ++pg)
    if (km[pg] != 0xffff) {
      es.first_evicted = (int64_t)pg * s->P + __builtin_ctz(~(uint32_t)km[pg]);
      break;
    }
  es.tokens_masked = newly;
  q->kmask = std::move(km);
  q->n_masked += newly;
  if (q->n_masked == 0) q->kmask.clear();
  for (int32_t c : ids) {
    auto it = q->spans.find(c);
    if (it->second.second > it->second.first) q->nonempty.erase(it->second.first);
    q->spans.erase(it);
  }
  ++s->st.evict_calls;
  if (stats) *stats = es;
  if (!s->device || newly == 0) return SQ_OK;
  hipStream_t strm = static_cast<hipStream_t>(stream);
  s->last_stream = strm;
  return upload_mask_row(s, h, strm);
}
// Launches of an in-place eviction.  Tail page k reads old list indices
// lo(k) .. hi(k), all >= fp + k.  A round [a, b) of tail pages can run as
// one parallel launch when no page of it reads the old page of another page
// of it (each reads its own before writing it): with every page's read
// range taken whole, adding page b is safe unless [lo(a), max hi] covers
// fp + b.  Rounds grow with the evicted tokens before them; when the rounds
// number more than kMaxInplaceRounds, the first ones run as one sweep (each
// workgroup takes their pages in order).
constexpr int64_t kMaxInplaceRounds = 64;

sq_status evict_inplace_launches(sq_store *s, sq_seq h, int64_t fp, int64_t n_new, int64_t Lp,
                                 const std::function<int64_t(int64_t)> &src_index,
                                 const sq::NewIds &ids, hipStream_t strm) {
  const int64_t P = s->P;
  auto lo_of = [&](int64_t k) { return src_index((fp + k) * P) / P; };
  auto hi_of = [&](int64_t k) { return src_index(std::min((fp + k + 1) * P, Lp) - 1) / P; };
  std::vector<std::pair<int64_t, int64_t>> rounds;
  for (int64_t a = 0; a < n_new;) {
    const int64_t lo = lo_of(a);
    int64_t hi = hi_of(a), b = a + 1;
    while (b < n_new && !(lo <= fp + b && fp + b <= hi)) hi = std::max(hi, hi_of(b++));
    rounds.push_back({a, b});
    a = b;
  }
  size_t first = 0; // rounds before it go to one sweep
  if ((int64_t)rounds.size() > kMaxInplaceRounds) first = rounds.size() - (kMaxInplaceRounds - 1);
  auto launch = [&](int64_t k0, int64_t n, int sweep) {
    sq::InplaceArgs ia{};
    ia.fp = (int32_t)fp;
    ia.k0 = (int32_t)k0;
    ia.n_pages = (int32_t)n;
    ia.new_len = (int32_t)Lp;
    ia.sweep = sweep;
    ia.src_of = s->ev_src;
    ia.pt_row = s->pt_row(h);
    ia.ids = ids;
    ProfPair pp;
    const bool on = s->prof_begin(strm, &pp, kProfGather);
    hipError_t e = sq::launch_evict_inplace(s->pools, ia, strm);
    s->prof_end(strm, &pp, on);
    return e == hipSuccess ? SQ_OK : hip_fail(e, "in-place eviction");
  };
  if (first > 0) {
    sq_status r = launch(0, rounds[first].first, 1);
    if (r != SQ_OK) return r;
  }
  for (size_t i = first; i < rounds.size(); ++i) {
    sq_status r = launch(rounds[i].first, rounds[i].second - rounds[i].first, 0);
    if (r != SQ_OK) return r;
  }
  return SQ_OK;
}

} // namespace

sq_status sq_evict_spans_ex(sq_store *s, sq_seq h, const int32_t *cursor_ids, int32_t n,
                            uint32_t flags, void *stream, sq_evict_stats *stats) {
  SQ_TRACE_CALL("sq_evict_spans", "store=%p seq=%d n_cursors=%d flags=%u", (void *)s, h, n, flags);
  if (!s) return fail(SQ_ERR_INVALID, "null store");
  Seq *q = s->get(h);
  if (!q) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", h);
  ++s->gen; // ends a begun decode step even when the call fails
  if (n < 0 || n > SQ_MAX_EVICT_SPANS)
    return fail(SQ_ERR_INVALID, "cursor count %d outside [0, %d]", n, SQ_MAX_EVICT_SPANS);
  if (n > 0 && !cursor_ids) return fail(SQ_ERR_INVALID, "null cursor list");
  std::vector<int32_t> ids(cursor_ids, cursor_ids + n);
  std::sort(ids.begin(), ids.end());
  ids.erase(std::unique(ids.begin(), ids.end()), ids.end());
  for (int32_t c : ids)
    if (!q->spans.count(c)) return fail(SQ_ERR_UNKNOWN_CURSOR, "cursor %d not registered on sequence %d", c, h);
  if (flags & ~SQ_EVICT_DEFER) return fail(SQ_ERR_INVALID, "unknown eviction flags 0x%x", flags);
  std::vector<std::pair<int64_t, int64_t>> sp;
  for (int32_t c : ids) {
    auto se = q->spans[c];
    if (se.second > se.first) sp.push_back(se);
  }
  std::sort(sp.begin(), sp.end());
  if (flags & SQ_EVICT_DEFER) return evict_deferred(s, h, ids, sp, stream, stats);
  if (q->n_masked > 0) {
    // masked slots leave with the spans: the union, as maximal runs
    std::vector<std::pair<int64_t, int64_t>> all = masked_runs(*q, s->P);
    all.insert(all.end(), sp.begin(), sp.end());
    std::sort(all.begin(), all.end());
    sp.clear();
    for (const auto &se : all) {
      if (!sp.empty() && se.first <= sp.back().second) sp.back().second = std::max(sp.back().second, se.second);
      else sp.push_back(se);
    }
  }
  sq_evict_stats es{};
  es.first_evicted = q->length;
  const int64_t L = q->length;
  if (sp.empty()) {
    for (int32_t c : ids) q->spans.erase(c);
    if (stats) *stats = es;
    return SQ_OK;
  }
  int64_t removed = 0;
  std::vector<int64_t> prefix(sp.size());
  for (size_t i = 0; i < sp.size(); ++i) {
    prefix[i] = removed;
    removed += sp[i].second - sp[i].first;
  }
  const int64_t Lp = L - removed;
  const int64_t f = sp[0].first;
  const int64_t fp = f / s->P;
  const int64_t new_np = (Lp + s->P - 1) / s->P;
  const int64_t n_new = new_np - fp;
  // Old index of the kept token that lands at new index j: kept run k (the
  // gap after span k - 1) starts at new index gap_dst[k] and is shifted by
  // the tokens evicted before it.
  std::vector<int64_t> gap_dst(sp.size() + 1), gap_shift(sp.size() + 1);
  for (size_t k = 0; k <= sp.size(); ++k) {
    const int64_t g0 = k == 0 ? 0 : sp[k - 1].second;
    gap_shift[k] = k == 0 ? 0 : prefix[k - 1] + (sp[k - 1].second - sp[k - 1].first);
    gap_dst[k] = g0 - gap_shift[k];
  }
  auto src_index = [&](int64_t j) -> int64_t {
    const size_t k = std::upper_bound(gap_dst.begin(), gap_dst.end(), j) - gap_dst.begin() - 1;
    return j + gap_shift[k];
  };
  // Page-aligned remap: tail page k whose P tokens are one old page's P
  // tokens in order takes that page by reference (no fresh page, no copy).
  const bool remap = (s->cfg.flags & SQ_STORE_EVICT_REMAP) != 0;
  std::vector<int32_t> alias(n_new, -1);
  std::vector<char> old_aliased(q->pages.size() - fp, 0); // by old-tail index
  int64_t n_alias = 0;
  if (remap)
    for (int64_t k = 0; k < n_new; ++k) {
      const int64_t j0 = (fp + k) * s->P;
      if (j0 + s->P > Lp) continue;
      const int64_t a0 = src_index(j0);
      if (a0 % s->P == 0 && src_index(j0 + s->P - 1) == a0 + s->P - 1) {
        alias[k] = q->pages[a0 / s->P];
        old_aliased[a0 / s->P - fp] = 1;
        ++n_alias;
      }
    }
  // In-place: tail page k is the old page at list index fp + k, rewritten,
  // when this sequence alone holds it.
  const bool inplace = (s->cfg.flags & SQ_STORE_EVICT_INPLACE) != 0;
  int64_t n_inplace = 0;
  if (inplace)
    for (int64_t k = 0; k < n_new; ++k)
      if (s->refcount[q->pages[fp + k]] == 1) {
        alias[k] = q->pages[fp + k];
        old_aliased[k] = 1;
        ++n_inplace;
      }
  auto fresh_in = [&](int64_t k0, int64_t c) {
    int64_t n = 0;
    for (int64_t k = k0; k < k0 + c; ++k) n += alias[k] < 0;
    return n;
  };

  // The schedule: fresh pages per step and the old-tail pages released after
  // it.  One-shot (evict_chunk_pages = 0): every fresh page first, every old
  // page at the end.  Chunked: C fresh pages per step, then the old pages
  // whose tokens all lie before the next kept token to move.
  const std::vector<int32_t> old_tail(q->pages.begin() + fp, q->pages.end());
  const int64_t C = s->cfg.evict_chunk_pages > 0 ? s->cfg.evict_chunk_pages
                                                 : std::max<int64_t>(1, n_new);
  struct Step {
    int64_t k0, c;
    size_t rel_begin, rel_end;
  };
  std::vector<Step> steps;
  {
    size_t released = 0;
    for (int64_t k0 = 0; k0 < n_new; k0 += C) {
      const int64_t c = std::min(C, n_new - k0);
      size_t upto = released;
      if (C < n_new) {
        const int64_t j_end = std::min((fp + k0 + c) * s->P, Lp);
        const int64_t consumed = j_end < Lp ? src_index(j_end) : L;
        while (upto < old_tail.size() && (fp + (int64_t)upto + 1) * s->P <= consumed) ++upto;
      }
      steps.push_back({k0, c, released, upto});
      released = upto;
    }
    steps.push_back({n_new, 0, released, old_tail.size()});
  }
  {
    int64_t free_now = s->n_free;
    for (const Step &st : steps) {
      const int64_t c = fresh_in(st.k0, st.c);
      if (c > free_now)
        return fail(SQ_ERR_NO_PAGES, "eviction needs %lld fresh pages at once, %lld free",
                    (long long)c, (long long)free_now);
      free_now -= c;
      for (size_t i = st.rel_begin; i < st.rel_end; ++i)
        free_now += s->refcount[old_tail[i]] + old_aliased[i] == 1; // a remap adds a reference
    }
  }

  // ---- commit: allocate and release in schedule order, enqueue the device
  // work (stream order keeps every gather ahead of the reuse of what it read),
  // then the host bookkeeping ----
  std::vector<int32_t> new_ids(n_new);
  int64_t freed = 0;
  for (int64_t k = 0; k < n_new; ++k)
    if (alias[k] >= 0) {
      ++s->refcount[alias[k]];
      new_ids[k] = alias[k];
    }
  for (const Step &st : steps) {
    for (int64_t k = st.k0; k < st.k0 + st.c; ++k)
      if (alias[k] < 0) s->alloc_pages(1, &new_ids[k]);
    for (size_t i = st.rel_begin; i < st.rel_end; ++i) s->unref(old_tail[i], &freed);
  }

  if (s->device) {
    hipStream_t strm = static_cast<hipStream_t>(stream);
    s->last_stream = strm;
    sq::EvictArgs ea{};
    ea.n_tokens = (int32_t)L;
    ea.n_spans = (int32_t)sp.size();
    ea.keep = s->ev_keep;
    ea.dst = s->ev_dst;
    ea.src_of = s->ev_src;
    // fresh ids of tail pages [k0, k0 + n) as runs of consecutive ids, or as
    // a list in the workspace when there are too many runs
    auto runs_of = [&](int64_t k0, int64_t n, sq::NewIds *ids) {
      *ids = sq::NewIds{};
      for (int64_t i = 0; i < n; ++i) {
        const int32_t id = new_ids[k0 + i];
        if (i == 0 || id != new_ids[k0 + i - 1] + 1) {
          if (ids->n_runs == sq::kInlineRanges) return false;
          ids->first[ids->n_runs] = id;
          ids->before[ids->n_runs] = (int32_t)i;
          ++ids->n_runs;
        }
      }
      return true;
    };
    sq::NewIds all{};
    const bool all_inline = runs_of(0, n_new, &all);
    // what does not fit in the kernel arguments goes up in one copy:
    // spans [nsp][3] (start, end, evicted before) | fresh ids [n_new]
    std::vector<int32_t> up;
    const bool spans_inline = sp.size() <= (size_t)sq::kInlineSpans;
    for (size_t k = 0; k < sp.size(); ++k) {
      const int32_t tmp[3] = {(int32_t)sp[k].first, (int32_t)sp[k].second, (int32_t)prefix[k]};
      if (spans_inline) std::copy(tmp, tmp + 3, ea.inl + 3 * k);
      else up.insert(up.end(), tmp, tmp + 3);
    }
    const size_t off_new = up.size();
    if (!all_inline) {
      up.insert(up.end(), new_ids.begin(), new_ids.end());
      all = sq::NewIds{};
      all.list = s->ev_upload + off_new;
    }
    if (!up.empty()) {
      sq_status us = upload(s, s->ev_upload, up.data(), up.size(), strm);
      if (us != SQ_OK) return us;
    }
    ea.spans = spans_inline ? nullptr : s->ev_upload;
    // A small first gather launch (one layer's pages, say) takes each kept
    // token's source from the spans in its kernel arguments, and the index
    // (keep, dst, src_of: for later gather launches, the in-place kernel and
    // the debug read) runs as extra workgroups of that launch, which saves
    // the index kernel and the gap after it (8-9 us).  Searching the spans
    // lengthens each gather workgroup, though: on the 64K compaction (11K
    // workgroups) the launch took 39.5 us against 33 us for the gather
    // alone, a cost that grows with the launch.  So a launch of more than
    // kFuseIndexMaxWgs workgroups keeps the index kernel, as do the
    // in-place kernel, an eviction that copies no page, and spans too many
    // to travel in the arguments; the gathers then read src_of.
    constexpr int64_t kFuseIndexMaxWgs = 12288;
    int64_t first_wgs = 0;
    if (!inplace)
      for (const Step &st : steps)
        if (st.c != 0 && fresh_in(st.k0, st.c) != 0) {
          first_wgs = st.c * (int64_t)s->cfg.num_layers * s->cfg.num_kv_heads;
          break;
        }
    const bool fuse_index = first_wgs > 0 && first_wgs <= kFuseIndexMaxWgs && spans_inline;
    ProfPair pp;
    bool on = false;
    hipError_t e = hipSuccess;
    if (!fuse_index) {
      on = s->prof_begin(strm, &pp, kProfScan);
      e = sq::launch_evict_index(ea, strm);
      s->prof_end(strm, &pp, on);
      if (e != hipSuccess) return hip_fail(e, "eviction index");
    }
    int32_t index_blocks = fuse_index ? (int32_t)((L + sq::kScanBlock - 1) / sq::kScanBlock) : 0;
    if (inplace) {
      sq_status is = evict_inplace_launches(s, h, fp, n_new, Lp, src_index, all, strm);
      if (is != SQ_OK) return is;
    }
    for (const Step &st : steps) {
      if (inplace) break;
      if (st.c == 0 || fresh_in(st.k0, st.c) == 0) continue; // nothing to copy
      sq::GatherArgs ga{};
      ga.fp = (int32_t)fp;
      ga.pi0 = (int32_t)st.k0;
      ga.n_new = (int32_t)st.c;
      ga.new_len = (int32_t)Lp;
      ga.index_blocks = index_blocks;
      index_blocks = 0; // the first launch writes the index
      ga.ev = ea;
      ga.pt_row = s->pt_row(h);
      ga.remap = remap ? 1 : 0;
      if (all_inline) {
        runs_of(st.k0, st.c, &ga.ids); // a sub-range has no more runs than the whole
      } else {
        ga.ids.list = all.list + st.k0;
      }
      on = s->prof_begin(strm, &pp, kProfGather);
      e = sq::launch_evict_gather(s->pools, ga, strm);
      s->prof_end(strm, &pp, on);
      if (e != hipSuccess) return hip_fail(e, "eviction gather");
    }
    // the page-table row takes the fresh ids after the last gather has read the old
    e = sq::launch_write_ids(s->pt_row(h) + fp, all, (int32_t)n_new, strm);
    if (e != hipSuccess) return hip_fail(e, "page-table update");
    s->have_last_evict = true;
    s->last_evict_L = L;
    s->last_evict_Lp = Lp;
  }

  q->pages.resize(fp);
  q->pages.insert(q->pages.end(), new_ids.begin(), new_ids.end());
  // positions: drop the evicted index ranges, re-index the rest
  {
    std::vector<PosRun> out;
    size_t k = 0;
    for (const PosRun &r : q->runs) {
      int64_t i = r.idx0;
      const int64_t iend = r.idx0 + r.n;
      while (i < iend) {
        while (k < sp.size() && sp[k].second <= i) ++k;
        int64_t stop = iend;
        if (k < sp.size()) {
          if (sp[k].first <= i) { // inside an evicted span: skip it
            i = std::min(iend, sp[k].second);
            continue;
          }
          stop = std::min(stop, sp[k].first);
        }
        const int64_t ni = i - evicted_before(sp, prefix, i);
        const int64_t np = r.pos0 + (i - r.idx0);
        if (!out.empty() && out.back().idx0 + out.back().n == ni &&
            out.back().pos0 + out.back().n == np)
          out.back().n += stop - i;
        else
          out.push_back({ni, np, stop - i});
        i = stop;
      }
    }
    q->runs = std::move(out);
  }
  q->length = Lp;
  for (int32_t c : ids) q->spans.erase(c);
  q->nonempty.clear();
  for (auto &kv : q->spans) {
    auto &se = kv.second;
    const int64_t ns = se.first - evicted_before(sp, prefix, se.first);
    const int64_t ne = se.second - evicted_before(sp, prefix, se.second);
    se = {ns, ne};
    if (ne > ns) q->nonempty[ns] = ne;
  }
  q->kmask.clear(); // the masked slots are gone (their device row stays dirty)
  q->n_masked = 0;
  const int64_t moved = Lp - fp * s->P - n_alias * s->P; // in-place pages are rewritten
  const int64_t per_tok =
      (int64_t)s->cfg.num_layers * s->cfg.num_kv_heads * s->cfg.head_dim * 2 * s->elem_bytes() + 4;
  es.tokens_removed = removed;
  es.tokens_moved = moved;
  es.bytes_moved = moved * per_tok;
  es.pages_allocated = n_new - n_alias - n_inplace;
  es.pages_remapped = n_alias;
  es.pages_freed = freed;
  es.first_evicted = f;
  ++s->st.evict_calls;
  s->st.evict_tokens_removed += removed;
  s->st.evict_tokens_moved += moved;
  s->st.evict_bytes_moved += es.bytes_moved;
  if (stats) *stats = es;
  return SQ_OK;
}

sq_status sq_decode_plan_info(sq_store *s, const sq_seq *seqs, int32_t batch, int32_t mode,
                              sq_plan_info *out) {
  if (!s || !seqs || !out) return fail(SQ_ERR_INVALID, "null argument");
  if (batch < 1 || batch > SQ_MAX_BATCH) return fail(SQ_ERR_INVALID, "batch must be in [1, %d]", SQ_MAX_BATCH);
  if (mode < SQ_ATTN_AUTO || mode > SQ_ATTN_MFMA) return fail(SQ_ERR_INVALID, "unknown mode %d", mode);
  for (int b = 0; b < batch; ++b)
    if (!s->get(seqs[b])) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", seqs[b]);
  Plan plan;
  sq_status r = build_plan(s, seqs, batch, mode, &plan, -1, 2); // as sq_decode_attn plans
  if (r != SQ_OK) return r;
  *out = sq_plan_info{};
  out->n_segments = (int32_t)plan.segs.size();
  out->n_groups = plan.n_groups;
  out->n_items_valu = plan.n_wg[0];
  out->n_items_mfma = plan.n_wg[1];
  out->chunk_pages = plan.n_wg[1] ? (int32_t)(plan.total[1] / plan.n_wg[1])
                                   : plan.n_wg[0] ? (int32_t)(plan.total[0] / plan.n_wg[0]) : 0;
  out->n_slots = plan.n_slots;
  out->kv_bytes = plan.kv_bytes;
  out->kv_bytes_logical = plan.kv_bytes_logical;
  out->kv_bytes_valu = plan.kv_bytes_valu;
  out->kv_bytes_mfma = plan.kv_bytes_mfma;
  out->io_bytes = plan.io_bytes;
  return SQ_OK;
}

sq_status sq_decode_attn(sq_store *s, int32_t layer, const sq_seq *seqs, int32_t batch,
                         const void *q, float *out, float scale, int32_t mode, void *stream) {
  return sq_decode_attn_ex(s, layer, seqs, batch, q, out, scale, mode, nullptr, stream);
}

sq_status sq_decode_attn_ex(sq_store *s, int32_t layer, const sq_seq *seqs, int32_t batch,
                            const void *q, float *out, float scale, int32_t mode,
                            const sq_attn_opts *opts, void *stream) {
  SQ_TRACE_CALL("sq_decode_attn", "store=%p layer=%d batch=%d mode=%d window=%d sinks=%d", (void *)s, layer, batch, mode, opts ? opts->window : 0, opts && opts->sinks ? 1 : 0);
  return decode_call(s, layer, seqs, batch, q, out, scale, mode, opts, stream, nullptr);
}

sq_status sq_decode_attn_noalloc(sq_store *s, int32_t layer, const sq_seq *seqs, int32_t batch,
                                 const void *q, float *out, float scale, int32_t mode,
                                 void *stream) {
  SQ_TRACE_CALL("sq_decode_attn_noalloc", "store=%p layer=%d batch=%d mode=%d", (void *)s, layer, batch, mode);
  if (s && s->device && s->spart_err != hipSuccess)
    return hip_fail(s->spart_err, "allocation-free partials (hipGetSymbolAddress at store creation)");
  return decode_call(s, layer, seqs, batch, q, out, scale, mode, nullptr, stream,
                     s ? &s->spart : nullptr);
}

sq_status sq_step_begin(sq_store *s, const sq_seq *seqs, int32_t batch, int32_t mode,
                        void *stream) {
  return sq_step_begin_ex(s, seqs, batch, mode, 0, stream);
}

sq_status sq_step_begin_ex(sq_store *s, const sq_seq *seqs, int32_t batch, int32_t mode,
                           int32_t window, void *stream) {
  SQ_TRACE_CALL("sq_step_begin", "store=%p batch=%d mode=%d window=%d", (void *)s, batch, mode, window);
  sq_status r = check_one_token_each(s, seqs, batch);
  if (r != SQ_OK) return r;
  if (mode < SQ_ATTN_AUTO || mode > SQ_ATTN_MFMA) return fail(SQ_ERR_INVALID, "unknown mode %d", mode);
  if (window < 0) return fail(SQ_ERR_INVALID, "window %d < 0", window);
  // attention over the tokens before the step; the new ones join in the
  // merge (a window of W keys: the new token and the last W - 1 old ones)
  Plan plan, plan_w;
  r = build_plan(s, seqs, batch, mode, &plan);
  if (r != SQ_OK) return r;
  if (window > 0) {
    if (plan.masked)
      return fail(SQ_ERR_INVALID, "a window over a sequence with masked slots (compact it first)");
    r = build_plan(s, seqs, batch, mode, &plan_w, window - 1);
    if (r != SQ_OK) return r;
  }
  // which launches a layer makes depends on the mode only, so that a
  // captured step replays for every later step of the same batch and mode
  const bool launch[2] = {mode == SQ_ATTN_STREAM || mode == SQ_ATTN_SHARED_PREFIX,
                          mode != SQ_ATTN_STREAM};
  for (int L = 0; L < 2; ++L)
    if ((plan.n_wg[L] > 0 || plan_w.n_wg[L] > 0) && !launch[L])
      return fail(SQ_ERR_INVALID, "internal: step plan needs an unlaunched kernel");
  const int sb = s->step_buf;
  if (s->device && s->step_pending[sb]) { // this staging copy's last upload
    hipError_t e = hipEventSynchronize(s->step_ev[sb]);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(step plan)");
    s->step_pending[sb] = false;
  }
  sq::StepPlan *sp = s->device ? s->step_staging[sb] : nullptr;
  if (sp) {
    std::memset(sp, 0, sizeof(*sp));
    fill_dyn(s, plan, sp->dec, &sp->merge);
    if (window > 0) fill_dyn(s, plan_w, sp->dec_w, &sp->merge_w);
  }
  const int64_t tok_bytes = (int64_t)s->cfg.num_kv_heads * s->cfg.head_dim * 2 * s->elem_bytes();
  TokenSlots t;
  take_one_token_each(s, seqs, batch, &t);
  if (sp) {
    for (int b = 0; b < batch; ++b) {
      sp->app.page[b] = t.page[b];
      sp->app.slot[b] = t.slot[b];
      sp->app.pos[b] = t.pos[b];
    }
    sp->batch = batch;
  }
  sq_store::Step &st = s->step;
  st = sq_store::Step{};
  st.active = true;
  st.gen = s->gen;
  st.batch = batch;
  st.mode = mode;
  for (int L = 0; L < 2; ++L) {
    st.launch[L] = launch[L];
    st.grid[L] = s->cus * s->wg_per_cu[L]; // >= plan.n_wg[L]
  }
  st.kv_bytes = plan.kv_bytes + batch * tok_bytes;
  st.kv_bytes_logical = plan.kv_bytes_logical + batch * tok_bytes;
  st.window = window;
  st.kv_bytes_w = plan_w.kv_bytes + batch * tok_bytes;
  st.kv_bytes_logical_w = plan_w.kv_bytes_logical + batch * tok_bytes;
  if (!s->device) return SQ_OK;
  hipStream_t strm = static_cast<hipStream_t>(stream);
  s->last_stream = strm;
  if (plan.masked) {
    r = clean_mask_rows(s, seqs, batch, strm);
    if (r != SQ_OK) return r;
  }
  // pages the step opens enter the page-table mirror now, whatever happens
  // to the step's layers
  sq::SetEntries se{};
  se.base = s->pt_dev;
  for (int b = 0; b < batch; ++b)
    if (t.pt_index[b] >= 0) {
      se.index[se.n] = t.pt_index[b];
      se.value[se.n] = t.page[b];
      ++se.n;
    }
  hipError_t e = sq::launch_set_entries(se, strm);
  if (e != hipSuccess) return hip_fail(e, "page-table entries");
  e = hipMemcpyAsync(s->step_dev, sp, sizeof(*sp), hipMemcpyHostToDevice, strm);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync(step plan)");
  e = hipEventRecord(s->step_ev[sb], strm);
  if (e != hipSuccess) return hip_fail(e, "hipEventRecord(step plan)");
  s->step_pending[sb] = true;
  s->step_buf = 1 - sb;
  return SQ_OK;
}

sq_status sq_step_attn(sq_store *s, int32_t layer, const void *k_new, const void *v_new,
                       const void *q, float *out, float scale, void *stream) {
  return sq_step_attn_ex(s, layer, k_new, v_new, q, out, scale, nullptr, stream);
}

sq_status sq_step_attn_ex(sq_store *s, int32_t layer, const void *k_new, const void *v_new,
                          const void *q, float *out, float scale, const sq_attn_opts *opts,
                          void *stream) {
  SQ_TRACE_CALL("sq_step_attn", "store=%p layer=%d window=%d sinks=%d", (void *)s, layer, opts ? opts->window : 0, opts && opts->sinks ? 1 : 0);
  sq_attn_opts o{};
  sq_status r = take_opts(opts, &o);
  if (r != SQ_OK) return r;
  if (!s) return fail(SQ_ERR_INVALID, "null store");
  if (!s->device) return fail(SQ_ERR_INVALID, "metadata-only store cannot run attention");
  const sq_store::Step &st = s->step;
  if (!st.active || st.gen != s->gen)
    return fail(SQ_ERR_INVALID, "no decode step is open (none begun, or the store changed since)");
  if (layer < 0 || layer >= s->cfg.num_layers) return fail(SQ_ERR_INVALID, "layer %d out of range", layer);
  if (!k_new || !v_new || !q || !out || !aligned16(k_new) || !aligned16(v_new) || !aligned16(q) ||
      !aligned16(out))
    return fail(SQ_ERR_INVALID, "k_new, v_new, q and out must be non-null and 16-byte aligned");
  if (!std::isfinite(scale)) return fail(SQ_ERR_INVALID, "scale must be finite");
  if (o.window != 0 && o.window != st.window)
    return fail(SQ_ERR_INVALID, "window %d: the step was begun with window %d", o.window, st.window);
  const bool win = o.window != 0;
  hipStream_t strm = static_cast<hipStream_t>(stream);
  s->last_stream = strm;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  (void)hipStreamIsCapturing(strm, &cap);
  const bool prof = cap == hipStreamCaptureStatusNone; // no timing events in a capture
  const sq::DecodeStatic ds = decode_static(s, layer, q, scale, true);
  for (int L = 0; L < 2; ++L) {
    if (!st.launch[L]) continue;
    ProfPair pp;
    const bool on = prof && s->prof_begin(strm, &pp, L == 0 ? kProfValu : kProfMfma);
    const sq::DecodeDyn *dd = win ? s->step_dev->dec_w : s->step_dev->dec;
    hipError_t e = L == 0 ? sq::launch_step_valu(s->D, s->G, ds, &dd[0], st.grid[0], strm)
                          : sq::launch_step_mfma(s->D, s->G, ds, &dd[1], st.grid[1], strm);
    s->prof_end(strm, &pp, on);
    if (e != hipSuccess) return hip_fail(e, "decode step kernel");
  }
  sq::StepMergeArgs ma{};
  ma.st = merge_static(s, layer, out, o.sinks);
  ma.plan = s->step_dev;
  ma.windowed = win ? 1 : 0;
  ma.q = static_cast<const uint16_t *>(q);
  ma.k_new = static_cast<const uint16_t *>(k_new);
  ma.v_new = static_cast<const uint16_t *>(v_new);
  ma.k = layer_pool(s, s->pools.k, layer);
  ma.v = layer_pool(s, s->pools.v, layer);
  ma.inv_k = s->inv(s->k_scale(layer));
  ma.inv_v = s->inv(s->v_scale(layer));
  ma.pos = s->pools.pos;
  ma.page_stride = s->pools.page_stride;
  ma.head_stride = s->pools.head_stride;
  ma.scale_log2 = ds.scale_log2;
  ProfPair pp;
  const bool on = prof && s->prof_begin(strm, &pp, kProfMerge);
  hipError_t e = sq::launch_step_merge(s->D, st.batch, ma, s->kv8, strm);
  s->prof_end(strm, &pp, on);
  if (e != hipSuccess) return hip_fail(e, "decode step merge");
  ++s->st.decode_calls;
  s->st.decode_kv_bytes += win ? st.kv_bytes_w : st.kv_bytes;
  s->st.decode_kv_bytes_logical += win ? st.kv_bytes_logical_w : st.kv_bytes_logical;
  return SQ_OK;
}

sq_status sq_extend_attn(sq_store *s, int32_t layer, sq_seq seq, int32_t n_new, const void *q,
                         float *out, float scale, void *stream) {
  return sq_extend_attn_ex(s, layer, seq, n_new, q, out, scale, nullptr, stream);
}

sq_status sq_extend_attn_ex(sq_store *s, int32_t layer, sq_seq seq, int32_t n_new, const void *q,
                            float *out, float scale, const sq_attn_opts *opts, void *stream) {
  SQ_TRACE_CALL("sq_extend_attn", "store=%p layer=%d seq=%d n_new=%d window=%d sinks=%d", (void *)s, layer, seq, n_new, opts ? opts->window : 0, opts && opts->sinks ? 1 : 0);
  sq_attn_opts o{};
  sq_status r = take_opts(opts, &o);
  if (r != SQ_OK) return r;
  if (!s) return fail(SQ_ERR_INVALID, "null store");
  if (!s->device) return fail(SQ_ERR_INVALID, "metadata-only store cannot run attention");
  if (layer < 0 || layer >= s->cfg.num_layers) return fail(SQ_ERR_INVALID, "layer %d out of range", layer);
  Seq *sqn = s->get(seq);
  if (!sqn) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", seq);
  if (n_new < 0 || n_new > sqn->length)
    return fail(SQ_ERR_INVALID, "n_new %d outside [0, %lld]", n_new, (long long)sqn->length);
  if (n_new == 0) return SQ_OK;
  if (!q || !out || !aligned16(q) || !aligned16(out))
    return fail(SQ_ERR_INVALID, "q and out must be non-null and 16-byte aligned");
  if (!std::isfinite(scale) || !(scale > 0.f))
    return fail(SQ_ERR_INVALID, "scale must be finite and positive");
  hipStream_t strm = static_cast<hipStream_t>(stream);
  s->last_stream = strm;
  sq::ExtendArgs a{};
  a.q = static_cast<const uint16_t *>(q);
  a.k = layer_pool(s, s->pools.k, layer);
  a.v = layer_pool(s, s->pools.v, layer);
  a.pt = s->pt_row(seq);
  a.out = out;
  a.page_stride = s->pools.page_stride;
  a.head_stride = s->pools.head_stride;
  a.n_pages = (int32_t)sqn->pages.size();
  a.L = (int32_t)sqn->length;
  a.n = n_new;
  a.hq = s->cfg.num_q_heads;
  a.hkv = s->cfg.num_kv_heads;
  const int tq = sq::kExtRows / s->G;
  a.n_qblocks = (n_new + tq - 1) / tq;
  a.scale_log2 = (float)((double)scale * 1.4426950408889634 * (double)s->k_scale(layer));
  a.sinks = o.sinks;
  a.window = o.window;
  a.sink_scale = 1.4426950408889634f;
  a.kv8 = s->kv8 ? 1 : 0;
  a.out_scale = s->v_scale(layer);
  a.mask_row = s->mask_row(seq);
  a.masked = sqn->n_masked > 0 ? 1 : 0;
  if (a.masked && o.window > 0)
    return fail(SQ_ERR_INVALID, "a window over a sequence with masked slots (compact it first)");
  // A chunk too short to give every CU two rounds of workgroups (one fits a
  // CU) splits the key range of each query block (at least 4 blocks of 64
  // keys per split) and merges the partial rows in a second launch.
  int64_t key_blocks = (sqn->length + sq::kExtKeys - 1) / sq::kExtKeys; // the last query block's
  if (o.window > 0) // a query block's keys span at most W + TQ - 1 indices
    key_blocks = std::min<int64_t>(key_blocks, ((int64_t)o.window + tq - 2) / sq::kExtKeys + 2);
  const int64_t base_wg = (int64_t)a.n_qblocks * a.hkv;
  const int64_t target = 2LL * s->cus;
  int64_t split = 1;
  if (base_wg < target) {
    split = (target + base_wg - 1) / base_wg;
    split = std::min<int64_t>(split, std::max<int64_t>(1, key_blocks / 4));
    split = std::min<int64_t>(split, 64);
    split = std::min<int64_t>(split, (int64_t)sq::kMaxItems * sq::kRows / sq::kExtRows / base_wg);
    split = std::max<int64_t>(split, 1);
  }
  a.n_split = (int32_t)split;
  a.split_blocks = (int32_t)((key_blocks + split - 1) / split);
  a.part_m = s->part_m;
  a.part_l = s->part_l;
  a.part_acc = s->part_acc;
  ProfPair pp;
  const bool on = s->prof_begin(strm, &pp, kProfExtend);
  hipError_t e = sq::launch_extend(s->D, s->G, a, strm);
  if (e == hipSuccess) e = sq::launch_extend_merge(s->D, s->G, a, strm);
  s->prof_end(strm, &pp, on);
  if (e != hipSuccess) return hip_fail(e, "extend kernel");
  ++s->st.extend_calls;
  s->st.extend_tokens += n_new;
  const int64_t keys_read = o.window > 0 ? std::min<int64_t>(sqn->length, (int64_t)n_new + o.window - 1)
                                         : sqn->length;
  s->st.extend_kv_bytes += keys_read * (int64_t)s->cfg.num_kv_heads * s->D * 2 * s->elem_bytes();
  return SQ_OK;
}

sq_status sq_seq_info(sq_store *s, sq_seq h, sq_seq_desc *out) {
  if (!s || !out) return fail(SQ_ERR_INVALID, "null argument");
  Seq *q = s->get(h);
  if (!q) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", h);
  *out = sq_seq_desc{};
  out->length = q->length;
  out->next_pos = q->next_pos;
  out->n_pages = (int32_t)q->pages.size();
  out->parent = q->parent;
  out->n_spans = (int32_t)q->spans.size();
  out->n_masked = (int32_t)q->n_masked;
  return SQ_OK;
}

sq_status sq_keep_flags(sq_store *s, sq_seq h, uint8_t *out, int64_t cap, int64_t *n) {
  if (!s || !n) return fail(SQ_ERR_INVALID, "null argument");
  Seq *q = s->get(h);
  if (!q) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", h);
  if (cap > 0 && !out) return fail(SQ_ERR_INVALID, "null output with cap > 0");
  *n = q->length;
  for (int64_t i = 0; i < std::min(cap, q->length); ++i) out[i] = slot_kept(*q, i, s->P) ? 1 : 0;
  return SQ_OK;
}

sq_status sq_page_table(sq_store *s, sq_seq h, int32_t *out, int32_t cap, int32_t *n) {
  if (!s || !n) return fail(SQ_ERR_INVALID, "null argument");
  Seq *q = s->get(h);
  if (!q) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", h);
  *n = (int32_t)q->pages.size();
  for (int32_t i = 0; i < std::min(cap, *n); ++i) out[i] = q->pages[i];
  return SQ_OK;
}

sq_status sq_positions(sq_store *s, sq_seq h, int64_t *out, int64_t cap, int64_t *n) {
  if (!s || !n) return fail(SQ_ERR_INVALID, "null argument");
  Seq *q = s->get(h);
  if (!q) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", h);
  *n = q->length;
  int64_t i = 0;
  for (const PosRun &r : q->runs)
    for (int64_t j = 0; j < r.n && i < cap; ++j, ++i) out[i] = r.pos0 + j;
  return SQ_OK;
}

sq_status sq_seq_spans(sq_store *s, sq_seq h, int32_t *cursors, int64_t *starts, int64_t *ends,
                       int32_t cap, int32_t *n) {
  if (!s || !n) return fail(SQ_ERR_INVALID, "null argument");
  Seq *q = s->get(h);
  if (!q) return fail(SQ_ERR_UNKNOWN_SEQ, "unknown sequence %d", h);
  *n = (int32_t)q->spans.size();
  int32_t i = 0;
  for (auto &kv : q->spans) {
    if (i >= cap) break;
    cursors[i] = kv.first;
    starts[i] = kv.second.first;
    ends[i] = kv.second.second;
    ++i;
  }
  return SQ_OK;
}

sq_status sq_refcounts(sq_store *s, int32_t *out, int32_t cap) {
  if (!s || !out) return fail(SQ_ERR_INVALID, "null argument");
  for (int32_t i = 0; i < std::min(cap, s->cfg.num_pages); ++i) out[i] = s->refcount[i];
  return SQ_OK;
}

sq_status sq_stats_get(sq_store *s, sq_stats *out) {
  if (!s || !out) return fail(SQ_ERR_INVALID, "null argument");
  *out = s->st;
  out->live_pages = s->live_pages();
  out->peak_pages = s->peak_pages;
  out->free_pages = s->n_free;
  return SQ_OK;
}

sq_status sq_debug_last_evict(sq_store *s, uint8_t *keep, int32_t *dst, int32_t *src_of,
                              int64_t cap, int64_t *n_tokens, int64_t *n_kept) {
  if (!s || !keep || !dst || !src_of || !n_tokens || !n_kept) return fail(SQ_ERR_INVALID, "null argument");
  if (!s->device || !s->have_last_evict) return fail(SQ_ERR_INVALID, "no eviction has moved tokens yet");
  if (cap < s->last_evict_L) return fail(SQ_ERR_INVALID, "cap %lld < %lld tokens", (long long)cap,
                                         (long long)s->last_evict_L);
  hipStream_t strm = s->last_stream;
  hipError_t e = hipMemcpyAsync(keep, s->ev_keep, s->last_evict_L, hipMemcpyDeviceToHost, strm);
  if (e == hipSuccess)
    e = hipMemcpyAsync(dst, s->ev_dst, s->last_evict_L * 4, hipMemcpyDeviceToHost, strm);
  if (e == hipSuccess)
    e = hipMemcpyAsync(src_of, s->ev_src, s->last_evict_Lp * 4, hipMemcpyDeviceToHost, strm);
  if (e == hipSuccess) e = hipStreamSynchronize(strm);
  if (e != hipSuccess) return hip_fail(e, "debug copy");
  *n_tokens = s->last_evict_L;
  *n_kept = s->last_evict_Lp;
  return SQ_OK;
}

sq_status sq_profile_enable(sq_store *s, int32_t on) {
  if (!s) return fail(SQ_ERR_INVALID, "null store");
  if (!s->device && on) return fail(SQ_ERR_INVALID, "metadata-only store has no kernels to time");
  s->prof_on = on != 0;
  return SQ_OK;
}

sq_status sq_profile_read(sq_store *s, sq_profile *out) {
  if (!s || !out) return fail(SQ_ERR_INVALID, "null argument");
  for (auto &pp : s->prof_pending) {
    hipError_t e = hipEventSynchronize(pp.b);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize(profile)");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, pp.a, pp.b);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    s->prof_ms[pp.kind] += ms;
    s->prof_n[pp.kind] += 1;
    s->ev_pool.push_back(pp.a);
    s->ev_pool.push_back(pp.b);
  }
  s->prof_pending.clear();
  *out = sq_profile{};
  out->decode_valu_ms = s->prof_ms[kProfValu];
  out->decode_mfma_ms = s->prof_ms[kProfMfma];
  out->decode_merge_ms = s->prof_ms[kProfMerge];
  out->evict_scan_ms = s->prof_ms[kProfScan];
  out->evict_gather_ms = s->prof_ms[kProfGather];
  out->append_ms = s->prof_ms[kProfAppend];
  out->decode_valu_launches = s->prof_n[kProfValu];
  out->decode_mfma_launches = s->prof_n[kProfMfma];
  out->decode_merge_launches = s->prof_n[kProfMerge];
  out->evict_scan_launches = s->prof_n[kProfScan];
  out->evict_gather_launches = s->prof_n[kProfGather];
  out->append_launches = s->prof_n[kProfAppend];
  out->extend_ms = s->prof_ms[kProfExtend];
  out->extend_launches = s->prof_n[kProfExtend];
  for (int k = 0; k < kProfKinds; ++k) {
    s->prof_ms[k] = 0;
    s->prof_n[k] = 0;
  }
  return SQ_OK;
}

} // extern "C"
