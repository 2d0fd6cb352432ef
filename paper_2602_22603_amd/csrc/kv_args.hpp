// kv_args.hpp - kernel arguments and launchers of the append, fork-copy and eviction
// kernels (kv_kernels.hip).
// Internal to libsq.
#pragma once

#include "sq_common.hpp"

namespace sq {

constexpr int kScanBlock = 2048;     // tokens per block of the eviction scan
constexpr int kScanThreads = 256;

// ---- append ---------------------------------------------------------------
// Tokens [tok0, tok0 + n_tok) of an append of n_total tokens, landing in
// pages page_ids[0..n_pages) starting at slot slot0 of the first page.
struct AppendArgs {
  int32_t n_tok;
  int32_t n_total;
  int32_t tok0;
  int32_t slot0;
  int32_t pos0;      // position of token tok0
  int32_t n_pages;
  int32_t pt_first;  // page-list index of page_ids[0]
  int32_t new_from;  // page_ids[i] with i >= new_from are new: write them to the mirror
  int32_t *pt_row;   // device page-table row of the sequence
  int32_t page_ids[kMaxAppendPages];
};

// One token for each of n sequences.
struct AppendBatchArgs {
  int32_t n;
  int32_t page[kMaxBatch];
  int32_t slot[kMaxBatch];
  int32_t pos[kMaxBatch];
  int32_t pt_index[kMaxBatch]; // row * max_pages + index, or -1 if the page is not new
  int32_t *pt;                 // device page-table mirror base
};

// base[index[i]] = value[i] for i < n (a decode step's new page-table
// entries).
struct SetEntries {
  int32_t *base;
  int32_t n;
  int32_t index[kMaxBatch];
  int32_t value[kMaxBatch];
};

// ---- eviction -------------------------------------------------------------
// Evicted spans as [n_spans][3] = (start, end, evicted tokens before start),
// sorted, disjoint and non-empty: up to kInlineSpans travel in the kernel
// arguments, more are read from device memory.
constexpr int kInlineSpans = 96;
constexpr int kInlineRanges = 60;

struct EvictArgs {
  int32_t n_tokens;     // L
  int32_t n_spans;
  const int32_t *spans; // device copy when n_spans > kInlineSpans
  uint8_t *keep;        // [L]
  int32_t *dst;         // [L]
  int32_t *src_of;      // [L']
  int32_t inl[3 * kInlineSpans];
};

// The fresh page ids of an eviction: a device list, or (when they form at
// most kInlineRanges runs of consecutive ids) the runs themselves.
struct NewIds {
  const int32_t *list;            // device, or null when the runs are used
  int32_t n_runs;
  int32_t first[kInlineRanges];   // first id of run r
  int32_t before[kInlineRanges];  // fresh pages before run r
};

struct GatherArgs {
  int32_t fp;             // first affected page index
  int32_t pi0;            // first fresh page (of the tail) this launch fills
  int32_t n_new;          // fresh pages this launch fills; ids[i] is tail page pi0 + i
  int32_t new_len;        // L'
  int32_t index_blocks;   // > 0 (spans in ev.inl only): the launch's first
                          //      index_blocks workgroups write the eviction
                          //      index (keep, dst, src_of) of ev, and the
                          //      others take sources from the spans; 0: the
                          //      sources are read from ev.src_of
  int32_t pad0;
  EvictArgs ev;           // the spans (each kept token's source comes from them)
  const int32_t *pt_row;  // device page-table row, still holding the old ids
  int32_t remap;          // 1: skip tail pages that are one old page in order
                          //    (the host maps them to that page; same rule)
  int32_t pad;
  NewIds ids;
};

// In-place eviction: tail pages [k0, k0 + n_pages) of the compacted
// sequence, each filled from its kept tokens' old slots and written to
// ids(k) (the old page at list index fp + k, or a fresh page).  Round mode
// (sweep = 0): one workgroup per (page, layer * Hkv + head); no page of the
// launch is read by another page of the launch.  Sweep mode (sweep = 1):
// one workgroup per layer * Hkv + head takes the pages in order.
struct InplaceArgs {
  int32_t fp;
  int32_t k0;
  int32_t n_pages;
  int32_t new_len;
  int32_t sweep;
  int32_t pad;
  const int32_t *src_of;
  const int32_t *pt_row;  // device page-table row, still holding the old ids
  NewIds ids;             // destination id of tail page k (k counted from 0)
};

static_assert(sizeof(AppendArgs) < 4096, "append kernel arguments too large");
static_assert(sizeof(InplaceArgs) + sizeof(Pools) < 4096, "in-place arguments too large");
static_assert(sizeof(AppendBatchArgs) < 4096, "append-batch kernel arguments too large");
static_assert(sizeof(EvictArgs) < 4096, "eviction index arguments too large");
static_assert(sizeof(GatherArgs) + sizeof(Pools) < 4096, "gather arguments too large");

hipError_t launch_append(const Pools &p, const AppendArgs &a, const void *k_new,
                         const void *v_new, hipStream_t s);
hipError_t launch_append_batch(const Pools &p, const AppendBatchArgs &a, const void *k_new,
                               const void *v_new, hipStream_t s);
hipError_t launch_set_entries(const SetEntries &a, hipStream_t s);
hipError_t launch_copy_i32(int32_t *dst, const int32_t *src, int32_t n, int32_t tail_index,
                           int32_t tail_value, hipStream_t s);
hipError_t launch_copy_page(const Pools &p, int32_t src_page, int32_t dst_page, hipStream_t s);
// dst[i] = value for i < n.
hipError_t launch_fill_i32(int32_t *dst, int32_t value, int32_t n, hipStream_t s);
hipError_t launch_evict_index(const EvictArgs &a, hipStream_t s);
hipError_t launch_write_ids(int32_t *dst, const NewIds &ids, int32_t n, hipStream_t s);
hipError_t launch_evict_gather(const Pools &p, const GatherArgs &a, hipStream_t s);
hipError_t launch_evict_inplace(const Pools &p, const InplaceArgs &a, hipStream_t s);

} // namespace sq
