// sq_kernels.hpp - kernel-argument structs and launchers shared by the host
// library (store.cpp) and the gfx950 kernels (kv_kernels.hip,
// decode_kernels.hip).  Everything here is internal to libsq.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace sq {

constexpr int kPage = 16;            // tokens per page in device mode
constexpr int kMaxAppendPages = 240; // pages one append launch may touch
constexpr int kMaxBatch = 64;        // queries per decode call
constexpr int kMaxSegs = 128;        // (page range, query rows) units per decode
constexpr int kMaxMembers = 4;       // sequences stacked in one MFMA tile
constexpr int kRows = 16;            // query rows per partial slot (MFMA N)
constexpr int kMaxItems = 8192;      // partial slots in the workspace
constexpr int kScanBlock = 2048;     // tokens per block of the eviction scan
constexpr int kScanThreads = 256;

// Device pools and shapes.  K: [NL][Hkv][NP][P][D]; V: [NL][Hkv][NP][D][P];
// pos: [NP][P].  Element strides are in bf16 units.  Head-major: the pages of
// one KV head are contiguous, so a decode work item streams one region.
struct Pools {
  uint16_t *k;
  uint16_t *v;
  int32_t *pos;
  int32_t nl, hkv, d, np;
  int64_t layer_stride; // Hkv * NP * P * D
  int64_t page_stride;  // P * D
  int64_t head_stride;  // NP * P * D
};

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
  int32_t n_new;          // fresh pages
  int32_t new_len;        // L'
  const int32_t *src_of;
  const int32_t *pt_row;  // device page-table row, still holding the old ids
  NewIds ids;
};

// ---- decode ---------------------------------------------------------------
// A segment: `ntok` tokens read from page-table row `row` from page index
// `page0` on, attended by `nmem` query sequences (batch indices packed as
// bytes in `mem`).  Its Hkv rows (one per KV head g) occupy the flattened
// page range [start + g * npages, start + (g + 1) * npages) of its launch.
struct Seg {
  int32_t row;
  int32_t page0;
  int32_t ntok;
  int32_t start;
  int32_t nmem;
  uint32_t mem; // byte j = batch index of member j
};

// A launch splits its flattened pages [0, total) evenly over n_wg <= total
// workgroups: workgroup w takes [w * total / n_wg, (w + 1) * total / n_wg).
// The piece of row r = segment * Hkv + g that workgroup w processes writes
// the partial slot slot_base + w + r.
struct DecodeArgs {
  const uint16_t *q;   // [B][Hq][D] bf16
  const uint16_t *k;   // K pool at this layer
  const uint16_t *v;   // V pool at this layer
  const int32_t *pt;   // page-table mirror base
  float *part_m;       // [kMaxItems][kRows]  (log2 domain)
  float *part_l;       // [kMaxItems][kRows]
  float *part_acc;     // [kMaxItems][kRows][D]
  int64_t page_stride; // P * D elements
  int64_t head_stride; // NP * P * D elements
  int32_t max_pages;   // page-table row pitch
  int32_t hq;
  int32_t hkv;
  int32_t n_segs;
  int32_t total;       // flattened pages of this launch
  int32_t n_wg;        // workgroups of this launch
  int32_t slot_base;   // first partial slot of this launch
  int32_t nontemporal; // 1: every page is read once in this launch
  float scale_log2;    // scale * log2(e)
  Seg segs[kMaxSegs];
};

// The workgroup whose range holds flattened page x.
__host__ __device__ inline int32_t wg_of(int64_t x, int64_t total, int64_t n_wg) {
  return (int32_t)(((x + 1) * n_wg - 1) / total);
}

struct MergeArgs {
  float *out;  // [B][Hq][D]
  const float *part_m;
  const float *part_l;
  const float *part_acc;
  int32_t hq;
  int32_t group; // G
  int32_t hkv;
  int32_t pad;
  int32_t total[2], n_wg[2], slot_base[2]; // per launch (0: VALU, 1: MFMA)
  // per batch entry: up to two segments it attends (launch, segment index,
  // flattened start, pages, member index inside the segment)
  int32_t n_src[kMaxBatch];
  int32_t src_launch[kMaxBatch][2];
  int32_t src_seg[kMaxBatch][2];
  int32_t src_start[kMaxBatch][2];
  int32_t src_npages[kMaxBatch][2];
  int32_t src_member[kMaxBatch][2];
};

// ---- extend (causal attention of an appended chunk) ------------------------
// The chunk is the last n of the sequence's L tokens; new token j attends to
// logical keys 0 .. L - n + j.  A workgroup takes 128 query rows (128 / G
// tokens x the G query heads of one KV head) against the whole key range.
constexpr int kExtRows = 128;
constexpr int kExtKeys = 64; // keys per LDS block (4 pages)

struct ExtendArgs {
  const uint16_t *q;  // bf16 [n][Hq][D]
  const uint16_t *k;  // K pool of the layer
  const uint16_t *v;  // V pool of the layer
  const int32_t *pt;  // device page-table row of the sequence
  float *out;         // fp32 [n][Hq][D]
  int64_t page_stride;
  int64_t head_stride;
  int32_t n_pages;    // pages in the sequence's list
  int32_t L;          // tokens in the sequence (the chunk included)
  int32_t n;          // new tokens
  int32_t hq;
  int32_t hkv;
  int32_t n_qblocks;  // ceil(n / (kExtRows / G))
  float scale_log2;
};

// Kernel arguments are passed by value; keep each well under 4 KiB.
static_assert(sizeof(AppendArgs) < 4096, "append kernel arguments too large");
static_assert(sizeof(AppendBatchArgs) < 4096, "append-batch kernel arguments too large");
static_assert(sizeof(DecodeArgs) < 4096, "decode kernel arguments too large");
static_assert(sizeof(MergeArgs) < 4096, "merge kernel arguments too large");
static_assert(sizeof(EvictArgs) < 4096, "eviction index arguments too large");
static_assert(sizeof(GatherArgs) + sizeof(Pools) < 4096, "gather arguments too large");

// ---- launchers (return the launch status) ------------------------------------
hipError_t launch_append(const Pools &p, const AppendArgs &a, const void *k_new,
                         const void *v_new, hipStream_t s);
hipError_t launch_append_batch(const Pools &p, const AppendBatchArgs &a, const void *k_new,
                               const void *v_new, hipStream_t s);
hipError_t launch_copy_i32(int32_t *dst, const int32_t *src, int32_t n, int32_t tail_index,
                           int32_t tail_value, hipStream_t s);
hipError_t launch_copy_page(const Pools &p, int32_t src_page, int32_t dst_page, hipStream_t s);
hipError_t launch_evict_index(const EvictArgs &a, hipStream_t s);
hipError_t launch_write_ids(int32_t *dst, const NewIds &ids, int32_t n, hipStream_t s);
hipError_t launch_evict_gather(const Pools &p, const GatherArgs &a, hipStream_t s);
hipError_t launch_decode_valu(int d, int group, const DecodeArgs &a, hipStream_t s);
hipError_t launch_decode_mfma(int d, int group, int waves, const DecodeArgs &a, hipStream_t s);
hipError_t launch_decode_merge(int d, int batch, const MergeArgs &a, hipStream_t s);
hipError_t launch_extend(int d, int group, const ExtendArgs &a, hipStream_t s);
// Workgroups of a decode kernel (kind 0: VALU, 1: MFMA) that fit on one CU.
hipError_t decode_blocks_per_cu(int kind, int d, int group, int waves, int *out);

} // namespace sq
