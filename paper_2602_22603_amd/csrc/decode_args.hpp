// decode_args.hpp - kernel arguments and launchers of the decode kernels
// (decode_kernels.hip).
// Internal to libsq.
#pragma once

#include "sq_common.hpp"

namespace sq {

// ---- decode ---------------------------------------------------------------
// A segment: `ntok` tokens read from page-table row `row` from page index
// `page0` on, attended by `nmem` query sequences (batch indices packed as
// bytes in `mem`).  Its Hkv rows (one per KV head g) occupy the flattened
// page ranges [start + g * (npages + row_pad), ... + npages) of its launch;
// each row is followed by row_pad flattened pages that map to nothing.  They
// stand for the fixed start-up cost of a piece (its query, page-id and
// first page loads), so that the even split gives a workgroup that covers
// many short rows fewer pages.
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
  int32_t row_pad;     // flattened pages after each row that map to nothing
  float scale_log2;    // scale * log2(e)
  Seg segs[kMaxSegs];
};

// The workgroup whose range holds flattened page x.
__host__ __device__ inline int32_t wg_of(int64_t x, int64_t total, int64_t n_wg) {
  return (int32_t)(((x + 1) * n_wg - 1) / total);
}

// A batch entry attends to the segments on its path through the tree of
// shared page runs: at most kMaxSrc (shared levels, then its own suffix).
constexpr int kMaxSrc = 4;

struct MergeArgs {
  float *out;  // [B][Hq][D]
  const float *part_m;
  const float *part_l;
  const float *part_acc;
  int32_t hq;
  int32_t group; // G
  int32_t hkv;
  int32_t pad;
  int32_t total[2], n_wg[2], slot_base[2], row_pad[2]; // per launch (0: VALU, 1: MFMA)
  // per batch entry: the segments it attends; meta packs the launch (bit 0),
  // the segment index inside that launch (bits 1-8) and the member index
  // inside the segment (bits 9-10)
  int32_t n_src[kMaxBatch];
  int32_t src_meta[kMaxBatch][kMaxSrc];
  int32_t src_start[kMaxBatch][kMaxSrc];  // flattened start of the segment's rows
  int32_t src_npages[kMaxBatch][kMaxSrc];
};

static_assert(sizeof(DecodeArgs) < 4096, "decode kernel arguments too large");
static_assert(sizeof(MergeArgs) < 4096, "merge kernel arguments too large");

hipError_t launch_decode_valu(int d, int group, const DecodeArgs &a, hipStream_t s);
hipError_t launch_decode_mfma(int d, int group, int waves, const DecodeArgs &a, hipStream_t s);
hipError_t launch_decode_merge(int d, int batch, const MergeArgs &a, hipStream_t s);
// Workgroups of a decode kernel (kind 0: VALU, 1: MFMA) that fit on one CU.
hipError_t decode_blocks_per_cu(int kind, int d, int group, int waves, int *out);

} // namespace sq
