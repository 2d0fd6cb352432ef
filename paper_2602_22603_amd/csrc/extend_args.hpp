// extend_args.hpp - kernel arguments and launcher of the extend kernel
// (extend_kernels.hip).
// Internal to libsq.
#pragma once

#include "sq_common.hpp"

namespace sq {

// ---- extend (causal attention of an appended chunk) ------------------------
// The chunk is the last n of the sequence's L tokens; new token j attends to
// logical keys 0 .. L - n + j.  A workgroup of kExtWaves waves takes 32
// query rows per wave (kExtRows / G tokens x the G query heads of one KV
// head) against the whole key range; one workgroup fits a CU.
constexpr int kExtWaves = 8;
constexpr int kExtRows = 32 * kExtWaves;
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
  // Split of the key range (chunks too short to fill the GPU): each (query
  // block, KV head) runs n_split workgroups over split_blocks key blocks
  // each and writes partial (m, l, acc) rows; k_extend_merge combines them.
  // n_split == 1: the workgroup writes out directly.
  int32_t n_split;
  int32_t split_blocks;
  float *part_m;      // [slots][kExtRows] (log2 units), slot = (qb * Hkv + g) * n_split + s
  float *part_l;      // [slots][kExtRows]
  float *part_acc;    // [slots][kExtRows][D]
  // Model variants: a window of `window` keys (0: none) ends at each
  // token's own index; sinks[h] (or null) joins each softmax as a term with
  // no value, scaled by sink_scale into the log2 units of the scores.
  const float *sinks;
  int32_t window;
  float sink_scale;
  // Keep masks of deferred evictions: entry i of the sequence's mask row
  // holds bit s = slot s of its page i attended; read only when masked.
  const int32_t *mask_row;
  int32_t masked;
  int32_t kv8;        // 1: the pools hold E4M3 codes (K scale in scale_log2)
  float out_scale;    // the layer's V scale in an 8-bit store (1 otherwise)
  int32_t pad;
};

static_assert(sizeof(ExtendArgs) < 4096, "extend kernel arguments too large");

hipError_t launch_extend(int d, int group, const ExtendArgs &a, hipStream_t s);
// Partial rows of the split key range -> out (no-op when n_split == 1).
hipError_t launch_extend_merge(int d, int group, const ExtendArgs &a, hipStream_t s);

} // namespace sq
