// decode_args.hpp - kernel arguments and launchers of the decode kernels
// (decode_kernels.hip).
// Internal to libsq.
#pragma once

#include "sq_common.hpp"

namespace sq {

// ---- decode ---------------------------------------------------------------
// A segment: tokens [tok0, ntok) counted from the first slot of page index
// `page0` of page-table row `row` (tok0 < 16: a window may start inside
// its first page), attended by `nmem` query sequences (batch indices packed
// as bytes in `mem`).  Its Hkv rows (one per KV head g) occupy the flattened
// page ranges [start + g * (npages + row_pad), ... + npages) of its launch;
// each row is followed by row_pad flattened pages that map to nothing.  They
// stand for the fixed start-up cost of a piece (its query, page-id and
// first page loads), so that the even split gives a workgroup that covers
// many short rows fewer pages.  row (< 256), nmem (<= kMaxMembers) and tok0
// share one word.
struct Seg {
  int32_t page0;
  int32_t ntok;
  int32_t start;
  uint32_t rmt;    // row | nmem << 8 | tok0 << 16
  uint32_t mem[2]; // byte j of the pair = batch index of member j
  __host__ __device__ int row() const { return (int)(rmt & 0xff); }
  __host__ __device__ int nmem() const { return (int)((rmt >> 8) & 0xff); }
  __host__ __device__ int tok0() const { return (int)(rmt >> 16); }
  __host__ __device__ int member(int j) const { return (int)((mem[j >> 2] >> (8 * (j & 3))) & 0xff); }
};

// What a decode launch needs that does not change from call to call.
struct DecodeStatic {
  const uint16_t *q;   // [B][Hq][D] bf16
  const uint16_t *k;   // K pool at this layer
  const uint16_t *v;   // V pool at this layer
  const int32_t *pt;   // page-table mirror base
  const int32_t *mask; // keep-mask mirror, the page table's shape: bit s of an
                       // entry = slot s attended (read only when the plan says)
  float *part_m;       // [kMaxItems][kRows]  (log2 domain)
  float *part_l;       // [kMaxItems][kRows]
  float *part_acc;     // [kMaxItems][kRows][D]
  int64_t page_stride; // P * D elements
  int64_t head_stride; // NP * P * D elements
  int32_t max_pages;   // page-table row pitch
  int32_t hq;
  int32_t hkv;
  int32_t nontemporal; // 1: every page is read once in this launch
  float scale_log2;    // scale * log2(e) (times the layer's K scale in an 8-bit store)
  int32_t kv8;         // 1: the pools hold E4M3 codes
};

// The plan of one launch.  It splits its flattened pages [0, total) evenly
// over n_wg <= total workgroups: workgroup w takes [w * total / n_wg,
// (w + 1) * total / n_wg).  The piece of row r = segment * Hkv + g that
// workgroup w processes writes the partial slot slot_base + w + r.  A launch
// may have more workgroups than n_wg (a step launch is sized once for every
// step); the extra ones do nothing.
struct DecodeDyn {
  int32_t n_segs;
  int32_t total;     // flattened pages of this launch
  int32_t n_wg;      // workgroups that share them
  int32_t slot_base; // first partial slot of this launch
  int32_t row_pad;   // flattened pages after each row that map to nothing
  int32_t masked;    // 1: some segment's sequence has masked slots (read the masks)
  int32_t rb;        // row blocks of 16 query rows per tile (MFMA launch: 1 or 2;
                     // a piece then owns rb consecutive partial slots)
  int32_t pad;
  Seg segs[kMaxSegs];
};

// A plain decode call passes its plan with the launch.
struct DecodeArgs {
  DecodeStatic st;
  DecodeDyn dyn;
};

// The workgroup whose range holds flattened page x.
__host__ __device__ inline int32_t wg_of(int64_t x, int64_t total, int64_t n_wg) {
  return (int32_t)(((x + 1) * n_wg - 1) / total);
}

// A batch entry attends to the segments on its path through the tree of
// shared page runs: at most kMaxSrc (shared levels, then its own suffix).
constexpr int kMaxSrc = 8;

struct MergeStatic {
  float *out; // [B][Hq][D]
  const float *part_m;
  const float *part_l;
  const float *part_acc;
  const float *sinks; // [Hq] learned softmax sink logits (log2 units after sink_scale), or null
  float sink_scale;   // log2(e): the sinks are in the units of the scaled scores
  float out_scale;    // V scale of the layer in an 8-bit store (1 otherwise)
  int32_t pad;
  int32_t hq;
  int32_t group; // G
  int32_t hkv;
};

struct MergeDyn {
  int32_t total[2], n_wg[2], slot_base[2], row_pad[2]; // per launch (0: VALU, 1: MFMA)
  int32_t rb[2];                                       // row blocks per launch
  // every segment of the call (both launches, plan order): flattened start
  // of its rows, pages, and its launch (bit 0) and index inside that launch
  // Every field is a whole 32-bit word: a kernel reads these tables with
  // scalar loads, which address dwords.
  int32_t seg_start[kMaxSegs];
  int32_t seg_npages[kMaxSegs];
  int32_t seg_meta[kMaxSegs];
  // per batch entry: the segments it attends, each as the segment's plan
  // index (bits 0-7) and the entry's member index inside it (bits 8-11),
  // two to a word (source e in half e % 2 of word e / 2)
  uint32_t src[kMaxBatch][kMaxSrc / 2];
  int32_t n_src[kMaxBatch];
};

// The row lists of a small call's merge, one entry per (batch entry b, KV
// head g) at index b * kInlineG + g: for each of the entry's sources e, the
// partial row of its first piece for query head g * G (a workgroup adds its
// head's offset within the group), and the piece count (bits 0-15) and row
// step (bits 16-31).  A source past the entry's count has no pieces.  With
// them, and the grid giving (head in group, KV head, entry), a merge
// workgroup reads all it needs in one round: each dependent round of
// argument reads costs a trip to HBM, since the arguments are written anew
// for every launch.
struct MergeRows {
  int32_t base[kMaxSrc];
  int32_t cnt_step[kMaxSrc];
};
constexpr int kInlineRows = 16;
constexpr int kInlineG = 8; // entry stride: calls with Hkv <= 8 and at most 2 entries

struct MergeArgs {
  MergeStatic st;
  int32_t n_inline; // 1: rows[b * kInlineG + g] hold the row lists
  int32_t pad[3];
  MergeRows rows[kInlineRows];
  MergeDyn dyn;
};

// ---- decode step (append fused) -------------------------------------------
// One decode step appends a token to every entry and attends over the old
// tokens plus the new one.  The decode launches read the old tokens from
// the pools; the merge adds the new token as one more partial (its score
// against the entry's query, weight 1, value v_new) and stores its K, V and
// position.  (A page the step opens enters the page-table mirror when the
// step begins, so the mirror never holds an unset entry.)
struct StepAppend {
  int32_t page[kMaxBatch]; // physical page of the new token
  int32_t slot[kMaxBatch]; // its slot in that page
  int32_t pos[kMaxBatch];  // its position
};

// The step plan, in device memory: written once per step, read by every
// layer's launches, whose arguments therefore stay the same from step to
// step.
struct StepPlan {
  DecodeDyn dec[2];   // VALU, MFMA launch over every old token
  MergeDyn merge;
  DecodeDyn dec_w[2]; // the same over the window's old tokens (a windowed step)
  MergeDyn merge_w;
  StepAppend app;
  int32_t batch;      // entries of the step; merge workgroups past it do nothing
  int32_t pad;
};

struct StepMergeArgs {
  MergeStatic st;
  const StepPlan *plan;
  int32_t windowed; // 1: the plan's windowed merge sources
  float inv_k;      // 8-bit store: 1 / K and 1 / V scale of the layer (the new
  float inv_v;      // token is stored as E4M3 codes and attended as stored)
  int32_t pad2;
  const uint16_t *q;     // [B][Hq][D] bf16
  const uint16_t *k_new; // [B][Hkv][D] bf16
  const uint16_t *v_new; // [B][Hkv][D] bf16
  uint16_t *k;           // K pool at this layer
  uint16_t *v;           // V pool at this layer
  int32_t *pos;          // position pool [NP][P]
  int64_t page_stride;
  int64_t head_stride;
  float scale_log2;
  int32_t pad;
};

static_assert(sizeof(DecodeArgs) < 4096, "decode kernel arguments too large");
static_assert(sizeof(MergeArgs) < 4096, "merge kernel arguments too large");

hipError_t launch_decode_valu(int d, int group, const DecodeArgs &a, hipStream_t s);
// The MFMA tile kernels run kMfmaWaves waves per workgroup.
constexpr int kMfmaWaves = 4;
hipError_t launch_decode_mfma(int d, int group, const DecodeArgs &a, hipStream_t s);
hipError_t launch_decode_merge(int d, int batch, const MergeArgs &a, hipStream_t s);
// Step launches: `n_wg` workgroups (at least the plan's), the plan in device
// memory at `dyn`.
hipError_t launch_step_valu(int d, int group, const DecodeStatic &st, const DecodeDyn *dyn,
                            int n_wg, hipStream_t s);
hipError_t launch_step_mfma(int d, int group, const DecodeStatic &st, const DecodeDyn *dyn,
                            int n_wg, hipStream_t s);
hipError_t launch_step_merge(int d, int batch, const StepMergeArgs &a, bool kv8, hipStream_t s);
// Split-partial buffers of one decode call: m, l [slots][kRows] and acc
// [slots][kRows][D].
struct StaticPartials {
  float *m = nullptr, *l = nullptr, *acc = nullptr;
  int32_t slots = 0;
};
// Partial slots of the device array behind the allocation-free entry point.
constexpr int kStaticSlots = 4096;
// That array on the current device (its address looked up once per device).
hipError_t static_partials(StaticPartials *out);

// Workgroups of a decode kernel that fit on one CU.  kind: 0 VALU, 1 MFMA,
// 2 the 8-bit MFMA kernel (four waves), 3 the 8-bit VALU kernel, 4 the
// two-row-block MFMA kernel
hipError_t decode_blocks_per_cu(int kind, int d, int group, int *out);

} // namespace sq
