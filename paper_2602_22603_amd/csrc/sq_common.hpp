// sq_common.hpp - constants and pool layout shared by the host library and every gfx950
// kernel file.
// Internal to libsq.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace sq {

constexpr int kPage = 16;            // tokens per page in device mode
constexpr int kMaxAppendPages = 240; // pages one append launch may touch
constexpr int kMaxBatch = 64;        // queries per decode call
constexpr int kMaxSegs = 128;        // (page range, query rows) units per decode
constexpr int kMaxMembers = 8;       // sequences stacked in one MFMA tile
constexpr int kRows = 16;            // query rows per partial slot (MFMA N)
constexpr int kMaxItems = 8192;      // partial slots in the workspace

// Device pools and shapes.  K: [NL][Hkv][NP][P][D]; V: [NL][Hkv][NP][D][P];
// pos: [NP][P].  Element strides are in elements: bf16 (2 bytes), or E4M3
// bytes in an 8-bit store (kv8).  Head-major: the pages of one KV head are
// contiguous, so a decode work item streams one region.
struct Pools {
  uint16_t *k;
  uint16_t *v;
  int32_t *pos;
  int32_t nl, hkv, d, np;
  int64_t layer_stride; // Hkv * NP * P * D
  int64_t page_stride;  // P * D
  int64_t head_stride;  // NP * P * D
  int32_t kv8;          // 1: elements are E4M3 codes
  int32_t pad;
  const float *scales;  // 8-bit store: device [NL][4] = K scale, V scale, 1 / K scale, 1 / V scale
};

} // namespace sq
