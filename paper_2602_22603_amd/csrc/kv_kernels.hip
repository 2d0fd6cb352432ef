// kv_kernels.hip - gfx950 kernels that write and move KV-cache pages:
//   append (Algorithm 1, Phase 3: the context grows by the response R and the
//   tool output O), the fork's tail-page copy (Phase 2, C_aux <- C + p), and
//   span eviction clear_kv (Phase 1): keep-mask -> exclusive prefix sum ->
//   inverse map -> page-level gather into fresh pages.
//
// Layouts (elements are bf16 stored as uint16_t):
//   K pool [NL][Hkv][NP][P][D]   one 16-token page of one head is P*D
//                                 contiguous values, token-major; the pages
//                                 of one head are contiguous (head-major)
//   V pool [NL][Hkv][NP][D][P]   the same page stored channel-major: the P
//                                 tokens of one channel are contiguous
//   pos    [NP][P]               int32 position of each cached token
// The page size is 16 throughout.
#include "fp8.hpp"
#include "kv_args.hpp"

namespace sq {
namespace {

constexpr int P = kPage;

__device__ inline const uint16_t *k_chunk(const Pools &p, int layer, int page, int head) {
  return p.k + layer * p.layer_stride + (int64_t)page * p.page_stride + head * p.head_stride;
}
__device__ inline const uint16_t *v_chunk(const Pools &p, int layer, int page, int head) {
  return p.v + layer * p.layer_stride + (int64_t)page * p.page_stride + head * p.head_stride;
}
__device__ inline uint16_t *k_chunk_w(const Pools &p, int layer, int page, int head) {
  return p.k + layer * p.layer_stride + (int64_t)page * p.page_stride + head * p.head_stride;
}
__device__ inline uint16_t *v_chunk_w(const Pools &p, int layer, int page, int head) {
  return p.v + layer * p.layer_stride + (int64_t)page * p.page_stride + head * p.head_stride;
}

// ---------------------------------------------------------------------------
// Append: one block per (page touched, layer * Hkv + head).  New tokens come
// token-major [NL][n_total][Hkv][D]; K rows are copied as 16-byte units, V is
// transposed through LDS when a whole page is written and scattered per
// element when only some slots of a page are (the other slots of that page
// already hold earlier tokens of the sequence).
template <int D>
__global__ __launch_bounds__(256) void k_append(Pools p, AppendArgs a,
                                                const uint16_t *__restrict__ kn,
                                                const uint16_t *__restrict__ vn) {
  constexpr int U = D / 8; // 16-byte units per row
  __shared__ uint16_t tile[P][D + 8];
  const int pi = blockIdx.x;
  const int lh = blockIdx.y;
  const int layer = lh / p.hkv;
  const int head = lh % p.hkv;
  const int page = a.page_ids[pi];
  const int s_begin = pi == 0 ? a.slot0 : 0;
  const int t_begin = pi == 0 ? 0 : pi * P - a.slot0; // launch-local token of s_begin
  int s_end = s_begin + (a.n_tok - t_begin);
  if (s_end > P) s_end = P;
  const int ns = s_end - s_begin;
  const int64_t tok_stride = (int64_t)p.hkv * D;
  const int64_t src0 = ((int64_t)layer * a.n_total + a.tok0 + t_begin) * tok_stride + head * D;

  uint16_t *kd = k_chunk_w(p, layer, page, head);
  for (int idx = threadIdx.x; idx < ns * U; idx += blockDim.x) {
    const int j = idx / U, u = idx % U;
    const uint4 val = *(reinterpret_cast<const uint4 *>(kn + src0 + j * tok_stride) + u);
    *(reinterpret_cast<uint4 *>(kd + (s_begin + j) * D) + u) = val;
  }

  uint16_t *vd = v_chunk_w(p, layer, page, head);
  if (ns == P) {
    for (int idx = threadIdx.x; idx < P * U; idx += blockDim.x) {
      const int j = idx / U, u = idx % U;
      const uint4 val = *(reinterpret_cast<const uint4 *>(vn + src0 + j * tok_stride) + u);
      *reinterpret_cast<uint4 *>(&tile[j][u * 8]) = val;
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < D * 2; idx += blockDim.x) {
      const int d = idx >> 1, h = idx & 1;
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e)
        w[e] = (uint32_t)tile[h * 8 + 2 * e][d] | ((uint32_t)tile[h * 8 + 2 * e + 1][d] << 16);
      *reinterpret_cast<uint4 *>(vd + d * P + h * 8) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  } else {
    for (int idx = threadIdx.x; idx < ns * D; idx += blockDim.x) {
      const int j = idx % ns, d = idx / ns;
      vd[d * P + s_begin + j] = vn[src0 + j * tok_stride + d];
    }
  }

  if (lh == 0) {
    for (int j = threadIdx.x; j < ns; j += blockDim.x)
      p.pos[(int64_t)page * P + s_begin + j] = a.pos0 + t_begin + j;
    if (threadIdx.x == 0 && pi >= a.new_from) a.pt_row[a.pt_first + pi] = page;
  }
}

// The same for an 8-bit store: each bf16 value x becomes the E4M3 code of
// float(x) * (1 / scale) of its layer (K and V scales apart).
__device__ inline float bf16_val(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ inline uint2 quant8(uint4 w, float inv) { // 8 bf16 -> 8 codes
  const uint32_t x[4] = {w.x, w.y, w.z, w.w};
  uint32_t c[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    c[2 * i] = e4m3_encode(__uint_as_float(x[i] << 16) * inv);
    c[2 * i + 1] = e4m3_encode(__uint_as_float(x[i] & 0xffff0000u) * inv);
  }
  return make_uint2(c[0] | c[1] << 8 | c[2] << 16 | c[3] << 24,
                    c[4] | c[5] << 8 | c[6] << 16 | c[7] << 24);
}

template <int D>
__global__ __launch_bounds__(256) void k_append8(Pools p, AppendArgs a,
                                                 const uint16_t *__restrict__ kn,
                                                 const uint16_t *__restrict__ vn) {
  constexpr int U = D / 8; // 8-element units per row
  __shared__ uint16_t tile[P][D + 8];
  const int pi = blockIdx.x;
  const int lh = blockIdx.y;
  const int layer = lh / p.hkv;
  const int head = lh % p.hkv;
  const float inv_k = p.scales[4 * layer + 2], inv_v = p.scales[4 * layer + 3];
  const int page = a.page_ids[pi];
  const int s_begin = pi == 0 ? a.slot0 : 0;
  const int t_begin = pi == 0 ? 0 : pi * P - a.slot0;
  int s_end = s_begin + (a.n_tok - t_begin);
  if (s_end > P) s_end = P;
  const int ns = s_end - s_begin;
  const int64_t tok_stride = (int64_t)p.hkv * D;
  const int64_t src0 = ((int64_t)layer * a.n_total + a.tok0 + t_begin) * tok_stride + head * D;
  const int64_t chunk = layer * p.layer_stride + (int64_t)page * p.page_stride + head * p.head_stride;

  uint8_t *kd = reinterpret_cast<uint8_t *>(p.k) + chunk;
  for (int idx = threadIdx.x; idx < ns * U; idx += blockDim.x) {
    const int j = idx / U, u = idx % U;
    const uint4 val = *(reinterpret_cast<const uint4 *>(kn + src0 + j * tok_stride) + u);
    *reinterpret_cast<uint2 *>(kd + (s_begin + j) * D + 8 * u) = quant8(val, inv_k);
  }

  uint8_t *vd = reinterpret_cast<uint8_t *>(p.v) + chunk;
  if (ns == P) {
    for (int idx = threadIdx.x; idx < P * U; idx += blockDim.x) {
      const int j = idx / U, u = idx % U;
      const uint4 val = *(reinterpret_cast<const uint4 *>(vn + src0 + j * tok_stride) + u);
      *reinterpret_cast<uint4 *>(&tile[j][u * 8]) = val;
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < D * 2; idx += blockDim.x) {
      const int d = idx >> 1, h = idx & 1;
      uint32_t w[2] = {0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e)
        w[e >> 2] |= e4m3_encode(bf16_val(tile[h * 8 + e][d]) * inv_v) << (8 * (e & 3));
      *reinterpret_cast<uint2 *>(vd + d * P + h * 8) = make_uint2(w[0], w[1]);
    }
  } else {
    for (int idx = threadIdx.x; idx < ns * D; idx += blockDim.x) {
      const int j = idx % ns, d = idx / ns;
      vd[d * P + s_begin + j] = (uint8_t)e4m3_encode(bf16_val(vn[src0 + j * tok_stride + d]) * inv_v);
    }
  }

  if (lh == 0) {
    for (int j = threadIdx.x; j < ns; j += blockDim.x)
      p.pos[(int64_t)page * P + s_begin + j] = a.pos0 + t_begin + j;
    if (threadIdx.x == 0 && pi >= a.new_from) a.pt_row[a.pt_first + pi] = page;
  }
}

// One token for each of n sequences: block (b, layer * Hkv + head).
template <int D>
__global__ __launch_bounds__(64) void k_append_batch(Pools p, AppendBatchArgs a,
                                                     const uint16_t *__restrict__ kn,
                                                     const uint16_t *__restrict__ vn) {
  constexpr int U = D / 8;
  const int b = blockIdx.x;
  const int lh = blockIdx.y;
  const int layer = lh / p.hkv;
  const int head = lh % p.hkv;
  const int page = a.page[b];
  const int slot = a.slot[b];
  const int64_t src = (((int64_t)layer * a.n + b) * p.hkv + head) * D;
  uint16_t *kd = k_chunk_w(p, layer, page, head) + slot * D;
  for (int u = threadIdx.x; u < U; u += blockDim.x)
    *(reinterpret_cast<uint4 *>(kd) + u) = *(reinterpret_cast<const uint4 *>(kn + src) + u);
  uint16_t *vd = v_chunk_w(p, layer, page, head) + slot;
  for (int d = threadIdx.x; d < D; d += blockDim.x) vd[d * P] = vn[src + d];
  if (lh == 0 && threadIdx.x == 0) {
    p.pos[(int64_t)page * P + slot] = a.pos[b];
    if (a.pt_index[b] >= 0) a.pt[a.pt_index[b]] = page;
  }
}

template <int D>
__global__ __launch_bounds__(64) void k_append_batch8(Pools p, AppendBatchArgs a,
                                                      const uint16_t *__restrict__ kn,
                                                      const uint16_t *__restrict__ vn) {
  constexpr int U = D / 8;
  const int b = blockIdx.x;
  const int lh = blockIdx.y;
  const int layer = lh / p.hkv;
  const int head = lh % p.hkv;
  const float inv_k = p.scales[4 * layer + 2], inv_v = p.scales[4 * layer + 3];
  const int page = a.page[b];
  const int slot = a.slot[b];
  const int64_t src = (((int64_t)layer * a.n + b) * p.hkv + head) * D;
  const int64_t chunk = layer * p.layer_stride + (int64_t)page * p.page_stride + head * p.head_stride;
  uint8_t *kd = reinterpret_cast<uint8_t *>(p.k) + chunk + slot * D;
  for (int u = threadIdx.x; u < U; u += blockDim.x)
    *reinterpret_cast<uint2 *>(kd + 8 * u) = quant8(*(reinterpret_cast<const uint4 *>(kn + src) + u), inv_k);
  uint8_t *vd = reinterpret_cast<uint8_t *>(p.v) + chunk + slot;
  for (int d = threadIdx.x; d < D; d += blockDim.x)
    vd[d * P] = (uint8_t)e4m3_encode(bf16_val(vn[src + d]) * inv_v);
  if (lh == 0 && threadIdx.x == 0) {
    p.pos[(int64_t)page * P + slot] = a.pos[b];
    if (a.pt_index[b] >= 0) a.pt[a.pt_index[b]] = page;
  }
}

// dst[i] = src[i] for i < n, then dst[n] = tail_value when tail_value >= 0.
__global__ __launch_bounds__(64) void k_set_entries(SetEntries a) {
  if ((int)threadIdx.x < a.n) a.base[a.index[threadIdx.x]] = a.value[threadIdx.x];
}

__global__ __launch_bounds__(256) void k_copy_i32(int32_t *dst, const int32_t *src, int32_t n,
                                                  int32_t tail_value) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
  if (i == n && tail_value >= 0) dst[n] = tail_value;
}

__global__ __launch_bounds__(256) void k_fill_i32(int32_t *dst, int32_t value, int32_t n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = value;
}

// Element E of the pools (bf16 bits, or E4M3 bytes): the chunk of one
// (layer, page, head), strides counted in elements.
template <class E> __device__ inline E *chunk_of(uint16_t *pool, const Pools &p, int layer, int page,
                                                 int head) {
  return reinterpret_cast<E *>(pool) + layer * p.layer_stride + (int64_t)page * p.page_stride +
         head * p.head_stride;
}

// Whole-page copy (every layer and head, K, V and pos): the fork's tail page.
template <int D, class E>
__global__ __launch_bounds__(256) void k_copy_page(Pools p, int32_t src_page, int32_t dst_page) {
  constexpr int U = P * D * (int)sizeof(E) / 16;
  const int lh = blockIdx.x;
  const int layer = lh / p.hkv;
  const int head = lh % p.hkv;
  const uint4 *ks = reinterpret_cast<const uint4 *>(chunk_of<E>(p.k, p, layer, src_page, head));
  const uint4 *vs = reinterpret_cast<const uint4 *>(chunk_of<E>(p.v, p, layer, src_page, head));
  uint4 *kd = reinterpret_cast<uint4 *>(chunk_of<E>(p.k, p, layer, dst_page, head));
  uint4 *vd = reinterpret_cast<uint4 *>(chunk_of<E>(p.v, p, layer, dst_page, head));
  for (int u = threadIdx.x; u < U; u += blockDim.x) {
    kd[u] = ks[u];
    vd[u] = vs[u];
  }
  if (lh == 0 && threadIdx.x < P)
    p.pos[(int64_t)dst_page * P + threadIdx.x] = p.pos[(int64_t)src_page * P + threadIdx.x];
}

// ---------------------------------------------------------------------------
// Eviction index.  keep[i] = 0 iff token i lies in one of the evicted spans;
// dst = exclusive prefix sum of keep; src_of[dst[i]] = i for kept i.  The
// keep mask is a union of sorted spans, so its prefix sum at i is
// i - (evicted tokens before i): the span-level exclusive prefix sums of the
// span lengths (spans[k][2]) plus the part of the span that contains i.
// Every token is independent, so one pass over the tokens suffices.
constexpr int kPerThread = kScanBlock / kScanThreads; // 8

__device__ inline int span_search(const int32_t *spans, int n_spans, int i) {
  // index of the last span whose start <= i, or -1
  int lo = 0, hi = n_spans - 1, ans = -1;
  while (lo <= hi) {
    const int mid = (lo + hi) >> 1;
    if (spans[3 * mid] <= i) {
      ans = mid;
      lo = mid + 1;
    } else {
      hi = mid - 1;
    }
  }
  return ans;
}

// The span list where a workgroup reads it: copied to LDS (lsp, 3 *
// kInlineSpans ints) from the kernel arguments when it travels there, else
// the device copy.  Every thread of the workgroup must call it.
__device__ inline const int32_t *stage_spans(const EvictArgs &a, int32_t *lsp) {
  const bool inl = a.n_spans <= kInlineSpans;
  if (inl)
    for (int i = threadIdx.x; i < 3 * a.n_spans; i += blockDim.x) lsp[i] = a.inl[i];
  __syncthreads();
  return inl ? lsp : a.spans;
}

// The old index of the kept token that lands at new index d: the last span k
// whose start lies at or before d once the tokens evicted before it are
// taken out (start_k - before_k <= d; non-decreasing in k) has every span up
// to it evicted before that token, so it is d + before_k + (end_k - start_k);
// with no such span it is d.
__device__ inline int source_of(const int32_t *spans, int n_spans, int d) {
  int lo = 0, hi = n_spans - 1, k = -1;
  while (lo <= hi) {
    const int mid = (lo + hi) >> 1;
    if (spans[3 * mid] - spans[3 * mid + 2] <= d) {
      k = mid;
      lo = mid + 1;
    } else {
      hi = mid - 1;
    }
  }
  return k < 0 ? d : d + spans[3 * k + 2] + (spans[3 * k + 1] - spans[3 * k]);
}

// Block blk (kScanBlock tokens) of the eviction index, by a workgroup of
// kScanThreads threads (the gather's too).
static_assert(kScanThreads == 256, "gather workgroups also run index blocks");
__device__ inline void evict_index_block(const EvictArgs &a, const int32_t *spans, int blk) {
  const int base = blk * kScanBlock + threadIdx.x * kPerThread;
  if (base >= a.n_tokens) return;
  int s = span_search(spans, a.n_spans, base);
  for (int e = 0; e < kPerThread; ++e) {
    const int i = base + e;
    if (i >= a.n_tokens) break;
    while (s + 1 < a.n_spans && spans[3 * (s + 1)] <= i) ++s;
    int before = 0; // evicted tokens before i
    bool inside = false;
    if (s >= 0) {
      const int st = spans[3 * s], en = spans[3 * s + 1];
      inside = i < en;
      before = spans[3 * s + 2] + (inside ? i - st : en - st);
    }
    const int d = i - before;
    a.keep[i] = inside ? 0 : 1;
    a.dst[i] = d;
    if (!inside) a.src_of[d] = i;
  }
}

__global__ __launch_bounds__(kScanThreads) void k_evict_index(EvictArgs a) {
  __shared__ int32_t lsp[3 * kInlineSpans];
  evict_index_block(a, stage_spans(a, lsp), blockIdx.x);
}

// Fresh page id number i of an eviction.
__device__ inline int32_t new_page_id(const NewIds &ids, int i) {
  if (ids.list) return ids.list[i];
  int r = 0;
  while (r + 1 < ids.n_runs && ids.before[r + 1] <= i) ++r;
  return ids.first[r] + (i - ids.before[r]);
}

// dst[i] = fresh id i: the page-table row takes the fresh ids after the gather.
__global__ __launch_bounds__(256) void k_write_ids(int32_t *dst, NewIds ids, int32_t n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = new_page_id(ids, i);
}

// One destination page's sources, staged: each slot's source page id and
// slot (LDS, written by the first P threads from src_of and the page-table
// row, which still holds the old ids), and the distinct
// source pages in order, which every thread finds itself from LDS (the kept
// tokens are in old order, and a page list holds a page once, so the source
// page changes exactly where the id does).
constexpr int kMaxStaged = 4; // source pages of one destination page staged whole
struct PageSources {
  int nv;                  // valid slots
  int nu;                  // distinct source pages (may exceed kMaxStaged)
  int u0, u1, u2, u3;      // their ids, the first kMaxStaged of them (scalars,
                           // so that nothing is indexed at run time)
  __device__ int up(int u) const { return u == 0 ? u0 : u == 1 ? u1 : u == 2 ? u2 : u3; }
};
static_assert(kMaxStaged == 4, "PageSources holds four staged pages");

__device__ inline void load_sources(const int32_t *src_of, const int32_t *pt_row, int t0, int nv,
                                    int *spage, int *sslot) {
  if ((int)threadIdx.x < nv) {
    const int src = src_of[t0 + threadIdx.x];
    spage[threadIdx.x] = pt_row[src / P];
    sslot[threadIdx.x] = src % P;
  }
}

__device__ inline PageSources distinct_sources(int nv, const int *spage) {
  PageSources ps{};
  ps.nv = nv;
  for (int j = 0; j < nv; ++j)
    if (j == 0 || spage[j] != spage[j - 1]) {
      const int id = spage[j];
      if (ps.nu == 0) ps.u0 = id;
      else if (ps.nu == 1) ps.u1 = id;
      else if (ps.nu == 2) ps.u2 = id;
      else if (ps.nu == 3) ps.u3 = id;
      ++ps.nu;
    }
  return ps;
}

// Staged source page of slot j: the page changes among slots 1..j.
__device__ inline int staged_of(int j, const int *spage) {
  int f = 0;
  for (int i = 1; i <= j; ++i) f += spage[i] != spage[i - 1];
  return f;
}

// The destination page's V^T units from the staged source pages (or, with
// more than kMaxStaged of them, element by element from the pools).
template <int D, class E>
__device__ inline void assemble_v(const Pools &p, int layer, int head, E *vd, const PageSources &ps,
                                  const uint4 (*vbuf)[D * P * sizeof(E) / 16], const int *spage,
                                  const int *sslot) {
  constexpr int VU = D * P * (int)sizeof(E) / 16;
  constexpr int EPU = 16 / (int)sizeof(E);
  for (int idx = threadIdx.x; idx < VU; idx += blockDim.x) {
    const int d = idx / (P / EPU), c = idx % (P / EPU);
    E out[EPU];
    int f = staged_of(c * EPU, spage);
#pragma unroll
    for (int e = 0; e < EPU; ++e) {
      const int j = c * EPU + e;
      if (e > 0 && j < ps.nv) f += spage[j] != spage[j - 1];
      if (j >= ps.nv) out[e] = (E)0;
      else if (ps.nu <= kMaxStaged) out[e] = reinterpret_cast<const E *>(vbuf[f])[d * P + sslot[j]];
      else out[e] = chunk_of<E>(p.v, p, layer, spage[j], head)[d * P + sslot[j]];
    }
    uint4 o;
    __builtin_memcpy(&o, out, 16);
    *reinterpret_cast<uint4 *>(vd + d * P + c * EPU) = o;
  }
}

// ---------------------------------------------------------------------------
// Gather: a workgroup per (fresh page pi0 + b, layer * Hkv + head) fills
// destination page fp + pi0 + b with the kept tokens (fp + pi0 + b) * P + j,
// j < P, j below L'.  K rows move as 16-byte units; V^T rows are assembled
// in LDS from the (at most four, usually one or two) source pages staged
// whole with 16-byte loads, then written as 16-byte units (more source pages
// fall back to element moves).  Kept token t comes from old token
// source_of(t) of the old pages, whose ids the page-table row still holds
// (the new ids are written there after the last gather).  When the spans
// travel in the kernel arguments, the first launch of an eviction also
// writes the eviction index (keep, dst, src_of) in its first index_blocks
// workgroups, alongside the copies, and takes the sources from the span
// list so that it does not wait for the index; later launches of a chunked
// eviction, and every launch after a separate index kernel, read src_of.  A fresh page is never a page
// this or a later gather reads: it is either a page nothing held or an old
// page whose tokens earlier gathers have all moved, so nothing is read after
// being written.
template <int D, class E>
__global__ __launch_bounds__(256) void k_evict_gather(Pools p, GatherArgs a) {
  constexpr int U = D * (int)sizeof(E) / 16;      // 16-byte units per K row
  constexpr int VU = D * P * (int)sizeof(E) / 16; // 16-byte units of one page's V^T
  constexpr int EPU = 16 / (int)sizeof(E);        // V^T elements per unit
  constexpr int kMaxSrc = 4;                       // source pages staged in LDS
  __shared__ int spage[P];
  __shared__ int sslot[P];
  __shared__ int sidx[P];  // the source's page index in the old list
  __shared__ int nvalid;
  __shared__ int upage[P]; // the distinct source pages, in order
  __shared__ int uidx[P];  // slot j's source page in upage
  __shared__ int n_up;
  __shared__ uint4 vbuf[kMaxSrc][VU];
  __shared__ int32_t lsp[3 * kInlineSpans];
  const int n = a.n_new;
  const int lin = blockIdx.x + blockIdx.y * gridDim.x;
  // the launch that writes the index takes the sources from the spans; later
  // launches of a chunked eviction read them from src_of (one round of loads)
  const bool from_spans = a.index_blocks > 0;
  const int32_t *spans = from_spans ? stage_spans(a.ev, lsp) : nullptr;
  if (lin < a.index_blocks) {
    evict_index_block(a.ev, spans, lin);
    return;
  }
  // Work item w = (KV row lh, tail page pl), page fastest.  Workgroups are
  // dealt to the 8 XCDs in turn, so each XCD takes a contiguous range of
  // w: neighbouring destination pages, which share source pages, then hit
  // the same L2.  (Workgroups past the last item, which round the grid up
  // to whole rows, have nothing to do.)
  const int total = n * p.nl * p.hkv;
  const int gl = lin - a.index_blocks;
  if (gl >= total) return;
  const int x = gl % 8, q = total / 8, r = total % 8;
  const int w = x * q + min(x, r) + gl / 8;
  const int pl = w % n;
  const int lh = w / n;
  const int pi = a.pi0 + pl;
  const int layer = lh / p.hkv;
  const int head = lh % p.hkv;
  const int t0 = (a.fp + pi) * P;
  const int ns = a.ev.n_spans;
  auto src_of = [&](int t) { return from_spans ? source_of(spans, ns, t) : a.ev.src_of[t]; };
  if (a.remap && t0 + P <= a.new_len) {
    const int s0 = src_of(t0);
    if (s0 % P == 0 && src_of(t0 + P - 1) == s0 + P - 1) return; // remapped, not copied
  }
  const int dst_page = new_page_id(a.ids, pl);
  if (threadIdx.x < P) {
    const int t = t0 + threadIdx.x;
    if (t < a.new_len) {
      const int src = src_of(t);
      spage[threadIdx.x] = a.pt_row[src / P];
      sslot[threadIdx.x] = src % P;
      sidx[threadIdx.x] = src / P;
    }
  }
  if (threadIdx.x == 0) nvalid = min(P, a.new_len - t0);
  __syncthreads();
  const int nv = nvalid;
  if ((int)threadIdx.x < nv) {
    // sources are in increasing old order, so slot j's source page is the
    // number of page changes among slots 1..j
    int f = 0;
    for (int i = 1; i <= (int)threadIdx.x; ++i) f += sidx[i] != sidx[i - 1];
    uidx[threadIdx.x] = f;
    upage[f] = spage[threadIdx.x];
    if ((int)threadIdx.x == nv - 1) n_up = f + 1;
  }

  E *kd = chunk_of<E>(p.k, p, layer, dst_page, head);
  for (int idx = threadIdx.x; idx < nv * U; idx += blockDim.x) {
    const int j = idx / U, u = idx % U;
    const uint4 *ks = reinterpret_cast<const uint4 *>(chunk_of<E>(p.k, p, layer, spage[j], head) +
                                                      sslot[j] * D);
    *(reinterpret_cast<uint4 *>(kd + j * D) + u) = ks[u];
  }
  __syncthreads();
  const int nu = n_up;
  E *vd = chunk_of<E>(p.v, p, layer, dst_page, head);
  if (nu <= kMaxSrc) {
    // stage the source pages' V^T (16-byte loads), then assemble each
    // destination unit of EPU slots of one channel from LDS
    for (int u = 0; u < nu; ++u) {
      const uint4 *vs = reinterpret_cast<const uint4 *>(chunk_of<E>(p.v, p, layer, upage[u], head));
      for (int idx = threadIdx.x; idx < VU; idx += blockDim.x) vbuf[u][idx] = vs[idx];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < VU; idx += blockDim.x) {
      const int d = idx / (P / EPU), c = idx % (P / EPU);
      E out[EPU];
#pragma unroll
      for (int e = 0; e < EPU; ++e) {
        const int j = c * EPU + e;
        out[e] = j < nv ? reinterpret_cast<const E *>(vbuf[uidx[j]])[d * P + sslot[j]] : (E)0;
      }
      uint4 o;
      __builtin_memcpy(&o, out, 16);
      *reinterpret_cast<uint4 *>(vd + d * P + c * EPU) = o;
    }
  } else {
    for (int idx = threadIdx.x; idx < D * P; idx += blockDim.x) {
      const int j = idx % P, d = idx / P;
      if (j < nv) vd[d * P + j] = chunk_of<E>(p.v, p, layer, spage[j], head)[d * P + sslot[j]];
    }
  }
  if (lh == 0 && threadIdx.x < nv)
    p.pos[(int64_t)dst_page * P + threadIdx.x] =
        p.pos[(int64_t)spage[threadIdx.x] * P + sslot[threadIdx.x]];
}

// ---------------------------------------------------------------------------
// In-place eviction: tail page k of the compacted sequence is written to
// ids(k), normally the old page at list index fp + k itself.  Its kept
// tokens come from old list indices >= fp + k, so a page is never read after
// a page before it in the tail has been rewritten, as long as the pages of
// one launch read no page of the launch but their own: the host cuts the
// tail into such runs (round mode, one workgroup per page and layer * Hkv +
// head, like the gather), or hands a run of short ones to sweep mode, where
// one workgroup per layer * Hkv + head takes the pages in order.  Either way
// a workgroup loads everything a page needs (K rows, the V^T of its source
// pages, positions) in one round into LDS, waits at a barrier until every
// load of the page has landed there, and only then writes the page, which
// may be one of its own sources.
template <int D, class E>
__global__ __launch_bounds__(256) void k_evict_inplace(Pools p, InplaceArgs a) {
  constexpr int U = D * (int)sizeof(E) / 16;      // 16-byte units per K row
  constexpr int VU = D * P * (int)sizeof(E) / 16; // 16-byte units of one page's V^T
  __shared__ int spage[P];
  __shared__ int sslot[P];
  __shared__ uint4 kbuf[P * U];
  __shared__ uint4 vbuf[kMaxStaged][VU];
  __shared__ int32_t pbuf[P];
  int pl0, pl1, lh;
  if (a.sweep) {
    pl0 = 0;
    pl1 = a.n_pages;
    lh = blockIdx.x;
  } else {
    // consecutive pages of one KV row to one XCD, as in the gather
    const int n = gridDim.x;
    const int total = n * gridDim.y;
    const int lin = blockIdx.x + blockIdx.y * n;
    const int x = lin % 8, q = total / 8, r = total % 8;
    const int w = x * q + min(x, r) + lin / 8;
    pl0 = w % n;
    pl1 = pl0 + 1;
    lh = w / n;
  }
  const int layer = lh / p.hkv;
  const int head = lh % p.hkv;
  for (int pl = pl0; pl < pl1; ++pl) {
    const int k = a.k0 + pl;
    const int t0 = (a.fp + k) * P;
    const int dst_page = new_page_id(a.ids, k);
    const int nv = min(P, a.new_len - t0);
    load_sources(a.src_of, a.pt_row, t0, nv, spage, sslot);
    __syncthreads();
    const PageSources ps = distinct_sources(nv, spage);
    // ---- read: everything the page needs, into LDS, in one round ----
    for (int idx = threadIdx.x; idx < nv * U; idx += blockDim.x) {
      const int j = idx / U, u = idx % U;
      kbuf[idx] = reinterpret_cast<const uint4 *>(chunk_of<E>(p.k, p, layer, spage[j], head) +
                                                  sslot[j] * D)[u];
    }
    if (ps.nu <= kMaxStaged) {
#pragma unroll
      for (int u = 0; u < kMaxStaged; ++u) {
        if (u >= ps.nu) break;
        const uint4 *vs = reinterpret_cast<const uint4 *>(chunk_of<E>(p.v, p, layer, ps.up(u), head));
        for (int idx = threadIdx.x; idx < VU; idx += blockDim.x) vbuf[u][idx] = vs[idx];
      }
    } else {
      E *vo = reinterpret_cast<E *>(&vbuf[0][0]);
      for (int idx = threadIdx.x; idx < D * P; idx += blockDim.x) {
        const int j = idx % P, d = idx / P;
        vo[idx] = j < nv ? chunk_of<E>(p.v, p, layer, spage[j], head)[d * P + sslot[j]] : (E)0;
      }
    }
    if (lh == 0 && (int)threadIdx.x < nv)
      pbuf[threadIdx.x] = p.pos[(int64_t)spage[threadIdx.x] * P + sslot[threadIdx.x]];
    // every load of this page's sources has been written to LDS by now: the
    // page itself may be overwritten
    __syncthreads();
    // ---- write ----
    uint4 *kd = reinterpret_cast<uint4 *>(chunk_of<E>(p.k, p, layer, dst_page, head));
    for (int idx = threadIdx.x; idx < nv * U; idx += blockDim.x) kd[idx] = kbuf[idx];
    E *vd = chunk_of<E>(p.v, p, layer, dst_page, head);
    if (ps.nu <= kMaxStaged) {
      assemble_v<D, E>(p, layer, head, vd, ps, vbuf, spage, sslot);
    } else {
      for (int idx = threadIdx.x; idx < VU; idx += blockDim.x)
        reinterpret_cast<uint4 *>(vd)[idx] = vbuf[0][idx];
    }
    if (lh == 0 && (int)threadIdx.x < nv) p.pos[(int64_t)dst_page * P + threadIdx.x] = pbuf[threadIdx.x];
    __syncthreads(); // the next page reuses the LDS
  }
}

} // namespace

// ---------------------------------------------------------------------------
hipError_t launch_append(const Pools &p, const AppendArgs &a, const void *k_new,
                         const void *v_new, hipStream_t s) {
  dim3 grid(a.n_pages, p.nl * p.hkv);
  const auto *kn = static_cast<const uint16_t *>(k_new);
  const auto *vn = static_cast<const uint16_t *>(v_new);
  if (p.kv8) {
    if (p.d == 128)
      hipLaunchKernelGGL(k_append8<128>, grid, dim3(256), 0, s, p, a, kn, vn);
    else
      hipLaunchKernelGGL(k_append8<64>, grid, dim3(256), 0, s, p, a, kn, vn);
  } else if (p.d == 128)
    hipLaunchKernelGGL(k_append<128>, grid, dim3(256), 0, s, p, a, kn, vn);
  else
    hipLaunchKernelGGL(k_append<64>, grid, dim3(256), 0, s, p, a, kn, vn);
  return hipGetLastError();
}

hipError_t launch_append_batch(const Pools &p, const AppendBatchArgs &a, const void *k_new,
                               const void *v_new, hipStream_t s) {
  dim3 grid(a.n, p.nl * p.hkv);
  const auto *kn = static_cast<const uint16_t *>(k_new);
  const auto *vn = static_cast<const uint16_t *>(v_new);
  if (p.kv8) {
    if (p.d == 128)
      hipLaunchKernelGGL(k_append_batch8<128>, grid, dim3(64), 0, s, p, a, kn, vn);
    else
      hipLaunchKernelGGL(k_append_batch8<64>, grid, dim3(64), 0, s, p, a, kn, vn);
  } else if (p.d == 128)
    hipLaunchKernelGGL(k_append_batch<128>, grid, dim3(64), 0, s, p, a, kn, vn);
  else
    hipLaunchKernelGGL(k_append_batch<64>, grid, dim3(64), 0, s, p, a, kn, vn);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t *dst, int32_t value, int32_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_i32, dim3((n + 255) / 256), dim3(256), 0, s, dst, value, n);
  return hipGetLastError();
}

hipError_t launch_set_entries(const SetEntries &a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  if (a.n > kMaxBatch) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_set_entries, dim3(1), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_copy_i32(int32_t *dst, const int32_t *src, int32_t n, int32_t tail_index,
                           int32_t tail_value, hipStream_t s) {
  (void)tail_index;
  const int total = n + 1;
  hipLaunchKernelGGL(k_copy_i32, dim3((total + 255) / 256), dim3(256), 0, s, dst, src, n,
                     tail_value);
  return hipGetLastError();
}

hipError_t launch_copy_page(const Pools &p, int32_t src_page, int32_t dst_page, hipStream_t s) {
  const dim3 grid(p.nl * p.hkv), block(256);
  if (p.kv8) {
    if (p.d == 128)
      hipLaunchKernelGGL((k_copy_page<128, uint8_t>), grid, block, 0, s, p, src_page, dst_page);
    else
      hipLaunchKernelGGL((k_copy_page<64, uint8_t>), grid, block, 0, s, p, src_page, dst_page);
  } else if (p.d == 128)
    hipLaunchKernelGGL((k_copy_page<128, uint16_t>), grid, block, 0, s, p, src_page, dst_page);
  else
    hipLaunchKernelGGL((k_copy_page<64, uint16_t>), grid, block, 0, s, p, src_page, dst_page);
  return hipGetLastError();
}

hipError_t launch_evict_index(const EvictArgs &a, hipStream_t s) {
  const int nblk = (a.n_tokens + kScanBlock - 1) / kScanBlock;
  if (nblk == 0) return hipSuccess;
  hipLaunchKernelGGL(k_evict_index, dim3(nblk), dim3(kScanThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_write_ids(int32_t *dst, const NewIds &ids, int32_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_write_ids, dim3((n + 255) / 256), dim3(256), 0, s, dst, ids, n);
  return hipGetLastError();
}

hipError_t launch_evict_inplace(const Pools &p, const InplaceArgs &a, hipStream_t s) {
  if (a.n_pages <= 0) return hipSuccess;
  const dim3 grid = a.sweep ? dim3(p.nl * p.hkv) : dim3(a.n_pages, p.nl * p.hkv);
  if (p.kv8) {
    if (p.d == 128)
      hipLaunchKernelGGL((k_evict_inplace<128, uint8_t>), grid, dim3(256), 0, s, p, a);
    else
      hipLaunchKernelGGL((k_evict_inplace<64, uint8_t>), grid, dim3(256), 0, s, p, a);
  } else if (p.d == 128)
    hipLaunchKernelGGL((k_evict_inplace<128, uint16_t>), grid, dim3(256), 0, s, p, a);
  else
    hipLaunchKernelGGL((k_evict_inplace<64, uint16_t>), grid, dim3(256), 0, s, p, a);
  return hipGetLastError();
}

hipError_t launch_evict_gather(const Pools &p, const GatherArgs &a, hipStream_t s) {
  if (a.n_new == 0) return hipSuccess;
  // rows of n_new workgroups: the copies' (layer, head) rows, then enough
  // for the index blocks
  const int rows = p.nl * p.hkv + (a.index_blocks + a.n_new - 1) / a.n_new;
  dim3 grid(a.n_new, rows);
  if (p.kv8) {
    if (p.d == 128)
      hipLaunchKernelGGL((k_evict_gather<128, uint8_t>), grid, dim3(256), 0, s, p, a);
    else
      hipLaunchKernelGGL((k_evict_gather<64, uint8_t>), grid, dim3(256), 0, s, p, a);
  } else if (p.d == 128)
    hipLaunchKernelGGL((k_evict_gather<128, uint16_t>), grid, dim3(256), 0, s, p, a);
  else
    hipLaunchKernelGGL((k_evict_gather<64, uint16_t>), grid, dim3(256), 0, s, p, a);
  return hipGetLastError();
}

} // namespace sq
