/*
 * sq.h - C ABI of libsq, the SideQuest KV-cache hot path for MI355X (gfx950).
 *
 * SideQuest (arXiv 2602.22603) lets a reasoning model fork an auxiliary
 * thread on its own shared context; the auxiliary thread names stale tool
 * responses ("cursors") and, once the main thread's turn has finished, their
 * tokens are cleared from the KV cache (Algorithm 1; §3.1).  This library
 * holds that KV cache and runs the data-parallel work under it:
 *
 *   - a paged KV store in which an auxiliary branch aliases the main thread's
 *     pages without copying them (sq_fork; storage claim of §3.4),
 *   - span eviction, clear_kv(Delta_ids) of Algorithm 1 Phase 1: keep-mask ->
 *     exclusive prefix sum -> page-level gather into fresh pages, kept keys
 *     keeping their original positions (sq_evict_spans),
 *   - decode-step attention of a batch of main and auxiliary queries over the
 *     shared, compacted cache: GQA split-K flash decoding plus a cross-split
 *     merge, and a multi-query MFMA tile for a prefix that several queries
 *     share (sq_decode_attn; the memory-bound step of §1 and §3.4, whose
 *     shared-prefix optimisation §3.4 points to).
 *
 * Conventions for every call
 * --------------------------
 *  - Every call returns an sq_status.  All validation happens before any
 *    change: a call that fails with SQ_ERR_INVALID, SQ_ERR_NO_PAGES,
 *    SQ_ERR_UNKNOWN_SEQ, SQ_ERR_UNKNOWN_CURSOR or SQ_ERR_SPAN changes nothing.
 *    SQ_ERR_HIP means a HIP call failed after validation; the device state of
 *    the store is then undefined and the store should be destroyed.
 *    sq_last_error() gives a thread-local message for the last failure.
 *  - Device buffers (pools, workspace, q, out, new K/V) are allocated and
 *    owned by the caller and must outlive the store or the call.  The library
 *    owns host metadata only; it never allocates device memory.  In device
 *    mode it allocates one pinned host staging buffer at sq_store_create.
 *  - Host metadata changes when a call returns; device work is enqueued on
 *    the given HIP stream (a hipStream_t passed as void*; NULL = the null
 *    stream).  All device work of one store must go to ONE stream, in call
 *    order: stream order is what makes an eviction issued after a decode read
 *    the old pages after that decode has read them (§3.1, step 4), and what
 *    lets a released page be reused safely.
 *  - A store is not thread-safe.
 *
 * Data layout in HBM (caller-allocated, sizes from sq_pool_bytes)
 * ---------------------------------------------------------------
 *   K pool  bf16  [NL][Hkv][num_pages][P][D]   token-major rows of D values
 *                                               (E4M3 bytes with SQ_STORE_KV_FP8)
 *   V pool  bf16  [NL][Hkv][num_pages][D][P]   page-transposed: the P tokens
 *                                               of one channel are contiguous
 *   pos     int32 [num_pages][P]               position of each cached token
 * Head-major: all pages of one KV head of one layer form one contiguous
 * region, which decode attention streams.
 * P (page_size) is 16 in device mode; D (head_dim) is 64 or 128; the query
 * group G = Hq / Hkv is 1, 2, 4 or 8.  Query head h reads KV head h / G.
 */
#ifndef SQ_H
#define SQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SQ_ABI_VERSION 8

typedef struct sq_store sq_store; /* opaque, library-owned host metadata */
typedef int32_t sq_seq;           /* sequence handle: main thread or aux branch */

typedef enum {
  SQ_OK = 0,
  SQ_ERR_INVALID = 1,        /* bad argument, capacity or configuration */
  SQ_ERR_NO_PAGES = 2,       /* the page pool cannot hold the result */
  SQ_ERR_UNKNOWN_SEQ = 3,    /* handle not live */
  SQ_ERR_UNKNOWN_CURSOR = 4, /* cursor not registered on the sequence */
  SQ_ERR_SPAN = 5,           /* span outside the sequence or overlapping */
  SQ_ERR_HIP = 6             /* a HIP runtime call failed */
} sq_status;

/* sq_store_config.flags */
#define SQ_STORE_METADATA_ONLY 1u /* host bookkeeping only: no pools, no
                                     workspace, no HIP calls; any page size;
                                     sq_decode_attn is rejected */
#define SQ_STORE_EVICT_REMAP 2u   /* page-aligned remap in sq_evict_spans: a
                                     tail page whose P kept tokens are one old
                                     page's P tokens in order (the tokens
                                     evicted before it are a multiple of P)
                                     takes that old page by reference instead
                                     of a fresh page and a copy.  Logical
                                     views are the same; page tables and
                                     refcounts differ from the default. */
#define SQ_STORE_EVICT_INPLACE 8u /* in-place eviction in sq_evict_spans: tail
                                     page k of the compacted sequence is the
                                     old page at the same list index (its
                                     kept tokens rewritten there) whenever the
                                     sequence alone holds that page; a fresh
                                     page only replaces one another branch
                                     still holds.  With no shared tail page
                                     the eviction takes no page at all, so it
                                     succeeds on a full pool.  Logical views
                                     are the same; page tables differ from the
                                     default.  Excludes SQ_STORE_EVICT_REMAP
                                     and evict_chunk_pages > 0. */
#define SQ_STORE_KV_FP8 4u        /* 8-bit KV cache (a model-serving option;
                                     the paper states no precision): the K and
                                     V pools hold E4M3 codes, one byte per
                                     element in the same layouts.  Appends
                                     take bf16 and store the code nearest to
                                     float(x) * float(1 / scale) (ties to
                                     even, saturating at 448) with the
                                     layer's scale from kv_scales; attention
                                     reads code * scale.  Every mode runs;
                                     SQ_ATTN_AUTO reads every segment on the
                                     MFMA tile. */

/* sq_decode_attn modes */
#define SQ_ATTN_AUTO 0          /* shared-prefix tiles where queries share
                                   pages, per-sequence tiles elsewhere */
#define SQ_ATTN_STREAM 1        /* per-sequence VALU split-K kernel */
#define SQ_ATTN_SHARED_PREFIX 2 /* shared prefixes on the MFMA multi-query
                                   tile, suffixes on the VALU kernel */
#define SQ_ATTN_MFMA 3          /* per-sequence, MFMA tile (no grouping) */

/* Limits. */
#define SQ_MAX_BATCH 64           /* sequences per sq_decode_attn / append_batch */
#define SQ_MAX_EVICT_SPANS 16384  /* distinct cursors per sq_evict_spans call */

typedef struct {
  int32_t num_layers;        /* NL >= 1 */
  int32_t num_q_heads;       /* Hq, a multiple of num_kv_heads */
  int32_t num_kv_heads;      /* Hkv >= 1 */
  int32_t head_dim;          /* D: 64 or 128 (device mode) */
  int32_t page_size;         /* P: 16 (device mode) */
  int32_t num_pages;         /* physical pages in the pools */
  int32_t max_seqs;          /* live sequence handles at once */
  int32_t max_pages_per_seq; /* longest page list of one sequence */
  void *k_pool;              /* device, see layout above (device mode) */
  void *v_pool;              /* device */
  int32_t *pos_pool;         /* device */
  void *workspace;           /* device scratch of sq_workspace_bytes() bytes */
  uint64_t workspace_bytes;
  uint32_t flags;            /* SQ_STORE_* */
  int32_t evict_chunk_pages; /* 0: sq_evict_spans allocates every fresh page
                                of the compacted tail before releasing old
                                ones.  C > 0: C fresh pages at a time, and the
                                old pages whose tokens are all gathered are
                                released between chunks (and may be reused by
                                the next chunk), so an eviction holds at most
                                C transient pages; one gather launch per
                                chunk.  The resulting page ids differ. */
  const float *kv_scales;    /* SQ_STORE_KV_FP8: host [num_layers][2], the K
                                and V scale of each layer (finite, > 0),
                                copied at creation; ignored otherwise */
} sq_store_config;

typedef struct {
  int64_t length;   /* tokens in the sequence */
  int64_t next_pos; /* position the next appended token gets */
  int32_t n_pages;  /* entries in its page list */
  int32_t parent;   /* handle it was forked from, -1 if none */
  int32_t n_spans;  /* registered cursor spans */
  int32_t n_masked; /* slots masked by deferred evictions (still in length) */
} sq_seq_desc;

typedef struct {
  int64_t tokens_removed;  /* L - L' */
  int64_t tokens_moved;    /* kept tokens gathered into new pages: L' - P*floor(f/P),
                              less P per remapped page */
  int64_t bytes_moved;     /* bytes written by the gather: tokens_moved * (NL*Hkv*D*2*E + 4),
                              E = 2 bytes per element (1 in an 8-bit store);
                              the gather reads as many */
  int64_t pages_allocated; /* fresh pages taken for the compacted tail */
  int64_t pages_freed;     /* old pages whose last reference went away */
  int64_t first_evicted;   /* f, the first evicted index (L if none) */
  int64_t pages_remapped;  /* tail pages taken by reference (SQ_STORE_EVICT_REMAP) */
  int64_t tokens_masked;   /* SQ_EVICT_DEFER: slots this call masked (0 otherwise) */
} sq_evict_stats;

typedef struct {
  int64_t live_pages, peak_pages, free_pages, live_seqs;
  int64_t append_tokens;                     /* tokens appended so far */
  int64_t fork_calls, fork_tail_copies;      /* forks; forks that copied a tail page */
  int64_t evict_calls, evict_tokens_removed, evict_tokens_moved, evict_bytes_moved;
  int64_t decode_calls;
  int64_t decode_kv_bytes;    /* K/V bytes decode must read, shared prefixes once */
  int64_t decode_kv_bytes_logical; /* same with every query's own tokens counted */
  int64_t extend_calls, extend_tokens; /* sq_extend_attn calls; query tokens they served */
  int64_t extend_kv_bytes;    /* K/V bytes of the keys those calls attended, each key once */
} sq_stats;

typedef struct {
  int32_t n_segments;       /* (page range, query rows) work units */
  int32_t n_groups;         /* shared-prefix groups (>= 2 sequences) */
  int32_t n_items_valu;     /* work items of the VALU split kernel */
  int32_t n_items_mfma;     /* work items of the MFMA tile kernel */
  int32_t chunk_pages;      /* pages per work item */
  int32_t n_slots;          /* partial slots (16 query rows each) the launches write */
  int64_t kv_bytes;         /* K/V bytes the call reads, shared pages once */
  int64_t kv_bytes_logical; /* K/V bytes with every sequence's pages counted */
  int64_t kv_bytes_valu;    /* part of kv_bytes read by the VALU kernel */
  int64_t kv_bytes_mfma;    /* part of kv_bytes read by the MFMA kernel */
  int64_t io_bytes;         /* q, out and page-id bytes */
} sq_plan_info;

typedef struct {
  /* Sums of kernel durations (ms) measured with HIP events recorded on the
     store's stream around each launch, over the calls made since profiling
     was enabled or last read.  evict_scan counts the eviction index kernel
     where it runs on its own (in-place evictions, or when no page is
     copied); otherwise the index is written inside the first gather launch
     and counts in evict_gather. */
  double decode_valu_ms, decode_mfma_ms, decode_merge_ms;
  double evict_scan_ms, evict_gather_ms, append_ms;
  int64_t decode_valu_launches, decode_mfma_launches, decode_merge_launches;
  int64_t evict_scan_launches, evict_gather_launches, append_launches;
  double extend_ms;
  int64_t extend_launches;
} sq_profile;

/* ---- store -------------------------------------------------------------
 * The paged KV store shared by the main thread and its auxiliary branches
 * (§3.4, "Storage Costs": the branch does not duplicate the cache). */

/* Bytes of device workspace a store with this configuration needs.
 * Returns 0 for an invalid configuration. */
uint64_t sq_workspace_bytes(const sq_store_config *cfg);

/* Bytes of the K pool (which = 0), V pool (1) or position pool (2).
 * Returns 0 for an invalid configuration or which. */
uint64_t sq_pool_bytes(const sq_store_config *cfg, int32_t which);

/* Create a store over caller-owned pools.  *out receives the handle.
 * SQ_ERR_INVALID: bad shape, capacity, missing buffer or workspace too small. */
sq_status sq_store_create(const sq_store_config *cfg, sq_store **out);

/* Destroy a store (host metadata only; does not touch the caller's buffers).
 * Waits for the store's last enqueued work before freeing its staging buffer. */
sq_status sq_store_destroy(sq_store *store);

/* New empty sequence (the context C <- [Q] of Algorithm 1 starts here).
 * Handles are the lowest free integers.  SQ_ERR_INVALID when max_seqs are live. */
sq_status sq_seq_create(sq_store *store, sq_seq *out);

/* ---- growth (Algorithm 1, Phase 3: C <- C + R, C <- C + O) --------------
 * Append n tokens to seq.  k_new, v_new: device bf16 [NL][n][Hkv][D].
 * Pages are taken lowest free id first, in page-list order; token i gets
 * position next_pos + i.  SQ_ERR_NO_PAGES if the pool is short,
 * SQ_ERR_INVALID if the page list would exceed max_pages_per_seq. */
sq_status sq_append(sq_store *store, sq_seq seq, int32_t n, const void *k_new,
                    const void *v_new, void *stream);

/* Append one token to each of `batch` distinct sequences (a decode step).
 * k_new, v_new: device bf16 [NL][batch][Hkv][D].  Pages are taken in batch
 * order.  SQ_ERR_INVALID for a repeated sequence or batch > SQ_MAX_BATCH. */
sq_status sq_append_batch(sq_store *store, const sq_seq *seqs, int32_t batch,
                          const void *k_new, const void *v_new, void *stream);

/* Register cursor `cursor` (a tool call and its response, §3 footnote on
 * "tool response"; the [Cursor n] indexing of §4.2) as the tokens
 * [start, end) of seq, in its current coordinates.  Empty spans are allowed.
 * SQ_ERR_INVALID: cursor < 0 or already registered on seq.
 * SQ_ERR_SPAN: outside [0, length] or overlapping a non-empty registered span. */
sq_status sq_span_mark(sq_store *store, sq_seq seq, int32_t cursor, int64_t start,
                       int64_t end);

/* ---- auxiliary thread (Algorithm 1, Phase 2: C_aux <- C + p) ------------
 * Fork a branch on the first fork_len tokens of parent.  The child aliases
 * the parent's first fork_len/P pages (refcount + 1, nothing copied, §3.4).
 * If fork_len % P != 0 the child gets one new page with a copy of the first
 * fork_len % P slots of the parent's page fork_len/P.  The child's next
 * position is the parent's if fork_len == parent length, else the position of
 * the parent's token fork_len.  The child inherits the cursor spans that end
 * at or before fork_len.  SQ_ERR_INVALID: fork_len outside [0, length] or no
 * free handle; SQ_ERR_NO_PAGES: no page for the tail copy. */
sq_status sq_fork(sq_store *store, sq_seq parent, int64_t fork_len, sq_seq *child,
                  void *stream);

/* Drop a branch when its thread finishes (§3.4: its transient tokens are
 * discarded; Algorithm 1 Phase 1 sets S_thread <- None).  Every page loses one
 * reference; pages reaching zero return to the pool.  Host-only. */
sq_status sq_release(sq_store *store, sq_seq seq);

/* ---- eviction (Algorithm 1, Phase 1: C.clear_kv(Delta_ids)) --------------
 * Remove from seq the tokens of the n cursors in cursor_ids (host array).
 * Duplicates are ignored.  With L tokens, keep[i] = 0 inside an evicted span,
 * dst = exclusive prefix sum of keep, L' = sum keep and src_of[dst[i]] = i.
 * With f the first evicted index, pages [0, f/P) stay; ceil(L'/P) - f/P fresh
 * pages (lowest ids, taken before any old page is released) receive the kept
 * tokens [P*floor(f/P), L') from the old pages: K, V of every layer and head
 * and their positions, which are carried unchanged.  Then every old page
 * from f/P on loses one reference.  Pages another live branch still holds
 * survive, so other branches keep attending to what they saw.  With
 * evict_chunk_pages > 0 the fresh pages come in chunks (see the config).
 * With SQ_STORE_EVICT_INPLACE the tail is written into the sequence's own
 * old pages instead (fresh pages only for pages another branch holds), one
 * launch per run of tail pages that read no page the run writes except
 * their own (each workgroup stages a page's sources before it writes it),
 * or one pass in page order per (layer, KV head) where such runs are short.
 * With SQ_STORE_EVICT_REMAP a full tail page whose P kept tokens are one old
 * page's P tokens in order takes that old page by reference (no fresh page,
 * nothing copied): this happens behind every evicted run whose evicted
 * tokens so far are a multiple of P, e.g. spans that start and end on
 * pages.  Remaining spans shift left by the evicted tokens before them.
 * Evicting only empty
 * spans (or none) only unregisters the cursors.  Issue it after the main
 * thread's turn (§3.1 step 4).  stats may be NULL.
 * SQ_ERR_UNKNOWN_CURSOR: a cursor is not registered on seq;
 * SQ_ERR_NO_PAGES: the pool cannot hold the compacted tail;
 * SQ_ERR_INVALID: n < 0 or n > SQ_MAX_EVICT_SPANS. */
sq_status sq_evict_spans(sq_store *store, sq_seq seq, const int32_t *cursor_ids,
                         int32_t n, void *stream, sq_evict_stats *stats);

/* ---- deferred eviction (a variant of clear_kv) ---------------------------
 * sq_evict_spans_ex with SQ_EVICT_DEFER masks the spans' slots instead of
 * removing them: from the call on, decode, step and extend attention skip
 * those slots (the §3.3 masking of evicted tokens, exactly: attention over
 * the kept slots equals attention after a physical eviction), while pages,
 * slot indices, length, positions and the other spans stay as they are, so
 * the call moves nothing and needs no page.  Its cursors are unregistered.
 * A fork inherits the masks of its slots.  The masked slots leave the store
 * at the sequence's next physical eviction, which removes them together
 * with its own spans, or at sq_compact, which removes only them; remaining
 * spans then shift left by the slots removed before each end.  Windowed
 * attention (sq_attn_opts.window > 0) on a sequence with masked slots is
 * rejected (a window counts kept tokens).  A sequence may hold at most
 * SQ_MAX_EVICT_SPANS maximal runs of masked slots: a deferred call that
 * would exceed it fails with SQ_ERR_INVALID and changes nothing, as does
 * one on a metadata-only store with page_size > 16 (masks are 16-bit words
 * per page).
 * flags: 0 (= sq_evict_spans) or SQ_EVICT_DEFER; the other arguments,
 * stats and errors as for sq_evict_spans. */
#define SQ_EVICT_DEFER 1u
sq_status sq_evict_spans_ex(sq_store *store, sq_seq seq, const int32_t *cursor_ids, int32_t n,
                            uint32_t flags, void *stream, sq_evict_stats *stats);

/* Physical eviction of the slots deferred evictions masked on seq (no
 * cursor); nothing to do when there are none.  Enqueued on stream like
 * sq_evict_spans, with the same stats (tokens_removed = the masked slots)
 * and errors (SQ_ERR_NO_PAGES). */
sq_status sq_compact(sq_store *store, sq_seq seq, void *stream, sq_evict_stats *stats);

/* Host copy of seq's per-slot keep flags (1 attended, 0 masked): up to cap
 * bytes into out; *n = its length. */
sq_status sq_keep_flags(sq_store *store, sq_seq seq, uint8_t *out, int64_t cap, int64_t *n);

/* ---- decode attention (the memory-bound decode step of §1 / §3.4) --------
 * One decode step of layer `layer` for `batch` sequences (main threads and
 * auxiliary branches together, §3.1 "Parallel Execution"):
 *   out[b][h] = sum_i softmax_i(scale * q[b][h] . K[i][h/G]) * V[i][h/G]
 * over all length(seqs[b]) cached tokens of seqs[b] (the caller appends the
 * current token first).  q: device bf16 [batch][Hq][D]; out: device fp32
 * [batch][Hq][D].  An empty sequence gives zeros.  mode: SQ_ATTN_*.  Pages
 * that several queries share as a common prefix are read once per group in
 * AUTO and SHARED_PREFIX modes (§3.4 cites shared-prefix kernels for this).
 * SQ_ERR_INVALID: batch outside [1, SQ_MAX_BATCH], bad layer or mode,
 * metadata-only store. */
sq_status sq_decode_attn(sq_store *store, int32_t layer, const sq_seq *seqs, int32_t batch,
                         const void *q, float *out, float scale, int32_t mode, void *stream);

/* ---- decode attention without the workspace's partial buffers ----------
 * For callers that cannot allocate device memory around a call (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * sq_decode_attn with the same arguments, kernels and result (bit for bit),
 * whose split partials (m, l, acc of every workgroup's piece) live in a
 * device array the library holds on each GPU it runs on, instead of the
 * store's workspace.  The array holds SQ_NOALLOC_PARTIAL_SLOTS slots of 16
 * query rows (34 MB) and stays allocated until the process ends; nothing in
 * it needs clearing (every slot a call reads, the same call writes first).
 * Every call on one GPU, from any store, uses the same array: calls that
 * may overlap on one GPU (other streams, other host threads) race, so order
 * them on one stream.  The call allocates nothing and records no profiling
 * events.  SQ_ERR_INVALID as sq_decode_attn, and for a call whose work
 * split needs more than SQ_NOALLOC_PARTIAL_SLOTS slots (with up to 8 KV
 * heads every mode fits); SQ_ERR_HIP if the array's address could not be
 * found when the store was created. */
#define SQ_NOALLOC_PARTIAL_SLOTS 4096
sq_status sq_decode_attn_noalloc(sq_store *store, int32_t layer, const sq_seq *seqs,
                                 int32_t batch, const void *q, float *out, float scale,
                                 int32_t mode, void *stream);

/* ---- decode step with the append fused (graph-capturable) ----------------
 * The decode loop of §3.1 appends one token to every running thread and
 * attends over the result.  sq_step_begin does the host part of that for
 * `batch` distinct sequences once per step: it appends one token slot to
 * each (length + 1, a new page when the last one is full, positions
 * continue) and writes the step's attention plan to device memory on
 * stream.  sq_step_attn then runs one layer: it stores the new token's K
 * and V in that layer and attends with q over every token of each
 * sequence, the new one included - the same result as sq_append_batch
 * followed by sq_decode_attn.  The new token joins in the merge kernel as
 * one more partial of the split softmax (score q . k_new, weight 1, value
 * v_new), so a layer costs two launches (one when the plan needs both the
 * VALU and MFMA kernels: three) and no separate append.
 *
 * The launches of sq_step_attn and their arguments depend on (layer,
 * pointers, scale, the step's batch size and mode) only: a stream capture
 * (hipStreamBeginCapture) of one step's sq_step_attn calls replays correctly
 * for every later step of the same batch size and mode, each after its own
 * sq_step_begin on the same stream, with the caller's q / k_new / v_new /
 * out buffers at the same addresses.  Replays do not update sq_stats.
 *
 * Between sq_step_begin and the last layer's sq_step_attn the new tokens'
 * slots hold stale K/V (a page the step opens is in the page table from
 * sq_step_begin on): every other call that changes a sequence (append,
 * fork, release, evict, a new step) ends the step, and sq_step_attn then
 * fails.  A replay sized for a larger batch than the open step's leaves the
 * extra entries untouched; one sized for a smaller batch misses entries.  mode: SQ_ATTN_*.  sq_step_begin errors change nothing;
 * SQ_ERR_INVALID for a repeated sequence, batch outside [1, SQ_MAX_BATCH],
 * a sequence at its page-list capacity; SQ_ERR_NO_PAGES; in a
 * metadata-only store it updates the metadata only. */
sq_status sq_step_begin(sq_store *store, const sq_seq *seqs, int32_t batch, int32_t mode,
                        void *stream);

/* One layer of the open step.  k_new, v_new: device bf16 [batch][Hkv][D];
 * q: device bf16 [batch][Hq][D]; out: device fp32 [batch][Hq][D]; all
 * 16-byte aligned, caller-owned; entry b is seqs[b] of sq_step_begin.
 *   out[b][h] = sum_i softmax_i(scale * q[b][h] . K[i][h/G]) * V[i][h/G]
 * over the L_b + 1 tokens of the sequence after the append.
 * SQ_ERR_INVALID: no open step, bad layer, null or misaligned buffers,
 * scale not finite, metadata-only store. */
sq_status sq_step_attn(sq_store *store, int32_t layer, const void *k_new, const void *v_new,
                       const void *q, float *out, float scale, void *stream);

/* Causal attention of a chunk that was just appended: Algorithm 1 grows the
 * context by whole chunks (Phase 3: C <- C + R, then C <- C + O), and every
 * token of such a chunk attends to the cached prefix (compacted by Phase 1's
 * evictions) and to the chunk's earlier tokens before decoding resumes.
 *
 * The chunk is the last n_new of seq's L tokens (append it with sq_append
 * first).  For new token j (0 <= j < n_new) and query head h:
 *   out[j][h] = sum_t softmax_t(scale * q[j][h] . k[t][h / G]) v[t][h / G]
 * over the keys at logical indices t = 0 .. L - n_new + j, G = Hq / Hkv.
 * Causality is by logical index: positions carried through evictions are
 * increasing in that order, so the two agree.
 *   q    device bf16 [n_new][Hq][D], 16-byte aligned (caller-owned)
 *   out  device fp32 [n_new][Hq][D], 16-byte aligned (caller-owned)
 * Work is enqueued on stream.  n_new = 0 does nothing.
 * SQ_ERR_UNKNOWN_SEQ: seq is not live.  SQ_ERR_INVALID: n_new outside
 * [0, L], bad layer, null or misaligned q / out, scale not finite and
 * positive, metadata-only store. */
sq_status sq_extend_attn(sq_store *store, int32_t layer, sq_seq seq, int32_t n_new,
                         const void *q, float *out, float scale, void *stream);

/* ---- attention options (model variants) ---------------------------------
 * Some models change the softmax of the attention above in two ways; the
 * paper's method (eviction, fork, shared prefixes) applies unchanged.
 *   sinks   device fp32 [Hq] (caller-owned, finite), or NULL: a learned
 *           logit per query head, in the units of the scaled scores, that
 *           joins each softmax as one more term with no value:
 *             out = sum_i e^(s_i - M) v_i / (e^(sink - M) + sum_i e^(s_i - M)),
 *           M = max(sink, max_i s_i).  A query with no keys still gets 0.
 *   window  0: every key; W > 0: a query at logical index t attends only
 *           to the keys at indices t - W + 1 .. t (the W most recent ones,
 *           its own included).  A decode query of a sequence of L tokens
 *           is at index L - 1; extend token j at L - n_new + j.
 *   reserved  must be 0.
 * The window is over logical indices of the (compacted) cache, as the
 * causal mask is.  SQ_ERR_INVALID: window < 0, reserved != 0, or a sinks
 * pointer that is not 4-byte aligned. */
typedef struct sq_attn_opts {
  const float *sinks;
  int32_t window;
  int32_t reserved;
} sq_attn_opts;

/* sq_decode_attn with options; opts NULL = sq_decode_attn.  A windowed
 * batch reads each entry's window on its own (no shared-prefix tiles). */
sq_status sq_decode_attn_ex(sq_store *store, int32_t layer, const sq_seq *seqs, int32_t batch,
                            const void *q, float *out, float scale, int32_t mode,
                            const sq_attn_opts *opts, void *stream);

/* sq_extend_attn with options; opts NULL = sq_extend_attn. */
sq_status sq_extend_attn_ex(sq_store *store, int32_t layer, sq_seq seq, int32_t n_new,
                            const void *q, float *out, float scale, const sq_attn_opts *opts,
                            void *stream);

/* sq_step_begin for a step whose layers may use a window of `window` keys
 * (0: none): besides the full plan it writes a windowed one, and every
 * sq_step_attn_ex of the step may then pick either (models alternate
 * windowed and full layers).  sq_step_begin = window 0.
 * SQ_ERR_INVALID also for window < 0. */
sq_status sq_step_begin_ex(sq_store *store, const sq_seq *seqs, int32_t batch, int32_t mode,
                           int32_t window, void *stream);

/* sq_step_attn with options; opts NULL = sq_step_attn.  opts->window is 0
 * (every key) or the window of sq_step_begin_ex.  A capture replays with
 * the same options, each step begun with the same window.
 * SQ_ERR_INVALID also for any other window. */
sq_status sq_step_attn_ex(sq_store *store, int32_t layer, const void *k_new, const void *v_new,
                          const void *q, float *out, float scale, const sq_attn_opts *opts,
                          void *stream);

/* Host-only description of the work sq_decode_attn would do for this batch. */
sq_status sq_decode_plan_info(sq_store *store, const sq_seq *seqs, int32_t batch,
                              int32_t mode, sq_plan_info *out);

/* ---- introspection -------------------------------------------------------*/
sq_status sq_seq_info(sq_store *store, sq_seq seq, sq_seq_desc *out);

/* Host copy of seq's page list: up to cap ids into out; *n = its length. */
sq_status sq_page_table(sq_store *store, sq_seq seq, int32_t *out, int32_t cap, int32_t *n);

/* Host copy of the positions of seq's tokens (the library's host record):
 * up to cap values into out; *n = length. */
sq_status sq_positions(sq_store *store, sq_seq seq, int64_t *out, int64_t cap, int64_t *n);

/* Registered spans of seq, ordered by cursor id: up to cap entries. */
sq_status sq_seq_spans(sq_store *store, sq_seq seq, int32_t *cursors, int64_t *starts,
                       int64_t *ends, int32_t cap, int32_t *n);

/* Refcount of every page: up to cap values into out (host array). */
sq_status sq_refcounts(sq_store *store, int32_t *out, int32_t cap);

sq_status sq_stats_get(sq_store *store, sq_stats *out);

/* Device keep / dst / src_of arrays of the last eviction that removed tokens,
 * copied to host buffers of cap entries (synchronises the store's stream).
 * *n_tokens = L before that eviction, *n_kept = L'.  SQ_ERR_INVALID if no
 * such eviction happened or cap < L. */
sq_status sq_debug_last_evict(sq_store *store, uint8_t *keep, int32_t *dst, int32_t *src_of,
                              int64_t cap, int64_t *n_tokens, int64_t *n_kept);

/* Kernel timing with HIP events on the store's stream (off by default). */
sq_status sq_profile_enable(sq_store *store, int32_t on);
/* Synchronises the recorded events, returns the sums and resets them. */
sq_status sq_profile_read(sq_store *store, sq_profile *out);

/* Message for the last failed call on this thread ("" if none). */
const char *sq_last_error(void);

/* SQ_ABI_VERSION of the loaded library. */
int32_t sq_abi_version(void);

/* Host call trace (off by default).  While open, every state-changing or
 * compute call (store create/destroy, sequence create, appends, span marks,
 * forks, releases, evictions, compaction, decode, decode steps, extend)
 * writes one line: "sq <call>(<arguments>) host_us=<time> ok" or
 * "... error: <message>", the time being the call's host time (device work
 * is only enqueued).  path "-" traces to stderr, another path appends to
 * that file, NULL closes the trace.  The environment variable SQ_TRACE,
 * read once when the library loads, opens one the same way ("1" or "-":
 * stderr; "0" or empty: none; otherwise a file path).  Lines are written
 * whole by concurrent threads.  SQ_ERR_INVALID if the file cannot be
 * opened (the previous trace stays open). */
sq_status sq_trace_open(const char *path);

#ifdef __cplusplus
}
#endif

#endif /* SQ_H */
