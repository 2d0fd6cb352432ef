"""A page-level model of the shared KV store, in plain Python.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What the paper fixes
--------------------
* The auxiliary thread runs on the *shared* context: it does not duplicate the
  KV cache of the conversation; its only extra storage is its own transient
  tokens, discarded when it finishes (§3.4 "Storage Costs"; Algorithm 1,
  Phase 2 ``C_aux <- C + p``).
* ``clear_kv(Delta_ids)`` removes the tokens of the named tool responses from
  the cache after the main thread's turn has finished (Algorithm 1, Phase 1;
  §3.1 step 4 "Synchronization").
* The context grows by appends: the main thread's response R and the tool
  output O (Algorithm 1, Phase 3).

Readings adopted where the paper is silent (also listed in the design notes)
-------------------------------------------------------------------------
* Storage is paged: P tokens per page; a sequence (main thread or auxiliary
  branch) is a list of page ids, a length and a position counter.
* Page allocation takes the lowest free page id first; an operation that needs
  several pages takes them one at a time, in the order they appear in the
  sequence's page list.
* Fork at F: the child aliases the parent's first F // P pages (refcount + 1,
  no copy).  If F % P != 0 the child gets one new page holding a copy of slots
  [0, F % P) of the parent's page F // P.  The child's position counter is the
  parent's if F equals the parent's length, otherwise the position of the
  parent's token F.  The child inherits the cursor spans that end at or before F.
* Eviction is out of place: with f the first evicted index and fp = f // P,
  pages [0, fp) are kept as they are; ceil(L'/P) - fp new pages are allocated
  (before any old page is released) and filled with the kept tokens
  [fp*P, L') gathered from the old pages; then every old page from fp on
  loses one reference and is freed at zero.  Pages still referenced by another
  live branch survive, so evicting one branch never changes what another
  branch attends to.
* Chunked eviction (a store option: chunk C > 0 pages) bounds the transient
  pages: the new tail's pages are allocated C at a time, in page-list order;
  once the kept tokens of a chunk's pages are gathered, every old page from
  fp on whose tokens all lie before the old index of the next kept token to
  move loses its reference (and is freed at zero, so the next chunk may take
  it again); the old pages left lose theirs at the end.  Live pages never
  exceed the count before the call plus C.  C = 0 is the one-shot rule
  above.
* Positions are carried, never recomputed: a kept token keeps its position and
  new tokens continue from the counter.
* Deferred eviction (NEXT-2 variant; the paper evicts at once, and masks
  tokens only to simulate eviction, §3.3 and Algorithm 2): ``evict(...,
  deferred=True)`` clears the keep flags of the spans' slots and drops their
  cursors; pages, slots, length and the other spans stay as they are, and
  attention sees the kept slots only (``view``).  A fork inherits the flags
  of its slots.  The masked slots leave the store at the next physical
  eviction of the sequence, which removes them together with its own spans
  (the union, as maximal runs), or at ``compact``, which removes only them;
  every remaining span then shifts left by the slots removed before its
  ends.
* Validation happens before any change: a failing call leaves the model as it
  was.  Error kinds: Invalid, NoPages, UnknownSeq, UnknownCursor, SpanError.
* Sequence handles are small integers, lowest free handle first.
"""

from __future__ import annotations

import heapq
import math

import numpy as np

from . import evict as _evict
from . import fp8 as _fp8


class OracleError(Exception):
    code = 0


class Invalid(OracleError):
    code = 1


class NoPages(OracleError):
    code = 2


class UnknownSeq(OracleError):
    code = 3


class UnknownCursor(OracleError):
    code = 4


class SpanError(OracleError):
    code = 5


class Seq:
    __slots__ = ("pages", "length", "next_pos", "pos", "spans", "parent", "keep")

    def __init__(self):
        self.pages = []
        self.length = 0
        self.next_pos = 0
        self.pos = []  # logical position of each token
        self.spans = {}  # cursor id -> (start, end), current coordinates
        self.parent = -1
        self.keep = []  # per slot: False once a deferred eviction masked it


class PageModel:
    """Page allocator, refcounts and sequences; optionally the K/V/pos data.

    With ``with_data`` the physical pools are held as float64 arrays
    K, V: [num_pages, P, NL, Hkv, D] and pos: [num_pages, P].
    """

    def __init__(self, num_pages, page_size, max_seqs, max_pages_per_seq,
                 layers=1, kv_heads=1, head_dim=1, with_data=False, evict_chunk_pages=0,
                 evict_remap=False, kv_scales=None, evict_inplace=False):
        self.num_pages = int(num_pages)
        self.evict_chunk_pages = int(evict_chunk_pages)
        self.evict_remap = bool(evict_remap)
        self.evict_inplace = bool(evict_inplace)
        if self.evict_inplace and (self.evict_remap or self.evict_chunk_pages):
            raise Invalid("in-place eviction takes neither chunks nor remaps")
        self.P = int(page_size)
        self.max_seqs = int(max_seqs)
        self.max_pages_per_seq = int(max_pages_per_seq)
        self.layers, self.kv_heads, self.head_dim = layers, kv_heads, head_dim
        self.refcount = np.zeros(self.num_pages, dtype=np.int64)
        self._free = list(range(self.num_pages))
        heapq.heapify(self._free)
        self.seqs = {}
        self.peak_pages = 0
        self.last_schedule = []  # the last eviction's (allocated, released) pages per step
        self.with_data = with_data
        # 8-bit cache: [NL][2] scales (K, V); appended K/V are stored as
        # their E4M3 round trip (see the fp8 module)
        self.kv_scales = None if kv_scales is None else np.asarray(kv_scales, dtype=np.float32)
        if with_data:
            shape = (self.num_pages, self.P, layers, kv_heads, head_dim)
            self.K = np.zeros(shape)
            self.V = np.zeros(shape)
            self.POS = np.zeros((self.num_pages, self.P), dtype=np.int64)

    # -- allocator ---------------------------------------------------------
    def free_pages(self):
        return len(self._free)

    def live_pages(self):
        return self.num_pages - len(self._free)

    def _alloc(self):
        page = heapq.heappop(self._free)
        assert self.refcount[page] == 0
        self.refcount[page] = 1
        self.peak_pages = max(self.peak_pages, self.live_pages())
        return page

    def _unref(self, page):
        self.refcount[page] -= 1
        assert self.refcount[page] >= 0
        if self.refcount[page] == 0:
            heapq.heappush(self._free, page)
            return 1
        return 0

    def _released_after(self, fp, released, n_old, consumed):
        """Old-tail pages [0, result) hold only tokens before old index
        ``consumed`` (the next kept token still to move): they may go."""
        upto = released
        while upto < n_old and (fp + upto + 1) * self.P <= consumed:
            upto += 1
        return upto

    def _remap_source(self, src_of, j0, new_len):
        """Page-aligned remap: the old index of the first of the P tokens that
        land at new indices j0 .. j0 + P - 1 when they are one whole old page
        in order (first at a page start, last P - 1 after it); else None."""
        if j0 + self.P > new_len:
            return None
        a0 = int(src_of[j0])
        if a0 % self.P == 0 and int(src_of[j0 + self.P - 1]) == a0 + self.P - 1:
            return a0
        return None

    def _seq(self, h):
        if h not in self.seqs:
            raise UnknownSeq(f"unknown sequence {h}")
        return self.seqs[h]

    # -- sequences ---------------------------------------------------------
    def seq_create(self):
        for h in range(self.max_seqs):
            if h not in self.seqs:
                self.seqs[h] = Seq()
                return h
        raise Invalid("no free sequence handle")

    def append(self, h, n, k_new=None, v_new=None):
        """Append n tokens.  k_new, v_new: [NL, n, Hkv, D] (with data)."""
        seq = self._seq(h)
        if n < 0:
            raise Invalid("negative token count")
        new_len = seq.length + n
        want = math.ceil(new_len / self.P)
        if want > self.max_pages_per_seq:
            raise Invalid("sequence would exceed its page-list capacity")
        if want - len(seq.pages) > self.free_pages():
            raise NoPages("not enough free pages")
        if seq.length % self.P:
            assert self.refcount[seq.pages[-1]] == 1, "partial tail page must be private"
        if self.with_data and self.kv_scales is not None and n:
            k_new = np.stack([_fp8.roundtrip(np.asarray(k_new)[l], self.kv_scales[l, 0])
                              for l in range(self.layers)])
            v_new = np.stack([_fp8.roundtrip(np.asarray(v_new)[l], self.kv_scales[l, 1])
                              for l in range(self.layers)])
        for i in range(n):
            if seq.length % self.P == 0:
                seq.pages.append(self._alloc())
            page, slot = seq.pages[seq.length // self.P], seq.length % self.P
            if self.with_data:
                self.K[page, slot] = np.asarray(k_new, dtype=np.float64)[:, i]
                self.V[page, slot] = np.asarray(v_new, dtype=np.float64)[:, i]
                self.POS[page, slot] = seq.next_pos
            seq.pos.append(seq.next_pos)
            seq.keep.append(True)
            seq.next_pos += 1
            seq.length += 1

    def span_mark(self, h, cursor, start, end):
        """Register cursor ``cursor`` as the tokens [start, end) of sequence h."""
        seq = self._seq(h)
        if cursor < 0 or cursor in seq.spans:
            raise Invalid("cursor id negative or already registered")
        if not (0 <= start <= end <= seq.length):
            raise SpanError("span outside the sequence")
        if end > start:
            for s, e in seq.spans.values():
                if e > s and s < end and start < e:
                    raise SpanError("span overlaps a registered span")
        seq.spans[cursor] = (int(start), int(end))

    def fork(self, parent, fork_len):
        """Open an auxiliary branch on the first ``fork_len`` tokens."""
        par = self._seq(parent)
        if not (0 <= fork_len <= par.length):
            raise Invalid("fork point outside the parent")
        if len(self.seqs) >= self.max_seqs:
            raise Invalid("no free sequence handle")
        tail = fork_len % self.P
        if tail and self.free_pages() < 1:
            raise NoPages("no page for the fork's tail copy")
        child_h = self.seq_create()
        child = self.seqs[child_h]
        full = fork_len // self.P
        for page in par.pages[:full]:
            self.refcount[page] += 1
        child.pages = list(par.pages[:full])
        if tail:
            page = self._alloc()
            src = par.pages[full]
            if self.with_data:
                self.K[page, :tail] = self.K[src, :tail]
                self.V[page, :tail] = self.V[src, :tail]
                self.POS[page, :tail] = self.POS[src, :tail]
            child.pages.append(page)
        child.length = fork_len
        child.pos = list(par.pos[:fork_len])
        child.keep = list(par.keep[:fork_len])
        child.next_pos = par.next_pos if fork_len == par.length else par.pos[fork_len]
        child.spans = {c: se for c, se in par.spans.items() if se[1] <= fork_len}
        child.parent = parent
        return child_h

    def release(self, h):
        """Drop a branch: every page loses one reference."""
        seq = self._seq(h)
        freed = sum(self._unref(p) for p in seq.pages)
        del self.seqs[h]
        return freed

    @staticmethod
    def _masked_runs(keep, extra=()):
        """Maximal runs [s, e) of slots that are masked or inside one of the
        ``extra`` spans, in order."""
        out = np.logical_not(np.asarray(keep, dtype=bool))
        for s, e in extra:
            out[s:e] = True
        runs, i, n = [], 0, len(out)
        while i < n:
            if out[i]:
                j = i
                while j < n and out[j]:
                    j += 1
                runs.append((i, j))
                i = j
            else:
                i += 1
        return runs

    def compact(self, h):
        """Remove the slots deferred evictions masked (a physical eviction
        of no cursor)."""
        return self.evict(h, [])

    def evict(self, h, cursor_ids, deferred=False):
        """``clear_kv``: remove the tokens of ``cursor_ids`` from sequence h
        (and any slots earlier deferred evictions masked); ``deferred`` only
        masks them."""
        seq = self._seq(h)
        ids = list(dict.fromkeys(int(c) for c in cursor_ids))
        for c in ids:
            if c not in seq.spans:
                raise UnknownCursor(f"cursor {c} not registered")
        own = [seq.spans[c] for c in ids if seq.spans[c][1] > seq.spans[c][0]]
        stats = dict(tokens_removed=0, tokens_moved=0, pages_allocated=0,
                     pages_freed=0, first_evicted=seq.length, pages_remapped=0,
                     tokens_masked=0)
        if deferred:
            for s0, e0 in own:
                stats["tokens_masked"] += sum(seq.keep[s0:e0])
                seq.keep[s0:e0] = [False] * (e0 - s0)
            for c in ids:
                del seq.spans[c]
            masked = [i for i, k in enumerate(seq.keep) if not k]
            stats["first_evicted"] = masked[0] if masked else seq.length
            return stats
        spans = self._masked_runs(seq.keep, own)
        if not spans:
            for c in ids:
                del seq.spans[c]
            return stats

        # 1. What eviction computes, by its plain definition: the kept
        #    tokens in their order (keep, src_of) and their data, which is
        #    the old logical view under the keep mask.
        keep, _dst, src_of, new_len, first = _evict.plan(seq.length, spans)
        if self.with_data:
            old_k, old_v, old_pos = self.slot_view(h)
            new_k = _evict.compact(old_k, keep)
            new_v = _evict.compact(old_v, keep)
            new_pos = _evict.compact(old_pos, keep)

        # 2. Where the result lives.  Pages before fp = floor(f / P) hold
        #    only tokens before f and stay.  The tail (new indices from
        #    fp * P on) fills n_new pages; tail page k is an old page taken
        #    by reference (remap, in-place) or a fresh page.
        fp = first // self.P
        n_new = math.ceil(new_len / self.P) - fp
        old_tail = seq.pages[fp:]
        alias, kind = self._place_tail(seq, fp, n_new, src_of, new_len)
        steps = self._alloc_release_steps(seq, fp, n_new, old_tail, src_of, new_len)
        self._check_pages_suffice(alias, steps)

        # 3. Apply: references to the pages taken, fresh pages and releases
        #    in schedule order, then the tail tokens written to their pages.
        new_pages, freed = [], 0
        for a in alias:
            if a is not None:
                self.refcount[a] += 1
        self.last_schedule = []  # (pages allocated, pages released) per step
        for k0, c, rel in steps:
            got = []
            for k in range(k0, k0 + c):
                new_pages.append(alias[k] if alias[k] is not None else self._alloc())
                if alias[k] is None:
                    got.append(new_pages[-1])
            freed += sum(self._unref(page) for page in rel)
            self.last_schedule.append((got, list(rel)))
        if self.with_data and new_len > fp * self.P:
            j = np.arange(fp * self.P, new_len)
            dp = [new_pages[x // self.P - fp] for x in j]
            ds = list(j % self.P)
            self.K[dp, ds] = new_k[fp * self.P:]
            self.V[dp, ds] = new_v[fp * self.P:]
            self.POS[dp, ds] = new_pos[fp * self.P:]
        seq.pages = seq.pages[:fp] + new_pages
        seq.pos = [p for p, k in zip(seq.pos, keep) if k]
        seq.keep = [True] * new_len
        old_len = seq.length
        seq.length = new_len
        for c in ids:
            del seq.spans[c]
        seq.spans = {c: _evict.shift_span(s, e, spans) for c, (s, e) in seq.spans.items()}
        n_remap = kind.count("remap")
        stats.update(tokens_removed=old_len - new_len,
                     tokens_moved=new_len - fp * self.P - n_remap * self.P,
                     pages_allocated=kind.count("fresh"), pages_freed=freed, first_evicted=first,
                     pages_remapped=n_remap)
        return stats

    def _place_tail(self, seq, fp, n_new, src_of, new_len):
        """The page each tail page k < n_new is, when it is an old page taken
        by reference (else None: a fresh page), and the kind of each.

        * remap: a full tail page whose P tokens are one old page's P tokens
          in order is that old page, unchanged;
        * in-place: tail page k is the old page at the same list index,
          fp + k, rewritten, when this sequence alone holds it;
        * otherwise (and for a page another branch holds) a fresh page."""
        alias, kind = [None] * n_new, ["fresh"] * n_new
        for k in range(n_new):
            if self.evict_remap:
                a0 = self._remap_source(src_of, (fp + k) * self.P, new_len)
                if a0 is not None:
                    alias[k], kind[k] = seq.pages[a0 // self.P], "remap"
            elif self.evict_inplace and self.refcount[seq.pages[fp + k]] == 1:
                alias[k], kind[k] = seq.pages[fp + k], "inplace"
        return alias, kind

    def _alloc_release_steps(self, seq, fp, n_new, old_tail, src_of, new_len):
        """[(first tail page, pages, old pages released after them)]: one
        step taking every tail page, then the release of the old tail; with
        chunks of C pages, after each chunk the old pages whose tokens all
        lie before the next kept token still to move."""
        C = self.evict_chunk_pages if self.evict_chunk_pages > 0 else max(1, n_new)
        steps, released = [], 0
        for k0 in range(0, n_new, C):
            c = min(C, n_new - k0)
            j_end = min((fp + k0 + c) * self.P, new_len)
            consumed = int(src_of[j_end]) if j_end < new_len else seq.length
            upto = self._released_after(fp, released, len(old_tail), consumed) if C < n_new else released
            steps.append((k0, c, old_tail[released:upto]))
            released = upto
        steps.append((n_new, 0, old_tail[released:]))
        return steps

    def _check_pages_suffice(self, alias, steps):
        """Every step must find its fresh pages free, counting the pages
        released before it (nothing changes when one does not)."""
        free, refs = self.free_pages(), {}
        for a in alias:
            if a is not None:
                refs[a] = refs.get(a, self.refcount[a]) + 1
        for k0, c, rel in steps:
            fresh = sum(alias[k] is None for k in range(k0, k0 + c))
            if fresh > free:
                raise NoPages("not enough free pages for the compacted tail")
            free -= fresh
            for page in rel:
                refs[page] = refs.get(page, self.refcount[page]) - 1
                free += refs[page] == 0

    # -- inspection --------------------------------------------------------
    def page_table(self, h):
        return list(self._seq(h).pages)

    def info(self, h):
        seq = self._seq(h)
        return dict(length=seq.length, next_pos=seq.next_pos, n_pages=len(seq.pages),
                    parent=seq.parent, n_spans=len(seq.spans),
                    n_masked=len(seq.keep) - sum(seq.keep))

    def keep_flags(self, h):
        """Per slot: 1 = attended, 0 = masked by a deferred eviction."""
        return np.asarray(self._seq(h).keep, dtype=np.uint8)

    def spans(self, h):
        return dict(self._seq(h).spans)

    def view(self, h):
        """What attention sees of sequence h, its kept slots in order:
        (K [L, NL, Hkv, D], V, pos [L]).  Without data only pos is returned
        (K and V are None)."""
        k, v, pos = self.slot_view(h)
        keep = self.keep_flags(h).astype(bool)
        if keep.all():
            return k, v, pos
        return (None if k is None else k[keep]), (None if v is None else v[keep]), pos[keep]

    def slot_view(self, h):
        """Every slot of sequence h, masked ones included, as the pools hold
        them: (K [L, NL, Hkv, D], V, pos [L])."""
        seq = self._seq(h)
        if not self.with_data:
            return None, None, np.asarray(seq.pos, dtype=np.int64)
        idx_p = [seq.pages[i // self.P] for i in range(seq.length)]
        idx_s = [i % self.P for i in range(seq.length)]
        k = self.K[idx_p, idx_s] if seq.length else np.zeros((0,) + self.K.shape[2:])
        v = self.V[idx_p, idx_s] if seq.length else np.zeros((0,) + self.V.shape[2:])
        pos = self.POS[idx_p, idx_s] if seq.length else np.zeros(0, dtype=np.int64)
        return k, v, pos

    def stats(self):
        return dict(live_pages=self.live_pages(), peak_pages=self.peak_pages,
                    free_pages=self.free_pages(), live_seqs=len(self.seqs))
