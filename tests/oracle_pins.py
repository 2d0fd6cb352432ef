"""Checks that pin the oracle to facts other than itself.

Each ``check_*`` raises AssertionError when the oracle (as currently bound in
the ``oracle`` package) breaks a fact fixed by the mathematics or by the
paper's statement of the method:

* closed forms (uniform weights, two keys, a single key),
* invariants (weights sum to one, key-permutation invariance),
* an independent library routine (``torch.softmax`` in float64),
* brute force over tiny inputs (every subset of spans; a naive list model of
  the context for append / fork / evict / release),
* hand-worked page tables under the stated allocation convention.

``test_oracle_pins.py`` runs them on the oracle as written;
``test_oracle_mutants.py`` plants plausible mistakes in the oracle and shows
each is caught by at least one check.
"""

from __future__ import annotations

import copy
import itertools
import math

import numpy as np
import torch

from oracle import attention as att
from oracle import evict as ev
from oracle import extend as ex
from oracle import pages as pg


def _rand_qkv(rng, hq, hkv, d, n):
    q = rng.standard_normal((hq, d))
    k = rng.standard_normal((n, hkv, d))
    v = rng.standard_normal((n, hkv, d))
    return q, k, v


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------
def check_weights_sum_to_one(seed=1):
    rng = np.random.default_rng(seed)
    for hq, hkv, d, n in [(4, 1, 16, 37), (8, 2, 8, 5), (2, 2, 32, 300)]:
        q, k, v = _rand_qkv(rng, hq, hkv, d, n)
        p = att.weights(q, k, 1 / math.sqrt(d), hq // hkv)
        assert np.all(p >= 0)
        assert np.max(np.abs(p.sum(axis=1) - 1.0)) <= 1e-12
        ones = np.ones_like(v)
        out = att.attention(q, k, ones, 1 / math.sqrt(d), hq // hkv)
        assert np.max(np.abs(out - 1.0)) <= 1e-14


def check_single_key_returns_v(seed=2):
    rng = np.random.default_rng(seed)
    for hq, hkv, d in [(4, 1, 64), (8, 2, 8), (1, 1, 3)]:
        q, k, v = _rand_qkv(rng, hq, hkv, d, 1)
        out = att.attention(q, k, v, 0.37, hq // hkv)
        for h in range(hq):
            assert np.array_equal(out[h], v[0, h // (hq // hkv)])


def check_textbook_softmax(seed=3):
    """Equal to torch.softmax(scale q K^T) V in float64, K/V expanded per
    query head with repeat_interleave (consecutive heads share a KV head)."""
    rng = np.random.default_rng(seed)
    for hq, hkv, d, n, scale in [(4, 1, 64, 50, 1 / 8), (8, 2, 8, 17, 0.5),
                                 (6, 3, 16, 64, 1.7), (2, 2, 4, 1, 1.0),
                                 (32, 8, 128, 40, 1 / math.sqrt(128))]:
        q, k, v = _rand_qkv(rng, hq, hkv, d, n)
        g = hq // hkv
        out = att.attention(q, k, v, scale, g)
        kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(g, dim=0)
        vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(g, dim=0)
        qt = torch.from_numpy(q)[:, None, :]
        logits = scale * torch.bmm(qt, kt.transpose(1, 2).contiguous())
        ref = torch.bmm(torch.softmax(logits, dim=-1), vt)[:, 0, :].numpy()
        assert np.max(np.abs(out - ref)) <= 1e-12, np.max(np.abs(out - ref))


def check_uniform_closed_form(seed=4):
    """q = 0 gives equal scores, so the output is the mean of the values."""
    rng = np.random.default_rng(seed)
    q, k, v = _rand_qkv(rng, 4, 2, 8, 9)
    out = att.attention(np.zeros_like(q), k, v, 0.3, 2)
    for h in range(4):
        assert np.max(np.abs(out[h] - v[:, h // 2].mean(axis=0))) <= 1e-14


def check_two_key_closed_form():
    """Two keys with scores a, b: weight of the first is 1 / (1 + e^(b - a))."""
    d = 2
    q = np.array([[1.0, 0.0]])
    k = np.array([[[2.0, 5.0]], [[-1.0, 3.0]]])
    v = np.array([[[1.0, 0.0]], [[0.0, 1.0]]])
    scale = 0.5
    a, b = scale * 2.0, scale * -1.0
    w1 = 1.0 / (1.0 + math.exp(b - a))
    out = att.attention(q, k, v, scale, 1)
    assert abs(out[0, 0] - w1) <= 1e-15 and abs(out[0, 1] - (1 - w1)) <= 1e-15
    assert d == out.shape[1]


def check_permutation_invariance(seed=5):
    rng = np.random.default_rng(seed)
    q, k, v = _rand_qkv(rng, 8, 2, 16, 33)
    perm = rng.permutation(33)
    a = att.attention(q, k, v, 0.25, 4)
    b = att.attention(q, k[perm], v[perm], 0.25, 4)
    assert np.max(np.abs(a - b)) <= 1e-13


def check_masked_semantics(seed=6):
    """Masking keys equals dropping them (general inputs, to round-off), and a
    fully masked head returns zeros."""
    rng = np.random.default_rng(seed)
    q, k, v = _rand_qkv(rng, 4, 1, 8, 20)
    mask = rng.integers(0, 2, 20).astype(np.uint8)
    mask[3] = 1
    a = att.masked_attention(q, k, v, mask, 0.4, 4)
    keep = mask.astype(bool)
    b = att.attention(q, k[keep], v[keep], 0.4, 4)
    assert np.max(np.abs(a - b)) <= 1e-14
    z = att.masked_attention(q, k, v, np.zeros(20, np.uint8), 0.4, 4)
    assert np.array_equal(z, np.zeros_like(z))


def check_merge_identity(seed=7):
    """Partials of any partition of the keys merge to direct attention; empty
    parts are ignored."""
    rng = np.random.default_rng(seed)
    for trial in range(12):
        hq, hkv, d, n = [(4, 1, 8, 40), (8, 2, 16, 23), (2, 1, 4, 3)][trial % 3]
        q, k, v = _rand_qkv(rng, hq, hkv, d, n)
        g = hq // hkv
        direct = att.attention(q, k, v, 0.6, g)
        labels = rng.integers(0, 5, n)
        parts = []
        for s in range(6):  # part 5 is always empty
            sel = labels == s
            parts.append(att.partial(q, k[sel], v[sel], 0.6, g))
        merged = att.merge(parts)
        assert np.max(np.abs(merged - direct)) <= 1e-13
    empty = att.partial(q, k[:0], v[:0], 0.6, g)
    assert np.all(empty[0] == -np.inf) and np.all(empty[1] == 0)
    assert np.array_equal(att.merge([empty, empty]), np.zeros((hq, d)))


# --------------------------------------------------------------------------
# eviction index arithmetic
# --------------------------------------------------------------------------
def check_scan_and_inverse(seed=8):
    rng = np.random.default_rng(seed)
    for n in [0, 1, 2, 17, 100]:
        for _ in range(5):
            spans = []
            cut = sorted(rng.integers(0, n + 1, 6).tolist())
            for i in range(0, 6, 2):
                spans.append((cut[i], cut[i + 1]))
            keep = ev.keep_mask(n, spans)
            inside = [any(s <= i < e for s, e in spans) for i in range(n)]
            assert keep.tolist() == [0 if x else 1 for x in inside]
            dst = ev.exclusive_scan(keep)
            want = [0] + list(itertools.accumulate(keep.tolist()))[:-1] if n else []
            assert dst.tolist() == want
            src_of = ev.inverse_map(keep, dst)
            assert src_of.tolist() == np.flatnonzero(keep).tolist()
            _, _, _, n_kept, first = ev.plan(n, spans)
            assert n_kept == int(keep.sum()) == len(src_of)
            assert first == (inside.index(True) if any(inside) else n)


def check_span_shift(seed=9):
    rng = np.random.default_rng(seed)
    for _ in range(50):
        n = 40
        cuts = sorted(rng.choice(np.arange(n + 1), 8, replace=False).tolist())
        spans = [(cuts[i], cuts[i + 1]) for i in range(0, 8, 2)]
        gone = [spans[i] for i in range(4) if rng.random() < 0.5]
        stay = [s for s in spans if s not in gone]
        tokens = [i for i in range(n) if not any(s <= i < e for s, e in gone)]
        for s, e in stay:
            ns, ne = ev.shift_span(s, e, gone)
            assert tokens[ns:ne] == list(range(s, e))


# --------------------------------------------------------------------------
# page model
# --------------------------------------------------------------------------
class ListModel:
    """Naive context model: each sequence is a Python list of token records
    (K row, V row, position, attended); fork copies a prefix, evict filters,
    a deferred eviction clears the attended flags in place."""

    def __init__(self):
        self.seqs = {}
        self.next_pos = {}
        self.spans = {}

    def create(self, h):
        self.seqs[h], self.next_pos[h], self.spans[h] = [], 0, {}

    def append(self, h, k_new, v_new):
        for i in range(k_new.shape[1]):
            self.seqs[h].append((k_new[:, i].copy(), v_new[:, i].copy(), self.next_pos[h], True))
            self.next_pos[h] += 1

    def fork(self, parent, f, child):
        self.seqs[child] = list(self.seqs[parent][:f])
        par = self.seqs[parent]
        self.next_pos[child] = self.next_pos[parent] if f == len(par) else par[f][2]
        self.spans[child] = {c: se for c, se in self.spans[parent].items() if se[1] <= f}

    def defer(self, h, cursors):
        old = self.seqs[h]
        for c in cursors:
            s, e = self.spans[h][c]
            for i in range(s, e):
                old[i] = old[i][:3] + (False,)
        self.spans[h] = {c: se for c, se in self.spans[h].items() if c not in cursors}

    def evict(self, h, cursors):
        old = self.seqs[h]
        gone = {i for i, t in enumerate(old) if not t[3]}
        for c in cursors:
            s, e = self.spans[h][c]
            gone.update(range(s, e))
        # a span's new coordinates: count the surviving tokens before each end
        survivors_before = np.cumsum([0] + [0 if i in gone else 1 for i in range(len(old))])
        self.spans[h] = {c: (int(survivors_before[s]), int(survivors_before[e]))
                         for c, (s, e) in self.spans[h].items() if c not in cursors}
        self.seqs[h] = [t for i, t in enumerate(old) if i not in gone]

    def view(self, h):
        toks = [t for t in self.seqs[h] if t[3]]
        if not toks:
            return None
        return (np.stack([t[0] for t in toks]), np.stack([t[1] for t in toks]),
                np.array([t[2] for t in toks]))


def _state(model):
    return copy.deepcopy((model.refcount.tolist(), sorted(model._free),
                          {h: (s.pages, s.length, s.next_pos, s.pos, s.spans, s.parent)
                           for h, s in model.seqs.items()}, model.peak_pages))


def check_against_list_model(seed=10, n_ops=60, chunks=(0,), remap=False, deferred=False,
                             inplace=False):
    """Random op sequences: the page model's logical views equal a naive list
    model's, for page sizes 1, 2, 4 and 16 (and each eviction chunk size).
    With ``remap`` half the marked spans are whole multiples of the page size,
    so that page-aligned remaps happen; returns the pages remapped.  With
    ``deferred`` evictions are also deferred and compactions happen.  With
    ``inplace`` evictions rewrite the sequence's own pages; returns the
    evictions that moved tokens without taking a page."""
    rng = np.random.default_rng(seed)
    nl, hkv, d = 2, 2, 3
    remapped = 0
    in_place = 0
    for page, chunk in itertools.product([1, 2, 4, 16], chunks):
        model = pg.PageModel(num_pages=400, page_size=page, max_seqs=6,
                             max_pages_per_seq=400, layers=nl, kv_heads=hkv,
                             head_dim=d, with_data=True, evict_chunk_pages=chunk,
                             evict_remap=remap, evict_inplace=inplace)
        ref = ListModel()
        next_cursor = 0
        h0 = model.seq_create()
        ref.create(h0)
        for _ in range(n_ops):
            live = sorted(model.seqs)
            ops = ["append", "append", "mark", "fork", "evict", "release"]
            if deferred:
                ops += ["defer", "defer", "compact"]
            op = rng.choice(ops)
            h = int(rng.choice(live))
            if op == "append":
                n = int(rng.integers(0, 2 * page + 3))
                k = rng.standard_normal((nl, n, hkv, d))
                v = rng.standard_normal((nl, n, hkv, d))
                model.append(h, n, k, v)
                ref.append(h, k, v)
            elif op == "mark":
                length = model.info(h)["length"]
                s = int(rng.integers(0, length + 1))
                e = int(rng.integers(s, length + 1))
                if remap and rng.random() < 0.5:
                    s = s // page * page
                    e = s + (e - s) // page * page
                try:
                    model.span_mark(h, next_cursor, s, e)
                    ref.spans[h][next_cursor] = (s, e)
                except pg.SpanError:
                    pass
                next_cursor += 1
            elif op == "fork" and len(live) < 6:
                f = int(rng.integers(0, model.info(h)["length"] + 1))
                c = model.fork(h, f)
                ref.fork(h, f, c)
            elif op == "evict":
                cur = list(model.spans(h))
                pick = [c for c in cur if rng.random() < 0.5]
                st = model.evict(h, pick)
                remapped += st["pages_remapped"]
                in_place += st["tokens_moved"] > 0 and st["pages_allocated"] == 0
                ref.evict(h, pick)
            elif op == "defer":
                cur = list(model.spans(h))
                pick = [c for c in cur if rng.random() < 0.5]
                pages = model.page_table(h)
                model.evict(h, pick, deferred=True)
                assert model.page_table(h) == pages  # nothing moves
                ref.defer(h, pick)
            elif op == "compact":
                model.compact(h)
                ref.evict(h, [])
                assert model.info(h)["n_masked"] == 0
            elif op == "release" and len(live) > 1:
                model.release(h)
                del ref.seqs[h]
            for hh in model.seqs:
                k, v, pos = model.view(hh)
                want = ref.view(hh)
                assert model.info(hh)["length"] == len(ref.seqs[hh])
                assert model.keep_flags(hh).tolist() == [int(t[3]) for t in ref.seqs[hh]]
                if want is None:
                    assert len(pos) == 0
                    continue
                assert np.array_equal(k, want[0]) and np.array_equal(v, want[1])
                assert np.array_equal(pos, want[2])
                assert model.spans(hh) == ref.spans[hh]
                assert model.info(hh)["next_pos"] == ref.next_pos[hh]
        # every page referenced exactly as often as it appears in page lists
        counts = np.zeros(model.num_pages, dtype=np.int64)
        for hh in model.seqs:
            for p in model.page_table(hh):
                counts[p] += 1
        assert np.array_equal(counts, model.refcount)
        for h in list(model.seqs):
            model.release(h)
        assert model.live_pages() == 0
    return in_place if inplace else remapped


def check_hand_worked_page_tables():
    """Page ids under lowest-free-first allocation, worked by hand (P = 4)."""
    m = pg.PageModel(num_pages=16, page_size=4, max_seqs=4, max_pages_per_seq=16)
    a = m.seq_create()
    assert a == 0
    m.append(a, 10)                      # tokens 0..9 -> pages 0, 1, 2
    assert m.page_table(a) == [0, 1, 2]
    b = m.fork(a, 8)                     # aligned: aliases pages 0, 1
    assert b == 1 and m.page_table(b) == [0, 1]
    assert m.refcount[:3].tolist() == [2, 2, 1] and m.live_pages() == 3
    c = m.fork(a, 6)                     # 6 = 1 page + 2 tokens: copy into page 3
    assert c == 2 and m.page_table(c) == [0, 3]
    m.append(b, 3)                       # b: 8 -> 11, new page 4
    assert m.page_table(b) == [0, 1, 4]
    m.span_mark(a, 7, 1, 6)              # evict [1, 6): f = 1, fp = 0
    st = m.evict(a, [7])                 # L' = 5 -> 2 new pages: 5, 6
    assert m.page_table(a) == [5, 6]
    assert st == dict(tokens_removed=5, tokens_moved=5, pages_allocated=2,
                      pages_freed=1, first_evicted=1, pages_remapped=0,
                      tokens_masked=0)  # page 2 was a's alone
    assert m.view(a)[2].tolist() == [0, 6, 7, 8, 9]
    assert m.refcount[:7].tolist() == [2, 1, 0, 1, 1, 1, 1]
    m.release(c)                         # page 0 -> 1 ref, page 3 freed
    m.append(a, 4)                       # a: 5 -> 9: slot 1..3 of page 6, then page 2
    assert m.page_table(a) == [5, 6, 2]
    assert m.view(a)[2].tolist() == [0, 6, 7, 8, 9, 10, 11, 12, 13]
    assert m.peak_pages == 7


def check_fork_is_zero_copy_and_release_restores():
    m = pg.PageModel(num_pages=64, page_size=16, max_seqs=4, max_pages_per_seq=64)
    a = m.seq_create()
    m.append(a, 160)
    before = m.refcount.copy(), m.live_pages()
    b = m.fork(a, 160)
    assert m.live_pages() == before[1]          # aligned: no page
    c = m.fork(a, 150)
    assert m.live_pages() == before[1] + 1      # one tail page
    m.release(b)
    m.release(c)
    assert np.array_equal(m.refcount, before[0]) and m.live_pages() == before[1]


def check_all_keep_eviction_is_identity(seed=11):
    rng = np.random.default_rng(seed)
    m = pg.PageModel(num_pages=32, page_size=4, max_seqs=4, max_pages_per_seq=32,
                     layers=1, kv_heads=1, head_dim=2, with_data=True)
    a = m.seq_create()
    m.append(a, 23, rng.standard_normal((1, 23, 1, 2)), rng.standard_normal((1, 23, 1, 2)))
    m.span_mark(a, 1, 5, 5)
    m.span_mark(a, 2, 9, 9)
    m.span_mark(a, 3, 10, 14)
    snap = _state(m), m.K.copy(), m.V.copy(), m.POS.copy(), m.stats()
    for cursors in ([], [1], [2, 2]):
        st = m.evict(a, cursors)
        assert st["tokens_removed"] == 0 and st["tokens_moved"] == 0
        assert st["pages_allocated"] == 0 and st["pages_freed"] == 0
        assert m.page_table(a) == snap[0][2][a][0]
        assert np.array_equal(m.K, snap[1]) and np.array_equal(m.V, snap[2])
        assert np.array_equal(m.POS, snap[3]) and m.stats() == snap[4]
    assert set(m.spans(a)) == {3}


def check_positions_carried(seed=12):
    rng = np.random.default_rng(seed)
    m = pg.PageModel(num_pages=200, page_size=16, max_seqs=2, max_pages_per_seq=200)
    a = m.seq_create()
    m.append(a, 500)
    cursor = 0
    for _ in range(6):
        length = m.info(a)["length"]
        before = m.view(a)[2]
        cuts = sorted(rng.choice(np.arange(length + 1), 6, replace=False).tolist())
        spans = [(cuts[i], cuts[i + 1]) for i in range(0, 6, 2)]
        ids = []
        for s, e in spans:
            m.span_mark(a, cursor, s, e)
            ids.append(cursor)
            cursor += 1
        keep = ev.keep_mask(length, spans)
        m.evict(a, ids)
        after = m.view(a)[2]
        assert np.array_equal(after, before[keep.astype(bool)])
        assert np.all(np.diff(after) > 0)
        m.append(a, 20)
        assert m.view(a)[2][-1] == 500 + 20 * (_ + 1) - 1


def check_evict_parent_leaves_child(seed=13):
    rng = np.random.default_rng(seed)
    m = pg.PageModel(num_pages=64, page_size=4, max_seqs=4, max_pages_per_seq=64,
                     layers=1, kv_heads=1, head_dim=2, with_data=True)
    a = m.seq_create()
    m.append(a, 30, rng.standard_normal((1, 30, 1, 2)), rng.standard_normal((1, 30, 1, 2)))
    b = m.fork(a, 26)
    m.append(b, 5, rng.standard_normal((1, 5, 1, 2)), rng.standard_normal((1, 5, 1, 2)))
    child_view = [x.copy() for x in m.view(b)]
    m.span_mark(a, 0, 3, 20)             # straddles nothing, shared pages
    m.span_mark(a, 1, 24, 28)            # straddles the fork point 26
    m.evict(a, [0, 1])
    for x, y in zip(child_view, m.view(b)):
        assert np.array_equal(x, y)


def check_errors_leave_state_unchanged():
    m = pg.PageModel(num_pages=6, page_size=4, max_seqs=2, max_pages_per_seq=8)
    a = m.seq_create()
    m.append(a, 14)                      # 4 pages
    m.span_mark(a, 0, 0, 3)
    m.span_mark(a, 1, 8, 14)
    cases = [
        (lambda: m.append(a, 11), pg.NoPages),     # needs 3 more pages, 2 free
        (lambda: m.append(a, 19), pg.Invalid),     # beyond 8 pages per sequence
        (lambda: m.append(9, 1), pg.UnknownSeq),
        (lambda: m.span_mark(a, 2, 2, 5), pg.SpanError),
        (lambda: m.span_mark(a, 0, 4, 5), pg.Invalid),
        (lambda: m.span_mark(a, 3, 10, 15), pg.SpanError),
        (lambda: m.evict(a, [0, 5]), pg.UnknownCursor),
        (lambda: m.fork(a, 15), pg.Invalid),
        (lambda: m.release(7), pg.UnknownSeq),
    ]
    for fn, kind in cases:
        snap = _state(m)
        try:
            fn()
        except pg.OracleError as err:
            assert type(err) is kind, (type(err), kind)
        else:
            raise AssertionError(f"expected {kind.__name__}")
        assert _state(m) == snap
    b = m.fork(a, 13)                    # takes the 5th page (tail copy)
    assert m.free_pages() == 1
    snap = _state(m)
    try:
        m.evict(a, [1])                  # needs ceil(8/4) - 2 = 0 pages: fine
    except pg.OracleError:
        raise AssertionError("evicting the tail needs no page")
    assert _state(m) != snap
    del b


def check_masked_equals_compacted(page_sizes=(1, 2, 4, 16), seed=14, n_tokens=40):
    """The paper's train/serve equivalence: attention over the compacted cache
    is bit-identical to masked attention over the full cache, for every subset
    of up to 6 spans."""
    rng = np.random.default_rng(seed)
    heads = [(1, 1), (4, 1), (8, 2)]
    for page in page_sizes:
        for hq, hkv in heads:
            for d in (8, 64):
                base = pg.PageModel(num_pages=3 * n_tokens, page_size=page, max_seqs=2,
                                    max_pages_per_seq=n_tokens, layers=1, kv_heads=hkv,
                                    head_dim=d, with_data=True)
                a = base.seq_create()
                n = n_tokens
                base.append(a, n, rng.standard_normal((1, n, hkv, d)),
                            rng.standard_normal((1, n, hkv, d)))
                cuts = sorted(rng.choice(np.arange(n + 1), 12, replace=False).tolist())
                spans = [(cuts[i], cuts[i + 1]) for i in range(0, 12, 2)]
                for c, (s, e) in enumerate(spans):
                    base.span_mark(a, c, s, e)
                q = rng.standard_normal((hq, d))
                k_full, v_full, pos_full = base.view(a)
                scale = 1 / math.sqrt(d)
                for r in range(len(spans) + 1):
                    for subset in itertools.combinations(range(len(spans)), r):
                        m = copy.deepcopy(base)
                        m.evict(a, list(subset))
                        keep = ev.keep_mask(n, [spans[c] for c in subset])
                        k, v, pos = m.view(a)
                        assert np.array_equal(pos, pos_full[keep.astype(bool)])
                        got = att.attention(q, k[:, 0], v[:, 0], scale, hq // hkv)
                        want = att.masked_attention(q, k_full[:, 0], v_full[:, 0],
                                                    keep, scale, hq // hkv)
                        assert np.array_equal(got, want)


# --------------------------------------------------------------------------
# extend (causal chunk) attention
# --------------------------------------------------------------------------
def check_extend_textbook(seed=15):
    """Equal to torch's scaled_dot_product_attention in float64 with an
    explicit boolean mask that lets new token j see keys 0 .. L - n + j."""
    rng = np.random.default_rng(seed)
    for hq, hkv, d, L, n, scale in [(4, 1, 64, 40, 40, 1 / 8), (4, 1, 64, 40, 1, 1 / 8),
                                    (8, 2, 16, 57, 13, 0.3), (6, 3, 8, 20, 7, 1.1),
                                    (32, 8, 128, 48, 16, 1 / math.sqrt(128))]:
        g = hq // hkv
        q = rng.standard_normal((n, hq, d))
        k = rng.standard_normal((L, hkv, d))
        v = rng.standard_normal((L, hkv, d))
        out = ex.extend_attention(q, k, v, scale, g)
        allowed = torch.arange(L)[None, :] <= (L - n + torch.arange(n))[:, None]
        kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(g, dim=0)
        vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(g, dim=0)
        qt = torch.from_numpy(q).permute(1, 0, 2).contiguous()
        ref = torch.nn.functional.scaled_dot_product_attention(
            qt, kt, vt, attn_mask=allowed, scale=scale).permute(1, 0, 2).numpy()
        assert np.max(np.abs(out - ref)) <= 1e-12, np.max(np.abs(out - ref))


def check_extend_first_token_alone(seed=16):
    """With no prefix (n = L) the first new token sees only itself: its
    output is its own V row, exactly."""
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((9, 8, 16))
    k = rng.standard_normal((9, 2, 16))
    v = rng.standard_normal((9, 2, 16))
    out = ex.extend_attention(q, k, v, 0.25, 4)
    for h in range(8):
        assert np.array_equal(out[0, h], v[0, h // 4])


def check_extend_causal(seed=17):
    """Changing a key after new token j's own index leaves row j unchanged
    (bit for bit); changing its own key changes it."""
    rng = np.random.default_rng(seed)
    L, n = 30, 10
    q = rng.standard_normal((n, 4, 8))
    k = rng.standard_normal((L, 2, 8))
    v = rng.standard_normal((L, 2, 8))
    base = ex.extend_attention(q, k, v, 0.5, 2)
    for t in (L - n, L - n + 4, L - 1):
        k2, v2 = k.copy(), v.copy()
        k2[t] += 1.0
        v2[t] -= 2.0
        out = ex.extend_attention(q, k2, v2, 0.5, 2)
        for j in range(n):
            if L - n + j < t:
                assert np.array_equal(out[j], base[j])
            else:
                assert not np.array_equal(out[j], base[j])


def check_extend_compacted_equals_masked(seed=18):
    """A chunk appended after an eviction: extend attention over the
    compacted cache equals masked extend attention over the full cache, bit
    for bit, for every subset of 4 spans of the prefix."""
    rng = np.random.default_rng(seed)
    prefix, n, hq, hkv, d = 36, 6, 4, 2, 8
    cuts = sorted(rng.choice(np.arange(prefix + 1), 8, replace=False).tolist())
    spans = [(cuts[i], cuts[i + 1]) for i in range(0, 8, 2)]
    k = rng.standard_normal((prefix + n, hkv, d))
    v = rng.standard_normal((prefix + n, hkv, d))
    q = rng.standard_normal((n, hq, d))
    for r in range(len(spans) + 1):
        for subset in itertools.combinations(spans, r):
            keep = np.concatenate([ev.keep_mask(prefix, list(subset)),
                                   np.ones(n, np.uint8)]).astype(bool)
            got = ex.extend_attention(q, k[keep], v[keep], 0.35, hq // hkv)
            want = ex.extend_attention(q, k, v, 0.35, hq // hkv, mask=keep)
            assert np.array_equal(got, want)


# --------------------------------------------------------------------------
# chunked eviction (bounded transient pages)
# --------------------------------------------------------------------------
def check_chunked_eviction_against_list_model():
    """With chunked eviction every logical view, span and position still
    equals the naive list model's, and refcounts match the page lists."""
    check_against_list_model(seed=19, n_ops=50, chunks=(1, 2, 3))


def check_chunked_page_tables_by_hand():
    """P = 2, 8 tokens in pages [0, 1, 2, 3]; evicting tokens 1 and 2 keeps
    0, 3, 4, 5, 6, 7 (3 pages).  One-shot: fresh pages 4, 5, 6.  C = 1:
    page 4 takes tokens 0, 3; the next source is token 4, so old pages 0 and
    1 go; page 0 takes 4, 5 and old page 2 goes; page 1 takes 6, 7.  C = 2:
    pages 4, 5 take 0, 3, 4, 5; old pages 0-2 go; page 0 takes 6, 7.  The
    live count peaks at 4 + C."""
    want = {0: [4, 5, 6], 1: [4, 0, 1], 2: [4, 5, 0], 3: [4, 5, 6]}
    for chunk, table in want.items():
        m = pg.PageModel(num_pages=10, page_size=2, max_seqs=2, max_pages_per_seq=8,
                         with_data=True, evict_chunk_pages=chunk)
        a = m.seq_create()
        k = np.arange(8, dtype=np.float64).reshape(1, 8, 1, 1)
        m.append(a, 8, k, -k)
        m.span_mark(a, 0, 1, 3)
        st = m.evict(a, [0])
        assert m.page_table(a) == table, (chunk, m.page_table(a))
        assert m.peak_pages == 4 + (3 if chunk in (0, 3) else chunk), (chunk, m.peak_pages)
        assert st["pages_allocated"] == 3 and st["pages_freed"] == 4
        kv, vv, pos = m.view(a)
        assert kv[:, 0, 0, 0].tolist() == [0, 3, 4, 5, 6, 7]
        assert vv[:, 0, 0, 0].tolist() == [0, -3, -4, -5, -6, -7]
        assert pos.tolist() == [0, 3, 4, 5, 6, 7]
        assert m.live_pages() == 3


def _chunk_reads(old_pages, first, spans, length, P, schedule):
    """Old page ids each step's gather reads (from the plan, independently of
    the model): step k fills the fresh pages it allocated, in page order."""
    keep, _dst, src_of, new_len, _f = ev.plan(length, spans)
    fp = first // P
    reads, pi = [], 0
    for got, _rel in schedule:
        r = set()
        for _ in got:
            for j in range((fp + pi) * P, min((fp + pi + 1) * P, new_len)):
                r.add(old_pages[int(src_of[j]) // P])
            pi += 1
        reads.append(r)
    return reads


def check_chunked_eviction_never_overwrites_unread_tokens(seed=20):
    """Each step of a chunked eviction is one parallel gather, so no page it
    writes may be read by it or a later step, and no page released after a
    step may be read later.  A hand-built case (a sequence whose old tail
    pages are [5, 6, 0, 1], P = 2, C = 1) puts a page that is released too
    early at the bottom of the free list; random cases follow."""
    def one(m, h, cursor):
        seq = m.seqs[h]
        old_pages, length = list(seq.pages), seq.length
        spans = [m.spans(h)[cursor]]
        if spans[0][1] <= spans[0][0]:
            return
        m.evict(h, [cursor])
        reads = _chunk_reads(old_pages, spans[0][0], spans, length, m.P, m.last_schedule)
        for k, (got, rel) in enumerate(m.last_schedule):
            later = set().union(*reads[k:]) if reads[k:] else set()
            assert not set(got) & later, (k, got, later)
            after = set().union(*reads[k + 1:]) if reads[k + 1:] else set()
            assert not set(rel) & after, (k, rel, after)

    m = pg.PageModel(num_pages=12, page_size=2, max_seqs=3, max_pages_per_seq=12,
                     with_data=True, evict_chunk_pages=1)
    b = m.seq_create()
    m.append(b, 10, np.zeros((1, 10, 1, 1)), np.zeros((1, 10, 1, 1)))
    a = m.seq_create()
    k = np.arange(8, dtype=np.float64).reshape(1, 8, 1, 1)
    m.append(a, 4, k[:, :4], k[:, :4])
    m.release(b)
    m.append(a, 4, k[:, 4:], k[:, 4:])
    assert m.page_table(a) == [5, 6, 0, 1]
    m.span_mark(a, 0, 1, 2)
    one(m, a, 0)
    assert m.page_table(a) == [2, 3, 4, 0]
    assert m.view(a)[0][:, 0, 0, 0].tolist() == [0, 2, 3, 4, 5, 6, 7]
    rng = np.random.default_rng(seed)
    for trial in range(40):
        m = pg.PageModel(num_pages=80, page_size=2, max_seqs=3, max_pages_per_seq=80,
                         evict_chunk_pages=int(rng.integers(1, 4)))
        hs = [m.seq_create(), m.seq_create()]
        for step in range(14):
            h = hs[int(rng.integers(0, 2))]
            m.append(h, int(rng.integers(1, 9)))
            L = m.info(h)["length"]
            s0 = int(rng.integers(0, L))
            e0 = int(rng.integers(s0, L + 1))
            try:
                m.span_mark(h, step, s0, e0)
            except pg.SpanError:
                continue
            if rng.random() < 0.5:
                one(m, h, step)


def check_chunked_eviction_fits_where_one_shot_does_not():
    """With one free page the one-shot eviction above needs three and fails
    (changing nothing); chunks of one page recycle the old pages and fit."""
    for chunk, ok in ((0, False), (1, True)):
        m = pg.PageModel(num_pages=5, page_size=2, max_seqs=2, max_pages_per_seq=8,
                         with_data=True, evict_chunk_pages=chunk)
        a = m.seq_create()
        k = np.arange(8, dtype=np.float64).reshape(1, 8, 1, 1)
        m.append(a, 8, k, k)
        m.span_mark(a, 0, 1, 3)
        snap = _state(m)
        try:
            m.evict(a, [0])
            assert ok
            assert m.page_table(a) == [4, 0, 1]
            assert m.view(a)[0][:, 0, 0, 0].tolist() == [0, 3, 4, 5, 6, 7]
        except pg.NoPages:
            assert not ok
            assert _state(m) == snap


# --------------------------------------------------------------------------
# page-aligned remap
# --------------------------------------------------------------------------
def check_remap_against_list_model():
    """With page-aligned remap (alone and with chunks) every logical view,
    span and position equals the naive list model's, refcounts match the page
    lists, and remaps do happen."""
    assert check_against_list_model(seed=21, n_ops=60, chunks=(0, 2), remap=True) > 0


def check_remap_page_tables_by_hand():
    """P = 4, 16 tokens in pages [0, 1, 2, 3].  Evicting [0, 4) shifts by one
    page: pages 1, 2, 3 become the whole list, nothing is copied, page 0 is
    freed.  Evicting [2, 6) also shifts by 4: new page 0 holds tokens
    0, 1, 6, 7 (fresh page 4), new pages 1 and 2 are old pages 2 and 3.
    Evicting [1, 3) shifts by 2: nothing lines up, as without remap."""
    cases = [((0, 4), [1, 2, 3], dict(pages_remapped=3, pages_allocated=0, pages_freed=1,
                                      tokens_moved=0)),
             ((2, 6), [4, 2, 3], dict(pages_remapped=2, pages_allocated=1, pages_freed=2,
                                      tokens_moved=4)),
             ((1, 3), [4, 5, 6, 7], dict(pages_remapped=0, pages_allocated=4, pages_freed=4,
                                         tokens_moved=14))]
    for chunk in (0, 1):
        for (s0, e0), table, want in cases:
            m = pg.PageModel(num_pages=12, page_size=4, max_seqs=2, max_pages_per_seq=8,
                             with_data=True, evict_chunk_pages=chunk, evict_remap=True)
            a = m.seq_create()
            k = np.arange(16, dtype=np.float64).reshape(1, 16, 1, 1)
            m.append(a, 16, k, -k)
            m.span_mark(a, 0, s0, e0)
            st = m.evict(a, [0])
            keep = [t for t in range(16) if not s0 <= t < e0]
            assert m.view(a)[0][:, 0, 0, 0].tolist() == keep
            assert m.view(a)[1][:, 0, 0, 0].tolist() == [-t for t in keep]
            assert m.view(a)[2].tolist() == keep
            if chunk == 0 or want["pages_remapped"]:
                assert m.page_table(a) == table, (chunk, s0, m.page_table(a))
            for key, val in want.items():
                assert st[key] == val, (chunk, s0, key, st[key], val)
            assert m.refcount.sum() == len(m.page_table(a))


# --------------------------------------------------------------------------
# in-place eviction (no transient pages)
# --------------------------------------------------------------------------
def check_inplace_against_list_model():
    """In-place eviction, alone and with deferred evictions: every logical
    view, span and position equals the naive list model's, refcounts match
    the page lists (a branch's pages are never rewritten: its view is the
    list model's too), and evictions that take no page do happen."""
    assert check_against_list_model(seed=29, n_ops=60, inplace=True) > 0
    assert check_against_list_model(seed=30, n_ops=60, deferred=True, inplace=True) > 0


def check_inplace_page_tables_by_hand():
    """P = 2, 8 tokens in pages [0, 1, 2, 3]; evicting tokens 1 and 2 keeps
    0, 3, 4, 5, 6, 7.  In place: pages [0, 1, 2] hold (0, 3), (4, 5),
    (6, 7); page 3 is freed; no page is taken.  With an auxiliary branch
    forked at 4 (holding pages 0 and 1), those two pages stay as they are
    for the branch and the sequence takes fresh pages 4 and 5 for them:
    [4, 5, 2]."""
    for fork, table, alloc in ((False, [0, 1, 2], 0), (True, [4, 5, 2], 2)):
        m = pg.PageModel(num_pages=8, page_size=2, max_seqs=2, max_pages_per_seq=8,
                         with_data=True, evict_inplace=True)
        a = m.seq_create()
        k = np.arange(8, dtype=np.float64).reshape(1, 8, 1, 1)
        m.append(a, 8, k, -k)
        if fork:
            aux = m.fork(a, 4)
        m.span_mark(a, 0, 1, 3)
        st = m.evict(a, [0])
        assert m.page_table(a) == table, (fork, m.page_table(a))
        assert (st["pages_allocated"], st["pages_freed"], st["tokens_moved"]) == (alloc, 1, 6)
        kv, vv, pos = m.view(a)
        assert kv[:, 0, 0, 0].tolist() == [0, 3, 4, 5, 6, 7]
        assert vv[:, 0, 0, 0].tolist() == [0, -3, -4, -5, -6, -7]
        assert pos.tolist() == [0, 3, 4, 5, 6, 7]
        assert m.peak_pages == 4 + alloc
        if fork:
            assert m.page_table(aux) == [0, 1]
            assert m.view(aux)[0][:, 0, 0, 0].tolist() == [0, 1, 2, 3]
            assert m.refcount.tolist()[:6] == [1, 1, 1, 0, 1, 1]


def check_inplace_fits_a_full_pool():
    """A pool whose every page holds the sequence: the one-shot and chunked
    evictions need fresh pages and fail (changing nothing); in place needs
    none and succeeds."""
    for mode, ok in (({}, False), ({"evict_chunk_pages": 1}, False),
                     ({"evict_inplace": True}, True)):
        m = pg.PageModel(num_pages=4, page_size=2, max_seqs=2, max_pages_per_seq=8,
                         with_data=True, **mode)
        a = m.seq_create()
        k = np.arange(8, dtype=np.float64).reshape(1, 8, 1, 1)
        m.append(a, 8, k, k)
        m.span_mark(a, 0, 1, 3)
        assert m.free_pages() == 0
        snap = _state(m)
        try:
            m.evict(a, [0])
            assert ok, mode
            assert m.page_table(a) == [0, 1, 2]
            assert m.view(a)[0][:, 0, 0, 0].tolist() == [0, 3, 4, 5, 6, 7]
            assert m.peak_pages == 4 and m.live_pages() == 3
        except pg.NoPages:
            assert not ok, mode
            assert _state(m) == snap


def _inplace_reads(length, spans, P, n_new, first):
    """Old page-list indices each tail page's kept tokens come from (from
    the eviction plan alone)."""
    _keep, _dst, src_of, new_len, _f = ev.plan(length, spans)
    fp = first // P
    return [sorted({int(src_of[j]) // P
                    for j in range((fp + k) * P, min((fp + k + 1) * P, new_len))})
            for k in range(n_new)]


def _inplace_rounds(reads, fp):
    """Runs [a, b) of tail pages that one parallel launch may rewrite: taking
    each page's read range whole, page b joins unless the range of pages
    a .. b - 1 covers fp + b."""
    rounds, a = [], 0
    while a < len(reads):
        lo, hi, b = reads[a][0], reads[a][-1], a + 1
        while b < len(reads) and not (lo <= fp + b <= hi):
            hi = max(hi, reads[b][-1])
            b += 1
        rounds.append((a, b))
        a = b
    return rounds


def check_inplace_order_never_reads_a_rewritten_page(seed=31):
    """Tail page k's tokens come from old list indices >= fp + k, so a pass
    that rewrites the tail pages in order never reads a page it has already
    rewritten; replaying such a pass on the physical pages (each page's
    sources read, then the page written) gives the model's result.  Runs of
    pages rewritten in parallel read no page of the run but their own, and
    with a shift of s tokens a run spans about s / P pages."""
    rng = np.random.default_rng(seed)
    P = 4
    for trial in range(60):
        L = int(rng.integers(8, 120))
        m = pg.PageModel(num_pages=64, page_size=P, max_seqs=2, max_pages_per_seq=64,
                         head_dim=2, with_data=True, evict_inplace=True)
        a = m.seq_create()
        k = rng.standard_normal((1, L, 1, 2))
        m.append(a, L, k, -k)
        cuts = np.sort(rng.choice(np.arange(L + 1), size=2 * int(rng.integers(1, 4)),
                                  replace=False))
        spans = [(int(cuts[2 * i]), int(cuts[2 * i + 1])) for i in range(len(cuts) // 2)]
        spans = [(s0, e0) for s0, e0 in spans if e0 > s0]
        if not spans:
            continue
        for c, (s0, e0) in enumerate(spans):
            m.span_mark(a, c, s0, e0)
        old_pages = list(m.page_table(a))
        phys_k = m.K.copy()
        st = m.evict(a, list(range(len(spans))))
        new_len, fp = m.info(a)["length"], st["first_evicted"] // P
        n_new = math.ceil(new_len / P) - fp
        reads = _inplace_reads(L, spans, P, n_new, st["first_evicted"])
        assert m.page_table(a)[fp:] == old_pages[fp: fp + n_new]
        _keep, _dst, src_of, _nl, _f = ev.plan(L, spans)
        for kk in range(n_new):
            assert reads[kk][0] >= fp + kk, (trial, kk, reads[kk])
            # the pass: read page kk's sources from the current pages, write it
            toks = range((fp + kk) * P, min((fp + kk + 1) * P, new_len))
            vals = [phys_k[old_pages[int(src_of[j]) // P], int(src_of[j]) % P].copy() for j in toks]
            for j, v in zip(toks, vals):
                phys_k[old_pages[fp + kk], j % P] = v
        for j in range(new_len):
            pg_id = m.page_table(a)[j // P]
            assert np.array_equal(phys_k[pg_id, j % P], m.K[pg_id, j % P])
        rounds = _inplace_rounds(reads, fp)
        for r0, r1 in rounds:
            for kk in range(r0, r1):
                others = {fp + x for x in range(r0, r1) if x != kk}
                assert not (set(range(reads[kk][0], reads[kk][-1] + 1)) & others), (trial, kk)
    # a shift of one token: every run is one page; a shift of 8 pages: runs of 8
    for shift, want in ((1, 1), (8 * P, 8)):
        reads = _inplace_reads(64 * P, [(0, shift)], P, math.ceil((64 * P - shift) / P), 0)
        rounds = _inplace_rounds(reads, 0)
        assert max(r1 - r0 for r0, r1 in rounds) == want, (shift, rounds[:3])


# --------------------------------------------------------------------------
# sinks and windows (model variants)
# --------------------------------------------------------------------------
def check_sinks_textbook(seed=22):
    """Per-head sinks: equal to torch.softmax over the logits with the sink
    appended as one more column (dropped after the softmax) times V, in
    float64; a sink of -inf changes nothing at all."""
    rng = np.random.default_rng(seed)
    for hq, hkv, d, n, scale in [(4, 1, 64, 50, 1 / 8), (8, 2, 8, 17, 0.5),
                                 (64, 8, 64, 30, 1 / 8), (2, 2, 4, 1, 1.0)]:
        q, k, v = _rand_qkv(rng, hq, hkv, d, n)
        g = hq // hkv
        sinks = rng.standard_normal(hq) * 3
        out = att.attention(q, k, v, scale, g, sinks=sinks)
        kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(g, dim=0)
        vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(g, dim=0)
        qt = torch.from_numpy(q)[:, None, :]
        logits = scale * torch.bmm(qt, kt.transpose(1, 2).contiguous())
        logits = torch.cat([logits, torch.from_numpy(sinks)[:, None, None]], dim=-1)
        p = torch.softmax(logits, dim=-1)[:, :, :n]
        ref = torch.bmm(p, vt)[:, 0, :].numpy()
        assert np.max(np.abs(out - ref)) <= 1e-12, np.max(np.abs(out - ref))
        same = att.attention(q, k, v, scale, g, sinks=np.full(hq, -np.inf))
        assert np.array_equal(same, att.attention(q, k, v, scale, g))


def check_sink_closed_form():
    """One key of score s and a sink c: the output is v * e^s / (e^s + e^c),
    i.e. v times the logistic function of s - c."""
    q = np.array([[1.0, 0.5]])
    k = np.array([[[2.0, -1.0]]])
    v = np.array([[[3.0, -4.0]]])
    s = 0.7 * (1.0 * 2.0 + 0.5 * -1.0)
    for c in (-2.0, 0.0, s, 5.0):
        out = att.attention(q, k, v, 0.7, 1, sinks=np.array([c]))
        want = v[0, 0] / (1.0 + math.exp(c - s))
        assert np.max(np.abs(out[0] - want)) <= 1e-15, (c, out, want)


def check_windows(seed=23):
    """A window of W keys: W >= L changes nothing; W = 1 returns the last
    key's V exactly; otherwise equal to torch's scaled_dot_product_attention
    with the band mask, for decode and for extend (band and causal)."""
    rng = np.random.default_rng(seed)
    for hq, hkv, d, L, scale in [(4, 1, 16, 40, 0.25), (8, 2, 8, 17, 0.5), (64, 8, 64, 33, 1 / 8)]:
        q, k, v = _rand_qkv(rng, hq, hkv, d, L)
        g = hq // hkv
        full = att.decode_batch(q[None], [(k, v)], scale, g)
        assert np.array_equal(att.decode_batch(q[None], [(k, v)], scale, g, window=L), full)
        one = att.decode_batch(q[None], [(k, v)], scale, g, window=1)[0]
        assert np.array_equal(one, np.repeat(v[-1], g, axis=0))
        kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(g, dim=0)
        vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(g, dim=0)
        for w in (2, 5, L - 1):
            out = att.decode_batch(q[None], [(k, v)], scale, g, window=w)[0]
            allowed = (torch.arange(L) >= L - w)[None, :]
            ref = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(q)[:, None, :], kt, vt, attn_mask=allowed,
                scale=scale)[:, 0, :].numpy()
            assert np.max(np.abs(out - ref)) <= 1e-12, (w, np.max(np.abs(out - ref)))
        n = 9
        qn = rng.standard_normal((n, hq, d))
        for w in (1, 4, 12):
            out = ex.extend_attention(qn, k, v, scale, g, window=w)
            j = torch.arange(n)[:, None] + (L - n)
            key = torch.arange(L)[None, :]
            allowed = (key <= j) & (key > j - w)
            ref = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(qn).permute(1, 0, 2).contiguous(), kt, vt, attn_mask=allowed,
                scale=scale).permute(1, 0, 2).numpy()
            assert np.max(np.abs(out - ref)) <= 1e-12, (w, np.max(np.abs(out - ref)))
            sinks = rng.standard_normal(hq)
            with_s = ex.extend_attention(qn, k, v, scale, g, window=w, sinks=sinks)
            for jj in range(n):
                last = L - n + jj
                lo = max(0, last - w + 1)
                want = att.attention(qn[jj], k[lo: last + 1], v[lo: last + 1], scale, g,
                                     sinks=sinks)
                assert np.array_equal(with_s[jj], want)


def check_deferred_against_list_model():
    """Deferred evictions and compactions among the random ops (one-shot and
    chunked schedules, with and without remap)."""
    check_against_list_model(seed=24, n_ops=80, chunks=(0, 1), deferred=True)
    check_against_list_model(seed=25, n_ops=60, remap=True, deferred=True)


def check_deferred_by_hand():
    """P = 4, ten tokens: a deferred eviction masks in place, a fork keeps
    the masks of its slots, a later physical eviction removes the masked
    slots with its own span (their union), and compaction alone removes only
    the masked ones; worked by hand."""
    m = pg.PageModel(num_pages=16, page_size=4, max_seqs=4, max_pages_per_seq=16)
    a = m.seq_create()
    m.append(a, 10)                                      # pages 0, 1, 2
    m.span_mark(a, 1, 1, 3)
    m.span_mark(a, 2, 6, 7)
    m.span_mark(a, 3, 8, 9)
    st = m.evict(a, [1, 2], deferred=True)
    assert st["tokens_masked"] == 3 and st["tokens_removed"] == 0 and st["first_evicted"] == 1
    assert m.page_table(a) == [0, 1, 2] and m.info(a)["length"] == 10
    assert m.keep_flags(a).tolist() == [1, 0, 0, 1, 1, 1, 0, 1, 1, 1]
    assert m.spans(a) == {3: (8, 9)}                     # unshifted
    assert m.view(a)[2].tolist() == [0, 3, 4, 5, 7, 8, 9]
    b = m.fork(a, 7)                                     # 1 page + 3 slots: page 3
    assert m.page_table(b) == [0, 3]
    assert m.keep_flags(b).tolist() == [1, 0, 0, 1, 1, 1, 0]
    assert m.view(b)[2].tolist() == [0, 3, 4, 5]
    m.span_mark(a, 4, 2, 5)                              # covers masked slot 2
    st = m.evict(a, [4])                                 # removes [1, 5) and [6, 7)
    assert st["tokens_removed"] == 5 and st["first_evicted"] == 1
    assert m.info(a)["length"] == 5 and m.info(a)["n_masked"] == 0
    assert m.view(a)[2].tolist() == [0, 5, 7, 8, 9]
    assert m.spans(a) == {3: (3, 4)}                     # 8 - 5 removed before it
    st = m.compact(b)                                    # b: [1, 3) and [6, 7)
    assert st["tokens_removed"] == 3 and m.info(b)["length"] == 4
    assert m.view(b)[2].tolist() == [0, 3, 4, 5] and m.keep_flags(b).tolist() == [1, 1, 1, 1]


def check_deferred_then_compact_equals_immediate(seed=26):
    """Deferring then compacting a set of spans leaves exactly the state an
    immediate eviction of the same spans leaves (page tables, refcounts,
    data, spans, stats but tokens_masked)."""
    rng = np.random.default_rng(seed)
    for page in (1, 4, 16):
        models = [pg.PageModel(num_pages=600, page_size=page, max_seqs=4, max_pages_per_seq=300,
                               layers=1, kv_heads=1, head_dim=2, with_data=True) for _ in range(2)]
        k = rng.standard_normal((1, 200, 1, 2))
        spans = [(s0, s0 + int(rng.integers(1, 20))) for s0 in range(5, 180, 23)]
        for m in models:
            h = m.seq_create()
            m.append(h, 200, k, k)
            m.fork(h, 150)
            for c, (s0, e0) in enumerate(spans):
                m.span_mark(h, c, s0, e0)
        pick = [0, 2, 3, 7]
        models[0].evict(0, pick, deferred=True)
        st0 = models[0].compact(0)
        st1 = models[1].evict(0, pick)
        st0.pop("tokens_masked")
        st1.pop("tokens_masked")
        assert st0 == st1
        assert _state(models[0]) == _state(models[1])
        assert np.array_equal(models[0].K, models[1].K)


def check_fp8_decode_table():
    """All 256 E4M3 codes decode to what torch's float8_e4m3fn type holds
    (an independent implementation of the same format)."""
    import torch
    from oracle import fp8
    codes = np.arange(256, dtype=np.uint8)
    want = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = fp8.decode(codes)
    assert np.array_equal(np.isnan(got), np.isnan(want))
    ok = ~np.isnan(want)
    assert np.array_equal(got[ok], want[ok])
    assert np.array_equal(np.signbit(got[ok]), np.signbit(want[ok]))
    assert got[0x7E] == 448.0 and got[0x01] == 2.0 ** -9 and got[0x08] == 2.0 ** -6


def check_fp8_encode(seed=27):
    """Nearest-even encoding: equal to torch's conversion wherever torch does
    not overflow (|y| < 464), including exact ties and subnormals; equal to a
    brute-force nearest search over every finite code; saturating at 448."""
    import torch
    from oracle import fp8
    rng = np.random.default_rng(seed)
    mags = fp8.decode(np.arange(0x7F))
    mids = (mags[:-1] + mags[1:]) / 2                       # exact ties
    y = np.concatenate([
        rng.standard_normal(4000) * 30, rng.standard_normal(2000) * 1e-3,
        rng.uniform(-460, 460, 2000), mids, -mids, mags, -mags, [0.0, -0.0, 463.9, -463.9],
    ]).astype(np.float32)
    got = fp8.encode(y)
    want = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(got, want)
    finite = np.array([c for c in range(256) if (c & 0x7F) != 0x7F])
    vals = fp8.decode(finite)
    for x in y[::37]:
        d = np.abs(vals - np.float64(x))
        best = finite[d == d.min()]
        best = best[np.signbit(fp8.decode(best)) == np.signbit(x)] if len(best) > 1 else best
        if len(best) > 1:
            best = best[best % 2 == 0]
        assert fp8.encode(np.float32(x)) == best[0], x
    big = np.array([448.0, 464.0, 500.0, 1e6, -448.0, -1e30], dtype=np.float32)
    assert fp8.encode(big).tolist() == [0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0xFE]


def check_fp8_store_values(seed=28):
    """An 8-bit store holds each appended value's E4M3 round trip with its
    layer's scale (relative error <= 1/16 in the normal range), and fork and
    eviction move those values unchanged."""
    from oracle import fp8
    rng = np.random.default_rng(seed)
    scales = np.array([[0.05, 0.02], [0.5, 0.25]], dtype=np.float32)
    m = pg.PageModel(num_pages=40, page_size=4, max_seqs=3, max_pages_per_seq=40, layers=2,
                     kv_heads=2, head_dim=3, with_data=True, kv_scales=scales)
    a = m.seq_create()
    k = rng.standard_normal((2, 30, 2, 3))
    v = rng.standard_normal((2, 30, 2, 3))
    m.append(a, 30, k, v)
    kk, vv, _ = m.view(a)
    for l in range(2):
        assert np.array_equal(kk[:, l], fp8.roundtrip(k[l], scales[l, 0]))
        assert np.array_equal(vv[:, l], fp8.roundtrip(v[l], scales[l, 1]))
        y = np.abs(k[l] / scales[l, 0])
        normal = (y >= 2.0 ** -6) & (y < 448)
        assert np.all(np.abs(kk[:, l] - k[l])[normal] <= np.abs(k[l])[normal] / 16 + 1e-12)
    b = m.fork(a, 13)
    m.span_mark(a, 0, 2, 9)
    m.evict(a, [0])
    keep = np.ones(30, bool)
    keep[2:9] = False
    assert np.array_equal(m.view(a)[0], kk[keep]) and np.array_equal(m.view(b)[1], vv[:13])


ALL_CHECKS = [
    check_weights_sum_to_one, check_single_key_returns_v, check_textbook_softmax,
    check_uniform_closed_form, check_two_key_closed_form,
    check_permutation_invariance, check_masked_semantics, check_merge_identity,
    check_scan_and_inverse, check_span_shift, check_against_list_model,
    check_hand_worked_page_tables, check_fork_is_zero_copy_and_release_restores,
    check_all_keep_eviction_is_identity, check_positions_carried,
    check_evict_parent_leaves_child, check_errors_leave_state_unchanged,
    check_masked_equals_compacted, check_extend_textbook, check_extend_first_token_alone,
    check_extend_causal, check_extend_compacted_equals_masked,
    check_chunked_eviction_against_list_model, check_chunked_page_tables_by_hand,
    check_chunked_eviction_fits_where_one_shot_does_not,
    check_chunked_eviction_never_overwrites_unread_tokens,
    check_remap_against_list_model, check_remap_page_tables_by_hand,
    check_inplace_against_list_model, check_inplace_page_tables_by_hand,
    check_inplace_fits_a_full_pool, check_inplace_order_never_reads_a_rewritten_page,
    check_sinks_textbook, check_sink_closed_form, check_windows,
    check_deferred_against_list_model, check_deferred_by_hand,
    check_deferred_then_compact_equals_immediate,
    check_fp8_decode_table, check_fp8_encode, check_fp8_store_values,
]
