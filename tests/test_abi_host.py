"""Host logic of libsq against the oracle's page model (CPU only).

A metadata-only store runs every bookkeeping step of the library (allocator,
refcounts, page lists, positions, spans, eviction planning, decode planning)
without a GPU; page tables, refcounts, positions and spans must match the
oracle bit for bit, and failing calls must fail the same way and change
nothing.
"""

import math
import os
import re

import numpy as np
import pytest

from oracle import pages as pg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def sq():
    from paper_2602_22603_amd import build_lib, sq as sqmod
    if not os.path.exists(sqmod.LIB_PATH):
        build_lib.build()
    sqmod.lib()
    return sqmod


ERR_KIND = {1: pg.Invalid, 2: pg.NoPages, 3: pg.UnknownSeq, 4: pg.UnknownCursor, 5: pg.SpanError}


def test_library_exports_every_declared_symbol(sq):
    header = open(os.path.join(ROOT, "include", "sq.h")).read()
    declared = set(re.findall(r"^\s*(?:[\w\s\*]+?)\b(sq_\w+)\s*\(", header, flags=re.M))
    declared -= {"sq_store", "sq_seq"}
    assert len(declared) >= 20
    lib = sq.lib()
    for name in sorted(declared):
        assert hasattr(lib, name), name
    assert declared == set(sq.EXPORTED)
    version = int(re.search(r"#define SQ_ABI_VERSION (\d+)", header).group(1))
    assert lib.sq_abi_version() == version


def _store(sq, num_pages, page, max_seqs, max_pages, chunk=0, remap=False, inplace=False):
    return sq.Store(num_layers=2, num_q_heads=4, num_kv_heads=2, head_dim=8,
                    num_pages=num_pages, max_seqs=max_seqs, max_pages_per_seq=max_pages,
                    page_size=page, metadata_only=True, evict_chunk_pages=chunk,
                    evict_remap=remap, evict_inplace=inplace)


def _compare(store, model):
    assert store.refcounts().tolist() == model.refcount.tolist()
    st = store.stats()
    ms = model.stats()
    assert (st["live_pages"], st["peak_pages"], st["free_pages"], st["live_seqs"]) == (
        ms["live_pages"], ms["peak_pages"], ms["free_pages"], ms["live_seqs"])
    for h in model.seqs:
        assert store.page_table(h) == model.page_table(h)
        info = store.seq_info(h)
        want = model.info(h)
        for k in ("length", "next_pos", "n_pages", "parent", "n_spans", "n_masked"):
            assert info[k] == want[k], (k, info[k], want[k])
        assert store.positions(h).tolist() == model.slot_view(h)[2].tolist()
        assert store.keep_flags(h).tolist() == model.keep_flags(h).tolist()
        assert store.spans(h) == model.spans(h)


def _both(store, model, sq, fn_store, fn_model):
    """Run one op on both; same outcome (value or error kind)."""
    try:
        want = fn_model()
        err_m = None
    except pg.OracleError as e:
        want, err_m = None, type(e)
    try:
        got = fn_store()
        err_s = None
    except sq.SqError as e:
        got, err_s = None, ERR_KIND[e.code]
    assert err_s == err_m, (err_s, err_m)
    return got, want


@pytest.mark.parametrize("page", [1, 2, 4, 16])
@pytest.mark.parametrize("seed,chunk,remap,deferred,inplace",
                         [(0, 0, False, False, False), (1, 0, False, False, False),
                          (2, 1, False, False, False), (3, 2, False, False, False),
                          (4, 5, False, False, False), (5, 0, True, False, False),
                          (6, 2, True, False, False), (7, 0, False, True, False),
                          (8, 2, True, True, False), (9, 0, False, False, True),
                          (10, 0, False, True, True)])
def test_random_ops_match_oracle(sq, page, seed, chunk, remap, deferred, inplace):
    rng = np.random.default_rng(100 + seed * 7 + page)
    num_pages, max_seqs, max_pages = 300 // page + 40, 5, 400 // page + 8
    store = _store(sq, num_pages, page, max_seqs, max_pages, chunk, remap, inplace)
    model = pg.PageModel(num_pages, page, max_seqs, max_pages, evict_chunk_pages=chunk,
                         evict_remap=remap, evict_inplace=inplace)
    cursor = 0
    h0, _ = _both(store, model, sq, store.seq_create, model.seq_create)
    for _ in range(250):
        live = sorted(model.seqs)
        h = int(rng.choice(live)) if live else 0
        ops = ["append", "append", "mark", "mark", "fork", "evict", "release", "bad", "step"]
        if deferred:
            ops += ["defer", "defer", "compact"]
        op = rng.choice(ops)
        if op == "step":
            # a decode step opens one slot per sequence, all or nothing
            batch = [int(x) for x in rng.permutation(live)[:int(rng.integers(1, len(live) + 1))]]
            need = sum(model.info(x)["length"] % page == 0 for x in batch)
            full = any(model.info(x)["length"] // page + 1 > max_pages
                       for x in batch if model.info(x)["length"] % page == 0)
            before = [store.page_table(x) for x in batch], store.refcounts().tolist()
            if full or need > model.stats()["free_pages"]:
                with pytest.raises(sq.SqError):
                    store.step_begin(batch)
                assert before == ([store.page_table(x) for x in batch], store.refcounts().tolist())
            else:
                store.step_begin(batch)
                for x in batch:
                    model.append(x, 1)
        elif op == "append":
            n = int(rng.integers(0, 3 * page + 5))
            _both(store, model, sq, lambda: store.append(h, n=n), lambda: model.append(h, n))
        elif op == "mark":
            length = model.info(h)["length"]
            s = int(rng.integers(0, length + 1))
            e = int(rng.integers(s, min(length, s + 40) + 1))
            if remap and rng.random() < 0.5:  # whole pages: remaps happen
                s = s // page * page
                e = s + (e - s) // page * page
            c = cursor if rng.random() < 0.9 else int(rng.integers(0, cursor + 1))
            _both(store, model, sq, lambda: store.span_mark(h, c, s, e),
                  lambda: model.span_mark(h, c, s, e))
            cursor += 1
        elif op == "fork":
            f = int(rng.integers(0, model.info(h)["length"] + 2))
            _both(store, model, sq, lambda: store.fork(h, f), lambda: model.fork(h, f))
        elif op == "evict":
            cur = list(model.spans(h))
            pick = [c for c in cur if rng.random() < 0.4]
            if rng.random() < 0.1:
                pick.append(10_000 + cursor)  # unknown cursor
            pick += pick[:1]                   # a duplicate
            got, want = _both(store, model, sq, lambda: store.evict(h, pick),
                              lambda: model.evict(h, pick))
            if want is not None:
                for k in want:
                    assert got[k] == want[k], (k, got, want)
        elif op == "defer":
            cur = list(model.spans(h))
            pick = [c for c in cur if rng.random() < 0.5] + cur[:1]
            got, want = _both(store, model, sq, lambda: store.evict(h, pick, deferred=True),
                              lambda: model.evict(h, pick, deferred=True))
            if want is not None:
                for k in want:
                    assert got[k] == want[k], (k, got, want)
        elif op == "compact":
            got, want = _both(store, model, sq, lambda: store.compact(h), lambda: model.compact(h))
            if want is not None:
                for k in want:
                    assert got[k] == want[k], (k, got, want)
        elif op == "release" and len(live) > 1:
            _both(store, model, sq, lambda: store.release(h), lambda: model.release(h))
        elif op == "bad":
            _both(store, model, sq, lambda: store.release(99), lambda: model.release(99))
        _compare(store, model)
    for h in list(model.seqs):
        store.release(h)
        model.release(h)
    _compare(store, model)
    assert store.stats()["live_pages"] == 0


def test_hand_worked_page_tables(sq):
    s = _store(sq, 16, 4, 4, 16)
    a = s.seq_create()
    s.append(a, n=10)
    assert s.page_table(a) == [0, 1, 2]
    b = s.fork(a, 8)
    c = s.fork(a, 6)
    assert (b, c) == (1, 2) and s.page_table(b) == [0, 1] and s.page_table(c) == [0, 3]
    s.append(b, n=3)
    s.span_mark(a, 7, 1, 6)
    st = s.evict(a, [7])
    assert s.page_table(a) == [5, 6]
    assert (st["tokens_removed"], st["tokens_moved"], st["pages_allocated"],
            st["pages_freed"], st["first_evicted"]) == (5, 5, 2, 1, 1)
    assert st["bytes_moved"] == 5 * (2 * 2 * 8 * 2 * 2 + 4)
    s.release(c)
    s.append(a, n=4)
    assert s.page_table(a) == [5, 6, 2]
    assert s.positions(a).tolist() == [0, 6, 7, 8, 9, 10, 11, 12, 13]
    assert s.stats()["peak_pages"] == 7


def test_chunked_eviction_page_tables_by_hand(sq):
    """P = 2, 8 tokens: evicting tokens 1-2 takes fresh pages [4, 5, 6] in one
    shot, [4, 0, 1] one page at a time (old pages reused as soon as their
    tokens are moved) and [4, 5, 0] two at a time; peak 4 + chunk."""
    for chunk, table in ((0, [4, 5, 6]), (1, [4, 0, 1]), (2, [4, 5, 0])):
        s = _store(sq, 10, 2, 2, 8, chunk)
        a = s.seq_create()
        s.append(a, n=8)
        s.span_mark(a, 0, 1, 3)
        st = s.evict(a, [0])
        assert s.page_table(a) == table
        assert s.positions(a).tolist() == [0, 3, 4, 5, 6, 7]
        assert s.stats()["peak_pages"] == 4 + (chunk or 3)
        assert (st["pages_allocated"], st["pages_freed"]) == (3, 4)
    # one free page: one-shot fails and changes nothing, chunks of one fit
    for chunk in (0, 1):
        s = _store(sq, 5, 2, 2, 8, chunk)
        a = s.seq_create()
        s.append(a, n=8)
        s.span_mark(a, 0, 1, 3)
        if chunk == 0:
            with pytest.raises(sq.SqError) as ei:
                s.evict(a, [0])
            assert ei.value.code == sq.ERR_NO_PAGES
            assert s.page_table(a) == [0, 1, 2, 3]
        else:
            s.evict(a, [0])
            assert s.page_table(a) == [4, 0, 1]
    with pytest.raises(sq.SqError):
        _store(sq, 10, 2, 2, 8, -1)


def test_error_paths_leave_state_unchanged(sq):
    s = _store(sq, 6, 4, 2, 8)
    m = pg.PageModel(6, 4, 2, 8)
    a = s.seq_create()
    m.seq_create()
    s.append(a, n=14)
    m.append(a, 14)
    for c, (x, y) in enumerate([(0, 3), (8, 14)]):
        s.span_mark(a, c, x, y)
        m.span_mark(a, c, x, y)
    cases = [
        (lambda: s.append(a, n=11), lambda: m.append(a, 11)),
        (lambda: s.append(a, n=19), lambda: m.append(a, 19)),
        (lambda: s.append(9, n=1), lambda: m.append(9, 1)),
        (lambda: s.append(a, n=-1), lambda: m.append(a, -1)),
        (lambda: s.span_mark(a, 2, 2, 5), lambda: m.span_mark(a, 2, 2, 5)),
        (lambda: s.span_mark(a, 0, 4, 5), lambda: m.span_mark(a, 0, 4, 5)),
        (lambda: s.span_mark(a, 3, 10, 15), lambda: m.span_mark(a, 3, 10, 15)),
        (lambda: s.span_mark(a, -1, 4, 5), lambda: m.span_mark(a, -1, 4, 5)),
        (lambda: s.evict(a, [0, 5]), lambda: m.evict(a, [0, 5])),
        (lambda: s.fork(a, 15), lambda: m.fork(a, 15)),
        (lambda: s.fork(a, -1), lambda: m.fork(a, -1)),
        (lambda: s.release(7), lambda: m.release(7)),
    ]
    for fs, fm in cases:
        before = (s.page_table(a), s.refcounts().tolist(), s.spans(a), s.stats())
        _both(s, m, sq, fs, fm)
        assert before == (s.page_table(a), s.refcounts().tolist(), s.spans(a), s.stats())
    # pool exhaustion for an eviction: fill the pool, then ask for fresh pages
    b = s.fork(a, 13)
    m.fork(a, 13)
    s.append(b, n=4)
    m.append(b, 4)
    _compare(s, m)
    assert s.stats()["free_pages"] == 0
    s.span_mark(a, 9, 4, 6)
    m.span_mark(a, 9, 4, 6)
    before = (s.page_table(a), s.refcounts().tolist(), s.spans(a))
    with pytest.raises(sq.SqError) as ei:
        s.evict(a, [9])
    assert ei.value.code == sq.ERR_NO_PAGES
    with pytest.raises(pg.NoPages):
        m.evict(a, [9])
    assert before == (s.page_table(a), s.refcounts().tolist(), s.spans(a))


def test_attention_needs_a_device_store(sq):
    """Attention calls on a metadata-only store fail cleanly and change nothing."""
    import ctypes as C
    s = _store(sq, 8, 4, 2, 8)
    a = s.seq_create()
    s.append(a, n=6)
    before = (s.page_table(a), s.stats())
    rc = sq.lib().sq_extend_attn(s._handle, 0, a, 2, None, None, C.c_float(0.5), None)
    assert rc == sq.ERR_INVALID
    assert b"metadata-only" in sq.lib().sq_last_error()
    seqs = (C.c_int32 * 1)(a)
    rc = sq.lib().sq_decode_attn(s._handle, 0, seqs, 1, None, None, C.c_float(0.5), 0, None)
    assert rc == sq.ERR_INVALID
    assert before == (s.page_table(a), s.stats())


def test_deferred_run_limit(sq):
    """A deferred eviction that would leave more than SQ_MAX_EVICT_SPANS
    masked runs fails and changes nothing; compaction then removes them."""
    s = _store(sq, 3300, 16, 2, 2200)
    a = s.seq_create()
    s.append(a, n=2 * sq.MAX_EVICT_SPANS + 8)
    for c in range(sq.MAX_EVICT_SPANS + 1):
        s.span_mark(a, c, 2 * c + 1, 2 * c + 2)
    st = s.evict(a, list(range(sq.MAX_EVICT_SPANS)), deferred=True)
    assert st["tokens_masked"] == sq.MAX_EVICT_SPANS and st["first_evicted"] == 1
    before = (s.keep_flags(a).tolist(), s.spans(a), s.seq_info(a))
    with pytest.raises(sq.SqError) as ei:
        s.evict(a, [sq.MAX_EVICT_SPANS], deferred=True)
    assert ei.value.code == sq.ERR_INVALID
    assert before == (s.keep_flags(a).tolist(), s.spans(a), s.seq_info(a))
    st = s.compact(a)
    assert st["tokens_removed"] == sq.MAX_EVICT_SPANS
    assert s.spans(a) == {sq.MAX_EVICT_SPANS: (sq.MAX_EVICT_SPANS + 1, sq.MAX_EVICT_SPANS + 2)}


def test_new_entry_point_errors(sq):
    """Deferred eviction, compaction, keep flags and 8-bit configurations
    reject bad arguments without changing anything."""
    import ctypes as C
    s = _store(sq, 16, 4, 2, 8)
    a = s.seq_create()
    s.append(a, n=10)
    s.span_mark(a, 0, 2, 5)
    before = (s.page_table(a), s.spans(a), s.keep_flags(a).tolist(), s.stats())
    es = sq.EvictStats()
    ids = (C.c_int32 * 1)(0)
    assert sq.lib().sq_evict_spans_ex(s._handle, a, ids, 1, 2, None, C.byref(es)) == sq.ERR_INVALID
    assert b"flags" in sq.lib().sq_last_error()
    bad = (C.c_int32 * 1)(7)
    assert sq.lib().sq_evict_spans_ex(s._handle, a, bad, 1, sq.EVICT_DEFER, None,
                                      C.byref(es)) == sq.ERR_UNKNOWN_CURSOR
    assert sq.lib().sq_compact(s._handle, 9, None, C.byref(es)) == sq.ERR_UNKNOWN_SEQ
    n = C.c_int64()
    assert sq.lib().sq_keep_flags(s._handle, a, None, 4, C.byref(n)) == sq.ERR_INVALID
    assert sq.lib().sq_keep_flags(s._handle, 9, None, 0, C.byref(n)) == sq.ERR_UNKNOWN_SEQ
    assert before == (s.page_table(a), s.spans(a), s.keep_flags(a).tolist(), s.stats())
    st = s.compact(a)                      # nothing masked: nothing to do
    assert st["tokens_removed"] == 0 and s.page_table(a) == before[0]
    # an 8-bit store needs finite positive scales (checked in every mode)
    cfg = sq.StoreConfig(2, 4, 2, 8, 4, 16, 2, 8)
    cfg.flags = sq.STORE_METADATA_ONLY | sq.STORE_KV_FP8
    h = C.c_void_p()
    assert sq.lib().sq_store_create(C.byref(cfg), C.byref(h)) == sq.ERR_INVALID  # no scales
    for vals in ([1.0, 1.0, 0.0, 1.0], [1.0, float("inf"), 1.0, 1.0]):
        sc = (C.c_float * 4)(*vals)
        cfg.kv_scales = C.cast(sc, C.c_void_p)
        assert sq.lib().sq_store_create(C.byref(cfg), C.byref(h)) == sq.ERR_INVALID
    sc = (C.c_float * 4)(0.5, 0.25, 1.0, 2.0)
    cfg.kv_scales = C.cast(sc, C.c_void_p)
    assert sq.lib().sq_store_create(C.byref(cfg), C.byref(h)) == sq.OK
    assert sq.lib().sq_pool_bytes(C.byref(cfg), 0) == 2 * 16 * 2 * 4 * 8  # one byte per element
    sq.lib().sq_store_destroy(h)


def test_attention_options_are_checked_first(sq):
    """sq_attn_opts errors (negative window, reserved field, misaligned
    sinks) are reported before anything else and change nothing; a windowed
    step opens on a metadata-only store exactly like a plain one."""
    import ctypes as C
    s = _store(sq, 8, 4, 2, 8)
    a = s.seq_create()
    s.append(a, n=6)
    seqs = (C.c_int32 * 1)(a)
    before = (s.page_table(a), s.stats())
    for window, reserved, sinks, what in ((-1, 0, None, b"window"), (0, 1, None, b"reserved"),
                                          (4, 0, 6, b"aligned")):
        o = sq.AttnOpts()
        o.window, o.reserved, o.sinks = window, reserved, sinks
        rc = sq.lib().sq_decode_attn_ex(s._handle, 0, seqs, 1, None, None, C.c_float(0.5), 0,
                                        C.byref(o), None)
        assert rc == sq.ERR_INVALID and what in sq.lib().sq_last_error()
        rc = sq.lib().sq_extend_attn_ex(s._handle, 0, a, 2, None, None, C.c_float(0.5),
                                        C.byref(o), None)
        assert rc == sq.ERR_INVALID and what in sq.lib().sq_last_error()
        rc = sq.lib().sq_step_attn_ex(s._handle, 0, None, None, None, None, C.c_float(0.5),
                                      C.byref(o), None)
        assert rc == sq.ERR_INVALID and what in sq.lib().sq_last_error()
    assert sq.lib().sq_step_begin_ex(s._handle, seqs, 1, 0, -2, None) == sq.ERR_INVALID
    assert before == (s.page_table(a), s.stats())
    s.step_begin([a], window=3)
    assert s.seq_info(a)["length"] == 7


def test_decode_step_metadata(sq):
    """sq_step_begin opens one token slot per sequence exactly as
    sq_append_batch appends one token (pages, positions, refcounts, stats);
    its errors change nothing; the layers need a device store."""
    import ctypes as C
    stores = [_store(sq, 8, 4, 4, 4) for _ in range(2)]   # 8 pages of 4 tokens, 16 per sequence
    for s in stores:
        a = s.seq_create()
        s.append(a, n=7)               # pages [0, 1]
        s.fork(a, 4)                   # aliases page 0
        s.seq_create()                 # an empty sequence
    stores[0].append_batch([0, 1, 2])
    stores[1].step_begin([0, 1, 2])
    for h in (0, 1, 2):
        assert stores[0].page_table(h) == stores[1].page_table(h)
        assert stores[0].positions(h).tolist() == stores[1].positions(h).tolist()
        assert stores[0].seq_info(h) == stores[1].seq_info(h)
    assert stores[1].page_table(1) == [0, 2] and stores[1].page_table(2) == [3]
    assert stores[0].refcounts().tolist() == stores[1].refcounts().tolist()
    assert stores[0].stats()["append_tokens"] == stores[1].stats()["append_tokens"]
    s = stores[1]
    snap = lambda: ([s.page_table(h) for h in (0, 1, 2)], s.refcounts().tolist(), s.stats())
    before = snap()
    for bad, code in (([0, 0], sq.ERR_INVALID), ([0, 9], sq.ERR_UNKNOWN_SEQ), ([], sq.ERR_INVALID)):
        with pytest.raises(sq.SqError) as ei:
            s.step_begin(bad)
        assert ei.value.code == code
        assert snap() == before
    s.append(2, n=3)                   # sequence 2 fills its page: its next step opens one
    s.append(1, n=11)                  # sequence 1 reaches its capacity (16 tokens, pages 4 and 5 added)
    before = snap()
    with pytest.raises(sq.SqError) as ei:
        s.step_begin([2, 1])
    assert ei.value.code == sq.ERR_INVALID and snap() == before
    d = s.seq_create()
    s.append(d, n=8)                   # takes the last two free pages
    assert s.stats()["free_pages"] == 0
    before = snap()
    with pytest.raises(sq.SqError) as ei:
        s.step_begin([2])
    assert ei.value.code == sq.ERR_NO_PAGES and snap() == before
    rc = sq.lib().sq_step_attn(s._handle, 0, None, None, None, None, C.c_float(0.5), None)
    assert rc == sq.ERR_INVALID and b"metadata-only" in sq.lib().sq_last_error()


def test_decode_plan_worst_case_segments(sq):
    """Segments 64 entries can need: every shared run splits into at least
    two parts, so n entries make at most 2n - 1 segments (127 for 64), below
    the 128 one decode call holds.  Eight binary trees of root -> 2 -> 4 -> 8
    forks (P = 4, G = 2: one tile takes all 8 leaves of a tree) make 15 per
    tree: one run of 8, two of 4, four of 2 and 8 private tails."""
    s = _store(sq, 4000, 4, 255, 64)
    leaves = []
    for _ in range(8):
        r = s.seq_create()
        s.append(r, n=8)
        for _ in range(2):
            m = s.fork(r, 8)
            s.append(m, n=4)
            for _ in range(2):
                x = s.fork(m, 12)
                s.append(x, n=4)
                for _ in range(2):
                    y = s.fork(x, 16)
                    s.append(y, n=1)
                    leaves.append(y)
    info = s.plan_info(leaves)
    assert info["n_segments"] == 120 and info["n_groups"] == 56
    assert info["kv_bytes"] < info["kv_bytes_logical"]


@pytest.mark.parametrize("group,members,read_once", [(1, 8, True), (2, 8, True), (4, 8, True),
                                                     (8, 8, False)])
def test_deep_and_wide_trees(sq, group, members, read_once):
    """A fork chain seven deep (each branch forked from the previous one,
    page-aligned or mid-page) and a fan-out of eight branches at one point:
    with 8 members per tile (16 / G rows per block, two blocks) each
    distinct page is read once; with G = 8 a tile holds four members and
    the wide runs are read once per tile."""
    P, tok = 16, 2 * 128 * 2 * 2
    s = sq.Store(1, 2 * group, 2, 128, num_pages=800, max_seqs=20, max_pages_per_seq=120,
                 metadata_only=True)

    def distinct(batch):
        full, partial = set(), 0
        for b in batch:
            L = s.seq_info(b)["length"]
            full.update(s.page_table(b)[: L // P])
            partial += L % P
        return (len(full) * P + partial) * tok

    m = s.seq_create()
    s.append(m, n=300)
    chain = [m]
    for d in range(members - 1):
        nxt = s.fork(chain[-1], s.seq_info(chain[-1])["length"] - (7 if d % 2 else 0))
        s.append(nxt, n=40)
        chain.append(nxt)
    a = s.seq_create()
    s.append(a, n=700)
    fan = [a]
    for i in range(members - 1):
        c = s.fork(a, 640 if i % 2 else 700)
        s.append(c, n=5 + 7 * i)
        fan.append(c)
    for batch in (chain, fan):
        info = s.plan_info(batch, sq.ATTN_AUTO)
        assert (info["kv_bytes"] == distinct(batch)) == read_once, (batch, info)
        assert info["kv_bytes"] < info["kv_bytes_logical"]
    # the deepest entry of the chain attends to every level
    info = s.plan_info(chain, sq.ATTN_AUTO)
    assert info["n_groups"] >= (members - 1 if read_once else 1)


def test_invalid_configurations(sq):
    with pytest.raises(sq.SqError):
        sq.Store(1, 3, 2, 8, 16, 2, 4, page_size=4, metadata_only=True)  # 3 % 2
    with pytest.raises(sq.SqError):
        sq.Store(1, 4, 1, 8, 0, 2, 4, page_size=4, metadata_only=True)
    cfg = sq.StoreConfig(1, 4, 1, 96, 16, 64, 2, 8)  # head_dim 96: no device kernels
    assert sq.lib().sq_workspace_bytes(cfg) == 0
    cfg = sq.StoreConfig(1, 4, 1, 64, 8, 64, 2, 8)   # page size 8: device needs 16
    assert sq.lib().sq_workspace_bytes(cfg) == 0
    cfg = sq.StoreConfig(1, 4, 1, 64, 16, 64, 2, 8)
    assert sq.lib().sq_workspace_bytes(cfg) > 0


def test_decode_plan_shared_prefix_bytes(sq):
    """Eight tasks at 128K: main + auxiliary share their first 8176 pages; the
    shared-prefix plan reads each shared page once."""
    tasks, main_len, fork_at, aux = 8, 131072, 130816, 512
    per_task_pages = main_len // 16 + aux // 16
    s = sq.Store(1, 32, 8, 128, num_pages=tasks * per_task_pages + 64, max_seqs=32,
                 max_pages_per_seq=main_len // 16 + 64, page_size=16, metadata_only=True)
    batch = []
    for _ in range(tasks):
        m = s.seq_create()
        s.append(m, n=fork_at)
        a = s.fork(m, fork_at)
        s.append(m, n=main_len - fork_at)
        s.append(a, n=aux)
        batch += [m, a]
    tok = 8 * 128 * 2 * 2
    info = s.plan_info(batch, sq.ATTN_AUTO)
    assert info["n_groups"] == tasks
    assert info["kv_bytes"] == tasks * (main_len + aux) * tok == 4_311_744_512
    assert info["kv_bytes_logical"] == tasks * (main_len + fork_at + aux) * tok == 8_598_323_200
    stream = s.plan_info(batch, sq.ATTN_STREAM)
    assert stream["n_groups"] == 0 and stream["n_items_mfma"] == 0
    assert stream["kv_bytes"] == stream["kv_bytes_logical"] == info["kv_bytes_logical"]
    assert info["n_items_valu"] + info["n_items_mfma"] <= 16384
    mf = s.plan_info(batch, sq.ATTN_MFMA)
    assert mf["n_items_valu"] == 0 and mf["kv_bytes"] == info["kv_bytes_logical"]
    assert math.isclose(info["kv_bytes"] / info["kv_bytes_logical"], 0.5014, rel_tol=1e-3)


def test_decode_plan_after_eviction(sq):
    """After the main thread evicts, main and auxiliary share only the pages
    before the first evicted one."""
    s = sq.Store(1, 32, 8, 128, num_pages=400, max_seqs=4, max_pages_per_seq=200,
                 page_size=16, metadata_only=True)
    m = s.seq_create()
    s.append(m, n=1000)
    a = s.fork(m, 1000)
    s.span_mark(m, 0, 330, 500)
    s.evict(m, [0])
    pt_m, pt_a = s.page_table(m), s.page_table(a)
    assert pt_m[:20] == pt_a[:20] and pt_m[20] != pt_a[20]
    info = s.plan_info([m, a], sq.ATTN_AUTO)
    tok = 8 * 128 * 2 * 2
    assert info["n_groups"] == 1
    assert info["kv_bytes"] == (20 * 16 + (830 - 320) + (1000 - 320)) * tok


def test_decode_plan_reads_a_tree_of_shared_runs_once(sq):
    """M (1000 tokens); A forked from M at 640 (+200); B forked from A at
    800 (+100); C forked from M at 960 (+20).  All four share pages [0, 40),
    M and C share [40, 60), A and B share [40, 50): three shared runs, four
    own suffixes, 1320 tokens read instead of 3720 (or 1800 with one level)."""
    s = sq.Store(1, 8, 2, 128, num_pages=400, max_seqs=12, max_pages_per_seq=100,
                 metadata_only=True)
    m = s.seq_create()
    s.append(m, n=1000)
    a = s.fork(m, 640)
    s.append(a, n=200)
    b = s.fork(a, 800)
    s.append(b, n=100)
    c = s.fork(m, 960)
    s.append(c, n=20)
    tok = 2 * 128 * 2 * 2
    for mode in (sq.ATTN_AUTO, sq.ATTN_SHARED_PREFIX):
        info = s.plan_info([m, a, b, c], mode)
        assert (info["n_segments"], info["n_groups"]) == (7, 3)
        assert info["kv_bytes"] == 1320 * tok and info["kv_bytes_logical"] == 3720 * tok
    info = s.plan_info([m, a, b, c], sq.ATTN_STREAM)
    assert (info["n_segments"], info["n_groups"], info["kv_bytes"]) == (4, 0, 3720 * tok)
    # a chain of six nested forks: one tile holds all six entries (two
    # 16-row blocks when G = 4), so the runs nest five deep and each page is
    # read once: M's 1000 tokens, 40 private tokens per child, and the 8
    # tokens each of the three mid-page forks (at 1000, 1080, 1160) copied
    # into its own tail page
    chain = [m]
    for i in range(5):
        nxt = s.fork(chain[-1], s.seq_info(chain[-1])["length"])
        s.append(nxt, n=40)
        chain.append(nxt)
    info = s.plan_info(chain, sq.ATTN_AUTO)
    assert info["n_groups"] == 5 and info["kv_bytes"] == (1000 + 5 * 40 + 3 * 8) * tok


@pytest.mark.parametrize("seed", range(6))
def test_tree_plan_reads_every_distinct_page_once(sq, seed):
    """Random forests of forks, appends and evictions (metadata only): for
    any batch of at most eight entries (one tile of two 16-row blocks when
    G = 4) the shared-prefix plan reads each distinct page once; the count
    comes from the page tables alone: P tokens per distinct full page plus
    each entry's partial last page."""
    rng = np.random.default_rng(1000 + seed)
    P, tok = 16, 2 * 128 * 2 * 2
    s = sq.Store(1, 8, 2, 128, num_pages=3000, max_seqs=16, max_pages_per_seq=400,
                 metadata_only=True)
    live = [s.seq_create()]
    s.append(live[0], n=int(rng.integers(100, 2000)))
    cursor = 0
    for _ in range(40):
        h = live[int(rng.integers(0, len(live)))]
        op = rng.random()
        L = s.seq_info(h)["length"]
        if op < 0.35 and len(live) < 12:
            live.append(s.fork(h, int(rng.integers(0, L + 1))))
        elif op < 0.7:
            s.append(h, n=int(rng.integers(1, 300)))
        elif op < 0.85 and L > 2:
            a0 = int(rng.integers(0, L - 1))
            a1 = int(rng.integers(a0 + 1, L + 1))
            try:
                s.span_mark(h, cursor, a0, a1)
                s.evict(h, [cursor])
            except sq.SqError:
                pass
            cursor += 1
        elif len(live) > 2:
            s.release(h)
            live.remove(h)
        for _ in range(3):
            k = int(rng.integers(1, min(8, len(live)) + 1))
            batch = [live[i] for i in rng.choice(len(live), k, replace=False)]
            full = set()
            partial = 0
            for b in batch:
                L = s.seq_info(b)["length"]
                full.update(s.page_table(b)[: L // P])
                partial += L % P
            info = s.plan_info(batch, sq.ATTN_AUTO)
            assert info["kv_bytes"] == (len(full) * P + partial) * tok, (batch, info)


def test_host_call_trace(sq, tmp_path):
    """sq_trace_open: one line per state-changing call, in call order, with
    its arguments, host time and outcome; nothing once closed."""
    path = tmp_path / "trace.log"
    sq.trace_open(path)
    try:
        s = _store(sq, 40, 4, 4, 20)
        a = s.seq_create()
        s.append(a, n=30)
        s.span_mark(a, 7, 4, 12)
        b = s.fork(a, 16)
        with pytest.raises(sq.SqError):
            s.evict(a, [99])                     # unknown cursor: a failed call
        s.evict(a, [7])
        s.release(b)
        s.page_table(a)                          # introspection is not traced
    finally:
        sq.trace_open(None)
    s.append(a, n=1)                             # after the trace closed
    lines = path.read_text().splitlines()
    calls = [re.match(r"sq (\w+)\(", l).group(1) for l in lines]
    assert calls == ["sq_store_create", "sq_seq_create", "sq_append", "sq_span_mark", "sq_fork",
                     "sq_evict_spans", "sq_evict_spans", "sq_release"]
    assert "seq=0 n=30" in lines[2] and "cursor=7 start=4 end=12" in lines[3]
    assert "parent=0 fork_len=16" in lines[4]
    assert lines[5].split("host_us=")[1].split()[1] == "error:" and "99" in lines[5]
    for l in lines[:5] + lines[6:]:
        assert l.endswith(" ok"), l
        assert float(l.split("host_us=")[1].split()[0]) >= 0.0
    with pytest.raises(sq.SqError):
        sq.trace_open(tmp_path / "no_such_dir" / "trace.log")


def test_host_call_trace_from_environment(tmp_path):
    """SQ_TRACE names the trace file when the library loads."""
    import subprocess
    import sys
    path = tmp_path / "env_trace.log"
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2602_22603_amd import sq\n"
            "s = sq.Store(1, 4, 2, 8, num_pages=8, max_seqs=2, max_pages_per_seq=8,"
            " page_size=4, metadata_only=True)\n"
            "s.append(s.seq_create(), n=5)\n") % ROOT
    env = dict(os.environ, SQ_TRACE=str(path))
    subprocess.run([sys.executable, "-c", code], check=True, env=env, timeout=120)
    calls = [re.match(r"sq (\w+)\(", l).group(1) for l in path.read_text().splitlines()]
    assert calls[:3] == ["sq_store_create", "sq_seq_create", "sq_append"]
