"""GPU parity of in-place eviction (the sequence's own tail pages rewritten,
no transient pages) through the C ABI: page tables, refcounts and the K/V/pos
pools bit for bit against the oracle's in-place mode, decode within 5e-4."""

import numpy as np
import pytest

from oracle import evict as oev
from paper_2602_22603_amd import workload as wl
from tests import scenarios as sc

pytestmark = pytest.mark.gpu
TOL = 5e-4


@pytest.fixture(scope="module")
def sq():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_22603_amd import sq as sqmod
    sqmod.lib()
    return sqmod


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    import gc
    import torch
    gc.collect()
    if torch.cuda.is_available():
        torch.cuda.empty_cache()


def _random_evictions(t, h, rng, rounds, n_cuts=8, others=()):
    cursor = 1000 * (h + 1)
    for rnd in range(rounds):
        length = t.model.info(h)["length"]
        if length < n_cuts + 1:
            t.append(h, 64)
            length = t.model.info(h)["length"]
        cuts = sorted(rng.choice(np.arange(length + 1), n_cuts, replace=False).tolist())
        ids = []
        for i in range(0, n_cuts, 2):
            if t.try_mark(h, cursor, cuts[i], cuts[i + 1]) and rng.random() < 0.8:
                ids.append(cursor)
            cursor += 1
        spans = sorted(t.model.spans(h)[c] for c in ids)
        st = t.evict(h, ids)
        if st["tokens_removed"]:
            keep, dst, src_of = t.store.debug_last_evict()
            okeep, odst, osrc, _n, first = oev.plan(length, spans)
            assert np.array_equal(keep, okeep) and np.array_equal(dst, odst)
            assert np.array_equal(src_of, osrc) and st["first_evicted"] == first
        t.check_state()
        t.append(h, int(rng.integers(1, 40)))
        errs, _ = t.decode_errors([h, *others], layer=rnd % t.nl)
        assert max(errs.values()) <= TOL, errs


@pytest.mark.parametrize("hq,hkv,d", [(8, 2, 64), (32, 8, 128)])
def test_inplace_random_bitexact(sq, hq, hkv, d):
    """Random spans evicted in place from a main thread while a forked
    auxiliary thread still holds the prefix pages: the pages the branch
    holds are replaced by fresh ones, the rest rewritten where they are."""
    t = sc.Twin(sq, 2, hq, hkv, d, 700, 6, 220, seed=41 + d, evict_inplace=True)
    rng = np.random.default_rng(41)
    main = t.create()
    t.append(main, 2500)
    aux = t.fork(main, 1200)
    t.append(aux, 50)
    _random_evictions(t, main, rng, 5, others=(aux,))
    t.release(aux)
    _random_evictions(t, main, rng, 3)
    # evict everything but one token, then everything, then grow again
    t.evict(main, list(t.model.spans(main)))
    length = t.model.info(main)["length"]
    t.mark(main, 90000, 1, length)
    t.evict(main, [90000])
    t.check_state()
    t.mark(main, 90001, 0, 1)
    t.evict(main, [90001])
    assert t.model.info(main)["length"] == 0
    t.append(main, 37)
    t.check_state()
    errs, _ = t.decode_errors([main])
    assert max(errs.values()) <= TOL


def test_inplace_on_a_full_pool(sq):
    """Every page of the pool holds the sequence: in-place eviction takes no
    page and succeeds, several times in a row, with decode steps between."""
    pages = 3000 // 16 + 1
    t = sc.Twin(sq, 3, 16, 4, 128, pages, 2, pages, seed=51, evict_inplace=True)
    rng = np.random.default_rng(51)
    main = t.create()
    t.append(main, pages * 16)
    assert t.store.stats()["free_pages"] == 0
    cursor = 0
    for rnd in range(4):
        length = t.model.info(main)["length"]
        cuts = sorted(rng.choice(np.arange(length + 1), 6, replace=False).tolist())
        ids = []
        for i in range(0, 6, 2):
            if t.try_mark(main, cursor, cuts[i], cuts[i + 1]):
                ids.append(cursor)
            cursor += 1
        free = t.store.stats()["free_pages"]
        st = t.evict(main, ids)
        assert st["pages_allocated"] == 0
        assert t.store.stats()["peak_pages"] == pages
        assert t.store.stats()["free_pages"] == free + st["pages_freed"]
        t.check_state()
        err, _ = t.step([main])
        assert err <= TOL
        t.append(main, min(t.store.stats()["free_pages"] * 16, int(rng.integers(16, 200))))
        t.check_state()


@pytest.mark.parametrize("shift", [1, 5, 17, 300])
def test_inplace_short_runs_and_sweep(sq, shift):
    """A few tokens evicted near the front shift the rest by less than a
    page: every tail page reads the next one, so each run of pages rewritten
    in parallel is one page long and the first ones go to the in-order
    pass; larger shifts give longer runs."""
    t = sc.Twin(sq, 2, 8, 2, 64, 520, 2, 300, seed=61 + shift, evict_inplace=True)
    main = t.create()
    t.append(main, 4000)          # 250 pages: more runs than one call launches
    t.mark(main, 0, 3, 3 + shift)
    st = t.evict(main, [0])
    assert st["pages_allocated"] == 0 and st["tokens_moved"] == 4000 - shift
    t.check_state()
    errs, _ = t.decode_errors([main])
    assert max(errs.values()) <= TOL


def test_inplace_8bit_store(sq):
    """In-place eviction moves E4M3 codes bit for bit."""
    scales = np.array([[0.011, 0.0095], [0.02, 0.013]], dtype=np.float32)
    t = sc.Twin(sq, 2, 8, 2, 128, 500, 4, 240, seed=71, evict_inplace=True, kv_scales=scales)
    rng = np.random.default_rng(71)
    main = t.create()
    t.append(main, 3000)
    _random_evictions(t, main, rng, 3)


def test_inplace_compaction64k_full_size(sq):
    """The 64K compaction evicted in place: the page table is the old one's
    first pages, the compacted K/V/pos equal the kept input rows bit for
    bit, and no page is taken."""
    import torch
    from paper_2602_22603_amd import drivers
    store, base, w, k, v = drivers.build_compaction64k(evict_inplace=True)
    L = w.length
    old = store.page_table(base)
    live = store.stats()["live_pages"]
    st = store.evict(base, w.evict_ids)
    spans = [w.spans[c] for c in w.evict_ids]
    keep, _dst, _src, n_kept, first = oev.plan(L, spans)
    assert st["pages_allocated"] == 0 and st["first_evicted"] == first
    n_pages = -(-n_kept // 16)
    assert store.page_table(base) == old[:n_pages]
    assert store.stats()["peak_pages"] == live
    assert store.stats()["live_pages"] == n_pages
    keep_t = torch.from_numpy(keep.astype(bool)).to("cuda")
    vk, vv, vp = sc.seq_view(store, base)
    assert np.array_equal(vk[:, 0], wl.torch_bf16_to_f64(k[0][keep_t]))
    assert np.array_equal(vv[:, 0], wl.torch_bf16_to_f64(v[0][keep_t]))
    assert np.array_equal(vp, np.flatnonzero(keep))
    store.close()
