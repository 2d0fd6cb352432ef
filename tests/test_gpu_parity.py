"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Indexing (page tables, K/V/pos views, keep / dst / src_of) must match bit for
bit; fp32 attention outputs from bf16 K/V must be within 5e-4 (max abs) of
the oracle's float64 result.
"""

import math

import numpy as np
import pytest

from tests import scenarios as sc
from oracle import attention as oatt
from oracle import evict as oev
from paper_2602_22603_amd import workload as wl

pytestmark = pytest.mark.gpu
TOL = 5e-4


@pytest.fixture(scope="module")
def sq():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2602_22603_amd import sq as sqmod
    sqmod.lib()  # raises if libsq.so is missing
    return sqmod


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    import gc
    import torch
    gc.collect()
    if torch.cuda.is_available():
        torch.cuda.empty_cache()


def test_tiny_end_to_end(sq):
    res = sc.run_tiny(sq)
    errs = sc.check_tiny(res)
    print("tiny max abs error per mode:", errs)


@pytest.mark.parametrize("head_dim,group", [(64, 4), (128, 4), (128, 1), (64, 8), (128, 2)])
def test_single_key_returns_v_exactly(sq, head_dim, group):
    hkv = 2
    t = sc.Twin(sq, 1, hkv * group, hkv, head_dim, 32, 4, 8, seed=head_dim + group)
    a = t.create()
    t.append(a, 1)
    errs, ref = t.decode_errors([a])
    _, v, _ = t.model.view(a)
    for m, e in errs.items():
        assert e == 0.0, (m, e)
    for h in range(hkv * group):
        assert np.array_equal(ref[0, h], v[0, 0, h // group])


@pytest.mark.parametrize("n", [1, 15, 16, 17, 333, 4099])
def test_values_one_give_one(sq, n):
    t = sc.Twin(sq, 1, 32, 8, 128, 2 * (n // 16 + 2) + 8, 4, n // 16 + 4, seed=n)
    a = t.create()
    t.append(a, n, const_v=1.0)
    b = t.fork(a, n - n % 16)
    t.append(b, 5, const_v=1.0)
    import torch
    q = wl.to_torch_bf16(wl.normal_bf16(t.rng, (2, 32, 128)), "cuda")
    for m in (sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA):
        out = t.store.decode(0, [a, b], q, mode=m)
        torch.cuda.synchronize()
        assert float((out - 1.0).abs().max()) <= 1e-6, m


@pytest.mark.parametrize("nl,hq,hkv,d", [(1, 2, 2, 64), (2, 4, 1, 64), (1, 8, 4, 128),
                                         (1, 32, 8, 128), (2, 16, 2, 128), (1, 8, 1, 64)])
def test_random_shapes_with_forks(sq, nl, hq, hkv, d):
    t = sc.Twin(sq, nl, hq, hkv, d, 1200, 12, 300, seed=hq * 7 + d)
    seqs = []
    for n in (1, 15, 16, 17, 100, 1000, 4099):
        a = t.create()
        t.append(a, n)
        seqs.append(a)
    f1 = t.fork(seqs[5], 992)   # aligned fork of a 1000-token sequence
    t.append(f1, 40)
    f2 = t.fork(seqs[6], 4001)  # unaligned: tail page copied
    t.append(f2, 7)
    t.append(seqs[6], 3)
    f3 = t.fork(seqs[6], 4099)
    seqs += [f1, f2, f3]
    t.check_state()
    for layer in range(nl):
        errs, _ = t.decode_errors(seqs, layer=layer)
        print((nl, hq, hkv, d, layer), errs)
        for m, e in errs.items():
            assert e <= TOL, (m, e)


@pytest.mark.parametrize("chunk", [0, 1, 7])
def test_eviction_random_bitexact(sq, chunk):
    t = sc.Twin(sq, 2, 8, 2, 64, 900, 8, 200, seed=11, evict_chunk_pages=chunk)
    rng = np.random.default_rng(5)
    main = t.create()
    t.append(main, 1500)
    aux = t.fork(main, 1200)
    t.append(aux, 50)
    cursor = 0
    for rnd in range(6):
        length = t.model.info(main)["length"]
        cuts = sorted(rng.choice(np.arange(length + 1), 8, replace=False).tolist())
        ids = []
        for i in range(0, 8, 2):
            if t.try_mark(main, cursor, cuts[i], cuts[i + 1]) and rng.random() < 0.7:
                ids.append(cursor)
            cursor += 1
        spans = sorted(t.model.spans(main)[c] for c in ids)
        st = t.evict(main, ids)
        if st["tokens_removed"]:
            keep, dst, src_of = t.store.debug_last_evict()
            okeep, odst, osrc, n_kept, first = oev.plan(length, spans)
            assert np.array_equal(keep, okeep) and np.array_equal(dst, odst)
            assert np.array_equal(src_of, osrc) and st["first_evicted"] == first
        t.check_state()
        t.append(main, int(rng.integers(1, 40)))
        errs, _ = t.decode_errors([main, aux], layer=rnd % 2)
        assert max(errs.values()) <= TOL, errs
    # evict everything but one token, then everything
    t.evict(main, list(t.model.spans(main)))
    length = t.model.info(main)["length"]
    t.mark(main, 1000, 1, length)
    t.evict(main, [1000])
    t.check_state()
    errs, _ = t.decode_errors([main, aux])
    assert max(errs.values()) <= TOL
    t.mark(main, 1001, 0, 1)
    t.evict(main, [1001])
    assert t.model.info(main)["length"] == 0
    t.check_state()
    import torch
    out = t.store.decode(0, [main], wl.to_torch_bf16(wl.normal_bf16(rng, (1, 8, 64)), "cuda"))
    torch.cuda.synchronize()
    assert float(out.abs().max()) == 0.0
    t.append(main, 20)
    t.check_state()
    errs, _ = t.decode_errors([main, aux])
    assert max(errs.values()) <= TOL


@pytest.mark.parametrize("chunk", [1, 4, 32])
def test_chunked_eviction_recycles_pages_bitexact(sq, chunk):
    """With no other branch holding the pages, chunked eviction reuses old
    pages of the sequence inside the same call; the compacted K/V/pos must
    still equal the oracle's bit for bit, and the peak stays within chunk."""
    t = sc.Twin(sq, 3, 8, 2, 128, 420, 4, 400, seed=21 + chunk, evict_chunk_pages=chunk)
    rng = np.random.default_rng(chunk)
    main = t.create()
    t.append(main, 3000)
    aux = t.fork(main, 2995)
    t.append(aux, 40)
    t.release(aux)                        # Phase 1: the auxiliary thread is done
    cursor = 0
    for rnd in range(4):
        length = t.model.info(main)["length"]
        cuts = sorted(rng.choice(np.arange(length + 1), 12, replace=False).tolist())
        ids = []
        for i in range(0, 12, 2):
            if t.try_mark(main, cursor, cuts[i], cuts[i + 1]):
                ids.append(cursor)
            cursor += 1
        before = t.store.stats()["live_pages"]
        t.evict(main, ids)
        assert t.store.stats()["peak_pages"] == t.model.peak_pages
        t.check_state()
        errs, _ = t.decode_errors([main], layer=rnd % 3)
        assert max(errs.values()) <= TOL, errs
        t.append(main, int(rng.integers(100, 400)))
        assert before > 0


@pytest.mark.parametrize("chunk", [0, 2])
def test_remap_eviction_bitexact(sq, chunk):
    """Page-aligned remap: spans of whole pages (and some ragged ones) evicted
    from a main thread whose auxiliary fork is still alive; tail pages that
    are one old page in order are taken by reference, the rest gathered.
    Page tables, refcounts and the K/V/pos views equal the oracle's remap
    mode bit for bit; decode matches the oracle; forks and decode steps of
    the result too."""
    t = sc.Twin(sq, 2, 8, 2, 128, 700, 6, 200, seed=31 + chunk, evict_chunk_pages=chunk,
                evict_remap=True)
    rng = np.random.default_rng(31)
    main = t.create()
    t.append(main, 2000)
    aux = t.fork(main, 1600)
    t.append(aux, 21)
    cursor, remapped = 0, 0
    for rnd in range(5):
        length = t.model.info(main)["length"]
        cuts = sorted(rng.choice(np.arange(length // 16), 8, replace=False).tolist())
        ids = []
        for i in range(0, 8, 2):
            s0, e0 = 16 * cuts[i], 16 * cuts[i + 1]
            if i == 6 and rnd % 2:
                e0 -= 5                  # one ragged span per odd round
            if t.try_mark(main, cursor, s0, e0):
                ids.append(cursor)
            cursor += 1
        st = t.evict(main, ids)
        remapped += st["pages_remapped"]
        t.check_state()
        errs, _ = t.decode_errors([main, aux], layer=rnd % 2)
        assert max(errs.values()) <= TOL, errs
        t.append(main, 16 * int(rng.integers(1, 6)))
        err, _ = t.step([main, aux])
        assert err <= TOL
    assert remapped > 0
    c = t.fork(main, 160)              # a fork of remapped pages
    t.append(c, 9)
    t.check_state()
    errs, _ = t.decode_errors([main, aux, c])
    assert max(errs.values()) <= TOL, errs


def test_all_keep_eviction_leaves_bytes(sq):
    import torch
    t = sc.Twin(sq, 1, 4, 1, 64, 64, 4, 32, seed=3)
    a = t.create()
    t.append(a, 300)
    t.mark(a, 0, 10, 10)
    t.mark(a, 1, 40, 40)
    torch.cuda.synchronize()
    snap = [x.clone() for x in (t.store.k_pool, t.store.v_pool, t.store.pos_pool)]
    st0 = t.store.stats()
    for ids in ([], [0], [1, 1]):
        es = t.evict(a, ids)
        assert es["tokens_removed"] == 0 and es["pages_allocated"] == 0
    torch.cuda.synchronize()
    for x, y in zip(snap, (t.store.k_pool, t.store.v_pool, t.store.pos_pool)):
        assert torch.equal(x, y)
    st1 = t.store.stats()
    assert st0 == st1


def test_fork_zero_copy_and_tail_copy(sq):
    import torch
    t = sc.Twin(sq, 2, 8, 2, 128, 64, 4, 32, seed=4)
    a = t.create()
    t.append(a, 200)
    torch.cuda.synchronize()
    snap = t.store.k_pool.clone(), t.store.v_pool.clone()
    live = t.store.stats()["live_pages"]
    b = t.fork(a, 192)
    torch.cuda.synchronize()
    assert t.store.stats()["live_pages"] == live
    assert torch.equal(snap[0], t.store.k_pool) and torch.equal(snap[1], t.store.v_pool)
    c = t.fork(a, 199)
    assert t.store.stats()["live_pages"] == live + 1
    t.check_state()
    t.append(c, 9)
    t.append(b, 3)
    t.check_state()
    t.release(b)
    t.release(c)
    assert t.store.stats()["live_pages"] == live


def test_compacted_equals_masked_every_subset(sq):
    """Attention over the GPU-compacted cache against the oracle's masked
    attention over the uncompacted cache, for all 64 subsets of 6 spans."""
    import itertools
    import torch
    t = sc.Twin(sq, 1, 4, 1, 64, 80, 4, 8, seed=6)
    base = t.create()
    t.append(base, 64)
    rng = np.random.default_rng(6)
    cuts = sorted(rng.choice(np.arange(65), 12, replace=False).tolist())
    spans = [(cuts[i], cuts[i + 1]) for i in range(0, 12, 2)]
    for c, (s, e) in enumerate(spans):
        t.mark(base, c, s, e)
    k, v, _ = t.model.view(base)
    qb = wl.normal_bf16(rng, (1, 4, 64))
    q = wl.to_torch_bf16(qb, "cuda")
    qf = wl.bf16_value(qb)[0]
    worst = 0.0
    for r in range(7):
        for subset in itertools.combinations(range(6), r):
            f = t.fork(base, 64)
            t.evict(f, list(subset))
            keep = oev.keep_mask(64, [spans[c] for c in subset])
            want = oatt.masked_attention(qf, k[:, 0], v[:, 0], keep, 0.125, 4)
            for m in (sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA):
                out = t.store.decode(0, [f], q, scale=0.125, mode=m)
                torch.cuda.synchronize()
                worst = max(worst, sc.max_abs(out.cpu().numpy()[0], want))
            t.release(f)
    t.check_state()
    assert worst <= TOL, worst


def test_decode_is_deterministic(sq):
    import torch
    t = sc.Twin(sq, 1, 32, 8, 128, 600, 4, 300, seed=8)
    a = t.create()
    t.append(a, 3000)
    b = t.fork(a, 2992)
    t.append(b, 77)
    q = wl.to_torch_bf16(wl.normal_bf16(t.rng, (2, 32, 128)), "cuda")
    for m in (sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_MFMA):
        outs = [t.store.decode(0, [a, b], q, mode=m).clone() for _ in range(5)]
        torch.cuda.synchronize()
        for o in outs[1:]:
            assert torch.equal(o, outs[0]), m


def test_append_batch_matches_appends(sq):
    t = sc.Twin(sq, 2, 8, 2, 64, 200, 6, 40, seed=9)
    seqs = [t.create() for _ in range(3)]
    for h, n in zip(seqs, (15, 16, 40)):
        t.append(h, n)
    kb = wl.normal_bf16(t.rng, (2, 3, 2, 64))
    vb = wl.normal_bf16(t.rng, (2, 3, 2, 64))
    t.store.append_batch(seqs, wl.to_torch_bf16(kb, "cuda"), wl.to_torch_bf16(vb, "cuda"))
    for i, h in enumerate(seqs):
        t.model.append(h, 1, wl.bf16_value(kb[:, i:i + 1]), wl.bf16_value(vb[:, i:i + 1]))
    t.check_state()
    errs, _ = t.decode_errors(seqs, layer=1)
    assert max(errs.values()) <= TOL
