"""GPU parity of deferred eviction (sq_evict_spans_ex with SQ_EVICT_DEFER,
then sq_compact or a later physical eviction) through the C ABI against the
oracle's page model: attention over a sequence with masked slots equals the
oracle's attention over its kept slots (decode in every mode, the fused
step, extend; max abs error <= 5e-4), the pools and page tables are left
untouched by the deferred call and equal the oracle's bit for bit after the
compaction."""

import math

import numpy as np
import pytest

from oracle import extend as oex
from tests import scenarios as sc
from paper_2602_22603_amd import workload as wl

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


def _task(t, spans):
    """A main thread with tool spans marked (cursor ids 0..), and an
    auxiliary branch forked before the deferred eviction."""
    main = t.create()
    t.append(main, 900)
    for c, (s, e) in enumerate(spans):
        t.mark(main, c, s, e)
    aux = t.fork(main, 880)
    t.append(aux, 21)
    return main, aux


SPANS = [(3, 9), (40, 100), (128, 160), (161, 163), (300, 517), (700, 701), (850, 880)]


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (8, 2, 64), (64, 8, 64), (4, 4, 128)])
def test_deferred_decode_then_compact(sq, hq, hkv, d):
    """Mask five tool spans (whole pages, page-crossing and one-token spans)
    on the main thread while its auxiliary branch is alive: nothing moves,
    every mode attends to the kept slots; the branch is untouched; then the
    compaction's pools equal the oracle's bit for bit and attention agrees
    again."""
    t = sc.Twin(sq, 2, hq, hkv, d, 400, 6, 80, seed=600 + hq + d)
    main, aux = _task(t, SPANS)
    pt_before = t.store.page_table(main)
    st = t.evict(main, [0, 1, 2, 4, 5], deferred=True)
    assert st["tokens_masked"] == 6 + 60 + 32 + 217 + 1
    assert t.store.page_table(main) == pt_before
    t.check_state()
    for layer in (0, 1):
        errs, _ = t.decode_errors([main, aux], layer=layer)
        assert max(errs.values()) <= TOL, (layer, errs)
    errs, _ = t.decode_errors([main])
    assert max(errs.values()) <= TOL, errs
    t.compact(main)
    t.check_state()
    errs, _ = t.decode_errors([main, aux])
    assert max(errs.values()) <= TOL, errs


def test_deferred_fork_shares_masks_and_pages(sq):
    """A branch forked after the deferred eviction inherits the masks: main
    and branch still share their pages (read once, masks equal), and a second
    branch forked before it does not (its pages are the same, its masks are
    not): all three in one batch."""
    t = sc.Twin(sq, 1, 32, 8, 128, 400, 6, 80, seed=610)
    main, early = _task(t, SPANS)
    t.evict(main, [1, 4], deferred=True)
    late = t.fork(main, 896)
    t.append(late, 40)
    mid = t.fork(main, 310)            # mid-page, inside the masked span [300, 517)
    t.append(mid, 9)
    assert t.store.keep_flags(mid).tolist()[300:310] == [0] * 10
    t.check_state()
    for _ in range(2):
        errs, _ = t.decode_errors([main, early, late, mid])
        assert max(errs.values()) <= TOL, errs
    plan = t.store.plan_info([main, late], t.sq.ATTN_AUTO)
    assert plan["n_groups"] >= 1
    assert t.store.seq_info(late)["n_masked"] == t.store.seq_info(main)["n_masked"]


def test_deferred_then_immediate_eviction_takes_the_union(sq):
    """A physical eviction of other spans also removes the masked slots, and
    a span marked over masked slots is fine."""
    t = sc.Twin(sq, 1, 8, 2, 128, 400, 6, 80, seed=611)
    main, aux = _task(t, SPANS)
    t.evict(main, [0, 2], deferred=True)
    t.mark(main, 20, 140, 161)        # over masked slots 140..159
    st = t.evict(main, [3, 20])
    assert t.store.seq_info(main)["n_masked"] == 0
    assert st["tokens_removed"] == 6 + (163 - 128)  # the union: [3, 9) and [128, 163)
    t.check_state()
    errs, _ = t.decode_errors([main, aux])
    assert max(errs.values()) <= TOL, errs


@pytest.mark.parametrize("mi", [0, 1, 2, 3])
def test_deferred_steps(sq, mi):
    """Fused decode steps over masked sequences in every mode, a deferred
    eviction between steps, then compaction between steps."""
    mode = [sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA][mi]
    t = sc.Twin(sq, 2, 32, 8, 128, 400, 6, 80, seed=620 + mi)
    main, aux = _task(t, SPANS)
    other = t.create()
    t.append(other, 47)
    seqs = [main, aux, other]
    t.evict(main, [0, 4], deferred=True)
    for r in range(12):
        err, _ = t.step(seqs, mode)
        assert err <= TOL, (r, err)
        if r == 4:
            t.evict(main, [1, 6], deferred=True)
        if r == 8:
            t.compact(main)
    t.check_state()


def test_captured_step_replays_across_deferred_eviction(sq):
    """A step captured before any slot is masked replays correctly after a
    deferred eviction (the step kernels read the plan's mask flag) and after
    the compaction."""
    import torch
    nl, hq, hkv, d = 2, 8, 2, 128
    t = sc.Twin(sq, nl, hq, hkv, d, 400, 6, 80, seed=630)
    main, aux = _task(t, SPANS)
    seqs = [main, aux]
    err, _ = t.step(seqs)
    assert err <= TOL
    g = dict(k=torch.zeros((nl, 2, hkv, d), dtype=torch.bfloat16, device="cuda"),
             v=torch.zeros((nl, 2, hkv, d), dtype=torch.bfloat16, device="cuda"),
             q=torch.zeros((nl, 2, hq, d), dtype=torch.bfloat16, device="cuda"),
             out=[torch.zeros((2, hq, d), dtype=torch.float32, device="cuda") for _ in range(nl)],
             graph=torch.cuda.CUDAGraph())
    with torch.cuda.graph(g["graph"]):
        for l in range(nl):
            t.store.step_attn(l, g["k"][l], g["v"][l], g["q"][l], out=g["out"][l])
    for r in range(7):
        err, _ = t.step(seqs, graph=g)
        assert err <= TOL, (r, err)
        if r == 1:
            t.evict(main, [1, 2, 4], deferred=True)
        if r == 4:
            t.compact(main)
    t.check_state()


def test_masked_plan_cleans_reused_rows(sq):
    """A sequence handle released with masks and reused by an unmasked
    sequence: a batch with another masked sequence reads its keep-mask row,
    which must then hold no old masks."""
    t = sc.Twin(sq, 1, 8, 2, 64, 300, 4, 80, seed=640)
    a = t.create()
    t.append(a, 600)
    t.mark(a, 0, 0, 320)
    t.evict(a, [0], deferred=True)
    t.release(a)
    b = t.create()                    # reuses handle a
    assert b == a
    t.append(b, 500)
    c = t.create()
    t.append(c, 300)
    t.mark(c, 0, 10, 200)
    t.evict(c, [0], deferred=True)
    errs, _ = t.decode_errors([b, c])
    assert max(errs.values()) <= TOL, errs
    err, _ = t.step([b, c])
    assert err <= TOL


def test_fully_masked_sequence_and_pages(sq):
    """Every slot of a sequence masked: zeros, as for an empty sequence;
    whole masked pages inside a shared run."""
    t = sc.Twin(sq, 1, 8, 2, 128, 200, 4, 40, seed=650)
    a = t.create()
    t.append(a, 100)
    t.mark(a, 0, 0, 100)
    b = t.create()
    t.append(b, 256)
    t.mark(b, 0, 16, 64)
    t.evict(a, [0], deferred=True)
    t.evict(b, [0], deferred=True)
    errs, ref = t.decode_errors([a, b])
    assert max(errs.values()) <= TOL, errs
    assert np.all(ref[0] == 0)


@pytest.mark.parametrize("prefix,n", [(900, 1), (900, 33), (900, 200), (12000, 1), (12000, 7)])
def test_deferred_extend(sq, prefix, n):
    """Extend of a chunk appended after a deferred eviction attends to the
    kept prefix slots and the chunk (one launch, or a split key range for
    the short chunks after the long prefix)."""
    import torch
    t = sc.Twin(sq, 1, 32, 8, 128, prefix // 16 + 60, 2, prefix // 16 + 40, seed=660 + n)
    a = t.create()
    t.append(a, prefix)
    spans = [(s0, s0 + 37) for s0 in range(11, prefix - 40, prefix // 9)] + [(prefix - 16, prefix)]
    for c, (s0, e0) in enumerate(spans):
        t.mark(a, c, s0, e0)
    t.evict(a, list(range(len(spans))), deferred=True)
    t.append(a, n)
    qb = wl.normal_bf16(t.rng, (n, 32, 128))
    out = t.store.extend(0, a, wl.to_torch_bf16(qb, "cuda"))
    torch.cuda.synchronize()
    k, v, _ = t.model.view(a)
    ref = oex.extend_attention(wl.bf16_value(qb), k[:, 0], v[:, 0], 1 / math.sqrt(128), 4)
    err = float(np.max(np.abs(out.cpu().numpy() - ref)))
    print(f"deferred extend prefix={prefix} n={n}: {err:.2e}")
    assert err <= TOL


def test_windows_refused_on_masked_sequences(sq):
    import torch
    t = sc.Twin(sq, 1, 8, 2, 64, 100, 4, 40, seed=670)
    a = t.create()
    t.append(a, 100)
    t.mark(a, 0, 5, 9)
    t.evict(a, [0], deferred=True)
    q = wl.device_normal_bf16((1, 8, 64), 1, "cuda")
    with pytest.raises(sq.SqError):
        t.store.decode(0, [a], q, window=16)
    with pytest.raises(sq.SqError):
        t.store.step_begin([a], window=16)
    with pytest.raises(sq.SqError):
        t.store.extend(0, a, q, window=16)
    assert t.store.seq_info(a)["length"] == 100
    torch.cuda.synchronize()
