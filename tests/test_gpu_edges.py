"""GPU parity at the edges of the decode planner: the largest batch, empty
and one-token sequences, duplicate entries, shared-prefix groups wider than
one MFMA tile holds, sequences that share a workgroup's page range with a
long one, negative and unusual scales, and layers past the first.  Every
mode is compared with the oracle (max abs error <= 5e-4); page tables and
views bit for bit."""

import numpy as np
import pytest

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


def _check(t, seqs, **kw):
    errs, ref = t.decode_errors(seqs, **kw)
    for m, e in errs.items():
        assert e <= TOL, (m, e)
    return errs, ref


def test_largest_batch_with_empty_and_tiny_sequences(sq):
    """64 queries: 24 main threads of mixed lengths (0, 1, 15, 16, 17, ...)
    and 40 forks of them, some forked mid-page."""
    rng = np.random.default_rng(7)
    t = sc.Twin(sq, 1, 32, 8, 128, 2600, 64, 80, seed=71)
    mains = []
    lengths = [0, 1, 15, 16, 17, 31, 33, 64, 65, 100, 257, 500, 1023, 1024, 1025, 7, 2, 3, 48,
               49, 200, 300, 640, 900]
    for n in lengths:
        a = t.create()
        if n:
            t.append(a, n)
        mains.append(a)
    seqs = list(mains)
    while len(seqs) < 64:
        i = int(rng.integers(0, len(mains)))
        L = lengths[i]
        f = int(rng.integers(0, L + 1))
        c = t.fork(mains[i], f)
        extra = int(rng.integers(0, 40))
        if extra:
            t.append(c, extra)
        seqs.append(c)
    t.check_state()
    errs, ref = _check(t, seqs)
    assert np.all(ref[0] == 0)          # the empty sequence attends to nothing
    print("batch 64:", errs)


def test_duplicate_entries_in_one_batch(sq):
    t = sc.Twin(sq, 1, 8, 2, 64, 200, 4, 64, seed=72)
    a = t.create()
    t.append(a, 300)
    b = t.fork(a, 250)
    t.append(b, 11)
    _check(t, [a, b, a, a, b])   # each entry has its own query


@pytest.mark.parametrize("group", [2, 4, 8])
def test_wide_fork_fanout(sq, group):
    """One main thread with six auxiliary forks at the same point: more
    members than one 16-row MFMA tile holds (16 / G), split into groups."""
    hkv = 2
    t = sc.Twin(sq, 1, hkv * group, hkv, 128, 400, 12, 64, seed=73 + group)
    a = t.create()
    t.append(a, 700)
    seqs = [a]
    for i in range(6):
        c = t.fork(a, 640 if i % 2 else 700)
        t.append(c, 5 + 7 * i)
        seqs.append(c)
    info = t.store.plan_info(seqs, sq.ATTN_AUTO)
    assert info["n_groups"] >= 2
    _check(t, seqs)


def test_short_rows_share_a_workgroup_with_a_long_one(sq):
    """A 20K-token sequence among one-page sequences: the balanced split
    lays rows end to end, so one workgroup's range covers several short
    rows and the start of the long one."""
    t = sc.Twin(sq, 1, 32, 8, 128, 1400, 8, 1300, seed=74)
    long_ = t.create()
    t.append(long_, 20000)
    seqs = []
    for n in (1, 3, 16, 17, 5):
        a = t.create()
        t.append(a, n)
        seqs.append(a)
    seqs.insert(2, long_)
    _check(t, seqs)


def test_everything_evicted_then_regrown(sq):
    t = sc.Twin(sq, 1, 8, 2, 64, 200, 4, 64, seed=75)
    a = t.create()
    t.append(a, 100)
    t.mark(a, 0, 0, 60)
    t.mark(a, 1, 60, 100)
    t.evict(a, [0, 1])
    assert t.store.seq_info(a)["length"] == 0
    errs, ref = _check(t, [a])
    assert np.all(ref == 0)
    t.append(a, 1)
    t.check_state()
    _check(t, [a])


@pytest.mark.parametrize("scale", [-0.2, 0.37, 2.5])
def test_unusual_scales(sq, scale):
    t = sc.Twin(sq, 1, 8, 2, 128, 200, 4, 80, seed=76)
    a = t.create()
    t.append(a, 1000)
    b = t.fork(a, 992)
    t.append(b, 20)
    _check(t, [a, b], scale=scale)


def test_later_layers(sq):
    t = sc.Twin(sq, 4, 8, 2, 64, 300, 4, 80, seed=77)
    a = t.create()
    t.append(a, 777)
    b = t.fork(a, 700)
    t.append(b, 30)
    for layer in (3, 1):
        _check(t, [a, b], layer=layer)


def test_binding_rejects_bad_tensors(sq):
    """The C ABI trusts pointer sizes, so the binding checks shape, dtype,
    contiguity and device before any call; nothing changes on a rejection."""
    import torch
    s = sq.Store(1, 8, 2, 64, 64, 4, 16, device="cuda")
    a = s.seq_create()
    k = torch.zeros((1, 5, 2, 64), dtype=torch.bfloat16, device="cuda")
    bad_k = [k.float(), k[:, :4], k.transpose(2, 3).contiguous().transpose(2, 3), k.cpu(),
             torch.zeros((1, 5, 2, 65), dtype=torch.bfloat16, device="cuda")]
    for kb in bad_k:
        with pytest.raises(sq.SqError) as ei:
            s.append(a, kb, k, n=5)
        assert ei.value.code == sq.ERR_INVALID
    assert s.seq_info(a)["length"] == 0 and s.stats()["live_pages"] == 0
    s.append(a, k, k)
    q = torch.zeros((1, 8, 64), dtype=torch.bfloat16, device="cuda")
    for qb, ob in [(q.float(), None), (q[:, :4], None), (q, torch.zeros((1, 8, 64), device="cuda").half()),
                   (q, torch.zeros((1, 8, 64), device="cuda")[:, ::2]), (q.cpu(), None)]:
        with pytest.raises(sq.SqError):
            s.decode(0, [a], qb, out=ob if ob is not None else torch.zeros((1, 8, 64), device="cuda"))
    with pytest.raises(sq.SqError):
        s.extend(0, a, torch.zeros((2, 8, 64), dtype=torch.float32, device="cuda"))
    assert s.stats()["decode_calls"] == 0 and s.stats()["extend_calls"] == 0
    s.close()


@pytest.mark.parametrize("group", [1, 2, 4, 8])
def test_deep_chain_and_wide_fanout(sq, group):
    """A fork chain seven deep (page-aligned and mid-page fork points) and a
    fan-out of eight branches at one point, alone and together: up to
    eight members share one tile (two 16-row blocks when G = 4 or 8, the
    two-block kernel), entries merge up to eight partial sources; every
    mode against the oracle, page tables and views bit for bit."""
    hkv = 2
    t = sc.Twin(sq, 1, hkv * group, hkv, 128, 900, 20, 120, seed=90 + group)
    m = t.create()
    t.append(m, 300)
    chain = [m]
    for d in range(7):
        nxt = t.fork(chain[-1], t.model.info(chain[-1])["length"] - (7 if d % 2 else 0))
        t.append(nxt, 40)
        chain.append(nxt)
    a = t.create()
    t.append(a, 700)
    fan = [a]
    for i in range(7):
        c = t.fork(a, 640 if i % 2 else 700)
        t.append(c, 5 + 7 * i)
        fan.append(c)
    t.check_state()
    for seqs in (chain, fan, fan[:5], chain[3:] + fan[:4]):
        info = t.store.plan_info(seqs, sq.ATTN_AUTO)
        assert info["kv_bytes"] < info["kv_bytes_logical"]
        _check(t, seqs)
    # and a decode step (one-block tiles: the fused step keeps its launches)
    err, _ = t.step(fan)
    assert err <= TOL


@pytest.mark.parametrize("group", [1, 2, 4])
def test_tree_of_forks(sq, group):
    """Forks of forks at page-aligned and mid-page points: the shared-prefix
    plan reads a tree of shared runs (up to three levels deep) once each and
    merges up to four partial sources per entry."""
    hkv = 2
    t = sc.Twin(sq, 1, hkv * group, hkv, 128, 600, 12, 120, seed=80 + group)
    m = t.create()
    t.append(m, 1000)
    a = t.fork(m, 640)
    t.append(a, 200)
    b = t.fork(a, 800)
    t.append(b, 100)
    c = t.fork(m, 960)
    t.append(c, 20)
    d = t.fork(b, 853)          # mid-page: its tail page is a copy
    t.append(d, 33)
    chain = [m]
    for _ in range(3):
        nxt = t.fork(chain[-1], t.model.info(chain[-1])["length"])
        t.append(nxt, 32)
        chain.append(nxt)
    t.check_state()
    for seqs in ([m, a, b, c], [d, b, a, m, c], chain, [m, a, b, c] + chain[1:]):
        info = t.store.plan_info(seqs, sq.ATTN_AUTO)
        assert info["kv_bytes"] < info["kv_bytes_logical"]
        _check(t, seqs)


@pytest.mark.parametrize("hq,hkv", [(32, 8), (32, 16), (16, 16)])
def test_merge_row_lists_in_arguments_and_from_the_plan(sq, hq, hkv):
    """Calls of one or two entries with at most 8 KV heads carry each (entry,
    KV head)'s merge row lists in the merge's arguments; three entries, or
    16 KV heads, derive them from the plan's tables.  Both ways against the
    oracle in every mode, on a shared prefix whose rows split over many
    workgroups and private suffixes of a few tokens to a few hundred."""
    t = sc.Twin(sq, 1, hq, hkv, 64, num_pages=2 * (3100 // 16) + 64, max_seqs=4,
                max_pages_per_seq=3100 // 16 + 8, seed=173)
    a = t.create()
    t.append(a, 3000)
    b = t.fork(a, 2000)
    t.append(b, 300)
    c = t.fork(a, 3000)
    t.append(c, 17)
    for seqs in ([a], [b], [a, b], [c, a], [a, b, c]):
        errs, _ = _check(t, seqs)
        print(f"hq={hq} hkv={hkv} batch {len(seqs)}:", {m: f"{e:.1e}" for m, e in errs.items()})
