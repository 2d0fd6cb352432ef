"""GPU parity of the decode step with the append fused (sq_step_begin, then
sq_step_attn per layer) against the oracle's one-token append to every
sequence followed by attention over every token: max abs error <= 5e-4 on
the fp32 outputs, the pools bit for bit afterwards, and replays of a
captured step (one capture, many steps, the metadata changing in between)
checked the same way on every replay."""

import numpy as np
import pytest

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


def _modes(sq):
    return [sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA]


@pytest.mark.parametrize("mi", [0, 1, 2, 3])
@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (8, 2, 64), (4, 4, 128), (64, 8, 64),
                                      (8, 4, 128)])
def test_steps_match_oracle(sq, mi, hq, hkv, d):
    """A main thread, its forked auxiliary thread, a sequence ending mid-page
    and an empty one, stepped 20 times in every mode (page boundaries are
    crossed on the way); the pools equal the oracle's afterwards."""
    mode = _modes(sq)[mi]
    t = sc.Twin(sq, 2, hq, hkv, d, 300, 6, 80, seed=100 + mi + hq)
    main = t.create()
    t.append(main, 700)
    aux = t.fork(main, 640)
    t.append(aux, 29)
    other = t.create()
    t.append(other, 47)
    empty = t.create()
    seqs = [main, aux, other, empty]
    worst = 0.0
    for _ in range(20):
        err, _ = t.step(seqs, mode)
        worst = max(worst, err)
        assert err <= TOL
    t.check_state()
    print(f"steps mode {mode} hq={hq} hkv={hkv} d={d}: max abs err {worst:.2e}")


def test_first_token_attends_to_itself(sq):
    """An empty sequence's first step: its only key is the new token, weight
    exactly 1, so every head's output is v_new exactly."""
    import torch
    s = sq.Store(1, 8, 2, 128, 16, 4, 8, device="cuda")
    a = s.seq_create()
    kn = wl.device_normal_bf16((1, 2, 128), 5, "cuda")
    vn = wl.device_normal_bf16((1, 2, 128), 6, "cuda")
    q = wl.device_normal_bf16((1, 8, 128), 7, "cuda")
    s.step_begin([a])
    out = s.step_attn(0, kn, vn, q)
    torch.cuda.synchronize()
    want = vn.float().repeat_interleave(4, dim=1)
    assert torch.equal(out, want)
    assert s.seq_info(a)["length"] == 1
    s.close()


@pytest.mark.parametrize("group", [1, 4])
def test_step_tree_of_forks(sq, group):
    """Forks of forks (mid-page and aligned) and a fan-out wider than one
    MFMA tile, stepped together."""
    hkv = 2
    t = sc.Twin(sq, 1, hkv * group, hkv, 128, 700, 14, 120, seed=120 + group)
    m = t.create()
    t.append(m, 1000)
    a = t.fork(m, 640)
    t.append(a, 200)
    b = t.fork(a, 800)
    t.append(b, 100)
    c = t.fork(m, 960)
    d = t.fork(b, 853)
    t.append(d, 33)
    fan = [t.fork(m, 992) for _ in range(6)]
    seqs = [m, a, b, c, d] + fan
    for _ in range(6):
        err, _ = t.step(seqs, sq.ATTN_AUTO)
        assert err <= TOL
    t.check_state()


def test_step_long_sequence_among_short_ones(sq):
    """A 20K-token sequence and its fork among one-page sequences: the even
    split lays short rows and the long one into shared workgroup ranges."""
    t = sc.Twin(sq, 1, 32, 8, 128, 2800, 8, 1300, seed=131)
    long_ = t.create()
    t.append(long_, 20000)
    aux = t.fork(long_, 19984)
    seqs = [long_, aux]
    for n in (1, 3, 16, 17):
        a = t.create()
        t.append(a, n)
        seqs.append(a)
    for _ in range(3):
        err, _ = t.step(seqs, sq.ATTN_AUTO)
        assert err <= TOL


@pytest.mark.parametrize("mi", [0, 2])
def test_captured_step_replays(sq, mi):
    """The layers of one step captured once (three layers: decode and merge
    launches), then replayed for eight more steps, each after its own
    sq_step_begin, with eager work in between: appends to a sequence of the
    batch, an eager decode call on the same partial buffers, an eviction of a
    sequence outside the batch.  Every replay is checked against the oracle,
    and the pools against the oracle's at the end."""
    import torch
    mode = _modes(sq)[mi]
    nl, hq, hkv, d = 3, 8, 2, 128
    t = sc.Twin(sq, nl, hq, hkv, d, 500, 6, 100, seed=140 + mi)
    main = t.create()
    t.append(main, 500)
    aux = t.fork(main, 496)
    t.append(aux, 12)
    side = t.create()
    t.append(side, 300)
    for c, (x, y) in enumerate([(10, 40), (100, 180)]):
        t.mark(side, c, x, y)
    seqs = [main, aux]
    err, _ = t.step(seqs, mode)        # eager step: opens the step the capture records
    assert err <= TOL
    g = dict(k=torch.zeros((nl, 2, hkv, d), dtype=torch.bfloat16, device="cuda"),
             v=torch.zeros((nl, 2, hkv, d), dtype=torch.bfloat16, device="cuda"),
             q=torch.zeros((nl, 2, hq, d), dtype=torch.bfloat16, device="cuda"),
             out=[torch.zeros((2, hq, d), dtype=torch.float32, device="cuda") for _ in range(nl)],
             graph=torch.cuda.CUDAGraph())
    with torch.cuda.graph(g["graph"]):
        for l in range(nl):
            t.store.step_attn(l, g["k"][l], g["v"][l], g["q"][l], out=g["out"][l])
    for r in range(8):
        err, got = t.step(seqs, mode, graph=g)
        print(f"replay {r}: max abs err {err:.2e}")
        assert err <= TOL, (r, err)
        if r == 2:
            t.append(aux, 20)                           # the plan changes under the graph
        if r == 4:
            e2, _ = t.decode_errors([side, main], modes=[sq.ATTN_AUTO])
            assert max(e2.values()) <= TOL
        if r == 5:
            t.evict(side, [0, 1])
    t.check_state()


def _device_page_table(store, seq):
    """The device page-table mirror row of seq (the workspace starts with it:
    int32 [max_seqs][max_pages_per_seq])."""
    import torch
    n = store.max_seqs * store.max_pages_per_seq
    rows = store.workspace[: 4 * n].view(torch.int32).view(store.max_seqs, store.max_pages_per_seq)
    return rows[seq, : store.seq_info(seq)["n_pages"]].tolist()


def test_step_begin_sets_the_page_table_at_once(sq):
    """A step that opens pages writes their page-table entries when it
    begins, so a step whose layers never run leaves no unset entry behind:
    the device mirror equals the host page table right after sq_step_begin,
    and the regular calls afterwards work (the abandoned tokens' slots hold
    whatever the fresh page held: zeros here)."""
    import torch
    t = sc.Twin(sq, 1, 8, 2, 64, 64, 4, 16, seed=150)
    a = t.create()
    t.append(a, 32)                    # two full pages: the step opens a third
    b = t.create()
    t.append(b, 5)
    t.store.step_begin([a, b])
    torch.cuda.synchronize()
    for h in (a, b):
        assert _device_page_table(t.store, h) == t.store.page_table(h)
    z = np.zeros((1, 1, 2, 64))
    for h in (a, b):                   # the oracle's view of the abandoned tokens
        t.model.append(h, 1, z, z)
    errs, _ = t.decode_errors([a, b])
    assert max(errs.values()) <= TOL, errs
    t.append(a, 3)
    errs, _ = t.decode_errors([a, b])
    assert max(errs.values()) <= TOL, errs


def test_step_arguments(sq):
    import torch
    s = sq.Store(2, 8, 2, 64, 32, 4, 8, device="cuda")
    a = s.seq_create()
    k = wl.device_normal_bf16((2, 5, 2, 64), 1, "cuda")
    s.append(a, k, k)
    kn = torch.zeros((1, 2, 64), dtype=torch.bfloat16, device="cuda")
    q = torch.zeros((1, 8, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(sq.SqError):
        s.step_attn(0, kn, kn, q)                      # no step opened
    s.step_begin([a])
    with pytest.raises(sq.SqError) as ei:
        s.step_attn(2, kn, kn, q)                      # no layer 2
    assert ei.value.code == sq.ERR_INVALID
    for bad in (kn.float(), kn[:, :1], torch.zeros((2, 2, 64), dtype=torch.bfloat16, device="cuda")):
        with pytest.raises(sq.SqError):
            s.step_attn(0, bad, kn, q)                 # wrong dtype or shape
    s.step_attn(0, kn, kn, q)
    s.append(a, k[:, :1].contiguous(), k[:, :1].contiguous())   # ends the step
    with pytest.raises(sq.SqError) as ei:
        s.step_attn(1, kn, kn, q)
    assert ei.value.code == sq.ERR_INVALID
    with pytest.raises(sq.SqError):
        s.step_begin([a, 3])                           # unknown sequence: nothing opened
    with pytest.raises(sq.SqError):
        s.step_attn(0, kn, kn, q)
    torch.cuda.synchronize()
    s.close()
