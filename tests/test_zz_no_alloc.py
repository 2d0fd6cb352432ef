"""The allocation-free decode entry point, sq_decode_attn_noalloc, through the
C ABI: on two calls in a row (the second with a smaller input) it returns
what sq_decode_attn returns, bit for bit, and both stay within 5e-4 of the
float64 oracle; a call whose work split needs more partial slots than the
library's device array holds is rejected and writes nothing."""

import math

import numpy as np
import pytest

from oracle import attention as oatt
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


def _oracle(t, seqs, qb, layer):
    views = []
    for h in seqs:
        k, v, _ = t.model.view(h)
        views.append((k[:, layer], v[:, layer]))
    return oatt.decode_batch(wl.bf16_value(qb), views, 1 / math.sqrt(t.d), t.group)


@pytest.mark.parametrize("kv8", [False, True])
def test_noalloc_matches_decode_on_two_calls(sq, kv8):
    import torch
    scales = np.array([[0.011, 0.0095], [0.02, 0.013]], dtype=np.float32) if kv8 else None
    t = sc.Twin(sq, 2, 32, 8, 128, 1400, 6, 600, seed=81, kv_scales=scales)
    main = t.create()
    t.append(main, 6000)
    aux = t.fork(main, 5900)
    t.append(aux, 77)
    other = t.create()
    t.append(other, 1500)
    for c, (s0, e0) in enumerate([(100, 900), (2000, 2600)]):
        t.mark(main, c, s0, e0)
    t.evict(main, [0, 1])            # a compacted sequence in the first batch
    rng = np.random.default_rng(83)
    calls = [([main, aux, other], 1), ([other], 0)]  # the second input is smaller
    qs = [wl.normal_bf16(rng, (len(seqs), 32, 128)) for seqs, _ in calls]
    refs = [_oracle(t, seqs, qb, layer) for (seqs, layer), qb in zip(calls, qs)]
    for mode in (sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA):
        qt = [wl.to_torch_bf16(qb, "cuda") for qb in qs]
        want = [t.store.decode(layer, seqs, q, mode=mode) for (seqs, layer), q in zip(calls, qt)]
        got = [torch.full_like(w, float("nan")) for w in want]
        for (seqs, layer), q, o in zip(calls, qt, got):
            t.store.decode_noalloc(layer, seqs, q, o, mode=mode)
        torch.cuda.synchronize()
        for i in range(2):
            assert torch.equal(got[i], want[i]), (mode, i)
            err = sc.max_abs(got[i].cpu().numpy(), refs[i])
            assert err <= TOL, (mode, i, err)


def test_noalloc_rejects_a_split_beyond_its_slots(sq):
    """64 branches of one context with 32 KV heads, SHARED_PREFIX mode: the
    work split needs more partial slots than the device array holds; the
    call fails with SQ_ERR_INVALID and leaves out untouched, while
    sq_decode_attn (workspace partials) runs it."""
    import torch
    store = sq.Store(1, 32, 32, 64, num_pages=1200, max_seqs=70, max_pages_per_seq=200,
                     device="cuda")
    base = store.seq_create()
    kb = wl.device_normal_bf16((1, 3000, 32, 64), 85, "cuda")
    store.append(base, kb, kb)
    kids = []
    for i in range(64):
        c = store.fork(base, 3000)
        kn = wl.device_normal_bf16((1, 100, 32, 64), 86 + i, "cuda")
        store.append(c, kn, kn)
        kids.append(c)
    info = store.plan_info(kids, sq.ATTN_SHARED_PREFIX)
    assert info["n_slots"] > sq.NOALLOC_PARTIAL_SLOTS, info
    q = wl.device_normal_bf16((64, 32, 64), 87, "cuda")
    out = torch.full((64, 32, 64), 7.0, device="cuda")
    with pytest.raises(sq.SqError) as ei:
        store.decode_noalloc(0, kids, q, out, mode=sq.ATTN_SHARED_PREFIX)
    assert ei.value.code == sq.ERR_INVALID
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    ref = store.decode(0, kids, q, mode=sq.ATTN_SHARED_PREFIX)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(ref).all())
    store.close()
