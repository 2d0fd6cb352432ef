"""GPU parity at full workload sizes, in the launch configuration bench.py
times (AUTO mode, default work split), plus the other attention modes.

The oracle cannot attend over every head of every 128K sequence in seconds,
so attention is checked on sampled (sequence, KV-head) outputs computed one
by one; eviction is checked in full (keep / dst / src_of, the compacted K/V
and positions, bit for bit).
"""

import math

import numpy as np
import pytest

from oracle import attention as oatt
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


def _modes(sq):
    return [sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA]


def _oracle_group(qf, k_t, v_t, g, scale):
    """Oracle attention of query heads 4g..4g+3 over one KV head g; k_t, v_t:
    torch bf16 [L, Hkv, D] on any device."""
    kf = wl.torch_bf16_to_f64(k_t[:, g: g + 1])
    vf = wl.torch_bf16_to_f64(v_t[:, g: g + 1])
    return oatt.attention(qf[4 * g: 4 * g + 4], kf, vf, scale, 4)


def _rows128k():
    """(batch entry, KV head) rows the 128K checks compare: every KV head of
    task 0's main and auxiliary threads, and KV head 0 of all 16 entries.
    The launch splits its (segment, KV head) rows into equal shares that cut
    across row boundaries, so the rows sit at every kind of boundary."""
    rows = [(b, g) for b in (0, 1) for g in range(8)]
    rows += [(b, 0) for b in range(2, 16)]
    return rows


def _task_kv(inputs, b, extra=None):
    """Seeded K/V (torch bf16 [L, Hkv, D], host) that entry b attends to:
    the main thread of task b // 2, or its auxiliary thread (the prefix up
    to the fork, then its own tokens); ``extra`` = (k_new, v_new) [B, Hkv,
    D] appends entry b's step token."""
    import torch
    k, v, ka, va = inputs[b // 2]
    fork_at = k.shape[1] - 256
    if b % 2 == 0:
        kk, vv = k[0].cpu(), v[0].cpu()
    else:
        kk = torch.cat([k[0, :fork_at].cpu(), ka[0].cpu()])
        vv = torch.cat([v[0, :fork_at].cpu(), va[0].cpu()])
    if extra is not None:
        kk = torch.cat([kk, extra[0][b: b + 1].cpu()])
        vv = torch.cat([vv, extra[1][b: b + 1].cpu()])
    return kk, vv


def _bits(t):
    """torch bf16 tensor -> uint16 bit patterns (host numpy)."""
    import torch
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _refs128k(inputs, qf, scale, extra=None):
    """Oracle outputs of every row of _rows128k, one oracle evaluation per
    row in CPU worker processes."""
    from tests import oracle_pool
    rows = _rows128k()
    jobs, cache = [], {}
    for b, g in rows:
        if b not in cache:
            cache = {b: _task_kv(inputs, b, extra)}
        kk, vv = cache[b]
        jobs.append((qf[b][4 * g: 4 * g + 4], _bits(kk[:, g]), _bits(vv[:, g]), scale, 4))
    return dict(zip(rows, oracle_pool.attention_many(jobs)))


def test_shared128k_sampled_heads(sq):
    import torch
    from paper_2602_22603_amd import drivers
    store, seqs, inputs = drivers.build_shared128k(keep_inputs=tuple(range(8)))
    rng = np.random.default_rng([2602, 2, 11])
    qb = wl.normal_bf16(rng, (16, 32, 128))
    q = wl.to_torch_bf16(qb, "cuda")
    qf = wl.bf16_value(qb)
    scale = 1 / math.sqrt(128)
    refs = _refs128k(inputs, qf, scale)
    for mode in _modes(sq):
        out = store.decode(0, seqs, q, mode=mode)
        torch.cuda.synchronize()
        o = out.cpu().numpy()
        for (b, g), ref in refs.items():
            err = sc.max_abs(o[b, 4 * g: 4 * g + 4], ref)
            assert err <= TOL, (mode, b, g, err)
    info = store.plan_info(seqs, sq.ATTN_AUTO)
    assert info["n_groups"] == 8 and info["kv_bytes"] == 4_311_744_512
    # the fused decode step bench.py also times: one token appended to all 16
    # sequences inside the step, then attention over every token
    kn = wl.device_normal_bf16((16, 8, 128), 2602_301, "cuda")
    vn = wl.device_normal_bf16((16, 8, 128), 2602_302, "cuda")
    q2 = wl.device_normal_bf16((16, 32, 128), 2602_303, "cuda")
    q2f = wl.torch_bf16_to_f64(q2)
    store.step_begin(seqs)
    out = store.step_attn(0, kn, vn, q2)
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    for (b, g), ref in _refs128k(inputs, q2f, scale, extra=(kn, vn)).items():
        err = sc.max_abs(o[b, 4 * g: 4 * g + 4], ref)
        assert err <= TOL, ("step", b, g, err)
    store.close()


def test_shared128k_fp8_sampled_heads(sq):
    """The 8-bit store's decode step at full size (the bench's kv_fp8 leg):
    sampled heads against the oracle over the round-tripped K/V in every
    mode (STREAM on the VALU kernel, the branches' private suffixes too in
    SHARED_PREFIX), and the stored codes of those heads against the
    oracle's quantisation."""
    import torch
    from oracle import fp8 as of8
    from paper_2602_22603_amd import drivers
    scales = np.array([[0.011, 0.0095]], dtype=np.float32)
    store, seqs, inputs = drivers.build_shared128k(keep_inputs=(0,), kv_scales=scales)
    rng = np.random.default_rng([2602, 2, 12])
    qb = wl.normal_bf16(rng, (16, 32, 128))
    q = wl.to_torch_bf16(qb, "cuda")
    qf = wl.bf16_value(qb)
    scale = 1 / math.sqrt(128)
    k, v, ka, va = inputs[0]
    fork_at = k.shape[1] - 256
    main_k, main_v = k[0], v[0]
    pt = store.page_table(seqs[0])
    refs = {}
    g = 5  # one KV head (the round trip of 16.7M values takes the oracle ~15 s)
    rk = of8.roundtrip(wl.torch_bf16_to_f64(main_k[:, g: g + 1]), scales[0, 0])
    rv = of8.roundtrip(wl.torch_bf16_to_f64(main_v[:, g: g + 1]), scales[0, 1])
    refs[(0, g)] = oatt.attention(qf[0][4 * g: 4 * g + 4], rk, rv, scale, 4)
    # the branch: the shared prefix's round trip, then its own tokens'
    ak = np.concatenate([rk[:fork_at], of8.roundtrip(wl.torch_bf16_to_f64(ka[0][:, g: g + 1]),
                                                     scales[0, 0])])
    av = np.concatenate([rv[:fork_at], of8.roundtrip(wl.torch_bf16_to_f64(va[0][:, g: g + 1]),
                                                     scales[0, 1])])
    refs[(1, g)] = oatt.attention(qf[1][4 * g: 4 * g + 4], ak, av, scale, 4)
    for mode in (sq.ATTN_AUTO, sq.ATTN_MFMA, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX):
        out = store.decode(0, seqs, q, mode=mode)
        torch.cuda.synchronize()
        o = out.cpu().numpy()
        for (b, g), ref in refs.items():
            err = sc.max_abs(o[b, 4 * g: 4 * g + 4], ref)
            assert err <= TOL, (mode, b, g, err)
    # codes of KV head 5 of the main thread's first and last pages
    for i in (0, len(pt) - 1):
        got = store.k_pool[0, 5, pt[i]].cpu().numpy()
        toks = main_k[16 * i: 16 * i + 16, 5]
        want = of8.quantize(wl.torch_bf16_to_f64(toks), scales[0, 0])
        assert np.array_equal(got[: len(want)], want), i
    store.close()


def test_outlier32k_evict_and_steps(sq):
    import torch
    from paper_2602_22603_amd import drivers
    store, main, aux, w, stats = drivers.build_outlier32k()
    L = w.main_len
    spans = [w.spans[c] for c in w.evict_ids]
    keep, dst, src_of, n_kept, first = oev.plan(L, spans)
    gk, gd, gs = store.debug_last_evict()
    assert np.array_equal(gk, keep) and np.array_equal(gd, dst) and np.array_equal(gs, src_of)
    assert stats["tokens_removed"] == L - n_kept and stats["first_evicted"] == first
    assert stats["tokens_removed"] >= L / 2
    kf, vf = wl.bf16_value(w.main_k)[0], wl.bf16_value(w.main_v)[0]   # [L, Hkv, D]
    k_main, v_main = kf[keep.astype(bool)], vf[keep.astype(bool)]
    vk, vv, vp = sc.seq_view(store, main)
    assert np.array_equal(vk[:, 0], k_main) and np.array_equal(vv[:, 0], v_main)
    assert np.array_equal(vp, np.flatnonzero(keep))
    ak, av = wl.bf16_value(w.aux_k)[0], wl.bf16_value(w.aux_v)[0]
    k_aux, v_aux = np.concatenate([kf, ak]), np.concatenate([vf, av])
    scale = 1 / math.sqrt(128)
    for i in range(w.steps):
        store.append_batch([main, aux], wl.to_torch_bf16(w.step_k[i], "cuda"),
                           wl.to_torch_bf16(w.step_v[i], "cuda"))
        sk, sv = wl.bf16_value(w.step_k[i])[0], wl.bf16_value(w.step_v[i])[0]  # [2, Hkv, D]
        k_main, v_main = np.concatenate([k_main, sk[:1]]), np.concatenate([v_main, sv[:1]])
        k_aux, v_aux = np.concatenate([k_aux, sk[1:]]), np.concatenate([v_aux, sv[1:]])
        q = wl.to_torch_bf16(w.q[i], "cuda")
        out = store.decode(0, [main, aux], q, mode=sq.ATTN_AUTO)
        if i in (0, w.steps - 1):
            torch.cuda.synchronize()
            qf = wl.bf16_value(w.q[i])
            ref = oatt.decode_batch(qf, [(k_main, v_main), (k_aux, v_aux)], scale, 4)
            outs = {sq.ATTN_AUTO: out.cpu().numpy()}
            for m in _modes(sq)[1:]:
                outs[m] = store.decode(0, [main, aux], q, mode=m).cpu().numpy()
            for m, o in outs.items():
                err = sc.max_abs(o, ref)
                assert err <= TOL, (i, m, err)
    store.close()


def test_compaction64k_evict_and_decode(sq):
    import torch
    from paper_2602_22603_amd import drivers
    store, base, w, k, v = drivers.build_compaction64k()
    L = w.length
    f = store.fork(base, L)
    stats = store.evict(f, w.evict_ids)
    spans = [w.spans[c] for c in w.evict_ids]
    keep, dst, src_of, n_kept, first = oev.plan(L, spans)
    assert stats["tokens_removed"] == L - n_kept >= 0.65 * L
    gk, gd, gs = store.debug_last_evict()
    assert np.array_equal(gk, keep) and np.array_equal(gd, dst) and np.array_equal(gs, src_of)
    # the compacted view equals the kept input rows; the base (full) is intact
    keep_t = torch.from_numpy(keep.astype(bool)).to("cuda")
    vk, vv, vp = sc.seq_view(store, f)
    assert np.array_equal(vk[:, 0], wl.torch_bf16_to_f64(k[0][keep_t]))
    assert np.array_equal(vv[:, 0], wl.torch_bf16_to_f64(v[0][keep_t]))
    assert np.array_equal(vp, np.flatnonzero(keep))
    bk, bv, bp = sc.seq_view(store, base)
    assert np.array_equal(bk[:, 0], wl.torch_bf16_to_f64(k[0]))
    assert np.array_equal(bp, np.arange(L))
    del bk, bv, vk, vv
    rng = np.random.default_rng([2602, 3, 5])
    qb = wl.normal_bf16(rng, (2, 32, 128))
    q = wl.to_torch_bf16(qb, "cuda")
    qf = wl.bf16_value(qb)
    scale = 1 / math.sqrt(128)
    ref = {}
    for g in (0, 6):
        ref[(0, g)] = _oracle_group(qf[0], k[0][keep_t], v[0][keep_t], g, scale)
        ref[(1, g)] = _oracle_group(qf[1], k[0], v[0], g, scale)
        kf = wl.torch_bf16_to_f64(k[0][:, g: g + 1])
        vf = wl.torch_bf16_to_f64(v[0][:, g: g + 1])
        masked = oatt.masked_attention(qf[0][4 * g: 4 * g + 4], kf, vf, keep, scale, 4)
        assert sc.max_abs(masked, ref[(0, g)]) <= 1e-12
    for mode in _modes(sq):
        out = store.decode(0, [f, base], q, mode=mode)
        torch.cuda.synchronize()
        o = out.cpu().numpy()
        for (b, g), r in ref.items():
            err = sc.max_abs(o[b, 4 * g: 4 * g + 4], r)
            assert err <= TOL, (mode, b, g, err)
    store.close()


def test_compaction64k_chunked_in_place_recycling(sq):
    """The 64K compaction evicted in chunks of 64 pages with no other branch
    holding the pages: old pages are reused inside the call.  The compacted
    view equals the kept input rows bit for bit, the page table equals the
    oracle's chunked schedule, and at most 64 transient pages are live."""
    import torch
    from oracle import pages as opg
    from paper_2602_22603_amd import drivers
    store, base, w, k, v = drivers.build_compaction64k(evict_chunk_pages=64)
    L = w.length
    before = store.stats()["live_pages"]
    store.evict(base, w.evict_ids)
    spans = [w.spans[c] for c in w.evict_ids]
    keep, _dst, _src, n_kept, _first = oev.plan(L, spans)
    model = opg.PageModel(store.num_pages, 16, store.max_seqs, store.max_pages_per_seq,
                          evict_chunk_pages=64)
    h = model.seq_create()
    model.append(h, L)
    for c, (s0, e0) in enumerate(w.spans):
        model.span_mark(h, c, s0, e0)
    model.evict(h, w.evict_ids)
    assert store.page_table(base) == model.page_table(h)
    assert store.stats()["peak_pages"] == model.peak_pages <= before + 64
    keep_t = torch.from_numpy(keep.astype(bool)).to("cuda")
    vk, vv, vp = sc.seq_view(store, base)
    assert np.array_equal(vk[:, 0], wl.torch_bf16_to_f64(k[0][keep_t]))
    assert np.array_equal(vv[:, 0], wl.torch_bf16_to_f64(v[0][keep_t]))
    assert np.array_equal(vp, np.flatnonzero(keep))
    store.close()


def test_full_stack_sampled(sq):
    """36 layers, 16K prefix + 30 turns of 8K tokens with an auxiliary thread
    every 4 turns evicting >= 60% of the live tool tokens: positions against
    a replay of the logged evictions, compacted K/V of sampled layers and
    heads bit for bit against the regenerated inputs, and sampled decode
    outputs of main and auxiliary against the oracle."""
    import torch
    from paper_2602_22603_amd import drivers
    store, main, aux, log, w = drivers.run_full_stack(decode=True)
    assert aux is None  # the last auxiliary thread finished and was released
    # positions: replay appends and evictions on a plain list
    pos = list(range(w.prefix))
    nxt = w.prefix
    for rec in log:
        if "evicted_spans" in rec:
            keep = oev.keep_mask(len(pos), rec["evicted_spans"])
            pos = [p for p, k in zip(pos, keep) if k]
        pos += list(range(nxt, nxt + w.turn_len))
        nxt += w.turn_len
    got = store.positions(main)
    assert got.tolist() == pos
    assert sum("evict" in r for r in log) == 7
    # inputs of main, gathered by position, for sampled (layer, head)
    samples = [(0, 0), (17, 5), (35, 7)]
    pos_t = torch.tensor(pos, device="cuda")
    rows_k = {s: [] for s in samples}
    rows_v = {s: [] for s in samples}
    for turn in range(-1, w.turns):
        lo = 0 if turn < 0 else w.prefix + turn * w.turn_len
        hi = w.prefix if turn < 0 else lo + w.turn_len
        sel = pos_t[(pos_t >= lo) & (pos_t < hi)] - lo
        k, v = drivers.full_stack_inputs(w, turn)
        for (layer, g) in samples:
            rows_k[(layer, g)].append(k[layer, sel, g])
            rows_v[(layer, g)].append(v[layer, sel, g])
        del k, v
    main_kv = {s: (torch.cat(rows_k[s]), torch.cat(rows_v[s])) for s in samples}
    # the GPU pools hold exactly those rows
    for (layer, g), (kk, vv) in main_kv.items():
        gk, gv, gp = sc.seq_view(store, main, layers=[layer])
        assert np.array_equal(gk[:, 0, g], wl.torch_bf16_to_f64(kk)), (layer, g)
        assert np.array_equal(gv[:, 0, g], wl.torch_bf16_to_f64(vv)), (layer, g)
        del gk, gv
    # a new auxiliary thread on the final context, with its own private tokens
    fork_len = store.seq_info(main)["length"]
    aux = store.fork(main, fork_len)
    ka, va = drivers.full_stack_aux_inputs(w, w.turns)
    store.append(aux, ka, va)
    rng = np.random.default_rng([2602, 4, 9])
    qb = wl.normal_bf16(rng, (2, 32, 128))
    q = wl.to_torch_bf16(qb, "cuda")
    qf = wl.bf16_value(qb)
    scale = 1 / math.sqrt(128)
    for (layer, g), (kk, vv) in main_kv.items():
        qg_main = qf[0][4 * g: 4 * g + 4]
        qg_aux = qf[1][4 * g: 4 * g + 4]
        ref_main = _oracle_group(qg_main, kk[:, None], vv[:, None], 0, scale)
        ak = torch.cat([kk, ka[layer, :, g]])[:, None]
        av = torch.cat([vv, va[layer, :, g]])[:, None]
        ref_aux = _oracle_group(qg_aux, ak, av, 0, scale)
        for mode in _modes(sq):
            out = store.decode(layer, [main, aux], q, mode=mode)
            torch.cuda.synchronize()
            o = out.cpu().numpy()
            e1 = sc.max_abs(o[0, 4 * g: 4 * g + 4], ref_main)
            e2 = sc.max_abs(o[1, 4 * g: 4 * g + 4], ref_aux)
            assert e1 <= TOL and e2 <= TOL, (layer, g, mode, e1, e2)
    store.close()
