"""Scenario drivers shared by the GPU tests, ``__graft_entry__.smoke()`` and
``bench.py``: each replays one seeded workload through the library and, when
asked, through the oracle's page model, so the two can be compared.

Only test infrastructure may import this module (it calls the oracle).
"""

from __future__ import annotations

import math

import numpy as np

from oracle import attention as oatt
from oracle import evict as oev
from oracle import fp8 as of8
from oracle import pages as opg
from paper_2602_22603_amd import workload as wl


def seq_view(store, seq, layers=None):
    """Logical view of ``seq`` read back from the GPU pools, in the oracle's
    order: (K f64 [L, NL, Hkv, D], V f64 [L, NL, Hkv, D], pos int64 [L])."""
    import torch
    pt = store.page_table(seq)
    length = store.seq_info(seq)["length"]
    layers = list(range(store.num_layers)) if layers is None else list(layers)
    if length == 0:
        z = np.zeros((0, len(layers), store.num_kv_heads, store.head_dim))
        return z, z.copy(), np.zeros(0, dtype=np.int64)
    dev = store.k_pool.device
    tok = torch.arange(length, device=dev)
    pages = torch.tensor(pt, device=dev, dtype=torch.int64)[tok // 16]
    slots = tok % 16
    lt = torch.tensor(layers, device=dev)
    # K pool [NL, Hkv, NP, P, D]; V pool [NL, Hkv, NP, D, P] -> [NL, Hkv, NP, P, D]
    kx = store.k_pool[lt]
    vx = store.v_pool[lt].permute(0, 1, 2, 4, 3)
    k = kx[:, :, pages, slots, :].permute(2, 0, 1, 3)     # [L, NL, Hkv, D]
    v = vx[:, :, pages, slots, :].permute(2, 0, 1, 3)
    pos = store.pos_pool[pages, slots]
    if getattr(store, "kv_fp8", False):  # E4M3 codes times the layer's scales
        sc = store.kv_scales[layers].astype(np.float64)
        kf = of8.decode(k.cpu().numpy()) * sc[None, :, 0, None, None]
        vf = of8.decode(v.cpu().numpy()) * sc[None, :, 1, None, None]
        return kf, vf, pos.cpu().numpy().astype(np.int64)
    return (wl.torch_bf16_to_f64(k), wl.torch_bf16_to_f64(v),
            pos.cpu().numpy().astype(np.int64))


def oracle_model_for(store, with_data=True):
    return opg.PageModel(store.num_pages, store.page_size, store.max_seqs,
                         store.max_pages_per_seq, layers=store.num_layers,
                         kv_heads=store.num_kv_heads, head_dim=store.head_dim,
                         with_data=with_data, evict_chunk_pages=store.evict_chunk_pages,
                         evict_remap=store.evict_remap,
                         evict_inplace=getattr(store, "evict_inplace", False),
                         kv_scales=getattr(store, "kv_scales", None))


def run_tiny(sq, device="cuda", modes=None, with_oracle=True):
    """The tiny case through the library (and the oracle): returns a dict with
    page tables, views, eviction arrays and decode outputs of both sides."""
    import torch
    w = wl.tiny()
    modes = [sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA] if modes is None else modes
    num_pages = 2 * (w.main_len // 16) + 16
    store = sq.Store(w.num_layers, w.num_q_heads, w.num_kv_heads, w.head_dim, num_pages,
                     max_seqs=4, max_pages_per_seq=w.main_len // 16 + 8, device=device)
    kk = wl.to_torch_bf16(w.main_k, device)
    vv = wl.to_torch_bf16(w.main_v, device)
    main = store.seq_create()
    store.append(main, kk[:, : w.fork_at].contiguous(), vv[:, : w.fork_at].contiguous())
    aux = store.fork(main, w.fork_at)
    store.append(main, kk[:, w.fork_at:].contiguous(), vv[:, w.fork_at:].contiguous())
    store.append(aux, wl.to_torch_bf16(w.aux_k, device), wl.to_torch_bf16(w.aux_v, device))
    for c, (s, e) in enumerate(w.spans):
        store.span_mark(main, c, s, e)
    ev_stats = store.evict(main, w.evict_ids)
    q = wl.to_torch_bf16(w.q, device)
    outs = {m: store.decode(0, [main, aux], q, scale=w.scale, mode=m).cpu().numpy() for m in modes}
    torch.cuda.synchronize()
    res = dict(store=store, main=main, aux=aux, outs=outs, ev_stats=ev_stats,
               evict_arrays=store.debug_last_evict(),
               page_tables={main: store.page_table(main), aux: store.page_table(aux)},
               views={main: seq_view(store, main), aux: seq_view(store, aux)}, workload=w)
    if not with_oracle:
        return res
    m = oracle_model_for(store)
    om = m.seq_create()
    kf, vf = wl.bf16_value(w.main_k), wl.bf16_value(w.main_v)
    m.append(om, w.fork_at, kf[:, : w.fork_at], vf[:, : w.fork_at])
    oa = m.fork(om, w.fork_at)
    m.append(om, w.main_len - w.fork_at, kf[:, w.fork_at:], vf[:, w.fork_at:])
    m.append(oa, w.aux_private, wl.bf16_value(w.aux_k), wl.bf16_value(w.aux_v))
    for c, (s, e) in enumerate(w.spans):
        m.span_mark(om, c, s, e)
    before = m.view(om)
    o_stats = m.evict(om, w.evict_ids)
    keep, dst, src_of, _, _ = oev.plan(w.main_len, [w.spans[c] for c in w.evict_ids])
    views = {main: m.view(om), aux: m.view(oa)}
    qf = wl.bf16_value(w.q)
    group = w.num_q_heads // w.num_kv_heads
    ref = oatt.decode_batch(qf, [(views[main][0][:, 0], views[main][1][:, 0]),
                                 (views[aux][0][:, 0], views[aux][1][:, 0])], w.scale, group)
    masked = oatt.masked_attention(qf[0], before[0][:, 0], before[1][:, 0], keep, w.scale, group)
    res["oracle"] = dict(model=m, main=om, aux=oa, stats=o_stats, keep=keep, dst=dst,
                         src_of=src_of, views=views, out=ref, masked_main=masked,
                         page_tables={main: m.page_table(om), aux: m.page_table(oa)})
    return res


def max_abs(a, b):
    return float(np.max(np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))))


def check_tiny(res, tol=5e-4):
    """Assertions shared by the smoke run and the tiny GPU test."""
    o = res["oracle"]
    main, aux = res["main"], res["aux"]
    assert res["page_tables"][main] == o["page_tables"][main]
    assert res["page_tables"][aux] == o["page_tables"][aux]
    for h in (main, aux):
        gk, gv, gp = res["views"][h]
        ok, ov, op = o["views"][h]
        assert np.array_equal(gk, ok) and np.array_equal(gv, ov), f"K/V view of {h}"
        assert np.array_equal(gp, op), f"positions of {h}"
    keep, dst, src_of = res["evict_arrays"]
    assert np.array_equal(keep, o["keep"]) and np.array_equal(dst, o["dst"])
    assert np.array_equal(src_of, o["src_of"])
    for k in o["stats"]:
        assert res["ev_stats"][k] == o["stats"][k], k
    errs = {}
    for mode, out in res["outs"].items():
        errs[mode] = max_abs(out, o["out"])
        assert errs[mode] <= tol, (mode, errs[mode])
        # compacted (GPU) against masked attention over the uncompacted cache
        assert max_abs(out[0], o["masked_main"]) <= tol
    return errs


def scale_for(head_dim):
    return 1.0 / math.sqrt(head_dim)


class Twin:
    """Applies every operation to a GPU store and to the oracle's page model
    (with data), drawing the same seeded bf16 inputs for both."""

    def __init__(self, sq, num_layers, num_q_heads, num_kv_heads, head_dim, num_pages,
                 max_seqs, max_pages_per_seq, seed=0, device="cuda", evict_chunk_pages=0,
                 evict_remap=False, kv_scales=None, evict_inplace=False):
        self.sq = sq
        self.device = device
        self.store = sq.Store(num_layers, num_q_heads, num_kv_heads, head_dim, num_pages,
                              max_seqs, max_pages_per_seq, device=device,
                              evict_chunk_pages=evict_chunk_pages, evict_remap=evict_remap,
                              evict_inplace=evict_inplace,
                              kv_scales=kv_scales)
        self.model = oracle_model_for(self.store)
        self.rng = np.random.default_rng([2602, 900, seed])
        self.nl, self.hq, self.hkv, self.d = num_layers, num_q_heads, num_kv_heads, head_dim
        self.group = num_q_heads // num_kv_heads

    def create(self):
        a = self.store.seq_create()
        b = self.model.seq_create()
        assert a == b
        return a

    def append(self, h, n, const_v=None, outlier=False, k_scale=1):
        """n seeded tokens; ``outlier`` scales K channels 0-3 and V channels
        5-8 by 8 (exact in bf16), the outlier-channel shape; ``k_scale`` (a
        power of two, exact in bf16) scales every key."""
        kb = wl.normal_bf16(self.rng, (self.nl, n, self.hkv, self.d))
        vb = wl.normal_bf16(self.rng, (self.nl, n, self.hkv, self.d))
        if k_scale != 1:
            kb = wl.bf16_bits((wl.bf16_value(kb) * k_scale).astype(np.float32))
        if const_v is not None:
            vb[...] = wl.bf16_bits(np.full(vb.shape, const_v, np.float32))
        if outlier:
            kf, vf = wl.bf16_value(kb), wl.bf16_value(vb)
            kf[..., :4] *= 8
            vf[..., 5:9] *= 8
            kb, vb = wl.bf16_bits(kf.astype(np.float32)), wl.bf16_bits(vf.astype(np.float32))
        self.store.append(h, wl.to_torch_bf16(kb, self.device), wl.to_torch_bf16(vb, self.device))
        self.model.append(h, n, wl.bf16_value(kb), wl.bf16_value(vb))

    def fork(self, h, f):
        a = self.store.fork(h, f)
        b = self.model.fork(h, f)
        assert a == b
        return a

    def mark(self, h, cursor, s, e):
        self.store.span_mark(h, cursor, s, e)
        self.model.span_mark(h, cursor, s, e)

    def try_mark(self, h, cursor, s, e):
        """Mark where the oracle accepts the span; both sides must agree."""
        try:
            self.model.span_mark(h, cursor, s, e)
        except opg.OracleError as err:
            try:
                self.store.span_mark(h, cursor, s, e)
            except self.sq.SqError as serr:
                assert serr.code == err.code, (serr.code, err.code)
                return False
            raise AssertionError("the library accepted a span the oracle rejects")
        self.store.span_mark(h, cursor, s, e)
        return True

    def evict(self, h, ids, deferred=False):
        got = self.store.evict(h, ids, deferred=deferred)
        want = self.model.evict(h, ids, deferred=deferred)
        for k in want:
            assert got[k] == want[k], (k, got, want)
        return got

    def compact(self, h):
        got = self.store.compact(h)
        want = self.model.compact(h)
        for k in want:
            assert got[k] == want[k], (k, got, want)
        return got

    def release(self, h):
        self.store.release(h)
        self.model.release(h)

    def check_state(self):
        assert self.store.refcounts().tolist() == self.model.refcount.tolist()
        for h in self.model.seqs:
            assert self.store.page_table(h) == self.model.page_table(h), h
            assert self.store.keep_flags(h).tolist() == self.model.keep_flags(h).tolist()
            gk, gv, gp = seq_view(self.store, h)
            ok, ov, op = self.model.slot_view(h)
            assert np.array_equal(gp, op), f"positions of {h}"
            assert np.array_equal(gk, ok), f"K of {h}"
            assert np.array_equal(gv, ov), f"V of {h}"

    def sinks(self, spread=2.0):
        """Seeded fp32 sink logits [Hq] (float32 values, as the kernels read them)."""
        return (self.rng.standard_normal(self.hq) * spread).astype(np.float32)

    def decode_errors(self, seqs, modes=None, layer=0, scale=None, window=0, sinks=None):
        """Max abs error of sq_decode_attn in each mode against the oracle;
        window and sinks (fp32 [Hq] numpy) are the model-variant options."""
        import torch
        sq = self.sq
        modes = [sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA] if modes is None else modes
        scale = scale_for(self.d) if scale is None else scale
        qb = wl.normal_bf16(self.rng, (len(seqs), self.hq, self.d))
        q = wl.to_torch_bf16(qb, self.device)
        views = []
        for h in seqs:
            k, v, _ = self.model.view(h)
            views.append((k[:, layer], v[:, layer]))
        ref = oatt.decode_batch(wl.bf16_value(qb), views, scale, self.group, window=window,
                                sinks=None if sinks is None else sinks.astype(np.float64))
        sk = None if sinks is None else torch.from_numpy(sinks).to(self.device)
        errs = {}
        for m in modes:
            out = self.store.decode(layer, seqs, q, scale=scale, mode=m, window=window, sinks=sk)
            torch.cuda.synchronize()
            errs[m] = max_abs(out.cpu().numpy(), ref)
        return errs, ref

    def step(self, seqs, mode=None, scale=None, graph=None, window=0, layer_windows=None,
             sinks=None):
        """One decode step of every layer through sq_step_begin / sq_step_attn
        (or, with ``graph``, a replay of captured sq_step_attn calls: a dict
        with the graph and its fixed k/v/q/out buffers), mirrored in the
        oracle as a one-token append to each sequence followed by attention.
        ``window`` opens the step with a windowed plan, ``layer_windows[l]``
        (0 or window) is layer l's window, ``sinks`` (fp32 [Hq] numpy, or a
        list of one per layer) its sink logits.  Returns the max abs error
        over all layers and entries."""
        import torch
        sq = self.sq
        mode = sq.ATTN_AUTO if mode is None else mode
        scale = scale_for(self.d) if scale is None else scale
        b = len(seqs)
        kb = wl.normal_bf16(self.rng, (self.nl, b, self.hkv, self.d))
        vb = wl.normal_bf16(self.rng, (self.nl, b, self.hkv, self.d))
        qb = wl.normal_bf16(self.rng, (self.nl, b, self.hq, self.d))
        lw = [0] * self.nl if layer_windows is None else list(layer_windows)
        ls = sinks if isinstance(sinks, list) else [sinks] * self.nl
        self.store.step_begin(seqs, mode, window=window)
        if graph is None:
            k, v, q = (wl.to_torch_bf16(x, self.device) for x in (kb, vb, qb))
            sk = [None if x is None else torch.from_numpy(x).to(self.device) for x in ls]
            outs = [self.store.step_attn(l, k[l], v[l], q[l], scale=scale, window=lw[l], sinks=sk[l])
                    for l in range(self.nl)]
        else:
            for name, x in (("k", kb), ("v", vb), ("q", qb)):
                graph[name].copy_(wl.to_torch_bf16(x, self.device))
            graph["graph"].replay()
            outs = graph["out"]
        torch.cuda.synchronize()
        got = [o.cpu().numpy() for o in outs]
        kf, vf = wl.bf16_value(kb), wl.bf16_value(vb)
        for j, h in enumerate(seqs):
            self.model.append(h, 1, kf[:, j:j + 1], vf[:, j:j + 1])
        err = 0.0
        qf = wl.bf16_value(qb)
        for l in range(self.nl):
            views = []
            for h in seqs:
                kk, vv, _ = self.model.view(h)
                views.append((kk[:, l], vv[:, l]))
            ref = oatt.decode_batch(qf[l], views, scale, self.group, window=lw[l],
                                    sinks=None if ls[l] is None else ls[l].astype(np.float64))
            err = max(err, max_abs(got[l], ref))
        return err, got


def tiny_step_error(sq, res, device="cuda"):
    """One fused decode step (sq_step_begin + sq_step_attn) of the tiny case's
    main and auxiliary threads after its eviction, against the oracle's
    one-token append and attention; returns the max abs error."""
    import torch
    w, o = res["workload"], res["oracle"]
    store, model = res["store"], o["model"]
    rng = np.random.default_rng([2602, 0, 77])
    hkv, hq, d = w.num_kv_heads, w.num_q_heads, w.head_dim
    kb = wl.normal_bf16(rng, (1, 2, hkv, d))
    vb = wl.normal_bf16(rng, (1, 2, hkv, d))
    qb = wl.normal_bf16(rng, (2, hq, d))
    store.step_begin([res["main"], res["aux"]])
    out = store.step_attn(0, wl.to_torch_bf16(kb[0], device), wl.to_torch_bf16(vb[0], device),
                          wl.to_torch_bf16(qb, device), scale=w.scale)
    torch.cuda.synchronize()
    kf, vf = wl.bf16_value(kb), wl.bf16_value(vb)
    views = []
    for j, h in enumerate((o["main"], o["aux"])):
        model.append(h, 1, kf[:, j:j + 1], vf[:, j:j + 1])
        k, v, _ = model.view(h)
        views.append((k[:, 0], v[:, 0]))
    ref = oatt.decode_batch(wl.bf16_value(qb), views, w.scale, hq // hkv)
    return max_abs(out.cpu().numpy(), ref)
