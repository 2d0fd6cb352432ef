"""GPU parity of extend attention (a chunk appended to the cache attends
causally to the cached prefix and to itself) through the C ABI, against the
float64 oracle: max abs error <= 5e-4 on the fp32 outputs.

Every reference is computed from the seeded bf16 inputs themselves, never
from what the library's pools hold: the small cases replay each append,
fork and eviction in the oracle's page model (``scenarios.Twin``), whose
logical view supplies the keys and values; the full-size case removes the
evicted spans from the seeded inputs with the oracle's keep mask."""

import math

import numpy as np
import pytest

from tests import scenarios as sc
from oracle import evict as oev
from oracle import extend as oex
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


def _twin(sq, hq, hkv, d, tokens, nl=1, seqs=4, seed=0):
    """A GPU store and the oracle's page model (with data) side by side."""
    return sc.Twin(sq, nl, hq, hkv, d, num_pages=2 * (tokens // 16 + 8) + 16, max_seqs=seqs,
                   max_pages_per_seq=tokens // 16 + 8, seed=seed)


def _extend_error(tw, seq, n, layer=0, pairs=None):
    """Runs extend for the last n tokens of seq on the GPU store and returns
    the max abs error against the oracle over the page model's view of the
    same sequence (all rows, or the sampled (row, KV head) pairs)."""
    import torch
    hq, hkv, d = tw.hq, tw.hkv, tw.d
    g = hq // hkv
    qb = wl.normal_bf16(tw.rng, (n, hq, d))
    out = tw.store.extend(layer, seq, wl.to_torch_bf16(qb, tw.device))
    torch.cuda.synchronize()
    k, v, _ = tw.model.view(seq)
    k, v = k[:, layer], v[:, layer]
    assert k.shape[0] == tw.store.seq_info(seq)["length"]
    qf = wl.bf16_value(qb)
    got = out.cpu().numpy()
    scale = 1 / math.sqrt(d)
    assert np.all(np.isfinite(got))
    if pairs is None:
        ref = oex.extend_attention(qf, k, v, scale, g)
        return float(np.max(np.abs(got - ref)))
    L = k.shape[0]
    err = 0.0
    for j, kv in pairs:
        last = L - n + j
        hs = slice(kv * g, kv * g + g)
        ref = oex.extend_attention(qf[j:j + 1, hs], k[: last + 1, kv:kv + 1],
                                   v[: last + 1, kv:kv + 1], scale, g)
        err = max(err, float(np.max(np.abs(got[j, hs] - ref[0]))))
    return err


SHAPES = [(4, 1, 64), (8, 2, 128), (8, 8, 128), (16, 2, 64), (4, 2, 128)]
CHUNKS = [(0, 1), (0, 45), (37, 33), (250, 130)]


@pytest.mark.parametrize("hq,hkv,d", SHAPES)
@pytest.mark.parametrize("prefix,n", CHUNKS)
def test_extend_matches_oracle(sq, hq, hkv, d, prefix, n):
    tw = _twin(sq, hq, hkv, d, prefix + n, seed=11 + prefix + hq + d)
    a = tw.create()
    if prefix:
        tw.append(a, prefix)
    tw.append(a, n)
    err = _extend_error(tw, a, n)
    print(f"extend hq={hq} hkv={hkv} d={d} prefix={prefix} n={n}: max abs err {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("hq,hkv,d,prefix,n", [(8, 8, 128, 300, 257), (32, 8, 128, 900, 200),
                                                (16, 2, 64, 1000, 61)])
def test_extend_several_query_blocks(sq, hq, hkv, d, prefix, n):
    tw = _twin(sq, hq, hkv, d, prefix + n, seed=21)
    a = tw.create()
    tw.append(a, prefix)
    tw.append(a, n)
    err = _extend_error(tw, a, n)
    print(f"extend hq={hq} hkv={hkv} d={d} prefix={prefix} n={n}: max abs err {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("hq,hkv,d", [(8, 2, 128), (4, 1, 64)])
@pytest.mark.parametrize("length", [64, 128, 192, 200, 256, 300, 384, 420])
def test_extend_key_block_counts(sq, hq, hkv, d, length):
    """One query block (a 16-token chunk) against 1 to 7 blocks of 64 keys,
    full and ragged: the kernel cycles its three block buffers a whole turn
    at a time and takes the last one or two blocks after the loop, so every
    count of turns and of blocks left over is covered."""
    n = 16
    tw = _twin(sq, hq, hkv, d, length, seed=170 + length)
    a = tw.create()
    tw.append(a, length - n)
    tw.append(a, n)
    err = _extend_error(tw, a, n)
    print(f"extend hq={hq} hkv={hkv} d={d} length={length}: max abs err {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (8, 2, 64)])
def test_extend_scores_far_above_the_running_reference(sq, hq, hkv, d):
    """Keys scaled by 16 and by 64 (exact in bf16) after ordinary ones: a
    row's later scores exceed its running reference by tens and then
    hundreds of log2 units, so the weights of those half blocks first sum
    past the 2^64 guard and then overflow to infinity; the kernel must raise
    the reference and take them again.  Ordinary keys after that carry
    weights far below it.  Chunks of 256 and 200 tokens cover several query
    blocks and the chunk's own diagonal."""
    tw = _twin(sq, hq, hkv, d, 1500, seed=131)
    a = tw.create()
    tw.append(a, 400)
    tw.append(a, 200, k_scale=16)
    tw.append(a, 150, k_scale=64)
    tw.append(a, 300)
    tw.append(a, 256, k_scale=4)
    err = _extend_error(tw, a, 256)
    print(f"extend hq={hq} hkv={hkv} d={d} scaled keys: max abs err {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("hq,hkv,d,prefix,n", [(32, 8, 128, 20000, 1), (32, 8, 128, 20000, 7),
                                                (32, 8, 128, 20000, 512), (16, 2, 64, 300, 1000),
                                                (8, 8, 128, 5000, 130)])
def test_extend_split_key_range(sq, hq, hkv, d, prefix, n):
    """Short chunks over long prefixes split each query block's key range
    over several workgroups and merge the partial rows (an auxiliary
    thread's prompt is such a chunk); with a long chunk over a short prefix
    the first query blocks leave later splits empty."""
    tw = _twin(sq, hq, hkv, d, prefix + n, seed=91)
    a = tw.create()
    tw.append(a, prefix)
    tw.append(a, n)
    if prefix + n > 5000:
        pairs = [(j, g) for j in sorted({0, n // 2, n - 1}) for g in (0, hkv - 1)]
        err = _extend_error(tw, a, n, pairs=pairs)
    else:
        err = _extend_error(tw, a, n)
    print(f"extend split hq={hq} d={d} prefix={prefix} n={n}: max abs err {err:.2e}")
    assert err <= TOL


def test_extend_whole_sequence_prefill(sq):
    """n = L: the first token sees only itself, so its rows equal its V (to
    fp32 rounding: its weight is 2^r with r the rounding error of the scaled
    score, |r| < 1e-6)."""
    import torch
    tw = _twin(sq, 8, 2, 128, 300, seed=31)
    a = tw.create()
    tw.append(a, 300)
    qb = wl.normal_bf16(tw.rng, (300, 8, 128))
    out = tw.store.extend(0, a, wl.to_torch_bf16(qb, "cuda"))
    torch.cuda.synchronize()
    k, v, _ = tw.model.view(a)
    got = out.cpu().numpy()
    for h in range(8):
        assert np.max(np.abs(got[0, h] - v[0, 0, h // 4])) <= 1e-6
    ref = oex.extend_attention(wl.bf16_value(qb), k[:, 0], v[:, 0], 1 / math.sqrt(128), 4)
    assert float(np.max(np.abs(got - ref))) <= TOL


def test_extend_after_eviction(sq):
    """A chunk appended after Phase 1 compacted the prefix (positions
    carried): the oracle evicts the same spans from the seeded inputs, and
    the pools must hold its compacted view bit for bit."""
    tw = _twin(sq, 32, 8, 128, 1400, seed=41)
    a = tw.create()
    tw.append(a, 1200, outlier=True)
    spans = [(17, 100), (130, 131), (300, 520), (600, 640), (900, 1111)]
    for c, (x, y) in enumerate(spans):
        tw.mark(a, c, x, y)
    tw.evict(a, [0, 2, 4])
    L0 = tw.store.seq_info(a)["length"]
    assert L0 == 1200 - 83 - 220 - 211
    tw.append(a, 150, outlier=True)
    err = _extend_error(tw, a, 150)
    print(f"extend after eviction (prefix {L0}): max abs err {err:.2e}")
    assert err <= TOL
    tw.check_state()


def test_extend_after_deferred_then_compacted(sq):
    """Spans masked by a deferred eviction, then compacted, before the chunk
    is appended: the oracle's view is the seeded inputs without them."""
    tw = _twin(sq, 16, 2, 64, 1000, seed=42)
    a = tw.create()
    tw.append(a, 800)
    for c, (x, y) in enumerate([(5, 60), (200, 333), (500, 517)]):
        tw.mark(a, c, x, y)
    tw.evict(a, [1], deferred=True)
    tw.evict(a, [0, 2])
    tw.append(a, 90)
    err = _extend_error(tw, a, 90)
    print(f"extend after deferred + physical eviction: max abs err {err:.2e}")
    assert err <= TOL
    tw.check_state()


def test_extend_on_forked_branch(sq):
    """The auxiliary thread forked mid-page (tail page copied) appends a chunk
    and attends over the aliased prefix pages."""
    tw = _twin(sq, 8, 2, 64, 700, seed=51)
    m = tw.create()
    tw.append(m, 500)
    aux = tw.fork(m, 489)
    tw.append(aux, 77)
    tw.append(m, 20)
    err = _extend_error(tw, aux, 77)
    err_m = _extend_error(tw, m, 20)
    print(f"extend on aux: {err:.2e}, on main: {err_m:.2e}")
    assert err <= TOL and err_m <= TOL
    tw.check_state()


def test_extend_other_layers(sq):
    tw = _twin(sq, 8, 2, 128, 400, nl=3, seed=61)
    a = tw.create()
    tw.append(a, 333)
    tw.append(a, 40)
    for layer in (2, 0):
        err = _extend_error(tw, a, 40, layer=layer)
        assert err <= TOL, (layer, err)


def test_extend_arguments(sq):
    import torch
    tw = _twin(sq, 8, 2, 64, 64, seed=71)
    s = tw.store
    a = tw.create()
    tw.append(a, 20)
    q = wl.device_normal_bf16((21, 8, 64), 73, "cuda")
    with pytest.raises(sq.SqError) as ei:
        s.extend(0, a, q)              # more new tokens than cached
    assert ei.value.code == sq.ERR_INVALID
    with pytest.raises(sq.SqError) as ei:
        s.extend(1, a, q[:5])          # no layer 1
    assert ei.value.code == sq.ERR_INVALID
    with pytest.raises(sq.SqError) as ei:
        s.extend(0, 3, q[:5])          # unknown sequence
    assert ei.value.code == sq.ERR_UNKNOWN_SEQ
    with pytest.raises(sq.SqError) as ei:
        s.extend(0, a, q[:5], scale=-0.125)  # the kernel needs a positive scale
    assert ei.value.code == sq.ERR_INVALID
    out = torch.full((0, 8, 64), 7.0, device="cuda")
    s.extend(0, a, q[:0], out=out)     # empty chunk: nothing to do
    st = s.stats()
    assert st["extend_calls"] == 0


def test_extend_full_size_sampled(sq):
    """The measured configuration: an 8192-token chunk appended to the 64K
    context after its tool spans were evicted (>= 65% of the tokens), 32
    query / 8 KV heads, head_dim 128.  The reference keys are the seeded
    inputs with the oracle's keep mask of the evicted spans applied, then
    the chunk's own; sampled rows of every KV head against the oracle."""
    import torch
    from paper_2602_22603_amd import drivers
    store, base, w, k, v = drivers.build_compaction64k(extra_tokens=8192 + 64)
    L = w.length
    keep, _dst, _src, n_kept, _f = oev.plan(L, [w.spans[c] for c in w.evict_ids])
    kept = torch.from_numpy(keep.astype(bool))
    k_kept, v_kept = k[0].cpu()[kept], v[0].cpu()[kept]   # bf16 [L', Hkv, D]
    del k, v
    store.evict(base, w.evict_ids)
    L0 = store.seq_info(base)["length"]
    assert L0 == n_kept
    assert np.array_equal(store.positions(base), np.flatnonzero(keep))
    n = 8192
    kn = wl.device_normal_bf16((1, n, 8, 128), 81, "cuda")
    vn = wl.device_normal_bf16((1, n, 8, 128), 82, "cuda")
    store.append(base, kn, vn)
    kf = wl.torch_bf16_to_f64(torch.cat([k_kept, kn[0].cpu()]))   # [L' + n, Hkv, D]
    vf = wl.torch_bf16_to_f64(torch.cat([v_kept, vn[0].cpu()]))
    del kn, vn, k_kept, v_kept
    q = wl.device_normal_bf16((n, 32, 128), 83, "cuda")
    out = store.extend(0, base, q)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    qf = wl.torch_bf16_to_f64(q)
    scale = 1 / math.sqrt(128)
    rows = [0, 1, 31, 32, 127, 128, 4095, 4096, 8190, 8191]
    err = 0.0
    for j in rows:
        last = n_kept + j
        for kv in range(8):
            hs = slice(4 * kv, 4 * kv + 4)
            ref = oex.extend_attention(qf[j:j + 1, hs], kf[: last + 1, kv:kv + 1],
                                       vf[: last + 1, kv:kv + 1], scale, 4)
            err = max(err, float(np.max(np.abs(got[j, hs] - ref[0]))))
    print(f"extend 8192 over compacted prefix {L0}: sampled max abs err {err:.2e}")
    assert err <= TOL
    st = store.stats()
    assert st["extend_tokens"] == n
    store.close()
    torch.cuda.empty_cache()
