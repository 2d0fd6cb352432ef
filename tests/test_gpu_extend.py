"""GPU parity of extend attention (a chunk appended to the cache attends
causally to the cached prefix and to itself) through the C ABI, against the
float64 oracle on the same bf16 inputs: max abs error <= 5e-4 on the fp32
outputs."""

import math

import numpy as np
import pytest

from tests import scenarios as sc
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


def _store(sq, hq, hkv, d, tokens, nl=1, seqs=4):
    pages = 2 * (tokens // 16 + 8) + 16
    return sq.Store(nl, hq, hkv, d, num_pages=pages, max_seqs=seqs,
                    max_pages_per_seq=tokens // 16 + 8, device="cuda")


def _append(store, seq, n, seed, outlier=False):
    k = wl.device_normal_bf16((store.num_layers, n, store.num_kv_heads, store.head_dim), seed, "cuda")
    v = wl.device_normal_bf16((store.num_layers, n, store.num_kv_heads, store.head_dim), seed + 1, "cuda")
    if outlier:  # four channels x8 (exact in bf16)
        k[..., :4] *= 8
        v[..., 5:9] *= 8
    store.append(seq, k, v)


def _extend_error(store, seq, n, seed, layer=0, pairs=None):
    """Runs extend for the last n tokens of seq and returns the max abs error
    against the oracle (all rows, or the sampled (row, KV head) pairs)."""
    import torch
    hq, hkv, d = store.num_q_heads, store.num_kv_heads, store.head_dim
    g = hq // hkv
    q = wl.device_normal_bf16((n, hq, d), seed, "cuda")
    out = store.extend(layer, seq, q)
    torch.cuda.synchronize()
    k, v, _ = sc.seq_view(store, seq, layers=[layer])
    qf = wl.torch_bf16_to_f64(q)
    got = out.cpu().numpy()
    scale = 1 / math.sqrt(d)
    if pairs is None:
        ref = oex.extend_attention(qf, k[:, 0], v[:, 0], scale, g)
        assert np.all(np.isfinite(got))
        return float(np.max(np.abs(got - ref)))
    L = k.shape[0]
    err = 0.0
    for j, kv in pairs:
        last = L - n + j
        hs = slice(kv * g, kv * g + g)
        ref = oex.extend_attention(qf[j:j + 1, hs], k[: last + 1, 0, kv:kv + 1],
                                   v[: last + 1, 0, kv:kv + 1], scale, g)
        err = max(err, float(np.max(np.abs(got[j, hs] - ref[0]))))
    return err


SHAPES = [(4, 1, 64), (8, 2, 128), (8, 8, 128), (16, 2, 64), (4, 2, 128)]
CHUNKS = [(0, 1), (0, 45), (37, 33), (250, 130)]


@pytest.mark.parametrize("hq,hkv,d", SHAPES)
@pytest.mark.parametrize("prefix,n", CHUNKS)
def test_extend_matches_oracle(sq, hq, hkv, d, prefix, n):
    s = _store(sq, hq, hkv, d, prefix + n)
    a = s.seq_create()
    if prefix:
        _append(s, a, prefix, 11 + prefix)
    _append(s, a, n, 13 + n)
    err = _extend_error(s, a, n, 17 + hq + d)
    print(f"extend hq={hq} hkv={hkv} d={d} prefix={prefix} n={n}: max abs err {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("hq,hkv,d,prefix,n", [(8, 8, 128, 300, 257), (32, 8, 128, 900, 200),
                                                (16, 2, 64, 1000, 61)])
def test_extend_several_query_blocks(sq, hq, hkv, d, prefix, n):
    s = _store(sq, hq, hkv, d, prefix + n)
    a = s.seq_create()
    _append(s, a, prefix, 21)
    _append(s, a, n, 23)
    err = _extend_error(s, a, n, 29)
    print(f"extend hq={hq} hkv={hkv} d={d} prefix={prefix} n={n}: max abs err {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("hq,hkv,d,prefix,n", [(32, 8, 128, 20000, 1), (32, 8, 128, 20000, 7),
                                                (32, 8, 128, 20000, 512), (16, 2, 64, 300, 1000),
                                                (8, 8, 128, 5000, 130)])
def test_extend_split_key_range(sq, hq, hkv, d, prefix, n):
    """Short chunks over long prefixes split each query block's key range
    over several workgroups and merge the partial rows (an auxiliary
    thread's prompt is such a chunk); with a long chunk over a short prefix
    the first query blocks leave later splits empty."""
    s = _store(sq, hq, hkv, d, prefix + n)
    a = s.seq_create()
    _append(s, a, prefix, 91)
    _append(s, a, n, 93)
    if prefix + n > 5000:
        pairs = [(j, g) for j in sorted({0, n // 2, n - 1}) for g in (0, hkv - 1)]
        err = _extend_error(s, a, n, 97, pairs=pairs)
    else:
        err = _extend_error(s, a, n, 97)
    print(f"extend split hq={hq} d={d} prefix={prefix} n={n}: max abs err {err:.2e}")
    assert err <= TOL


def test_extend_whole_sequence_prefill(sq):
    """n = L: the first token sees only itself, so its rows equal its V (to
    fp32 rounding: its weight is 2^r with r the rounding error of the scaled
    score, |r| < 1e-6)."""
    import torch
    s = _store(sq, 8, 2, 128, 300)
    a = s.seq_create()
    _append(s, a, 300, 31)
    q = wl.device_normal_bf16((300, 8, 128), 37, "cuda")
    out = s.extend(0, a, q)
    torch.cuda.synchronize()
    k, v, _ = sc.seq_view(s, a, layers=[0])
    got = out.cpu().numpy()
    for h in range(8):
        assert np.max(np.abs(got[0, h] - v[0, 0, h // 4])) <= 1e-6
    ref = oex.extend_attention(wl.torch_bf16_to_f64(q), k[:, 0], v[:, 0], 1 / math.sqrt(128), 4)
    assert float(np.max(np.abs(got - ref))) <= TOL


def test_extend_after_eviction(sq):
    """A chunk appended after Phase 1 compacted the prefix (positions carried)."""
    s = _store(sq, 32, 8, 128, 1400)
    a = s.seq_create()
    _append(s, a, 1200, 41, outlier=True)
    spans = [(17, 100), (130, 131), (300, 520), (600, 640), (900, 1111)]
    for c, (x, y) in enumerate(spans):
        s.span_mark(a, c, x, y)
    s.evict(a, [0, 2, 4])
    L0 = s.seq_info(a)["length"]
    assert L0 == 1200 - 83 - 220 - 211
    _append(s, a, 150, 43, outlier=True)
    err = _extend_error(s, a, 150, 47)
    print(f"extend after eviction (prefix {L0}): max abs err {err:.2e}")
    assert err <= TOL


def test_extend_on_forked_branch(sq):
    """The auxiliary thread forked mid-page (tail page copied) appends a chunk
    and attends over the aliased prefix pages."""
    s = _store(sq, 8, 2, 64, 700)
    m = s.seq_create()
    _append(s, m, 500, 51)
    aux = s.fork(m, 489)
    _append(s, aux, 77, 53)
    _append(s, m, 20, 55)
    err = _extend_error(s, aux, 77, 57)
    err_m = _extend_error(s, m, 20, 59)
    print(f"extend on aux: {err:.2e}, on main: {err_m:.2e}")
    assert err <= TOL and err_m <= TOL


def test_extend_other_layers(sq):
    s = _store(sq, 8, 2, 128, 400, nl=3)
    a = s.seq_create()
    _append(s, a, 333, 61)
    _append(s, a, 40, 63)
    for layer in (2, 0):
        err = _extend_error(s, a, 40, 67 + layer, layer=layer)
        assert err <= TOL, (layer, err)


def test_extend_arguments(sq):
    import torch
    s = _store(sq, 8, 2, 64, 64)
    a = s.seq_create()
    _append(s, a, 20, 71)
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
    query / 8 KV heads, head_dim 128; sampled rows against the oracle."""
    import torch
    from paper_2602_22603_amd import drivers
    store, base, w, k, v = drivers.build_compaction64k(extra_tokens=8192 + 64)
    del k, v
    store.evict(base, w.evict_ids)
    L0 = store.seq_info(base)["length"]
    n = 8192
    kn = wl.device_normal_bf16((1, n, 8, 128), 81, "cuda")
    vn = wl.device_normal_bf16((1, n, 8, 128), 82, "cuda")
    store.append(base, kn, vn)
    del kn, vn
    pairs = [(0, 0), (1, 7), (31, 3), (32, 4), (4095, 1), (4096, 6), (8190, 2), (8191, 5)]
    err = _extend_error(store, base, n, 83, pairs=pairs)
    print(f"extend 8192 over compacted prefix {L0}: sampled max abs err {err:.2e}")
    assert err <= TOL
    st = store.stats()
    assert st["extend_tokens"] == n
    store.close()
    torch.cuda.empty_cache()
