"""GPU parity of the 8-bit (E4M3) KV store (SQ_STORE_KV_FP8) through the C
ABI against the oracle: the stored codes equal the oracle's quantisation
bit for bit (appends and fused steps), fork and eviction move codes
unchanged, every code converts exactly, and attention over the stored
values matches the oracle's (max abs error <= 5e-4) in every mode the store
runs."""

import numpy as np
import pytest

from oracle import fp8 as of8
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


def _scales(nl):
    """Per-layer scales near what a calibration of unit-variance K/V gives
    (largest |x| / 448 ~ 0.01), one layer with scale 1."""
    base = np.array([[0.011, 0.0095], [1.0, 1.0], [0.02, 0.013]], dtype=np.float32)
    return base[:nl]


def _codes(store, seq, layer):
    """The K codes [L, Hkv, D] and V codes [L, Hkv, D] the pools hold for seq."""
    import torch
    pt = store.page_table(seq)
    n = store.seq_info(seq)["length"]
    tok = torch.arange(n, device="cuda")
    pages = torch.tensor(pt, device="cuda", dtype=torch.int64)[tok // 16]
    slots = tok % 16
    k = store.k_pool[layer][:, pages, slots, :].permute(1, 0, 2)
    v = store.v_pool[layer].permute(0, 1, 3, 2)[:, pages, slots, :].permute(1, 0, 2)
    return k.cpu().numpy(), v.cpu().numpy()


def test_every_code_converts_exactly(sq):
    """One token whose 256 V values are the 256 E4M3 values (NaN codes
    replaced by +-448): quantising them with scale 1 gives back each code,
    and attention over one key returns v exactly."""
    import torch
    s = sq.Store(1, 4, 2, 128, 8, 2, 4, device="cuda", kv_scales=[[1.0, 1.0]])
    a = s.seq_create()
    codes = np.arange(256, dtype=np.int64)
    codes[0x7F], codes[0xFF] = 0x7E, 0xFE
    vals = of8.decode(codes).reshape(1, 1, 2, 128)
    vb = torch.from_numpy(vals.astype(np.float32)).to(torch.bfloat16).to("cuda")
    assert np.array_equal(vb.float().cpu().numpy().astype(np.float64), vals)  # exact in bf16
    kb = torch.zeros_like(vb)
    s.append(a, kb, vb)
    _, vc = _codes(s, a, 0)
    assert np.array_equal(vc.reshape(-1), codes.astype(np.uint8))
    q = wl.device_normal_bf16((1, 4, 128), 3, "cuda")
    for mode in (sq.ATTN_AUTO, sq.ATTN_MFMA):
        out = s.decode(0, [a], q, mode=mode)
        torch.cuda.synchronize()
        got = out.cpu().numpy()[0].astype(np.float64)
        want = np.repeat(vals[0, 0], 2, axis=0)  # query heads 0, 1 -> KV head 0; 2, 3 -> 1
        assert np.array_equal(got, want), mode
    s.close()


@pytest.mark.parametrize("d", [64, 128])
def test_appended_codes_are_the_oracle_quantisation(sq, d):
    """Codes of a long append (partial first page, whole pages, a ragged
    tail) and of single-token appends equal the oracle's, sign of zero
    included; values far beyond 448 * scale saturate."""
    import torch
    nl = 3
    scales = _scales(nl)
    s = sq.Store(nl, 8, 2, d, 64, 4, 32, device="cuda", kv_scales=scales)
    a = s.seq_create()
    rng = np.random.default_rng(700 + d)
    chunks = [5, 300, 1, 1, 27]
    ks, vs = [], []
    for n in chunks:
        k = wl.normal_bf16(rng, (nl, n, 2, d))
        v = wl.normal_bf16(rng, (nl, n, 2, d))
        kf = wl.bf16_value(k)
        if n == 300:  # outliers, tiny values and signed zeros
            kf2 = kf.copy()
            kf2[:, 3, 0, :4] = [1e6, -1e6, 0.0, -0.0]
            kf2[:, 4, 0, :2] = [1e-6, -1e-6]
            k = wl.bf16_bits(kf2.astype(np.float32))
        s.append(a, wl.to_torch_bf16(k, "cuda"), wl.to_torch_bf16(v, "cuda"))
        ks.append(wl.bf16_value(k))
        vs.append(wl.bf16_value(v))
    torch.cuda.synchronize()
    kall, vall = np.concatenate(ks, axis=1), np.concatenate(vs, axis=1)
    for l in range(nl):
        kc, vc = _codes(s, a, l)
        assert np.array_equal(kc, of8.quantize(kall[l], scales[l, 0])), l
        assert np.array_equal(vc, of8.quantize(vall[l], scales[l, 1])), l
    s.close()


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (8, 2, 64), (64, 8, 64), (4, 4, 128)])
def test_fp8_decode_fork_evict(sq, hq, hkv, d):
    """Main thread, its fork (aligned and mid-page), eviction while the
    branch lives and a deferred eviction: pools equal the oracle's values bit
    for bit, attention in every mode within 5e-4 (STREAM and the singletons
    of SHARED_PREFIX read the codes on the VALU kernel)."""
    import torch
    t = sc.Twin(sq, 2, hq, hkv, d, 400, 6, 80, seed=710 + hq + d, kv_scales=_scales(2))
    main = t.create()
    t.append(main, 700)
    aux = t.fork(main, 640)
    t.append(aux, 29)
    mid = t.fork(main, 333)
    t.append(mid, 3)
    for c, (x, y) in enumerate([(10, 90), (200, 230), (400, 433)]):
        t.mark(main, c, x, y)
    t.check_state()
    modes = [sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA]
    for layer in (0, 1):
        errs, _ = t.decode_errors([main, aux, mid], modes=modes, layer=layer)
        assert max(errs.values()) <= TOL, (layer, errs)
    t.evict(main, [0, 1])
    t.evict(main, [2], deferred=True)
    t.check_state()
    errs, _ = t.decode_errors([main, aux, mid], modes=modes)
    assert max(errs.values()) <= TOL, errs
    t.compact(main)
    t.check_state()
    errs, _ = t.decode_errors([main, aux, mid], modes=modes)
    assert max(errs.values()) <= TOL, errs
    torch.cuda.synchronize()


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (8, 2, 64), (64, 8, 64)])
@pytest.mark.parametrize("prefix,n,window", [(0, 45, 0), (250, 130, 0), (600, 300, 50),
                                             (9000, 7, 0)])
def test_fp8_extend(sq, hq, hkv, d, prefix, n, window):
    """Extend over an 8-bit store (codes converted as each block is staged):
    one launch, several query blocks, a window, a split key range; sinks."""
    import math
    import torch
    from oracle import extend as oex
    t = sc.Twin(sq, 2, hq, hkv, d, (prefix + n) // 16 + 24, 2, (prefix + n) // 16 + 8,
                seed=740 + prefix + n, kv_scales=_scales(2))
    a = t.create()
    if prefix:
        t.append(a, prefix)
    t.append(a, n)
    sinks = t.sinks()
    qb = wl.normal_bf16(t.rng, (n, hq, d))
    for layer in (0, 1):
        out = t.store.extend(layer, a, wl.to_torch_bf16(qb, "cuda"), window=window,
                             sinks=torch.from_numpy(sinks).to("cuda"))
        torch.cuda.synchronize()
        k, v, _ = t.model.view(a)
        ref = oex.extend_attention(wl.bf16_value(qb), k[:, layer], v[:, layer], 1 / math.sqrt(d),
                                   hq // hkv, window=window, sinks=sinks.astype(np.float64))
        err = float(np.max(np.abs(out.cpu().numpy() - ref)))
        print(f"fp8 extend layer={layer} prefix={prefix} n={n} window={window}: {err:.2e}")
        assert err <= TOL


@pytest.mark.parametrize("length", [128, 192, 256, 300])
def test_fp8_extend_key_block_counts(sq, length):
    """An 8-bit store's extend over 2 to 5 blocks of 64 keys (its converted
    copies rotate through the kernel's block buffers like the bf16 ones)."""
    import math
    import torch
    from oracle import extend as oex
    hq, hkv, d, n = 8, 2, 128, 16
    t = sc.Twin(sq, 1, hq, hkv, d, length // 16 + 24, 2, length // 16 + 8,
                seed=780 + length, kv_scales=_scales(1))
    a = t.create()
    t.append(a, length - n)
    t.append(a, n)
    qb = wl.normal_bf16(t.rng, (n, hq, d))
    out = t.store.extend(0, a, wl.to_torch_bf16(qb, "cuda"))
    torch.cuda.synchronize()
    k, v, _ = t.model.view(a)
    ref = oex.extend_attention(wl.bf16_value(qb), k[:, 0], v[:, 0], 1 / math.sqrt(d), hq // hkv)
    err = float(np.max(np.abs(out.cpu().numpy() - ref)))
    print(f"fp8 extend length={length}: {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("mi", [0, 1, 2, 3])
def test_fp8_steps(sq, mi):
    """Fused decode steps on an 8-bit store: the new token is stored as its
    codes in the merge and attended as stored (pools equal the oracle's after
    20 steps); windowed layers with sinks too."""
    mode = [sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA][mi]
    t = sc.Twin(sq, 2, 32, 8, 128, 300, 6, 80, seed=720 + mi, kv_scales=_scales(2))
    main = t.create()
    t.append(main, 700)
    aux = t.fork(main, 640)
    t.append(aux, 29)
    other = t.create()
    t.append(other, 47)
    seqs = [main, aux, other]
    sinks = [t.sinks(), None]
    for r in range(20):
        err, _ = t.step(seqs, mode, window=24, layer_windows=[24, 0], sinks=sinks)
        assert err <= TOL, (r, err)
    t.check_state()


def test_fp8_captured_step_replays(sq):
    import torch
    nl, hq, hkv, d = 2, 8, 2, 128
    t = sc.Twin(sq, nl, hq, hkv, d, 300, 6, 80, seed=730, kv_scales=_scales(2))
    main = t.create()
    t.append(main, 400)
    aux = t.fork(main, 390)
    t.append(aux, 5)
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
    for r in range(6):
        err, _ = t.step(seqs, graph=g)
        assert err <= TOL, (r, err)
        if r == 2:
            t.append(aux, 20)
    t.check_state()


def test_fp8_configuration_errors(sq):
    with pytest.raises(sq.SqError):
        sq.Store(2, 8, 2, 64, 16, 2, 8, device="cuda", kv_scales=[[1.0, 1.0], [0.0, 1.0]])
    with pytest.raises(sq.SqError):
        sq.Store(1, 8, 2, 64, 16, 2, 8, device="cuda", kv_scales=[[float("nan"), 1.0]])
