"""GPU parity of the attention options (per-head softmax sinks and key
windows, sq_attn_opts) through the C ABI against the oracle's
``decode_batch`` / ``extend_attention`` with the same options: max abs error
<= 5e-4 on the fp32 outputs, over decode in every mode, the fused decode
step (windowed and full layers in one step, eager and replayed from a
capture) and extend (one launch and split key ranges)."""

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


def _branches(t):
    """A main thread, its auxiliary fork with its own tokens, a sequence
    ending mid-page, a one-token one and an empty one."""
    main = t.create()
    t.append(main, 700)
    aux = t.fork(main, 640)
    t.append(aux, 29)
    other = t.create()
    t.append(other, 47)
    one = t.create()
    t.append(one, 1)
    empty = t.create()
    return [main, aux, other, one, empty]


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (8, 2, 64), (64, 8, 64), (4, 4, 128)])
@pytest.mark.parametrize("window", [0, 1, 5, 16, 17, 40, 100, 5000])
@pytest.mark.parametrize("with_sinks", [False, True])
def test_decode_window_sinks(sq, hq, hkv, d, window, with_sinks):
    """Every mode: windows inside the first page, on page boundaries, across
    the fork point and longer than every sequence; sinks on and off."""
    if window == 0 and not with_sinks:
        pytest.skip("no option: covered by the decode parity tests")
    t = sc.Twin(sq, 1, hq, hkv, d, 260, 6, 60, seed=400 + window + hq)
    seqs = _branches(t)
    sinks = t.sinks() if with_sinks else None
    errs, _ = t.decode_errors(seqs, window=window, sinks=sinks)
    print(f"decode window={window} sinks={with_sinks} hq={hq} hkv={hkv} d={d}: {errs}")
    assert max(errs.values()) <= TOL, errs


def test_decode_window_after_eviction(sq):
    """A window over a compacted sequence counts logical indices of the
    compacted cache (kept tokens only)."""
    t = sc.Twin(sq, 1, 8, 2, 128, 200, 4, 60, seed=431)
    a = t.create()
    t.append(a, 600)
    for c, (x, y) in enumerate([(500, 530), (560, 561), (570, 590)]):
        t.mark(a, c, x, y)
    t.evict(a, [0, 1, 2])
    for w in (7, 40, 64):
        errs, _ = t.decode_errors([a], window=w, sinks=t.sinks())
        assert max(errs.values()) <= TOL, (w, errs)


def test_decode_dominant_and_negligible_sinks(sq):
    """A sink far above every score takes almost all of the weight (outputs
    near 0), one far below leaves plain softmax; both match the oracle."""
    t = sc.Twin(sq, 1, 8, 2, 64, 100, 4, 40, seed=432)
    a = t.create()
    t.append(a, 300)
    b = t.fork(a, 288)
    t.append(b, 3)
    for level in (40.0, -40.0):
        sinks = np.full(8, level, np.float32)
        sinks[::3] = 0.5
        errs, _ = t.decode_errors([a, b], sinks=sinks)
        assert max(errs.values()) <= TOL, (level, errs)


def test_decode_long_window_shared_prefix(sq):
    """A 12K-token main thread and two forks near its end, window 4096 with
    sinks (the windows meet on the shared pages), next to a full-attention
    call on the same batch."""
    t = sc.Twin(sq, 1, 64, 8, 64, 1700, 4, 800, seed=433)
    m = t.create()
    t.append(m, 12000)
    a = t.fork(m, 11904)
    t.append(a, 100)
    b = t.fork(m, 11990)
    t.append(b, 7)
    sinks = t.sinks()
    errs, _ = t.decode_errors([m, a, b], window=4096, sinks=sinks)
    assert max(errs.values()) <= TOL, errs
    errs, _ = t.decode_errors([m, a, b], sinks=sinks)
    assert max(errs.values()) <= TOL, errs


@pytest.mark.parametrize("mi", [0, 1, 2, 3])
@pytest.mark.parametrize("window", [1, 2, 17, 64])
def test_step_windowed_and_full_layers(sq, mi, window):
    """Two layers per step, the first windowed, the second full, with sinks
    on the first: 20 steps cross page boundaries; the pools equal the
    oracle's afterwards.  Window 1 leaves only the new token."""
    mode = [sq.ATTN_AUTO, sq.ATTN_STREAM, sq.ATTN_SHARED_PREFIX, sq.ATTN_MFMA][mi]
    t = sc.Twin(sq, 2, 32, 8, 128, 300, 6, 80, seed=440 + mi + window)
    seqs = _branches(t)
    sinks = [t.sinks(), None]
    worst = 0.0
    for _ in range(20):
        err, _ = t.step(seqs, mode, window=window, layer_windows=[window, 0], sinks=sinks)
        worst = max(worst, err)
        assert err <= TOL
    t.check_state()
    print(f"windowed steps mode {mode} window {window}: max abs err {worst:.2e}")


def test_step_window_one_attends_to_the_new_token(sq):
    """Window 1: the only key is the new token, so without sinks the output
    is v_new exactly; with a sink s the weight is 1 / (1 + e^(s - score))."""
    import torch
    s = sq.Store(1, 8, 2, 128, 16, 4, 8, device="cuda")
    a = s.seq_create()
    k0 = wl.device_normal_bf16((1, 40, 2, 128), 1, "cuda")
    s.append(a, k0, k0)
    kn = wl.device_normal_bf16((1, 2, 128), 5, "cuda")
    vn = wl.device_normal_bf16((1, 2, 128), 6, "cuda")
    q = wl.device_normal_bf16((1, 8, 128), 7, "cuda")
    s.step_begin([a], window=1)
    out = s.step_attn(0, kn, vn, q, window=1)
    torch.cuda.synchronize()
    assert torch.equal(out, vn.float().repeat_interleave(4, dim=1))
    s.close()


def test_captured_windowed_step_replays(sq):
    """A capture of one step's windowed and full layers (with sinks) replays
    for six more steps, each begun with the same window."""
    import torch
    nl, hq, hkv, d, w = 2, 8, 2, 128, 24
    t = sc.Twin(sq, nl, hq, hkv, d, 400, 6, 100, seed=450)
    main = t.create()
    t.append(main, 400)
    aux = t.fork(main, 390)
    t.append(aux, 5)
    seqs = [main, aux]
    sinks = [t.sinks(), t.sinks()]
    err, _ = t.step(seqs, window=w, layer_windows=[w, 0], sinks=sinks)
    assert err <= TOL
    sk = [torch.from_numpy(x).to("cuda") for x in sinks]
    g = dict(k=torch.zeros((nl, 2, hkv, d), dtype=torch.bfloat16, device="cuda"),
             v=torch.zeros((nl, 2, hkv, d), dtype=torch.bfloat16, device="cuda"),
             q=torch.zeros((nl, 2, hq, d), dtype=torch.bfloat16, device="cuda"),
             out=[torch.zeros((2, hq, d), dtype=torch.float32, device="cuda") for _ in range(nl)],
             graph=torch.cuda.CUDAGraph())
    with torch.cuda.graph(g["graph"]):
        for l in range(nl):
            t.store.step_attn(l, g["k"][l], g["v"][l], g["q"][l], out=g["out"][l],
                              window=[w, 0][l], sinks=sk[l])
    for r in range(6):
        err, _ = t.step(seqs, window=w, layer_windows=[w, 0], sinks=sinks, graph=g)
        print(f"windowed replay {r}: max abs err {err:.2e}")
        assert err <= TOL, (r, err)
        if r == 2:
            t.append(aux, 20)
    t.check_state()


def _extend_case(sq, hq, hkv, d, prefix, n, window, with_sinks, seed):
    import torch
    t = sc.Twin(sq, 1, hq, hkv, d, (prefix + n) // 16 + 24, 2, (prefix + n) // 16 + 8, seed=seed)
    a = t.create()
    if prefix:
        t.append(a, prefix)
    t.append(a, n)
    sinks = t.sinks() if with_sinks else None
    qb = wl.normal_bf16(t.rng, (n, hq, d))
    q = wl.to_torch_bf16(qb, "cuda")
    sk = None if sinks is None else torch.from_numpy(sinks).to("cuda")
    out = t.store.extend(0, a, q, window=window, sinks=sk)
    torch.cuda.synchronize()
    k, v, _ = t.model.view(a)
    ref = oex.extend_attention(wl.bf16_value(qb), k[:, 0], v[:, 0], 1 / math.sqrt(d), hq // hkv,
                               window=window,
                               sinks=None if sinks is None else sinks.astype(np.float64))
    got = out.cpu().numpy()
    assert np.all(np.isfinite(got))
    return float(np.max(np.abs(got - ref)))


@pytest.mark.parametrize("hq,hkv,d", [(8, 2, 128), (64, 8, 64), (8, 8, 128)])
@pytest.mark.parametrize("prefix,n", [(0, 45), (37, 33), (250, 130), (600, 300)])
@pytest.mark.parametrize("window,with_sinks", [(1, False), (16, True), (50, False), (128, True),
                                               (0, True), (10000, True)])
def test_extend_window_sinks(sq, hq, hkv, d, prefix, n, window, with_sinks):
    """Windows shorter than a key block, a query block, the chunk and longer
    than the sequence; sinks on and off; several query blocks."""
    err = _extend_case(sq, hq, hkv, d, prefix, n, window, with_sinks, 460 + prefix + window)
    print(f"extend window={window} sinks={with_sinks} prefix={prefix} n={n}: {err:.2e}")
    assert err <= TOL


@pytest.mark.parametrize("prefix,n,window", [(20000, 1, 4096), (20000, 7, 128), (9000, 64, 700),
                                             (20000, 40, 0)])
def test_extend_window_split_key_range(sq, prefix, n, window):
    """Short chunks after long prefixes split their key range: with a window
    the split covers the window's blocks only (sinks join in the merge)."""
    err = _extend_case(sq, 32, 8, 128, prefix, n, window, True, 470 + n)
    print(f"extend split window={window} prefix={prefix} n={n}: {err:.2e}")
    assert err <= TOL


def test_option_arguments(sq):
    """Negative windows, a nonzero reserved field, misaligned sinks and a
    step window other than the step's are refused."""
    import ctypes as C
    import torch
    s = sq.Store(2, 8, 2, 64, 32, 4, 8, device="cuda")
    a = s.seq_create()
    k0 = wl.device_normal_bf16((2, 20, 2, 64), 1, "cuda")
    s.append(a, k0, k0)
    q = wl.device_normal_bf16((1, 8, 64), 2, "cuda")
    out = torch.zeros((1, 8, 64), dtype=torch.float32, device="cuda")
    with pytest.raises(sq.SqError):
        s.decode(0, [a], q, out=out, window=-1)
    with pytest.raises(sq.SqError):
        s.decode(0, [a], q, out=out, sinks=torch.zeros(7, device="cuda"))
    o = sq.AttnOpts()
    o.reserved = 1
    seqs = (C.c_int32 * 1)(a)
    assert sq.lib().sq_decode_attn_ex(s._handle, 0, seqs, 1, q.data_ptr(), out.data_ptr(),
                                      0.125, sq.ATTN_AUTO, C.byref(o), None) == sq.ERR_INVALID
    o.reserved = 0
    o.sinks = torch.zeros(16, device="cuda").data_ptr() + 2
    assert sq.lib().sq_decode_attn_ex(s._handle, 0, seqs, 1, q.data_ptr(), out.data_ptr(),
                                      0.125, sq.ATTN_AUTO, C.byref(o), None) == sq.ERR_INVALID
    with pytest.raises(sq.SqError):
        s.step_begin([a], window=-3)
    s.step_begin([a], window=8)
    kn = wl.device_normal_bf16((1, 2, 64), 3, "cuda")
    with pytest.raises(sq.SqError):
        s.step_attn(0, kn, kn, q, window=9)
    s.step_attn(0, kn, kn, q, window=8)
    s.step_attn(1, kn, kn, q)
    s.step_begin([a])                  # no windowed plan: a window is refused
    with pytest.raises(sq.SqError):
        s.step_attn(0, kn, kn, q, window=8)
    torch.cuda.synchronize()
    s.close()
