"""Decode-phase attention over a KV cache, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed
----------------
The paper treats decode-phase attention over the whole KV cache as the
memory-bound step that eviction shrinks (§1; §3.4 "Compute and Memory Movement
Cost"; §4.5 "KV Cache Memory Reads").  It does not restate attention itself;
the definition used is standard scaled dot-product softmax attention of one
new query per head, with grouped KV heads (GQA, named in §2.1):

    g(h)   = h // G                  (G = Hq / Hkv consecutive query heads
                                      share one KV head)
    s[h,i] = scale * sum_d q[h,d] * k[i, g(h), d]
    m[h]   = max_i s[h,i]
    p[h,i] = exp(s[h,i] - m[h]) / sum_j exp(s[h,j] - m[h])
    out[h] = sum_i p[h,i] * v[i, g(h), :]

Masked attention (Algorithm 2 ``BuildMask``; "Simulated Eviction" in §3.3)
is the same with s[h,i] = -inf where mask[i] == 0; a head with every key
masked returns zeros.

Summation order
---------------
Every sum over keys and over the head dimension is taken in ascending index
order (``np.cumsum`` is a running sum).  With that order, attention over a
compacted cache and masked attention over the uncompacted cache are
bit-identical in float64: a masked key contributes an exact +0.0 and leaves
the maximum over the kept keys unchanged.

Sinks and windows (model variants; the paper names only its model)
--------------------------------------------------------------------
Two options of the attention itself, as some models define it:

* a learned sink logit per query head, ``sinks[h]`` (in the units of the
  scaled scores), joins the softmax as one more term of its denominator with
  no value:  out[h] = sum_i e^(s[h,i] - M) v_i / (e^(sinks[h] - M) +
  sum_i e^(s[h,i] - M)),  M = max(sinks[h], max_i s[h,i]).  A head whose
  keys are all masked then returns zeros as before.
* a window of W keys: a query attends only to the W most recent keys up to
  and including its own position (for a decode step, the last W of the L
  keys); it is the band mask ``window_mask(L, W)``.

Split partials
--------------
``partial`` returns (m, l, acc) with l = sum_i exp(s_i - m) and
acc = sum_i exp(s_i - m) v_i, unnormalised.  ``merge`` combines the partials
of any partition of the keys:
    M = max_s m_s;  out = sum_s e^(m_s - M) acc_s / sum_s e^(m_s - M) l_s,
an empty part being (-inf, 0, 0) and an all-empty head giving zeros.
"""

from __future__ import annotations

import numpy as np


def _as_f64(x):
    return np.asarray(x, dtype=np.float64)


def scores(q, k, scale, group, mask=None):
    """s[h, i] for query heads h and keys i; masked keys get -inf.

    q: [Hq, D]; k: [L, Hkv, D]; group = Hq // Hkv; mask: [L] (nonzero = keep).
    """
    q = _as_f64(q)
    k = _as_f64(k)
    hq, d = q.shape
    n_keys = k.shape[0]
    if hq % group != 0 or k.shape[1] * group != hq:
        raise ValueError("query heads must be group * kv heads")
    s = np.empty((hq, n_keys), dtype=np.float64)
    for h in range(hq):
        g = h // group
        if n_keys:
            # running sum over d, ascending: identical for a key wherever it sits
            dots = np.cumsum(k[:, g, :] * q[h][None, :], axis=1)[:, -1]
        else:
            dots = np.zeros(0)
        s[h] = scale * dots
    if mask is not None:
        keep = np.asarray(mask).astype(bool)
        s[:, ~keep] = -np.inf
    return s


def partial(q, k, v, scale, group, mask=None):
    """Unnormalised attention state (m, l, acc) per query head.

    m: [Hq] (-inf for a head with no unmasked key), l: [Hq], acc: [Hq, D].
    """
    v = _as_f64(v)
    s = scores(q, k, scale, group, mask)
    hq, n_keys = s.shape
    d = v.shape[2] if v.ndim == 3 else _as_f64(q).shape[1]
    m = np.full(hq, -np.inf)
    l = np.zeros(hq)
    acc = np.zeros((hq, d))
    for h in range(hq):
        if n_keys == 0:
            continue
        mh = s[h].max()
        if mh == -np.inf:
            continue
        e = np.exp(s[h] - mh)  # exp(-inf) = +0.0 for masked keys
        m[h] = mh
        l[h] = np.cumsum(e)[-1]
        acc[h] = np.cumsum(e[:, None] * v[:, h // group, :], axis=0)[-1]
    return m, l, acc


def weights(q, k, scale, group, mask=None):
    """Softmax weights p[h, i] (rows sum to 1; an all-masked row is 0)."""
    s = scores(q, k, scale, group, mask)
    p = np.zeros_like(s)
    for h in range(s.shape[0]):
        if s.shape[1] == 0:
            continue
        mh = s[h].max()
        if mh == -np.inf:
            continue
        e = np.exp(s[h] - mh)
        p[h] = e / np.cumsum(e)[-1]
    return p


def attention(q, k, v, scale, group, mask=None, sinks=None):
    """out[h] = sum_i p[h, i] v[i, h // group]; zeros for an all-masked head.
    With ``sinks`` ([Hq]) each head's softmax has one more denominator term
    e^(sinks[h]) carrying no value."""
    m, l, acc = partial(q, k, v, scale, group, mask)
    out = np.zeros_like(acc)
    if sinks is not None:
        sinks = _as_f64(sinks)
        for h in range(acc.shape[0]):
            if l[h] == 0:
                continue
            big = max(m[h], sinks[h])
            scale_kv = np.exp(m[h] - big)    # rescales the keys' sum and values
            l_all = l[h] * scale_kv + np.exp(sinks[h] - big)
            out[h] = acc[h] * scale_kv / l_all
        return out
    live = l > 0
    out[live] = acc[live] / l[live][:, None]
    return out


def window_mask(n_keys, window):
    """Keep mask of a decode query over n_keys keys with a window of
    ``window`` keys (0: every key): the last ``window`` keys."""
    keep = np.ones(n_keys, dtype=np.uint8)
    if window > 0:
        keep[: max(0, n_keys - window)] = 0
    return keep


def masked_attention(q, k, v, mask, scale, group):
    """Attention with the keys where ``mask == 0`` removed by -inf scores."""
    return attention(q, k, v, scale, group, mask=mask)


def merge(parts):
    """Combine split partials [(m, l, acc), ...] of one set of heads.

    Each m: [Hq], l: [Hq], acc: [Hq, D].  Empty parts carry m = -inf.
    """
    ms = np.stack([_as_f64(p[0]) for p in parts])  # [S, Hq]
    ls = np.stack([_as_f64(p[1]) for p in parts])
    accs = np.stack([_as_f64(p[2]) for p in parts])  # [S, Hq, D]
    big_m = ms.max(axis=0)
    out = np.zeros(accs.shape[1:])
    for h in range(ms.shape[1]):
        if big_m[h] == -np.inf:
            continue
        w = np.exp(ms[:, h] - big_m[h])  # empty parts: exp(-inf) = 0
        num = np.cumsum(w[:, None] * accs[:, h, :], axis=0)[-1]
        den = np.cumsum(w * ls[:, h])[-1]
        out[h] = num / den
    return out


def decode_batch(q, views, scale, group, masks=None, window=0, sinks=None):
    """One decode step for a batch: q [B, Hq, D]; views[b] = (k, v) with
    k, v: [L_b, Hkv, D] (the sequence's logical view for one layer);
    optional window (in keys) and per-head sinks [Hq]."""
    q = _as_f64(q)
    out = np.zeros((q.shape[0], q.shape[1], q.shape[2]))
    for b, (k, v) in enumerate(views):
        mask = None if masks is None else masks[b]
        if window > 0:
            band = window_mask(np.asarray(k).shape[0], window)
            mask = band if mask is None else band * np.asarray(mask)
        out[b] = attention(q[b], k, v, scale, group, mask, sinks)
    return out
