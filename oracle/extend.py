"""Extend (chunked prefill) attention over a KV cache, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed
----------------
Algorithm 1 grows the main thread's context by whole chunks: the turn's
reasoning R and the tool's output O are appended (Phase 3).  Before those
tokens can be decoded from, the model runs one causal attention pass for the
n appended tokens over everything already cached (the compacted prefix, after
Phase 1's eviction) plus the earlier tokens of the chunk itself.  The paper
does not restate attention; the definition used is standard causal scaled
dot-product attention with grouped KV heads:

    the cache holds L tokens, the last n of which are the new ones;
    new token j (0 <= j < n) sits at logical index L - n + j and attends to
    the keys at logical indices 0 .. L - n + j (itself included);
    out[j, h] = decode attention of q[j, h] over those keys (see
    ``attention.attention``: scale, GQA mapping h -> h // G, softmax).

Causality is by logical index in the cache, not by stored position: after an
eviction the positions of the retained keys are no longer contiguous, but
they stay strictly increasing in logical order, so the two orders agree.

A key mask (the masked form of eviction, Algorithm 2 ``BuildMask``) removes
keys of the prefix for every query, exactly as in ``attention``.  A window
of W keys restricts new token j to the keys at logical indices
max(0, L - n + j - W + 1) .. L - n + j; per-head sinks join every softmax as
in ``attention``.
"""

from __future__ import annotations

import numpy as np

from . import attention as _att


def extend_attention(q, k, v, scale, group, mask=None, window=0, sinks=None):
    """Causal attention of the last n cached tokens.

    q: [n, Hq, D] (the new tokens' queries); k, v: [L, Hkv, D], the logical
    view of the cache after the n new tokens were appended (L >= n);
    mask: optional [L] (nonzero = keep); window: keys per query (0: all);
    sinks: optional [Hq].  Returns out [n, Hq, D].
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n, hq, d = q.shape
    n_keys = k.shape[0]
    if n > n_keys:
        raise ValueError("more new tokens than cached tokens")
    out = np.zeros((n, hq, d))
    for j in range(n):
        last = n_keys - n + j          # logical index of new token j
        lo = max(0, last - window + 1) if window > 0 else 0
        m = None if mask is None else np.asarray(mask)[lo: last + 1]
        out[j] = _att.attention(q[j], k[lo: last + 1], v[lo: last + 1], scale, group, m, sinks)
    return out
