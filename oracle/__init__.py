"""SideQuest KV-cache oracle: a plain, slow, float64 CPU statement of what the
hot path computes.

TEST INFRASTRUCTURE ONLY.  Nothing in the product (the ``paper_2602_22603_amd``
package, its HIP kernels or its C-ABI library) imports, links or calls this
package, and this package imports nothing from the product.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` use it.

Modules
-------
attention
    Decode-phase attention of one query per head over a KV cache with grouped
    KV heads, its masked form, split partials and their merge.
extend
    Causal attention of a chunk of newly appended tokens over the cache
    (the prefill of Algorithm 1's Phase 3 appends) with grouped KV heads.
evict
    The keep-mask, exclusive prefix sum and inverse map that ``clear_kv``
    (Algorithm 1, Phase 1) reduces to, and the compaction of a logical view.
fp8
    The 8-bit E4M3 code of the optional 8-bit KV cache: decode, nearest
    encode with saturation, per-layer scales.
pages
    A page-level model of the KV store: lowest-free-first page allocator,
    refcounts, per-sequence page lists, zero-copy fork of the auxiliary
    thread (§3.1, Algorithm 1 Phase 2; storage claim of §3.4), cursor spans,
    out-of-place span eviction and release.

Readings of points the paper leaves open are stated where they are used and
listed again, all together, in the repository's design notes.

Parity status
-------------
Every function here is pinned by the CPU tests in ``tests/test_oracle_*.py``
against closed forms, invariants, an independent library routine
(``torch.softmax`` in float64) or brute force over tiny inputs.  No function
is "parity unpinned".
"""

from . import attention, evict, extend, fp8, pages  # noqa: F401

__all__ = ["attention", "evict", "extend", "fp8", "pages"]
