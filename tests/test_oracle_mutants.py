"""Plant plausible mistakes in the oracle (on the CPU) and show the pins see them.

Each mutant replaces one oracle function with a subtly wrong version; the test
passes when at least one pin check fails on the mutated oracle.
"""

import heapq
import math

import numpy as np
import pytest

from oracle import attention as att
from oracle import evict as ev
from oracle import extend as ex
from oracle import fp8 as f8
from oracle import pages as pg
from tests import oracle_pins as pins

_ORIG_RUNS = pg.PageModel._masked_runs
_ORIG_DECODE = f8.decode
_ORIG_ENCODE = f8.encode
_ORIG_FORK = pg.PageModel.fork
_ORIG_EVICT = pg.PageModel.evict


def _scores_gqa_modulo(q, k, scale, group, mask=None):
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    hkv = k.shape[1]
    s = np.stack([scale * np.cumsum(k[:, h % hkv, :] * q[h], axis=1)[:, -1]
                  if k.shape[0] else np.zeros(0) for h in range(q.shape[0])])
    if mask is not None:
        s[:, ~np.asarray(mask).astype(bool)] = -np.inf
    return s


_orig_scores = att.scores
_orig_partial = att.partial


def _scores_no_scale(q, k, scale, group, mask=None):
    return _orig_scores(q, k, 1.0, group, mask)


def _scores_sign(q, k, scale, group, mask=None):
    return _orig_scores(q, k, -scale, group, mask)


def _partial_k_as_v(q, k, v, scale, group, mask=None):
    return _orig_partial(q, k, k, scale, group, mask)


def _attention_unnormalised(q, k, v, scale, group, mask=None):
    m, l, acc = _orig_partial(q, k, v, scale, group, mask)
    return acc


def _merge_no_rescale(parts):
    accs = sum(np.asarray(p[2]) for p in parts)
    ls = sum(np.asarray(p[1]) for p in parts)
    out = np.zeros_like(accs)
    live = ls > 0
    out[live] = accs[live] / ls[live][:, None]
    return out


def _scan_inclusive(keep):
    return np.cumsum(np.asarray(keep, dtype=np.int64))


def _keep_mask_end_inclusive(length, spans):
    keep = np.ones(int(length), dtype=np.uint8)
    for s, e in spans:
        keep[s:e + 1] = 0
    return keep


def _shift_span_wrong(start, end, evicted):
    before = sum(e - s for s, e in evicted if s <= start)
    return start - before, end - before + (1 if evicted else 0)


def _alloc_highest(self):
    page = max(self._free)
    self._free.remove(page)
    heapq.heapify(self._free)
    self.refcount[page] = 1
    self.peak_pages = max(self.peak_pages, self.live_pages())
    return page


_orig_fork = pg.PageModel.fork
_orig_evict = pg.PageModel.evict


def _fork_copies(self, parent, fork_len):
    child = _orig_fork(self, parent, fork_len)
    # a copying fork: take one fresh page per aliased page
    seq = self.seqs[child]
    for i, page in enumerate(list(seq.pages[: fork_len // self.P])):
        fresh = self._alloc()
        if self.with_data:
            self.K[fresh], self.V[fresh], self.POS[fresh] = self.K[page], self.V[page], self.POS[page]
        self._unref(page)
        seq.pages[i] = fresh
    return child


def _fork_next_pos_parent(self, parent, fork_len):
    child = _orig_fork(self, parent, fork_len)
    self.seqs[child].next_pos = self.seqs[parent].next_pos
    return child


def _evict_recompute_pos(self, h, cursor_ids):
    stats = _orig_evict(self, h, cursor_ids)
    seq = self.seqs[h]
    seq.pos = list(range(seq.length))
    if self.with_data:
        for i in range(seq.length):
            self.POS[seq.pages[i // self.P], i % self.P] = i
    return stats


def _evict_keeps_old_refs(self, h, cursor_ids):
    seq = self.seqs[h]
    old = list(seq.pages)
    stats = _orig_evict(self, h, cursor_ids)
    if stats["tokens_removed"]:
        fp = stats["first_evicted"] // self.P
        for page in old[fp:]:  # leak: take the references back
            if self.refcount[page] == 0:
                self._free.remove(page)
                heapq.heapify(self._free)
            self.refcount[page] += 1
    return stats


def _extend_excludes_self(q, k, v, scale, group, mask=None):
    q = np.asarray(q, np.float64)
    n, L = q.shape[0], np.asarray(k).shape[0]
    out = np.zeros(q.shape)
    for j in range(n):
        last = L - n + j
        out[j] = att.attention(q[j], k[:last], v[:last], scale, group,
                               None if mask is None else mask[:last])
    return out


def _extend_no_prefix_offset(q, k, v, scale, group, mask=None):
    q = np.asarray(q, np.float64)
    out = np.zeros(q.shape)
    for j in range(q.shape[0]):
        out[j] = att.attention(q[j], k[: j + 1], v[: j + 1], scale, group,
                               None if mask is None else mask[: j + 1])
    return out


def _extend_ignores_mask(q, k, v, scale, group, mask=None):
    return _orig_extend(q, k, v, scale, group)


_orig_extend = ex.extend_attention


def _released_one_page_early(self, fp, released, n_old, consumed):
    upto = released
    while upto < n_old and (fp + upto) * self.P <= consumed:
        upto += 1
    return upto


def _evict_chunk_never_recycles(self, h, cursor_ids):
    # allocate every fresh page before releasing any old one, even in chunks
    chunk = self.evict_chunk_pages
    self.evict_chunk_pages = 0
    try:
        return _orig_evict(self, h, cursor_ids)
    finally:
        self.evict_chunk_pages = chunk


def _remap_page_start_only(self, src_of, j0, new_len):
    # takes the old page whenever the first token starts one, runs or not
    if j0 + self.P > new_len:
        return None
    a0 = int(src_of[j0])
    return a0 if a0 % self.P == 0 else None


_orig_remap_source = pg.PageModel._remap_source


def _remap_next_page(self, src_of, j0, new_len):
    a0 = _orig_remap_source(self, src_of, j0, new_len)
    return None if a0 is None else a0 + self.P


_orig_attention = att.attention
_orig_window_mask = att.window_mask


def _sinks_ignored(q, k, v, scale, group, mask=None, sinks=None):
    return _orig_attention(q, k, v, scale, group, mask)


def _sink_carries_a_value(q, k, v, scale, group, mask=None, sinks=None):
    # as if the sink were a key whose value is all ones
    out = _orig_attention(q, k, v, scale, group, mask, sinks)
    if sinks is None:
        return out
    m, l, acc = att.partial(q, k, v, scale, group, mask)
    for h in range(out.shape[0]):
        if l[h] > 0:
            big = max(m[h], sinks[h])
            out[h] += np.exp(sinks[h] - big) / (l[h] * np.exp(m[h] - big) + np.exp(sinks[h] - big))
    return out


def _window_one_too_wide(n_keys, window):
    return _orig_window_mask(n_keys, window + 1 if window > 0 else 0)


def _runs_ignore_masks(keep, extra=()):
    return _ORIG_RUNS(np.ones(len(keep), dtype=bool), extra)


def _fork_drops_masks(self, parent, fork_len):
    h = _ORIG_FORK(self, parent, fork_len)
    self.seqs[h].keep = [True] * fork_len
    return h


def _deferred_shifts_spans(self, h, cursor_ids, deferred=False):
    seq = self.seqs[h]
    gone = sorted(seq.spans[c] for c in cursor_ids if c in seq.spans)
    st = _ORIG_EVICT(self, h, cursor_ids, deferred)
    if deferred:
        seq.spans = {c: ev.shift_span(a, b, gone) for c, (a, b) in seq.spans.items()}
    return st


def _fp8_decode_bias_8(codes):
    return _ORIG_DECODE(codes) / 2.0


def _fp8_ties_away(y):
    y = np.asarray(y, dtype=np.float32)
    code = _ORIG_ENCODE(y).astype(np.int64)
    mags = _ORIG_DECODE(np.arange(0x7F))
    a = np.abs(y.astype(np.float64))
    mid = np.isin(a, (mags[:-1] + mags[1:]) / 2)
    up = np.where(mid & ((code & 0x7F) < 0x7E), code + ((code & 1) == 0), code)
    return up.astype(np.uint8)


def _fp8_no_saturation(y):
    code = _ORIG_ENCODE(y)
    a = np.abs(np.asarray(y, dtype=np.float64))
    return np.where(a > 464, code | 0x7F, code).astype(np.uint8)


def _extend_window_one_too_wide(q, k, v, scale, group, mask=None, window=0, sinks=None):
    return _orig_extend(q, k, v, scale, group, mask, window + 1 if window > 0 else 0, sinks)


_ORIG_PLACE = pg.PageModel._place_tail


def _inplace_ignores_sharing(self, seq, fp, n_new, src_of, new_len):
    # rewrites the old tail page even when another branch still holds it
    alias, kind = _ORIG_PLACE(self, seq, fp, n_new, src_of, new_len)
    if self.evict_inplace:
        for k in range(n_new):
            alias[k], kind[k] = seq.pages[fp + k], "inplace"
    return alias, kind


def _inplace_next_page(self, seq, fp, n_new, src_of, new_len):
    # takes the old page one list index further on (the last one stays fresh)
    alias, kind = _ORIG_PLACE(self, seq, fp, n_new, src_of, new_len)
    if self.evict_inplace:
        for k in range(n_new):
            ok = fp + k + 1 < len(seq.pages) and self.refcount[seq.pages[fp + k + 1]] == 1
            alias[k], kind[k] = (seq.pages[fp + k + 1], "inplace") if ok else (None, "fresh")
    return alias, kind


def _inplace_counts_as_fresh(self, seq, fp, n_new, src_of, new_len):
    # never reuses a page: the one-shot rule under the in-place flag
    alias, kind = _ORIG_PLACE(self, seq, fp, n_new, src_of, new_len)
    if self.evict_inplace:
        alias, kind = [None] * n_new, ["fresh"] * n_new
    return alias, kind


MUTANTS = {
    "gqa_head_modulo": (att, "scores", _scores_gqa_modulo),
    "missing_scale": (att, "scores", _scores_no_scale),
    "score_sign": (att, "scores", _scores_sign),
    "k_used_as_v": (att, "partial", _partial_k_as_v),
    "unnormalised_output": (att, "attention", _attention_unnormalised),
    "merge_without_rescale": (att, "merge", _merge_no_rescale),
    "inclusive_scan": (ev, "exclusive_scan", _scan_inclusive),
    "span_end_inclusive": (ev, "keep_mask", _keep_mask_end_inclusive),
    "span_shift_wrong": (ev, "shift_span", _shift_span_wrong),
    "alloc_highest_first": (pg.PageModel, "_alloc", _alloc_highest),
    "fork_copies_pages": (pg.PageModel, "fork", _fork_copies),
    "fork_next_pos_from_parent": (pg.PageModel, "fork", _fork_next_pos_parent),
    "evict_recomputes_positions": (pg.PageModel, "evict", _evict_recompute_pos),
    "evict_leaks_old_pages": (pg.PageModel, "evict", _evict_keeps_old_refs),
    "extend_excludes_own_key": (ex, "extend_attention", _extend_excludes_self),
    "extend_drops_prefix_offset": (ex, "extend_attention", _extend_no_prefix_offset),
    "extend_ignores_mask": (ex, "extend_attention", _extend_ignores_mask),
    "evict_chunks_never_recycle": (pg.PageModel, "evict", _evict_chunk_never_recycles),
    "evict_chunk_releases_a_page_early": (pg.PageModel, "_released_after", _released_one_page_early),
    "remap_without_run_check": (pg.PageModel, "_remap_source", _remap_page_start_only),
    "remap_takes_the_next_page": (pg.PageModel, "_remap_source", _remap_next_page),
    "inplace_rewrites_a_shared_page": (pg.PageModel, "_place_tail", _inplace_ignores_sharing),
    "inplace_takes_the_next_page": (pg.PageModel, "_place_tail", _inplace_next_page),
    "inplace_takes_fresh_pages": (pg.PageModel, "_place_tail", _inplace_counts_as_fresh),
    "sinks_ignored": (att, "attention", _sinks_ignored),
    "sink_carries_a_value": (att, "attention", _sink_carries_a_value),
    "window_one_key_too_wide": (att, "window_mask", _window_one_too_wide),
    "extend_window_one_key_too_wide": (ex, "extend_attention", _extend_window_one_too_wide),
    "eviction_ignores_masked_slots": (pg.PageModel, "_masked_runs", staticmethod(_runs_ignore_masks)),
    "fork_drops_masks": (pg.PageModel, "fork", _fork_drops_masks),
    "deferred_eviction_shifts_spans": (pg.PageModel, "evict", _deferred_shifts_spans),
    "fp8_exponent_bias_8": (f8, "decode", _fp8_decode_bias_8),
    "fp8_ties_away_from_zero": (f8, "encode", _fp8_ties_away),
    "fp8_overflow_to_nan": (f8, "encode", _fp8_no_saturation),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    owner, attr, fn = MUTANTS[name]
    monkeypatch.setattr(owner, attr, fn)
    failed = []
    for check in pins.ALL_CHECKS:
        try:
            check()
        except Exception as err:  # noqa: BLE001 - any failure counts as caught
            failed.append((check.__name__, type(err).__name__))
    assert failed, f"mutant {name} passed every pin"


def test_pins_green_without_mutation():
    for check in pins.ALL_CHECKS:
        check()
    assert math.isfinite(1.0)
