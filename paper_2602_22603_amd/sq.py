"""Thin ctypes binding over libsq.so (include/sq.h).

Argument marshalling only: every step of the hot path runs in the library's
host code and HIP kernels.  PyTorch is used for device memory (pools,
workspace, inputs, outputs) and for the current HIP stream.  There is no
fallback: if ``libsq.so`` is missing or a call fails, an exception is raised.
"""

from __future__ import annotations

import ctypes as C
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsq.so")

OK, ERR_INVALID, ERR_NO_PAGES, ERR_UNKNOWN_SEQ, ERR_UNKNOWN_CURSOR, ERR_SPAN, ERR_HIP = range(7)
STORE_METADATA_ONLY = 1
STORE_EVICT_REMAP = 2
STORE_KV_FP8 = 4
STORE_EVICT_INPLACE = 8
NOALLOC_PARTIAL_SLOTS = 4096  # SQ_NOALLOC_PARTIAL_SLOTS
EVICT_DEFER = 1
ATTN_AUTO, ATTN_STREAM, ATTN_SHARED_PREFIX, ATTN_MFMA = 0, 1, 2, 3
MAX_BATCH = 64
MAX_EVICT_SPANS = 16384

_STATUS_NAMES = {
    ERR_INVALID: "SQ_ERR_INVALID", ERR_NO_PAGES: "SQ_ERR_NO_PAGES",
    ERR_UNKNOWN_SEQ: "SQ_ERR_UNKNOWN_SEQ", ERR_UNKNOWN_CURSOR: "SQ_ERR_UNKNOWN_CURSOR",
    ERR_SPAN: "SQ_ERR_SPAN", ERR_HIP: "SQ_ERR_HIP",
}


class SqError(RuntimeError):
    def __init__(self, code, message):
        super().__init__(f"{_STATUS_NAMES.get(code, code)}: {message}")
        self.code = code


class StoreConfig(C.Structure):
    _fields_ = [
        ("num_layers", C.c_int32), ("num_q_heads", C.c_int32), ("num_kv_heads", C.c_int32),
        ("head_dim", C.c_int32), ("page_size", C.c_int32), ("num_pages", C.c_int32),
        ("max_seqs", C.c_int32), ("max_pages_per_seq", C.c_int32),
        ("k_pool", C.c_void_p), ("v_pool", C.c_void_p), ("pos_pool", C.c_void_p),
        ("workspace", C.c_void_p), ("workspace_bytes", C.c_uint64), ("flags", C.c_uint32),
        ("evict_chunk_pages", C.c_int32), ("kv_scales", C.c_void_p),
    ]


class SeqDesc(C.Structure):
    _fields_ = [("length", C.c_int64), ("next_pos", C.c_int64), ("n_pages", C.c_int32),
                ("parent", C.c_int32), ("n_spans", C.c_int32), ("n_masked", C.c_int32)]


class EvictStats(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("tokens_removed", "tokens_moved", "bytes_moved",
                                         "pages_allocated", "pages_freed", "first_evicted",
                                         "pages_remapped", "tokens_masked")]


class Stats(C.Structure):
    _fields_ = [(n, C.c_int64) for n in (
        "live_pages", "peak_pages", "free_pages", "live_seqs", "append_tokens",
        "fork_calls", "fork_tail_copies", "evict_calls", "evict_tokens_removed",
        "evict_tokens_moved", "evict_bytes_moved", "decode_calls", "decode_kv_bytes",
        "decode_kv_bytes_logical", "extend_calls", "extend_tokens", "extend_kv_bytes")]


class PlanInfo(C.Structure):
    _fields_ = [("n_segments", C.c_int32), ("n_groups", C.c_int32),
                ("n_items_valu", C.c_int32), ("n_items_mfma", C.c_int32),
                ("chunk_pages", C.c_int32), ("n_slots", C.c_int32),
                ("kv_bytes", C.c_int64), ("kv_bytes_logical", C.c_int64),
                ("kv_bytes_valu", C.c_int64), ("kv_bytes_mfma", C.c_int64),
                ("io_bytes", C.c_int64)]


class AttnOpts(C.Structure):
    _fields_ = [("sinks", C.c_void_p), ("window", C.c_int32), ("reserved", C.c_int32)]


class Profile(C.Structure):
    _fields_ = ([(n, C.c_double) for n in ("decode_valu_ms", "decode_mfma_ms", "decode_merge_ms",
                                            "evict_scan_ms", "evict_gather_ms", "append_ms")] +
                [(n, C.c_int64) for n in ("decode_valu_launches", "decode_mfma_launches",
                                           "decode_merge_launches", "evict_scan_launches",
                                           "evict_gather_launches", "append_launches")] +
                [("extend_ms", C.c_double), ("extend_launches", C.c_int64)])


_LIB = None

# name -> (restype, argtypes)
_SIGS = {
    "sq_abi_version": (C.c_int32, []),
    "sq_last_error": (C.c_char_p, []),
    "sq_trace_open": (C.c_int, [C.c_char_p]),
    "sq_workspace_bytes": (C.c_uint64, [C.POINTER(StoreConfig)]),
    "sq_pool_bytes": (C.c_uint64, [C.POINTER(StoreConfig), C.c_int32]),
    "sq_store_create": (C.c_int, [C.POINTER(StoreConfig), C.POINTER(C.c_void_p)]),
    "sq_store_destroy": (C.c_int, [C.c_void_p]),
    "sq_seq_create": (C.c_int, [C.c_void_p, C.POINTER(C.c_int32)]),
    "sq_append": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p]),
    "sq_append_batch": (C.c_int, [C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.c_void_p,
                                  C.c_void_p, C.c_void_p]),
    "sq_span_mark": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, C.c_int64, C.c_int64]),
    "sq_fork": (C.c_int, [C.c_void_p, C.c_int32, C.c_int64, C.POINTER(C.c_int32), C.c_void_p]),
    "sq_release": (C.c_int, [C.c_void_p, C.c_int32]),
    "sq_evict_spans": (C.c_int, [C.c_void_p, C.c_int32, C.POINTER(C.c_int32), C.c_int32,
                                 C.c_void_p, C.POINTER(EvictStats)]),
    "sq_decode_attn": (C.c_int, [C.c_void_p, C.c_int32, C.POINTER(C.c_int32), C.c_int32,
                                 C.c_void_p, C.c_void_p, C.c_float, C.c_int32, C.c_void_p]),
    "sq_decode_attn_noalloc": (C.c_int, [C.c_void_p, C.c_int32, C.POINTER(C.c_int32), C.c_int32,
                                         C.c_void_p, C.c_void_p, C.c_float, C.c_int32,
                                         C.c_void_p]),
    "sq_step_begin": (C.c_int, [C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.c_int32,
                                C.c_void_p]),
    "sq_step_attn": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                               C.c_void_p, C.c_float, C.c_void_p]),
    "sq_extend_attn": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_void_p,
                                 C.c_void_p, C.c_float, C.c_void_p]),
    "sq_evict_spans_ex": (C.c_int, [C.c_void_p, C.c_int32, C.POINTER(C.c_int32), C.c_int32,
                                    C.c_uint32, C.c_void_p, C.POINTER(EvictStats)]),
    "sq_compact": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.POINTER(EvictStats)]),
    "sq_keep_flags": (C.c_int, [C.c_void_p, C.c_int32, C.POINTER(C.c_uint8), C.c_int64,
                                C.POINTER(C.c_int64)]),
    "sq_decode_attn_ex": (C.c_int, [C.c_void_p, C.c_int32, C.POINTER(C.c_int32), C.c_int32,
                                    C.c_void_p, C.c_void_p, C.c_float, C.c_int32,
                                    C.POINTER(AttnOpts), C.c_void_p]),
    "sq_extend_attn_ex": (C.c_int, [C.c_void_p, C.c_int32, C.c_int32, C.c_int32, C.c_void_p,
                                    C.c_void_p, C.c_float, C.POINTER(AttnOpts), C.c_void_p]),
    "sq_step_begin_ex": (C.c_int, [C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.c_int32,
                                   C.c_int32, C.c_void_p]),
    "sq_step_attn_ex": (C.c_int, [C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                                  C.c_void_p, C.c_float, C.POINTER(AttnOpts), C.c_void_p]),
    "sq_decode_plan_info": (C.c_int, [C.c_void_p, C.POINTER(C.c_int32), C.c_int32, C.c_int32,
                                      C.POINTER(PlanInfo)]),
    "sq_seq_info": (C.c_int, [C.c_void_p, C.c_int32, C.POINTER(SeqDesc)]),
    "sq_page_table": (C.c_int, [C.c_void_p, C.c_int32, C.POINTER(C.c_int32), C.c_int32,
                                C.POINTER(C.c_int32)]),
    "sq_positions": (C.c_int, [C.c_void_p, C.c_int32, C.POINTER(C.c_int64), C.c_int64,
                               C.POINTER(C.c_int64)]),
    "sq_seq_spans": (C.c_int, [C.c_void_p, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int64),
                               C.POINTER(C.c_int64), C.c_int32, C.POINTER(C.c_int32)]),
    "sq_refcounts": (C.c_int, [C.c_void_p, C.POINTER(C.c_int32), C.c_int32]),
    "sq_stats_get": (C.c_int, [C.c_void_p, C.POINTER(Stats)]),
    "sq_debug_last_evict": (C.c_int, [C.c_void_p, C.POINTER(C.c_uint8), C.POINTER(C.c_int32),
                                      C.POINTER(C.c_int32), C.c_int64, C.POINTER(C.c_int64),
                                      C.POINTER(C.c_int64)]),
    "sq_profile_enable": (C.c_int, [C.c_void_p, C.c_int32]),
    "sq_profile_read": (C.c_int, [C.c_void_p, C.POINTER(Profile)]),
}

EXPORTED = tuple(_SIGS)


def lib():
    """Load libsq.so (built in-tree); raises if it is missing."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2602_22603_amd.build_lib`")
        handle = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = handle
    return _LIB


def _check(status):
    if status != OK:
        msg = lib().sq_last_error().decode(errors="replace")
        raise SqError(status, msg)


def trace_open(path):
    """Host call trace: "-" to stderr, a path to append to, None to close."""
    _check(lib().sq_trace_open(None if path is None else str(path).encode()))


def _i32_array(values):
    arr = (C.c_int32 * max(1, len(values)))(*[int(v) for v in values])
    return arr


def _ptr(t):
    return C.c_void_p(0 if t is None else int(t.data_ptr()))


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


class Store:
    """A paged KV store (main thread plus auxiliary branches) on one GPU.

    Device mode allocates the pools and the workspace as torch tensors on
    ``device``.  ``metadata_only=True`` keeps host bookkeeping only (no GPU).
    """

    def __init__(self, num_layers, num_q_heads, num_kv_heads, head_dim, num_pages, max_seqs,
                 max_pages_per_seq, page_size=16, device="cuda", metadata_only=False,
                 evict_chunk_pages=0, evict_remap=False, kv_scales=None, evict_inplace=False):
        """kv_scales: [num_layers][2] K and V scales of an 8-bit (E4M3) store
        (None: bf16 pools)."""
        self.cfg = StoreConfig(num_layers, num_q_heads, num_kv_heads, head_dim, page_size,
                               num_pages, max_seqs, max_pages_per_seq)
        self.cfg.evict_chunk_pages = evict_chunk_pages
        self.evict_chunk_pages = evict_chunk_pages
        self.evict_remap = bool(evict_remap)
        self.evict_inplace = bool(evict_inplace)
        self.metadata_only = metadata_only
        self.num_layers, self.num_q_heads, self.num_kv_heads = num_layers, num_q_heads, num_kv_heads
        self.head_dim, self.page_size, self.num_pages = head_dim, page_size, num_pages
        self.max_seqs, self.max_pages_per_seq = max_seqs, max_pages_per_seq
        L = lib()
        self._handle = C.c_void_p()
        self.cfg.flags = (STORE_EVICT_REMAP if evict_remap else 0) | \
            (STORE_EVICT_INPLACE if evict_inplace else 0)
        self.kv_fp8 = kv_scales is not None
        self.kv_scales = None
        if self.kv_fp8:
            self.kv_scales = np.ascontiguousarray(np.asarray(kv_scales, dtype=np.float32)
                                                  .reshape(num_layers, 2))
            self.cfg.flags |= STORE_KV_FP8
            self.cfg.kv_scales = self.kv_scales.ctypes.data
        if metadata_only:
            self.cfg.flags |= STORE_METADATA_ONLY
            self.k_pool = self.v_pool = self.pos_pool = self.workspace = None
        else:
            import torch
            kb = L.sq_pool_bytes(C.byref(self.cfg), 0)
            pb = L.sq_pool_bytes(C.byref(self.cfg), 2)
            wb = L.sq_workspace_bytes(C.byref(self.cfg))
            if kb == 0 or wb == 0:
                raise SqError(ERR_INVALID, "invalid store configuration for device mode")
            dev = torch.device(device)
            shape_k = (num_layers, num_kv_heads, num_pages, page_size, head_dim)
            shape_v = (num_layers, num_kv_heads, num_pages, head_dim, page_size)
            kv_dtype = torch.uint8 if self.kv_fp8 else torch.bfloat16  # E4M3 codes as bytes
            self.k_pool = torch.zeros(shape_k, dtype=kv_dtype, device=dev)
            self.v_pool = torch.zeros(shape_v, dtype=kv_dtype, device=dev)
            self.pos_pool = torch.zeros((num_pages, page_size), dtype=torch.int32, device=dev)
            self.workspace = torch.empty(wb, dtype=torch.uint8, device=dev)
            assert self.k_pool.numel() * self.k_pool.element_size() == kb
            assert self.pos_pool.numel() * 4 == pb
            self.cfg.k_pool = self.k_pool.data_ptr()
            self.cfg.v_pool = self.v_pool.data_ptr()
            self.cfg.pos_pool = self.pos_pool.data_ptr()
            self.cfg.workspace = self.workspace.data_ptr()
            self.cfg.workspace_bytes = wb
        _check(L.sq_store_create(C.byref(self.cfg), C.byref(self._handle)))

    # -- lifetime -------------------------------------------------------------
    def close(self):
        if self._handle:
            _check(lib().sq_store_destroy(self._handle))
            self._handle = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:  # noqa: BLE001 - interpreter shutdown
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -- argument checks (the C ABI takes raw pointers and trusts the sizes) -----
    def _tensor(self, t, shape, dtype, what):
        """t must be a contiguous tensor of exactly this shape and dtype on the
        store's device; returns its pointer."""
        import torch
        if not isinstance(t, torch.Tensor):
            raise SqError(ERR_INVALID, f"{what} must be a torch tensor")
        if t.dtype != dtype:
            raise SqError(ERR_INVALID, f"{what} must be {dtype}, got {t.dtype}")
        if tuple(t.shape) != tuple(shape):
            raise SqError(ERR_INVALID, f"{what} must have shape {tuple(shape)}, got {tuple(t.shape)}")
        if not t.is_contiguous():
            raise SqError(ERR_INVALID, f"{what} must be contiguous")
        if t.device != self.k_pool.device:
            raise SqError(ERR_INVALID, f"{what} must be on {self.k_pool.device}, got {t.device}")
        return _ptr(t)

    def _kv_ptrs(self, k_new, v_new, n):
        import torch
        if self.metadata_only:
            return _ptr(None), _ptr(None)
        shape = (self.num_layers, n, self.num_kv_heads, self.head_dim)
        return (self._tensor(k_new, shape, torch.bfloat16, "k_new"),
                self._tensor(v_new, shape, torch.bfloat16, "v_new"))

    def _opts(self, window, sinks):
        """AttnOpts for (window, sinks) or None when neither is set; sinks is
        a float32 tensor [Hq] on the store's device."""
        import torch
        if not window and sinks is None:
            return None
        o = AttnOpts()
        o.window = int(window)
        if sinks is not None:
            o.sinks = (_ptr(sinks) if self.metadata_only else
                       self._tensor(sinks, (self.num_q_heads,), torch.float32, "sinks"))
        return o

    def _qo_ptrs(self, q, out, rows):
        import torch
        shape = (rows, self.num_q_heads, self.head_dim)
        return (self._tensor(q, shape, torch.bfloat16, "q"),
                self._tensor(out, shape, torch.float32, "out"))

    # -- sequences --------------------------------------------------------------
    def seq_create(self):
        out = C.c_int32()
        _check(lib().sq_seq_create(self._handle, C.byref(out)))
        return out.value

    def append(self, seq, k_new=None, v_new=None, n=None, stream=None):
        """Append tokens; k_new, v_new: bf16 [NL, n, Hkv, D] on the device."""
        if n is None:
            n = int(k_new.shape[1])
        kp, vp = self._kv_ptrs(k_new, v_new, n)
        st = C.c_void_p(0) if self.metadata_only else _stream(stream)
        _check(lib().sq_append(self._handle, seq, n, kp, vp, st))

    def append_batch(self, seqs, k_new=None, v_new=None, stream=None):
        """One token per sequence; k_new, v_new: bf16 [NL, B, Hkv, D]."""
        seqs = list(seqs)
        kp, vp = self._kv_ptrs(k_new, v_new, len(seqs))
        st = C.c_void_p(0) if self.metadata_only else _stream(stream)
        _check(lib().sq_append_batch(self._handle, _i32_array(seqs), len(seqs), kp, vp, st))

    def span_mark(self, seq, cursor, start, end):
        _check(lib().sq_span_mark(self._handle, seq, cursor, start, end))

    def fork(self, parent, fork_len, stream=None):
        out = C.c_int32()
        st = C.c_void_p(0) if self.metadata_only else _stream(stream)
        _check(lib().sq_fork(self._handle, parent, fork_len, C.byref(out), st))
        return out.value

    def release(self, seq):
        _check(lib().sq_release(self._handle, seq))

    def evict(self, seq, cursor_ids, stream=None, deferred=False):
        """Evict the cursors' spans (deferred: mask their slots, move nothing)."""
        es = EvictStats()
        st = C.c_void_p(0) if self.metadata_only else _stream(stream)
        ids = list(cursor_ids)
        if deferred:
            _check(lib().sq_evict_spans_ex(self._handle, seq, _i32_array(ids), len(ids),
                                           EVICT_DEFER, st, C.byref(es)))
        else:
            _check(lib().sq_evict_spans(self._handle, seq, _i32_array(ids), len(ids), st,
                                        C.byref(es)))
        return {n: getattr(es, n) for n, _ in EvictStats._fields_}

    def compact(self, seq, stream=None):
        """Remove the slots deferred evictions masked."""
        es = EvictStats()
        st = C.c_void_p(0) if self.metadata_only else _stream(stream)
        _check(lib().sq_compact(self._handle, seq, st, C.byref(es)))
        return {n: getattr(es, n) for n, _ in EvictStats._fields_}

    def keep_flags(self, seq):
        """Per slot: 1 attended, 0 masked by a deferred eviction."""
        n = C.c_int64()
        _check(lib().sq_keep_flags(self._handle, seq, None, 0, C.byref(n)))
        buf = np.zeros(max(1, n.value), dtype=np.uint8)
        _check(lib().sq_keep_flags(self._handle, seq, buf.ctypes.data_as(C.POINTER(C.c_uint8)),
                                   n.value, C.byref(n)))
        return buf[: n.value]

    def decode(self, layer, seqs, q, out=None, scale=None, mode=ATTN_AUTO, stream=None,
               window=0, sinks=None):
        """out[b, h] = attention of q[b, h] (bf16 [B, Hq, D]) over seqs[b]; fp32.
        window > 0: the last `window` keys only; sinks: fp32 [Hq] sink logits."""
        import torch
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        if scale is None:
            scale = 1.0 / float(self.head_dim) ** 0.5
        seqs = list(seqs)
        qp, op = (_ptr(q), _ptr(out)) if self.metadata_only else self._qo_ptrs(q, out, len(seqs))
        o = self._opts(window, sinks)
        if o is None:
            _check(lib().sq_decode_attn(self._handle, layer, _i32_array(seqs), len(seqs), qp, op,
                                        float(scale), mode, _stream(stream)))
        else:
            _check(lib().sq_decode_attn_ex(self._handle, layer, _i32_array(seqs), len(seqs), qp,
                                           op, float(scale), mode, C.byref(o), _stream(stream)))
        return out

    def decode_noalloc(self, layer, seqs, q, out, scale=None, mode=ATTN_AUTO, stream=None):
        """decode() through sq_decode_attn_noalloc: the split partials in the
        library's per-GPU device array instead of the store's workspace; the
        caller passes ``out`` (fp32 [B, Hq, D])."""
        if scale is None:
            scale = 1.0 / float(self.head_dim) ** 0.5
        seqs = list(seqs)
        qp, op = (_ptr(q), _ptr(out)) if self.metadata_only else self._qo_ptrs(q, out, len(seqs))
        _check(lib().sq_decode_attn_noalloc(self._handle, layer, _i32_array(seqs), len(seqs), qp,
                                            op, float(scale), mode, _stream(stream)))
        return out

    def step_begin(self, seqs, mode=ATTN_AUTO, stream=None, window=0):
        """Open a decode step: one token slot appended to each of seqs (their
        K/V arrive layer by layer through step_attn).  window > 0 also plans
        layers that attend to the last `window` keys only."""
        seqs = list(seqs)
        st = C.c_void_p(0) if self.metadata_only else _stream(stream)
        # the C side trusts buffer sizes: step_attn checks them against the
        # batch of the last step this binding opened, and refuses after a
        # failed step_begin
        self._step_batch = None
        if window:
            _check(lib().sq_step_begin_ex(self._handle, _i32_array(seqs), len(seqs), mode,
                                          int(window), st))
        else:
            _check(lib().sq_step_begin(self._handle, _i32_array(seqs), len(seqs), mode, st))
        self._step_batch = len(seqs)

    def step_attn(self, layer, k_new, v_new, q, out=None, scale=None, stream=None, window=0,
                  sinks=None):
        """One layer of the open step: store k_new, v_new (bf16 [B, Hkv, D])
        and attend with q (bf16 [B, Hq, D]) over every token, the new one
        included; returns out (fp32 [B, Hq, D]).  window: 0 or the step's
        window; sinks: fp32 [Hq] sink logits."""
        import torch
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        if scale is None:
            scale = 1.0 / float(self.head_dim) ** 0.5
        if self.metadata_only:
            ptrs = (_ptr(k_new), _ptr(v_new), _ptr(q), _ptr(out))
        else:
            b = getattr(self, "_step_batch", None)
            if b is None:
                raise SqError(ERR_INVALID, "no decode step opened by this binding")
            kv = (b, self.num_kv_heads, self.head_dim)
            ptrs = (self._tensor(k_new, kv, torch.bfloat16, "k_new"),
                    self._tensor(v_new, kv, torch.bfloat16, "v_new"), *self._qo_ptrs(q, out, b))
        o = self._opts(window, sinks)
        if o is None:
            _check(lib().sq_step_attn(self._handle, layer, *ptrs, float(scale), _stream(stream)))
        else:
            _check(lib().sq_step_attn_ex(self._handle, layer, *ptrs, float(scale), C.byref(o),
                                         _stream(stream)))
        return out

    def extend(self, layer, seq, q, out=None, scale=None, stream=None, window=0, sinks=None):
        """Causal attention of the last n = q.shape[0] tokens of seq (just
        appended) over the cache: q bf16 [n, Hq, D] -> out fp32 [n, Hq, D].
        window > 0: each token sees its last `window` keys; sinks: fp32 [Hq]."""
        import torch
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
        if scale is None:
            scale = 1.0 / float(self.head_dim) ** 0.5
        n = int(q.shape[0])
        qp, op = (_ptr(q), _ptr(out)) if self.metadata_only else self._qo_ptrs(q, out, n)
        o = self._opts(window, sinks)
        if o is None:
            _check(lib().sq_extend_attn(self._handle, layer, seq, n, qp, op, float(scale),
                                        _stream(stream)))
        else:
            _check(lib().sq_extend_attn_ex(self._handle, layer, seq, n, qp, op, float(scale),
                                           C.byref(o), _stream(stream)))
        return out

    def plan_info(self, seqs, mode=ATTN_AUTO):
        pi = PlanInfo()
        _check(lib().sq_decode_plan_info(self._handle, _i32_array(seqs), len(seqs), mode,
                                         C.byref(pi)))
        return {n: getattr(pi, n) for n, _ in PlanInfo._fields_}

    # -- introspection -------------------------------------------------------------
    def seq_info(self, seq):
        d = SeqDesc()
        _check(lib().sq_seq_info(self._handle, seq, C.byref(d)))
        return {n: getattr(d, n) for n, _ in SeqDesc._fields_}

    def page_table(self, seq):
        n = C.c_int32()
        _check(lib().sq_page_table(self._handle, seq, None, 0, C.byref(n)))
        buf = (C.c_int32 * max(1, n.value))()
        _check(lib().sq_page_table(self._handle, seq, buf, n.value, C.byref(n)))
        return list(buf[: n.value])

    def positions(self, seq):
        n = C.c_int64()
        _check(lib().sq_positions(self._handle, seq, None, 0, C.byref(n)))
        buf = np.zeros(max(1, n.value), dtype=np.int64)
        _check(lib().sq_positions(self._handle, seq, buf.ctypes.data_as(C.POINTER(C.c_int64)),
                                  n.value, C.byref(n)))
        return buf[: n.value]

    def spans(self, seq):
        n = C.c_int32()
        _check(lib().sq_seq_spans(self._handle, seq, None, None, None, 0, C.byref(n)))
        cap = max(1, n.value)
        cur = (C.c_int32 * cap)()
        s = (C.c_int64 * cap)()
        e = (C.c_int64 * cap)()
        _check(lib().sq_seq_spans(self._handle, seq, cur, s, e, cap, C.byref(n)))
        return {cur[i]: (s[i], e[i]) for i in range(n.value)}

    def refcounts(self):
        buf = (C.c_int32 * self.num_pages)()
        _check(lib().sq_refcounts(self._handle, buf, self.num_pages))
        return np.array(buf[:], dtype=np.int64)

    def stats(self):
        st = Stats()
        _check(lib().sq_stats_get(self._handle, C.byref(st)))
        return {n: getattr(st, n) for n, _ in Stats._fields_}

    def debug_last_evict(self):
        """(keep u8 [L], dst i32 [L], src_of i32 [L']) of the last eviction."""
        cap = self.max_pages_per_seq * self.page_size
        keep = np.zeros(cap, dtype=np.uint8)
        dst = np.zeros(cap, dtype=np.int32)
        src = np.zeros(cap, dtype=np.int32)
        n_tok, n_kept = C.c_int64(), C.c_int64()
        _check(lib().sq_debug_last_evict(
            self._handle, keep.ctypes.data_as(C.POINTER(C.c_uint8)),
            dst.ctypes.data_as(C.POINTER(C.c_int32)), src.ctypes.data_as(C.POINTER(C.c_int32)),
            cap, C.byref(n_tok), C.byref(n_kept)))
        return keep[: n_tok.value], dst[: n_tok.value], src[: n_kept.value]

    def profile_enable(self, on=True):
        _check(lib().sq_profile_enable(self._handle, 1 if on else 0))

    def profile_read(self):
        pr = Profile()
        _check(lib().sq_profile_read(self._handle, C.byref(pr)))
        return {n: getattr(pr, n) for n, _ in Profile._fields_}
