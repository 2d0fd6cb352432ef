"""Seeded synthetic agent-shaped inputs for the SideQuest KV hot path.

This module only draws inputs; it holds none of the method's arithmetic.
Both the HIP path and the CPU oracle consume the same arrays from here.

The paper's agentic traces (ReAct loops over web search; §4.1, Fig. 2) are
not available, so these contexts stand in for them with the shapes the paper
describes: contexts dominated by tool responses, of a few thousand to over a
hundred thousand tokens, reasoning text between tool calls (Algorithm 1,
Phase 3), and an auxiliary thread forked every K = 4 turns (§4.3).  Model
shapes (heads, head size, layers) are GQA shapes of a large model.

Conventions
-----------
* Seed: ``numpy.random.default_rng([2602, config_index])``.
* Draw order: span lengths, evicted-span choice, main-thread K then V (token
  order), auxiliary private K then V, queries.
* Values: N(0, 1) in float32, rounded to bfloat16 round-to-nearest-even.
  bf16 values are carried as uint16 bit patterns; ``bf16_value`` gives their
  exact float64 values.
* Span lengths "lognormal, normalised to fill": x_i ~ LogNormal(mu, sigma),
  len_i = largest-remainder rounding of x_i / sum(x) * total, each at least 1,
  summing exactly to total.
* Large configurations draw K/V on the GPU with a seeded torch generator
  (``device_normal_bf16``); checks against the oracle then copy the sampled
  slices of those input tensors to the host.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 2602


def rng_for(config_index):
    return np.random.default_rng([SEED_BASE, int(config_index)])


def bf16_bits(x):
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def bf16_value(bits):
    """Exact float64 values of bfloat16 bit patterns."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def normal_bf16(rng, shape):
    return bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def lognormal_lengths(rng, n, mu, sigma, total):
    """n positive integer lengths summing to ``total`` (largest remainder)."""
    if n > total:
        raise ValueError("more spans than tokens")
    x = rng.lognormal(mu, sigma, n)
    share = x / x.sum() * (total - n)  # one token reserved per span
    base = np.floor(share).astype(np.int64)
    rem = int(total - n - base.sum())
    order = np.argsort(-(share - base), kind="stable")
    base[order[:rem]] += 1
    return (base + 1).tolist()


def spans_from_lengths(lengths, start=0):
    out, pos = [], start
    for n in lengths:
        out.append((pos, pos + n))
        pos += n
    return out


def choose_until(rng, spans, candidates, target_tokens):
    """Seeded random order over ``candidates`` (indices into spans), taking
    whole spans until at least ``target_tokens`` tokens are chosen."""
    order = rng.permutation(len(candidates))
    chosen, got = [], 0
    for i in order:
        if got >= target_tokens:
            break
        c = candidates[i]
        chosen.append(c)
        got += spans[c][1] - spans[c][0]
    return sorted(chosen), got


# ---------------------------------------------------------------------------
# Tiny: 1 layer, 4 query heads / 1 KV head, head size 64, scale 1/8.
@dataclass
class Tiny:
    num_layers: int = 1
    num_q_heads: int = 4
    num_kv_heads: int = 1
    head_dim: int = 64
    scale: float = 1.0 / 8.0
    main_len: int = 2048
    fork_at: int = 2000
    aux_private: int = 48
    n_spans: int = 10
    n_evict: int = 4
    span_lengths: list = field(default_factory=list)
    spans: list = field(default_factory=list)
    evict_ids: list = field(default_factory=list)
    main_k: np.ndarray = None  # uint16 [NL, main_len, Hkv, D]
    main_v: np.ndarray = None
    aux_k: np.ndarray = None   # uint16 [NL, aux_private, Hkv, D]
    aux_v: np.ndarray = None
    q: np.ndarray = None       # uint16 [2, Hq, D]: main, aux


def tiny(config_index=0):
    """The tiny case: main 2048 tokens = 10 tool spans (LogNormal(4.5, 0.6)
    normalised to 2048); the auxiliary thread forks at 2000 and adds 48
    private tokens; 4 seeded spans are evicted; one decode step of [main, aux]."""
    w = Tiny()
    rng = rng_for(config_index)
    w.span_lengths = lognormal_lengths(rng, w.n_spans, 4.5, 0.6, w.main_len)
    w.spans = spans_from_lengths(w.span_lengths)
    w.evict_ids = sorted(rng.choice(w.n_spans, w.n_evict, replace=False).tolist())
    shape = (w.num_layers, w.main_len, w.num_kv_heads, w.head_dim)
    w.main_k = normal_bf16(rng, shape)
    w.main_v = normal_bf16(rng, shape)
    ashape = (w.num_layers, w.aux_private, w.num_kv_heads, w.head_dim)
    w.aux_k = normal_bf16(rng, ashape)
    w.aux_v = normal_bf16(rng, ashape)
    w.q = normal_bf16(rng, (2, w.num_q_heads, w.head_dim))
    return w


# ---------------------------------------------------------------------------
# Single-layer 32 query / 8 KV heads, head size 128.
GQA_SHAPE = dict(num_q_heads=32, num_kv_heads=8, head_dim=128)


@dataclass
class Shared128K:
    """8 tasks; each main thread reaches 131072 tokens; its auxiliary thread
    forks at 130816 (the main thread then decodes 256 more tokens in
    parallel) and adds 512 private tokens.  16 queries, no eviction."""
    n_tasks: int = 8
    main_len: int = 131072
    fork_at: int = 130816
    aux_private: int = 512
    num_layers: int = 1
    seed: int = SEED_BASE * 100 + 2


def shared128k(n_tasks=8, main_len=131072, fork_at=130816, aux_private=512):
    return Shared128K(n_tasks=n_tasks, main_len=main_len, fork_at=fork_at,
                      aux_private=aux_private)


@dataclass
class Outlier32K:
    """One task at 32768 tokens = 30 tool spans (LogNormal(7.0, 0.8)
    normalised); K and V carry 4 outlier channels per KV head scaled x8; the
    auxiliary thread forks at 32768 and adds 512 private tokens; whole spans
    are evicted in seeded order until at least half the tokens are gone;
    64 decode steps of [main, aux]."""
    main_len: int = 32768
    n_spans: int = 30
    aux_private: int = 512
    steps: int = 64
    span_lengths: list = field(default_factory=list)
    spans: list = field(default_factory=list)
    evict_ids: list = field(default_factory=list)
    outlier_k: np.ndarray = None  # [Hkv, 4] channel indices
    outlier_v: np.ndarray = None
    main_k: np.ndarray = None     # uint16 [1, L, Hkv, D]
    main_v: np.ndarray = None
    aux_k: np.ndarray = None
    aux_v: np.ndarray = None
    step_k: np.ndarray = None     # uint16 [steps, 1, 2, Hkv, D]
    step_v: np.ndarray = None
    q: np.ndarray = None          # uint16 [steps, 2, Hq, D]


def _with_outliers(rng, shape, channels):
    x = rng.standard_normal(shape, dtype=np.float32)
    for h in range(shape[2]):
        x[:, :, h, channels[h]] *= 8.0  # exact in binary floating point
    return bf16_bits(x)


def outlier32k(config_index=1, main_len=32768, steps=64):
    w = Outlier32K(main_len=main_len, steps=steps)
    rng = rng_for(config_index)
    hkv, d, hq = GQA_SHAPE["num_kv_heads"], GQA_SHAPE["head_dim"], GQA_SHAPE["num_q_heads"]
    w.span_lengths = lognormal_lengths(rng, w.n_spans, 7.0, 0.8, w.main_len)
    w.spans = spans_from_lengths(w.span_lengths)
    w.evict_ids, _ = choose_until(rng, w.spans, list(range(w.n_spans)), w.main_len / 2)
    w.outlier_k = np.stack([rng.choice(d, 4, replace=False) for _ in range(hkv)])
    w.outlier_v = np.stack([rng.choice(d, 4, replace=False) for _ in range(hkv)])
    w.main_k = _with_outliers(rng, (1, w.main_len, hkv, d), w.outlier_k)
    w.main_v = _with_outliers(rng, (1, w.main_len, hkv, d), w.outlier_v)
    w.aux_k = _with_outliers(rng, (1, w.aux_private, hkv, d), w.outlier_k)
    w.aux_v = _with_outliers(rng, (1, w.aux_private, hkv, d), w.outlier_v)
    w.step_k = np.stack([_with_outliers(rng, (1, 2, hkv, d), w.outlier_k) for _ in range(steps)])
    w.step_v = np.stack([_with_outliers(rng, (1, 2, hkv, d), w.outlier_v) for _ in range(steps)])
    w.q = normal_bf16(rng, (steps, 2, hq, d))
    return w


@dataclass
class Compaction64K:
    """64K tokens = 40 reasoning spans U[200, 800] interleaved (reasoning,
    tool, reasoning, tool, ...) with 40 tool spans (LogNormal(7.0, 0.8) scaled
    to fill the rest); whole tool spans evicted in seeded order until at least
    65% of all tokens are gone; 128 decode steps after the eviction."""
    length: int = 65536
    n_pairs: int = 40
    steps: int = 128
    evict_frac: float = 0.65
    reasoning: list = field(default_factory=list)
    tool: list = field(default_factory=list)
    spans: list = field(default_factory=list)   # [(start, end)] of the 40 tool spans
    evict_ids: list = field(default_factory=list)
    evicted_tokens: int = 0
    seed: int = SEED_BASE * 100 + 3


def compaction64k(config_index=3, length=65536, n_pairs=40, evict_frac=0.65):
    w = Compaction64K(length=length, n_pairs=n_pairs, evict_frac=evict_frac)
    rng = rng_for(config_index)
    w.reasoning = rng.integers(200, 801, n_pairs).tolist()
    w.tool = lognormal_lengths(rng, n_pairs, 7.0, 0.8, length - sum(w.reasoning))
    pos = 0
    for r, t in zip(w.reasoning, w.tool):
        pos += r
        w.spans.append((pos, pos + t))
        pos += t
    assert pos == length
    w.evict_ids, w.evicted_tokens = choose_until(rng, w.spans, list(range(n_pairs)),
                                                 math.ceil(evict_frac * length))
    return w


@dataclass
class FullStack:
    """36 layers x 8 KV heads x 128, 32 query heads; a non-evictable 16K
    prefix, then 30 turns of 8192 tokens (reasoning U[200, 800], the rest one
    tool span).  Every 4 turns an auxiliary thread forks (512 private tokens)
    and names seeded-random live tool spans until at least 60% of the live
    tool tokens are covered; they are evicted at the next turn's Phase 1."""
    num_layers: int = 36
    prefix: int = 16384
    turns: int = 30
    turn_len: int = 8192
    interval: int = 4
    aux_private: int = 512
    evict_frac: float = 0.60
    reasoning: list = field(default_factory=list)
    seed: int = SEED_BASE * 100 + 4


def full_stack(config_index=4, turns=30, turn_len=8192, prefix=16384, num_layers=36):
    w = FullStack(turns=turns, turn_len=turn_len, prefix=prefix, num_layers=num_layers)
    rng = rng_for(config_index)
    w.reasoning = rng.integers(200, 801, turns).tolist()
    w._rng = rng  # later choices continue the same stream
    return w


# ---------------------------------------------------------------------------
def device_normal_bf16(shape, seed, device):
    """N(0, 1) bfloat16 tensor drawn on ``device`` by a seeded torch generator."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    return torch.randn(shape, generator=gen, device=device, dtype=torch.float32).to(torch.bfloat16)


def to_torch_bf16(bits, device):
    """uint16 bf16 bit patterns -> torch.bfloat16 tensor on ``device``."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).to(device)


def torch_bf16_to_f64(t):
    """torch.bfloat16 tensor (any device) -> exact float64 numpy array."""
    import torch
    bits = t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return bf16_value(bits)
