"""Seeded synthetic inputs for position-free paged attention.

This module only *arranges* data: random values, paged-pool placement, block
tables, span descriptors and logical positions.  It performs none of the
method's arithmetic (no rotary embedding, no window rule, no attention), so
the CPU oracle and the HIP path can both consume what it builds without
sharing any computation.

Input recipe (stand-in for the paper's RAG workload of retrieved documents,
Sec. 4.1; no dataset items are reproduced): spans of 512 tokens (or the sizes
a case asks for), block-aligned to 16-token KV blocks, drawn from a pool of
shared cached spans in a seeded random order; Q/K/V i.i.d. N(0,1) times a
scale, rounded to the compute dtype; physical blocks handed out from a seeded
permutation of the pool; blocks no request uses (and fresh slots before they
are written) hold NaN when ``poison`` is set.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np
import torch

# Span flags of the batch descriptor (bit values shared with include/pic_attn.h).
SSEP = 1   # span separator: the span is detached from what precedes it
PDEP = 2   # prompt-depend: the span depends on the whole preceding prompt
QUERY = 4  # the span's tokens are computed in this call (they are queries)

BLOCK = 16


@dataclass
class Span:
    """One span of one request.

    ``key`` names a shared cached span (the same key in two requests means the
    same physical blocks); ``None`` makes the span private to its request.
    ``fresh`` spans have no cached KV yet: their K/V rows are produced in the
    call and written to the pool through the slot mapping.
    """
    length: int
    flags: int
    key: Optional[object] = None
    fresh: bool = False


@dataclass
class Workload:
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    rope_theta: float
    dtype: torch.dtype
    is_decode: bool
    seq_lens: np.ndarray        # int32 [R]
    cu_spans: np.ndarray        # int32 [R+1]
    span_start: np.ndarray      # int32 [S]
    span_flags: np.ndarray      # int32 [S]
    block_tables: np.ndarray    # int32 [R][max_blocks]
    positions: np.ndarray       # int32 [sum L]
    num_blocks: int
    k_pool: torch.Tensor        # [NB][Hkv][16][D] before the fresh rows are written
    v_pool: torch.Tensor
    k_new: torch.Tensor         # [n_new][Hkv][D]
    v_new: torch.Tensor
    slot_mapping: np.ndarray    # int32 [n_new], slot = block*16 + offset
    q: torch.Tensor             # prefill: [total_q][Hq][D]; decode: [R][Hq][D]
    q_tokens: np.ndarray        # int32 [rows of q, 2]: (request, sequence index)
    block_size: int = BLOCK
    softmax_scale: float = 0.0  # 0 means 1/sqrt(head_dim)
    span_window: Optional[np.ndarray] = None  # optional explicit window start per span
    rope_inv_freq: Optional[np.ndarray] = None  # optional RoPE frequencies [rotary_dim/2]
    rotary_dim: Optional[int] = None            # optional partial rotary width (None: head_dim)
    info: dict = field(default_factory=dict)

    @property
    def num_reqs(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def seq_offsets(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.seq_lens)]).astype(np.int64)


def _randn(gen: torch.Generator, shape, scale: float, dtype: torch.dtype) -> torch.Tensor:
    x = torch.randn(shape, generator=gen, dtype=torch.float32)
    if scale != 1.0:
        x.mul_(scale)
    return x.to(dtype)


def build(name: str, requests: Sequence[Sequence[Span]], *, num_q_heads: int, num_kv_heads: int,
          head_dim: int, rope_theta: float, dtype: torch.dtype, seed: int, value_scale: float = 1.0,
          num_blocks: Optional[int] = None, poison: bool = True, decode: bool = False,
          position_offsets: Optional[Sequence[int]] = None, shuffle_blocks: bool = True,
          softmax_scale: float = 0.0, max_blocks: Optional[int] = None,
          block_overrides: Optional[dict] = None) -> Workload:
    """Lay out ``requests`` (lists of spans) in a paged pool and draw values.

    Shared spans (same ``key``) must start on a block boundary and, unless they
    end the request, span whole blocks, so their physical blocks can be reused
    verbatim.  Value draws come from one ``torch.Generator`` in the order
    Q, K (cached, then fresh), V (cached, then fresh); layout randomness comes
    from ``numpy.random.default_rng(seed)``.
    """
    rng = np.random.default_rng(seed)
    gen = torch.Generator().manual_seed(seed)
    R = len(requests)
    seq_lens = np.array([sum(s.length for s in req) for req in requests], dtype=np.int64)
    nblk_req = [(int(L) + BLOCK - 1) // BLOCK for L in seq_lens]

    # ---- physical block allocation -------------------------------------------------
    shared_blocks = {}   # key -> list of physical blocks
    need = 0
    for req in requests:
        for s in req:
            if s.key is not None and s.key not in shared_blocks:
                shared_blocks[s.key] = None
                need += (s.length + BLOCK - 1) // BLOCK
    for r, req in enumerate(requests):
        priv = 0
        n = 0
        for s in req:
            if s.key is None:
                priv += 1
            n += s.length
        need += nblk_req[r]  # upper bound for private blocks
    if num_blocks is None:
        num_blocks = need
    order = rng.permutation(num_blocks) if shuffle_blocks else np.arange(num_blocks)
    cursor = 0

    def take(n):
        nonlocal cursor
        if cursor + n > num_blocks:
            raise ValueError("pool too small for the workload")
        out = order[cursor:cursor + n].tolist()
        cursor += n
        return out

    for key in shared_blocks:
        length = None
        for req in requests:
            for s in req:
                if s.key == key:
                    length = s.length
        shared_blocks[key] = take((length + BLOCK - 1) // BLOCK)

    maxb = max(nblk_req) if max_blocks is None else max_blocks
    block_tables = np.full((R, max(maxb, 1)), -1, dtype=np.int32)
    span_start, span_flags, cu_spans = [], [], [0]
    # token bookkeeping: (request, seq index) for cached-shared, cached-private and fresh tokens
    for r, req in enumerate(requests):
        n = 0
        for s in req:
            span_start.append(n)
            span_flags.append(s.flags)
            if s.key is not None:
                if n % BLOCK:
                    raise ValueError("shared span must start on a block boundary")
                blks = shared_blocks[s.key]
                for i, b in enumerate(blks):
                    bi = n // BLOCK + i
                    if bi < block_tables.shape[1]:
                        block_tables[r, bi] = b
            n += s.length
        cu_spans.append(len(span_start))
        # private blocks fill whatever the shared spans did not cover
        for bi in range(nblk_req[r]):
            if block_tables[r, bi] < 0:
                block_tables[r, bi] = take(1)[0]
    if block_overrides:
        for (r, bi), b in block_overrides.items():
            block_tables[r, bi] = b

    # ---- which tokens carry cached values, which are fresh ---------------------------
    # cached-shared values are drawn once per physical slot; cached-private per token.
    cached_slots = []   # physical slots holding cached values (drawn once each)
    seen_slots = set()
    fresh_tok = []      # (r, n)
    q_tok = []          # (r, n)
    for r, req in enumerate(requests):
        n = 0
        for s in req:
            for i in range(s.length):
                t = n + i
                slot = int(block_tables[r, t // BLOCK]) * BLOCK + t % BLOCK
                if s.fresh:
                    fresh_tok.append((r, t, slot))
                elif slot not in seen_slots:
                    seen_slots.add(slot)
                    cached_slots.append(slot)
                if (s.flags & QUERY) and not decode:
                    q_tok.append((r, t))
            n += s.length
    if decode:
        q_tok = [(r, int(seq_lens[r]) - 1) for r in range(R)]

    Hq, Hkv, D = num_q_heads, num_kv_heads, head_dim
    q = _randn(gen, (len(q_tok), Hq, D), value_scale, dtype)
    k_cached = _randn(gen, (len(cached_slots), Hkv, D), value_scale, dtype)
    k_new = _randn(gen, (len(fresh_tok), Hkv, D), value_scale, dtype)
    v_cached = _randn(gen, (len(cached_slots), Hkv, D), value_scale, dtype)
    v_new = _randn(gen, (len(fresh_tok), Hkv, D), value_scale, dtype)

    fill = float("nan") if poison else 0.0
    k_pool = torch.full((num_blocks, Hkv, BLOCK, D), fill, dtype=dtype)
    v_pool = torch.full((num_blocks, Hkv, BLOCK, D), fill, dtype=dtype)
    if cached_slots:
        cs = torch.as_tensor(np.array(cached_slots, dtype=np.int64))
        kp = k_pool.permute(0, 2, 1, 3).reshape(num_blocks * BLOCK, Hkv, D)
        vp = v_pool.permute(0, 2, 1, 3).reshape(num_blocks * BLOCK, Hkv, D)
        kp[cs] = k_cached
        vp[cs] = v_cached
        k_pool = kp.reshape(num_blocks, BLOCK, Hkv, D).permute(0, 2, 1, 3).contiguous()
        v_pool = vp.reshape(num_blocks, BLOCK, Hkv, D).permute(0, 2, 1, 3).contiguous()

    offs = [0] * R if position_offsets is None else list(position_offsets)
    positions = np.concatenate([np.arange(int(L), dtype=np.int64) + offs[r]
                                for r, L in enumerate(seq_lens)]).astype(np.int32)

    return Workload(
        name=name, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, rope_theta=float(rope_theta),
        dtype=dtype, is_decode=decode,
        seq_lens=seq_lens.astype(np.int32), cu_spans=np.array(cu_spans, dtype=np.int32),
        span_start=np.array(span_start, dtype=np.int32), span_flags=np.array(span_flags, dtype=np.int32),
        block_tables=block_tables, positions=positions, num_blocks=num_blocks,
        k_pool=k_pool, v_pool=v_pool, k_new=k_new, v_new=v_new,
        slot_mapping=np.array([s for (_, _, s) in fresh_tok], dtype=np.int32).reshape(-1),
        q=q, q_tokens=np.array(q_tok, dtype=np.int32).reshape(-1, 2),
        softmax_scale=softmax_scale,
        info={"seed": seed, "value_scale": value_scale,
              "fresh_tokens": np.array([(r, t) for (r, t, _) in fresh_tok], dtype=np.int32).reshape(-1, 2)},
    )


# ----------------------------------------------------------------------------------------
# The five benchmark-shaped workloads
# ----------------------------------------------------------------------------------------

def tiny_fp32(seed: int = 1000, tail_only: bool = False) -> Workload:
    """Tiny fp32 prefill: two SSEP spans of 64 tokens and a 32-token PDEP tail,
    4 query heads over 1 KV head, head_dim 64, theta 1e4, 16 pool blocks of which
    10 are used in shuffled order.  All 160 tokens are queries (fresh), or only the
    tail with the two spans cached when ``tail_only``."""
    if tail_only:
        spans = [Span(64, SSEP), Span(64, SSEP), Span(32, PDEP | QUERY, fresh=True)]
    else:
        spans = [Span(64, SSEP | QUERY, fresh=True), Span(64, SSEP | QUERY, fresh=True),
                 Span(32, PDEP | QUERY, fresh=True)]
    return build("tiny_fp32_prefill" + ("_tail" if tail_only else ""), [spans],
                 num_q_heads=4, num_kv_heads=1, head_dim=64, rope_theta=1e4,
                 dtype=torch.float32, seed=seed, value_scale=1.0, num_blocks=16)


def llama3_8b_rag(seed: int = 1001) -> Workload:
    """Llama-3-8B-shaped RAG prefill: 10 cached SSEP spans of 512 tokens and a fresh
    256-token PDEP query tail; 32/8 heads, head_dim 128, theta 5e5, bf16."""
    spans = [Span(512, SSEP, key=("doc", i)) for i in range(10)] + [Span(256, PDEP | QUERY, fresh=True)]
    return build("llama3_8b_rag_prefill", [spans], num_q_heads=32, num_kv_heads=8, head_dim=128,
                 rope_theta=5e5, dtype=torch.bfloat16, seed=seed, value_scale=0.5, num_blocks=512)


def concurrent_reuse(seed: int = 1002, num_reqs: int = 16, pool_spans: int = 32, per_req: int = 8,
            span_len: int = 512, tail: int = 128) -> Workload:
    """Concurrent reuse: each of 16 requests draws 8 of 32 shared cached spans
    (without replacement, random order) plus a private 128-token PDEP query tail."""
    rng = np.random.default_rng(seed + 7919)
    reqs = []
    for _ in range(num_reqs):
        pick = rng.choice(pool_spans, size=per_req, replace=False)
        reqs.append([Span(span_len, SSEP, key=("doc", int(i))) for i in pick]
                    + [Span(tail, PDEP | QUERY, fresh=True)])
    nb = pool_spans * span_len // BLOCK + num_reqs * ((tail + BLOCK - 1) // BLOCK) + 64
    return build("concurrent_reuse_prefill", reqs, num_q_heads=32, num_kv_heads=8, head_dim=128,
                 rope_theta=5e5, dtype=torch.bfloat16, seed=seed, value_scale=0.5, num_blocks=nb)


def decode_64req(seed: int = 1003, num_reqs: int = 64, num_spans: int = 16, span_len: int = 512,
            shared: bool = True) -> Workload:
    """Decode: 64 requests, each an 8192-token context of 16 shared 512-token spans in a
    per-request random order, plus the new token (written through the slot mapping)
    whose query attends to the whole 8193-token context.  ``shared=False`` gives every
    request its own copies of the spans (the unshared control)."""
    rng = np.random.default_rng(seed + 7919)
    reqs = []
    for r in range(num_reqs):
        order = rng.permutation(num_spans)
        if shared:
            spans = [Span(span_len, SSEP, key=("doc", int(i))) for i in order]
        else:
            spans = [Span(span_len, SSEP, key=("doc", r, int(i))) for i in order]
        spans.append(Span(1, PDEP, fresh=True))
        reqs.append(spans)
    n_unique = num_spans * (1 if shared else num_reqs)
    nb = n_unique * span_len // BLOCK + num_reqs + 16
    return build("decode" + ("" if shared else "_unshared"), reqs, num_q_heads=32, num_kv_heads=8,
                 head_dim=128, rope_theta=5e5, dtype=torch.bfloat16, seed=seed, value_scale=0.5,
                 num_blocks=nb, decode=True, poison=shared)


def llama3_70b_long(seed: int = 1004, num_spans: int = 64, span_len: int = 512, tail: int = 512,
                    part: str = "all") -> Workload:
    """Llama-3-70B-shaped long prefill: 64 SSEP spans of 512 tokens, a seeded half of
    them fresh (queried and written in the call), the other half cached, and a fresh
    512-token PDEP query tail; 64/8 heads, head_dim 128, theta 5e5, bf16.  ``part``
    "tail" or "fresh" keeps the same spans and positions but queries only the tail
    (the fresh spans are then cached) or only the fresh spans (the tail cached)."""
    assert part in ("all", "tail", "fresh")
    rng = np.random.default_rng(seed + 7919)
    fresh = set(rng.choice(num_spans, size=num_spans // 2, replace=False).tolist())
    spans = []
    for i in range(num_spans):
        if i in fresh and part != "tail":
            spans.append(Span(span_len, SSEP | QUERY, fresh=True))
        else:
            spans.append(Span(span_len, SSEP, key=("doc", i)))
    if part == "fresh":
        spans.append(Span(tail, PDEP, key=("tail",)))
    else:
        spans.append(Span(tail, PDEP | QUERY, fresh=True))
    L = num_spans * span_len + tail
    nb = L // BLOCK + 32
    name = "llama3_70b_long_prefill" + ("" if part == "all" else "_" + part)
    return build(name, [spans], num_q_heads=64, num_kv_heads=8, head_dim=128,
                 rope_theta=5e5, dtype=torch.bfloat16, seed=seed, value_scale=0.5, num_blocks=nb)


WORKLOADS = {"tiny_fp32": tiny_fp32, "llama3_8b_rag": llama3_8b_rag, "concurrent_reuse": concurrent_reuse,
             "decode_64req": decode_64req, "llama3_70b_long": llama3_70b_long,
             "llama3_70b_long_tail": lambda **kw: llama3_70b_long(part="tail", **kw),
             "llama3_70b_long_fresh": lambda **kw: llama3_70b_long(part="fresh", **kw)}


def make(name: str, **kw) -> Workload:
    """The named workload (a key of WORKLOADS)."""
    return WORKLOADS[name](**kw)


def small_case(name: str, requests: Sequence[Sequence[Span]], *, Hq=4, Hkv=2, D=64, theta=1e4,
               dtype=torch.float32, seed=0, **kw) -> Workload:
    """A small hand-shaped case for tests (same layout rules as the configs)."""
    return build(name, requests, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D, rope_theta=theta,
                 dtype=dtype, seed=seed, **kw)
