"""A synthetic RAG session over the span cache (Sec. 3.3.1 "Request submission"):
documents are prefilled once, then reused at new offsets in a later prompt.

Attention needs per-token q, K and V; with no model here they are drawn from a
generator seeded by the hash of the token's block (eq. (1)), so that every
block with the same hash holds the same unrotated K and V wherever it sits --
the property a real model gives an SSEP span, whose keys the position-free
cache stores before RoPE.  The trailing partial block, which is never hashed,
is seeded by its tokens.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass

import numpy as np
import torch

BLOCK = 16
SSEP_TOK, PDEP_TOK = 128011, 128012
SEED = hashlib.sha256(b"pic block hash seed").digest()


def rand_tokens(rng, n, lo=0, hi=128000):
    return rng.integers(lo, hi, size=n).astype(np.int64)


def rag_prompt(rng, docs, system_len=32, task_len=40):
    """[system pad][SSEP doc1 pad][SSEP doc2 pad]...[PDEP task]: every marker at a block start
    (padding token 5)."""
    toks = list(rand_tokens(rng, system_len))
    toks += [5] * ((-len(toks)) % BLOCK)
    for d in docs:
        toks += [SSEP_TOK] + list(d)
        toks += [5] * ((-len(toks)) % BLOCK)  # padding token 5
    toks += [PDEP_TOK] + list(rand_tokens(rng, task_len - 1))
    return np.array(toks, dtype=np.int64)


def _gen(key: bytes, salt: int) -> torch.Generator:
    g = torch.Generator()
    g.manual_seed(int.from_bytes(hashlib.sha256(key + bytes([salt])).digest()[:8], "little") & (2**63 - 1))
    return g


def block_rows(key: bytes, n: int, Hq: int, Hkv: int, D: int, dtype):
    """q [n][Hq][D], k, v [n][Hkv][D] of the n tokens of one block keyed by `key`."""
    q = torch.randn((BLOCK, Hq, D), generator=_gen(key, 0), dtype=torch.float32)[:n]
    k = torch.randn((BLOCK, Hkv, D), generator=_gen(key, 1), dtype=torch.float32)[:n] * 0.5
    v = torch.randn((BLOCK, Hkv, D), generator=_gen(key, 2), dtype=torch.float32)[:n]
    return q.to(dtype), k.to(dtype), v.to(dtype)


@dataclass
class Step:
    """One prompt of the session: its span descriptor and the call's inputs."""
    tokens: np.ndarray
    span_start: np.ndarray
    span_flags: np.ndarray
    table: np.ndarray          # int32 [nb] block ids
    fresh: np.ndarray          # int64 sequence indices computed in the call (q rows, k/v rows)
    slots: np.ndarray          # int32 [n_fresh]
    q: torch.Tensor
    k_new: torch.Tensor
    v_new: torch.Tensor
    n_hits: int


def plan_prompt(tokens, hashes, hit_ids, spans_fn, alloc, Hq, Hkv, D, dtype) -> Step:
    """Block table and fresh rows of one prompt given its block hashes (uint8 [nb_full][32]),
    the cache lookup (block id or -1 per full block) and a span builder
    spans_fn(tokens, hit) -> (span_start, span_flags)."""
    L = len(tokens)
    full, nb = L // BLOCK, -(-L // BLOCK)
    hit = np.asarray(hit_ids) >= 0
    starts, flags = spans_fn(tokens, hit)
    starts = np.asarray(starts, dtype=np.int32)
    flags = np.asarray(flags, dtype=np.int32)
    table = np.array([int(hit_ids[b]) if b < full and hit[b] else alloc() for b in range(nb)], dtype=np.int32)
    ends = np.append(starts[1:], L)
    fresh = np.concatenate([np.arange(s, e) for s, e, f in zip(starts, ends, flags) if f & 4] or
                           [np.zeros(0, dtype=np.int64)]).astype(np.int64)
    qs, ks, vs = [], [], []
    for b in sorted(set((fresh // BLOCK).tolist())):
        key = bytes(hashes[b]) if b < full else b"tail" + np.asarray(tokens[b * BLOCK:], dtype="<i4").tobytes()
        n = min(BLOCK, L - b * BLOCK)
        q, k, v = block_rows(key, n, Hq, Hkv, D, dtype)
        sel = fresh[(fresh // BLOCK) == b] - b * BLOCK
        qs.append(q[sel])
        ks.append(k[sel])
        vs.append(v[sel])
    slots = (table[fresh // BLOCK].astype(np.int64) * BLOCK + fresh % BLOCK).astype(np.int32)
    cat = lambda xs, h: torch.cat(xs) if xs else torch.zeros((0, h, D), dtype=dtype)  # noqa: E731
    return Step(np.asarray(tokens), starts, flags, table, fresh, slots, cat(qs, Hq), cat(ks, Hkv), cat(vs, Hkv),
                int(hit.sum()))
