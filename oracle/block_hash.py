"""CPU oracle of the block-hash rule and of span reuse decisions.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the
library's native span cache.

What it computes (paper, Sec. 3.1.1 "Three User-Facing Primitives", eq. (1)):
the hash h_i of KV block i (16 tokens, x_i) of a token sequence is

* H(h_0, x_i)            if the block's first token is the span separator SSEP,
* H(h_0, x_1 .. x_i)     if the block's first token is the prompt-depend PDEP,
* H(h_{i-1}, x_i)        otherwise (h_{i-1} = h_0 for the first block),

with h_0 a global seed and H a cryptographic hash; the markers act only as a
block's first token.  The byte encoding is a reading (the paper fixes none):
H is SHA-256 over the 32-byte chaining value followed by the tokens as int32
little-endian.  Only full blocks are hashed (a partial block is never reused).

``spans_from_blocks`` states which spans of a sequence are computed and which
are read from the cache given the per-block hits: spans begin at token 0 and
at each marker block (SSEP/PDEP span of Sec. 3.1.1, with the window that the
flag gives), and wherever hit and miss alternate inside one hash chain (an
unflagged span, which keeps the window of the span before it).  Computed spans
carry QUERY.
"""
from __future__ import annotations

import hashlib
from typing import List, Sequence, Tuple

import numpy as np

from workloads import PDEP, QUERY, SSEP

BLOCK = 16


def _H(chain: bytes, tokens: Sequence[int]) -> bytes:
    """H(chain, tokens): SHA-256 of the chaining value then the int32 LE tokens."""
    return hashlib.sha256(chain + np.asarray(tokens, dtype="<i4").tobytes()).digest()


def block_hashes(tokens: Sequence[int], ssep: int, pdep: int, seed: bytes) -> List[bytes]:
    """h_1 .. h_nb of the nb = len(tokens) // 16 full blocks, by eq. (1)."""
    assert len(seed) == 32 and ssep != pdep
    toks = [int(t) for t in tokens]
    nb = len(toks) // BLOCK
    out: List[bytes] = []
    h_prev = seed
    for i in range(nb):
        x_i = toks[i * BLOCK:(i + 1) * BLOCK]
        if x_i[0] == ssep:
            h = _H(seed, x_i)
        elif x_i[0] == pdep:
            h = _H(seed, toks[:(i + 1) * BLOCK])
        else:
            h = _H(h_prev, x_i)
        out.append(h)
        h_prev = h
    return out


def marker_of_block(tokens: Sequence[int], b: int, ssep: int, pdep: int) -> int:
    first = int(tokens[b * BLOCK])
    return SSEP if first == ssep else PDEP if first == pdep else 0


def spans_from_blocks(tokens: Sequence[int], ssep: int, pdep: int,
                      hits: Sequence[bool]) -> Tuple[List[int], List[int]]:
    """(span_start, span_flags) of a sequence given the hit flag of each full block."""
    n = len(tokens)
    assert n > 0
    nb = -(-n // BLOCK)
    full = n // BLOCK
    starts: List[int] = []
    flags: List[int] = []
    prev_cached = None
    for b in range(nb):
        marker = marker_of_block(tokens, b, ssep, pdep)
        cached = b < full and bool(hits[b])
        if b == 0 or marker or cached != prev_cached:
            starts.append(b * BLOCK)
            flags.append(marker | (0 if cached else QUERY))
        prev_cached = cached
    return starts, flags


def token_windows(tokens: Sequence[int], ssep: int, pdep: int) -> np.ndarray:
    """Window start of every token from the markers alone: the start of the last
    SSEP block at or before the token's block, 0 after a PDEP block or when no
    marker precedes (Sec. 3.1.1 span semantics, token by token)."""
    n = len(tokens)
    w = np.zeros(n, dtype=np.int64)
    cur = 0
    for t in range(n):
        if t % BLOCK == 0:
            m = marker_of_block(tokens, t // BLOCK, ssep, pdep)
            if m == SSEP:
                cur = t
            elif m == PDEP:
                cur = 0
        w[t] = cur
    return w
