"""fp64 CPU oracle for position-free paged attention.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library; the one thing it takes from outside is the input format (span flag
bit values) of the seeded input generator in ``workloads``.

What it computes (paper, Sec. 3.2.1 "Mechanism", the score equation, and
Sec. 3.1.1 "Three User-Facing Primitives", eq. (1) with the span semantics
around it; Sec. 3.3.1 for how spans are composed in a final request):

* the cache holds unrotated keys K~ and values V in 16-token pages reached
  through a per-request block table;
* queries and keys are rotated by RoPE at the token's per-request logical
  position (positions are only fed to RoPE, never to the mask);
* query t sees key j iff w(t) <= j <= t in sequence-index space, where the
  window start w is the span start for an SSEP span, 0 for a PDEP span, and
  inherited from the previous span for an unflagged span (its blocks continue
  the previous hash chain);
* softmax(score) V with score = (R_t q)^T (R_pi(j) k~_j) * scale, scale 1/sqrt(D)
  unless given.

Every step is written out in float64 with no blocking or fusion beyond
chunking the query rows so that score blocks stay small.  Where the paper leaves
a point open the oracle takes: NeoX half-split pairing (GPT-J on request),
omega_i = theta^(-2i/D), KV head g = h // (Hq/Hkv), and for decode a query at the
request's last token, which the call's kv_write has stored.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np

from workloads import PDEP, QUERY, SSEP

BLOCK = 16


# -------------------------------------------------------------------------------------
# RoPE (Sec. 3.2.1 score equation; rotation R_p of RoFormer with omega_i = theta^(-2i/D))
# -------------------------------------------------------------------------------------

def rope_inv_freq(head_dim: int, theta: float) -> np.ndarray:
    """omega_i = theta^(-2i/D), i = 0 .. D/2-1, in float64 (D: the rotated width)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(float(theta), -2.0 * i / head_dim)


def rope(x: np.ndarray, pos: np.ndarray, theta: float, style: str = "neox",
         inv_freq: Optional[Sequence[float]] = None, rotary_dim: Optional[int] = None) -> np.ndarray:
    """Rotate the last axis of ``x`` (float64) by R_p, p = ``pos`` broadcast over the
    leading axes.  Only the first R = ``rotary_dim`` (default: all D) elements turn;
    the rest pass through.  Within them NeoX pairs element i with i + R/2, GPT-J pairs
    2i with 2i+1, and pair i turns by the angle p * omega_i, omega_i = theta^(-2i/R)
    unless ``inv_freq`` (R/2 values) gives the frequencies (scaled RoPE variants)."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    R = D if rotary_dim is None else int(rotary_dim)
    om = rope_inv_freq(R, theta) if inv_freq is None else np.asarray(inv_freq, dtype=np.float64)
    assert om.shape == (R // 2,)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * om
    c, s = np.cos(ang), np.sin(ang)
    y = x.copy()
    if style == "neox":
        a, b = x[..., : R // 2], x[..., R // 2:R]
        y[..., :R] = np.concatenate([a * c - b * s, b * c + a * s], axis=-1)
        return y
    if style == "gptj":
        a, b = x[..., 0:R:2], x[..., 1:R:2]
        y[..., 0:R:2] = a * c - b * s
        y[..., 1:R:2] = b * c + a * s
        return y
    raise ValueError(f"unknown rope style {style!r}")


# -------------------------------------------------------------------------------------
# Span windows (Sec. 3.1.1, eq. (1) and the SSep / PDep semantics it implements)
# -------------------------------------------------------------------------------------

def span_windows(span_start: Sequence[int], span_flags: Sequence[int], seq_len: int,
                 span_window: Optional[Sequence[int]] = None) -> np.ndarray:
    """Window start w(n) for every token n of one request.

    SSEP: the span is detached from the preceding chain, so it sees only itself
    (w = its start).  PDEP: it depends on the whole preceding prompt (w = 0).
    Neither: its blocks hash through the previous block, so it keeps the window
    of the span before it (0 for the first span).  ``span_window`` entries >= 0
    override the rule (generalised windows)."""
    S = len(span_start)
    w = np.empty(seq_len, dtype=np.int64)
    prev = 0
    for k in range(S):
        b = int(span_start[k])
        e = int(span_start[k + 1]) if k + 1 < S else seq_len
        f = int(span_flags[k])
        if (f & SSEP) and (f & PDEP):
            raise ValueError("a span cannot be both SSEP and PDEP")
        if span_window is not None and int(span_window[k]) >= 0:
            wk = int(span_window[k])
        elif f & SSEP:
            wk = b
        elif f & PDEP:
            wk = 0
        else:
            wk = prev
        w[b:e] = wk
        prev = wk
    return w


def query_tokens(span_start, span_flags, seq_len) -> np.ndarray:
    """Sequence indices of the tokens computed in a prefill call: the tokens of the
    spans flagged QUERY, in sequence order."""
    S = len(span_start)
    out = []
    for k in range(S):
        if int(span_flags[k]) & QUERY:
            b = int(span_start[k])
            e = int(span_start[k + 1]) if k + 1 < S else seq_len
            out.append(np.arange(b, e, dtype=np.int64))
    return np.concatenate(out) if out else np.zeros(0, dtype=np.int64)


# -------------------------------------------------------------------------------------
# Paged cache
# -------------------------------------------------------------------------------------

def kv_write(k_pool: np.ndarray, v_pool: np.ndarray, k_new: np.ndarray, v_new: np.ndarray,
             slot_mapping: Sequence[int]) -> None:
    """Store row i of k_new / v_new (unrotated, Sec. 3.2.1) at slot s = block*16 + offset,
    i.e. pool[s // 16][:, s % 16, :]; negative slots are skipped.  Works on any dtype
    (bit-exact copy), in place."""
    for i, s in enumerate(slot_mapping):
        s = int(s)
        if s < 0:
            continue
        b, o = divmod(s, BLOCK)
        k_pool[b, :, o, :] = k_new[i]
        v_pool[b, :, o, :] = v_new[i]


def gather(pool: np.ndarray, block_row: np.ndarray, n_tokens: int, kv_head: int) -> np.ndarray:
    """Rows 0..n_tokens-1 of one request and one KV head, through its block table."""
    n = np.arange(n_tokens)
    return np.asarray(pool[block_row[n // BLOCK], kv_head, n % BLOCK, :], dtype=np.float64)


def blocks_gather(pool: np.ndarray, block_ids: Sequence[int]) -> np.ndarray:
    """Copy out whole cache blocks (Sec. 3.2.3, offloading): result[i] = pool[block_ids[i]],
    shape [n][Hkv][16][D], same dtype (bit-exact).  The blocks carry unrotated keys, so
    nothing about their positions travels with them."""
    out = np.empty((len(block_ids),) + pool.shape[1:], dtype=pool.dtype)
    for i, b in enumerate(block_ids):
        out[i] = pool[int(b)]
    return out


def blocks_scatter(pool: np.ndarray, block_ids: Sequence[int], src: np.ndarray) -> None:
    """Bring blocks back (Sec. 3.2.3): pool[block_ids[i]] = src[i], in place; the ids may
    differ from the ones the blocks were gathered from."""
    for i, b in enumerate(block_ids):
        pool[int(b)] = src[i]


# -------------------------------------------------------------------------------------
# Attention
# -------------------------------------------------------------------------------------

def _attend(qr: np.ndarray, kr: np.ndarray, v: np.ndarray, t: np.ndarray, w: np.ndarray,
            scale: float) -> np.ndarray:
    """Masked softmax attention for query rows qr [T][D] (already rotated) at sequence
    indices t with window starts w, against rotated keys kr [L][D] and values v [L][D]."""
    L = kr.shape[0]
    s = (qr @ kr.T) * scale
    j = np.arange(L)
    vis = (j[None, :] >= w[:, None]) & (j[None, :] <= t[:, None])
    s = np.where(vis, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    p = np.where(vis, np.exp(s - m), 0.0)
    return (p @ v) / p.sum(axis=1, keepdims=True)


def _attend_request(q_rows: np.ndarray, q_idx: np.ndarray, k_pool, v_pool, block_row, seq_len,
                    pos_row: np.ndarray, w_tok: np.ndarray, num_kv_heads: int, theta: float,
                    scale: float, style: str, chunk: int = 512, rope_kw: Optional[dict] = None) -> np.ndarray:
    """q_rows [T][Hq][D] at sequence indices q_idx of one request -> O [T][Hq][D]."""
    T, Hq, D = q_rows.shape
    G = Hq // num_kv_heads
    rk = rope_kw or {}
    out = np.empty((T, Hq, D), dtype=np.float64)
    if T == 0:
        return out
    hi = int(q_idx.max()) + 1                 # keys past the last query are never visible
    for g in range(num_kv_heads):
        kr = rope(gather(k_pool, block_row, hi, g), pos_row[:hi], theta, style, **rk)
        v = gather(v_pool, block_row, hi, g)
        for c0 in range(0, T, chunk):
            sl = slice(c0, min(T, c0 + chunk))
            t = q_idx[sl]
            w = w_tok[t]
            lo = int(w.min())
            top = int(t.max()) + 1
            for hl in range(G):
                h = g * G + hl
                qr = rope(np.asarray(q_rows[sl, h, :], dtype=np.float64), pos_row[t], theta, style, **rk)
                out[sl, h, :] = _attend(qr, kr[lo:top], v[lo:top], t - lo, w - lo, scale)
    return out


def _scale(head_dim: int, softmax_scale: float) -> float:
    return float(softmax_scale) if softmax_scale else 1.0 / math.sqrt(head_dim)


def prefill(q, k_pool, v_pool, block_tables, positions, seq_lens, cu_spans, span_start, span_flags,
            num_kv_heads: int, theta: float, softmax_scale: float = 0.0, style: str = "neox",
            span_window=None, rows: Optional[np.ndarray] = None, rope_kw: Optional[dict] = None) -> np.ndarray:
    """Prefill output for every query row (or only the rows listed in ``rows``).

    q [total_q][Hq][D] holds the unrotated queries of all requests, request-major, in
    the order of ``query_tokens``; the pools must already hold the call's fresh rows.
    Returns float64 [total_q][Hq][D] (or [len(rows)][Hq][D]).  ``rope_kw`` passes
    ``inv_freq`` / ``rotary_dim`` on to ``rope``."""
    q = np.asarray(q)
    D = q.shape[-1]
    scale = _scale(D, softmax_scale)
    offs = np.concatenate([[0], np.cumsum(seq_lens)]).astype(np.int64)
    want = None if rows is None else np.asarray(rows, dtype=np.int64)
    out_rows = []
    row0 = 0
    for r in range(len(seq_lens)):
        L = int(seq_lens[r])
        sb, se = int(cu_spans[r]), int(cu_spans[r + 1])
        ss, sf = span_start[sb:se], span_flags[sb:se]
        sw = None if span_window is None else span_window[sb:se]
        qi = query_tokens(ss, sf, L)
        n = qi.shape[0]
        sel = np.arange(n)
        if want is not None:
            sel = want[(want >= row0) & (want < row0 + n)] - row0
        if sel.shape[0]:
            w_tok = span_windows(ss, sf, L, sw)
            pos_row = np.asarray(positions[offs[r]:offs[r] + L], dtype=np.int64)
            o = _attend_request(np.asarray(q[row0 + sel], dtype=np.float64), qi[sel], k_pool, v_pool,
                                block_tables[r], L, pos_row, w_tok, num_kv_heads, theta, scale, style,
                                rope_kw=rope_kw)
            out_rows.append((row0 + sel, o))
        row0 += n
    total = row0 if want is None else want.shape[0]
    out = np.empty((total,) + q.shape[1:], dtype=np.float64)
    if want is None:
        for idx, o in out_rows:
            out[idx] = o
    else:
        where = {int(x): i for i, x in enumerate(want)}
        for idx, o in out_rows:
            out[[where[int(x)] for x in idx]] = o
    return out


def decode(q, k_pool, v_pool, block_tables, positions, seq_lens, cu_spans, span_start, span_flags,
           num_kv_heads: int, theta: float, softmax_scale: float = 0.0, style: str = "neox",
           span_window=None, reqs: Optional[Sequence[int]] = None, rope_kw: Optional[dict] = None) -> np.ndarray:
    """Decode output: one query per request at its last token n = L_r - 1 (which the
    call's ``kv_write`` has already stored), window taken from that token's span.
    q [R][Hq][D] -> float64 [R][Hq][D] (or only the requests in ``reqs``)."""
    q = np.asarray(q)
    D = q.shape[-1]
    scale = _scale(D, softmax_scale)
    offs = np.concatenate([[0], np.cumsum(seq_lens)]).astype(np.int64)
    rs = range(len(seq_lens)) if reqs is None else list(reqs)
    out = np.empty((len(rs),) + q.shape[1:], dtype=np.float64)
    for i, r in enumerate(rs):
        L = int(seq_lens[r])
        sb, se = int(cu_spans[r]), int(cu_spans[r + 1])
        sw = None if span_window is None else span_window[sb:se]
        w_tok = span_windows(span_start[sb:se], span_flags[sb:se], L, sw)
        pos_row = np.asarray(positions[offs[r]:offs[r] + L], dtype=np.int64)
        out[i] = _attend_request(np.asarray(q[r:r + 1], dtype=np.float64), np.array([L - 1]), k_pool,
                                 v_pool, block_tables[r], L, pos_row, w_tok, num_kv_heads, theta,
                                 scale, style, rope_kw=rope_kw)[0]
    return out


def visible_pairs(seq_lens, cu_spans, span_start, span_flags, decode_mode: bool = False,
                  span_window=None) -> int:
    """Number of visible (query token, key) pairs of a batch, the unit in which the
    prefill work 4*D*Hq*P is counted."""
    total = 0
    for r in range(len(seq_lens)):
        L = int(seq_lens[r])
        sb, se = int(cu_spans[r]), int(cu_spans[r + 1])
        sw = None if span_window is None else span_window[sb:se]
        w = span_windows(span_start[sb:se], span_flags[sb:se], L, sw)
        t = np.array([L - 1]) if decode_mode else query_tokens(span_start[sb:se], span_flags[sb:se], L)
        total += int(np.sum(t - w[t] + 1))
    return total
