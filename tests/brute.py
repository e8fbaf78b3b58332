"""Independent brute-force formulation used to pin the oracle (tests only).

Shares nothing with oracle/ except the input format.  Differences on purpose:
  * RoPE enters through the relative form: the score of (t, j) is
    Re sum_i conj(zq_i) zk_i exp(i (p_j - p_t) w_i) over complex pairs z, which is
    what (R_t q)^T (R_j k) equals for a rotation (Sec. 3.2.1 score equation);
  * visibility comes from walking the hash chain of eq. (1) backwards span by
    span instead of from a window array;
  * pages are gathered with an explicit per-token loop, softmax is
    scipy.special.softmax over the list of visible keys.
Only for tiny inputs (pure-Python loops).
"""
import math

import numpy as np
from scipy.special import softmax

from workloads import PDEP, QUERY, SSEP


def inv_freq(D, theta):
    return np.array([math.exp(-(2.0 * i / D) * math.log(theta)) for i in range(D // 2)])


def to_complex(x, style):
    D = x.shape[-1]
    if style == "neox":
        return x[..., : D // 2] + 1j * x[..., D // 2:]
    return x[..., 0::2] + 1j * x[..., 1::2]


def from_complex(z, style):
    D = z.shape[-1] * 2
    out = np.empty(z.shape[:-1] + (D,))
    if style == "neox":
        out[..., : D // 2], out[..., D // 2:] = z.real, z.imag
    else:
        out[..., 0::2], out[..., 1::2] = z.real, z.imag
    return out


def rotate_abs(x, pos, theta, style):
    """Absolute rotation through complex multiplication (used to pre-rotate)."""
    z = to_complex(np.asarray(x, dtype=np.float64), style)
    w = inv_freq(x.shape[-1], theta)
    return from_complex(z * np.exp(1j * np.asarray(pos, dtype=np.float64)[..., None] * w), style)


def visible(starts, flags, L, t, j):
    """Does token t see key j?  Walk eq. (1)'s chain back from t's span."""
    if j > t:
        return False
    k = max(i for i in range(len(starts)) if starts[i] <= t)
    while True:
        f = flags[k]
        if f & PDEP:
            return True
        if f & SSEP:
            return j >= starts[k]
        if k == 0:
            return True
        k -= 1


def page_row(pool, table_row, n, g):
    blk = table_row[n // 16]
    return np.asarray(pool[blk][g][n % 16], dtype=np.float64)


def attention(q, k_pool, v_pool, block_tables, positions, seq_lens, cu_spans, span_start, span_flags,
              num_kv_heads, theta, scale, style="neox", decode=False):
    q = np.asarray(q, dtype=np.float64)
    Hq, D = q.shape[1], q.shape[2]
    G = Hq // num_kv_heads
    w = inv_freq(D, theta)
    out = np.zeros_like(q)
    row = 0
    off = 0
    for r in range(len(seq_lens)):
        L = int(seq_lens[r])
        starts = [int(x) for x in span_start[cu_spans[r]:cu_spans[r + 1]]]
        flags = [int(x) for x in span_flags[cu_spans[r]:cu_spans[r + 1]]]
        pos = [int(positions[off + n]) for n in range(L)]
        if decode:
            toks = [L - 1]
        else:
            toks = []
            for k in range(len(starts)):
                if flags[k] & QUERY:
                    e = starts[k + 1] if k + 1 < len(starts) else L
                    toks.extend(range(starts[k], e))
        for t in toks:
            vis = [j for j in range(L) if visible(starts, flags, L, t, j)]
            for h in range(Hq):
                g = h // G
                zq = to_complex(q[row, h], style)
                sc = []
                for j in vis:
                    zk = to_complex(page_row(k_pool, block_tables[r], j, g), style)
                    sc.append(scale * float(np.sum(np.conj(zq) * zk * np.exp(1j * (pos[j] - pos[t]) * w)).real))
                p = softmax(np.array(sc))
                acc = np.zeros(D)
                for pj, j in zip(p, vis):
                    acc += pj * page_row(v_pool, block_tables[r], j, g)
                out[row, h] = acc
            row += 1
        off += L
    return out[:row]
