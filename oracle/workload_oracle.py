"""Run the fp64 oracle on a seeded workload (test infrastructure only).

Widens the workload's values to float64 (exact for bf16 and fp32), writes the
fresh rows into a copy of the pool with the oracle's own ``kv_write``, and
calls ``prefill`` / ``decode``.
"""
from __future__ import annotations

import numpy as np
import torch

from . import pic_oracle


def pools_after_write(wl):
    """float64 copies of the pools after the call's fresh rows are stored."""
    k = wl.k_pool.to(torch.float64).numpy().copy()
    v = wl.v_pool.to(torch.float64).numpy().copy()
    pic_oracle.kv_write(k, v, wl.k_new.to(torch.float64).numpy(), wl.v_new.to(torch.float64).numpy(),
                        wl.slot_mapping)
    return k, v


def run(wl, rows=None, style: str = "neox", pools=None):
    """Oracle output for a workload: prefill rows (all, or ``rows``) or decode requests."""
    k, v = pools_after_write(wl) if pools is None else pools
    q = wl.q.to(torch.float64).numpy()
    args = (k, v, wl.block_tables, wl.positions, wl.seq_lens, wl.cu_spans, wl.span_start, wl.span_flags,
            wl.num_kv_heads, wl.rope_theta, wl.softmax_scale, style, wl.span_window)
    rope_kw = {"inv_freq": getattr(wl, "rope_inv_freq", None), "rotary_dim": getattr(wl, "rotary_dim", None)}
    if wl.is_decode:
        return pic_oracle.decode(q, *args, reqs=rows, rope_kw=rope_kw)
    return pic_oracle.prefill(q, *args, rows=rows, rope_kw=rope_kw)


def flops(wl) -> float:
    """Algorithmic prefill work 4 * D * Hq * (visible pairs)."""
    P = pic_oracle.visible_pairs(wl.seq_lens, wl.cu_spans, wl.span_start, wl.span_flags,
                                 decode_mode=wl.is_decode, span_window=wl.span_window)
    return 4.0 * wl.head_dim * wl.num_q_heads * P
