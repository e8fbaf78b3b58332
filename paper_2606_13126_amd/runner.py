"""Run the library on a batch described by host arrays (device placement and
the call sequence only; every step of the computation runs in libpic_attn).

A batch object needs the attributes of ``workloads.Workload``: head counts,
head_dim, rope_theta, dtype, is_decode, the span descriptor arrays, block
tables, positions, pools, new K/V rows with their slot mapping, and q.
"""
from __future__ import annotations

import numpy as np
import torch

from . import _binding as B


def config_of(wl, k_prerotated: bool = False, rope_style: int = B.PIC_ROPE_NEOX):
    dtype = B.PIC_F32 if wl.dtype == torch.float32 else B.PIC_BF16
    return B.make_config(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, dtype=dtype, rope_theta=wl.rope_theta,
                         rope_style=rope_style, softmax_scale=wl.softmax_scale, k_prerotated=int(k_prerotated),
                         inv_freq=getattr(wl, "rope_inv_freq", None), rotary_dim=getattr(wl, "rotary_dim", None))


class DeviceBatch:
    """Device copies of a batch plus the host span descriptor; ``write()`` stores
    the fresh rows, ``attend()`` runs prefill or decode into ``self.o``."""

    def __init__(self, wl, device="cuda", rope_style: int = B.PIC_ROPE_NEOX, table_positions: int | None = None,
                 k_prerotated: bool = False):
        self.wl = wl
        self.cfg = config_of(wl, k_prerotated=k_prerotated, rope_style=rope_style)
        self.host = B.HostBatch(wl.seq_lens, wl.cu_spans, wl.span_start, wl.span_flags, wl.span_window)
        self.block_tables = torch.from_numpy(np.ascontiguousarray(wl.block_tables)).to(device)
        self.positions = torch.from_numpy(np.ascontiguousarray(wl.positions)).to(device)
        self.k_pool = wl.k_pool.to(device)
        self.v_pool = wl.v_pool.to(device)
        self.k_new = wl.k_new.to(device)
        self.v_new = wl.v_new.to(device)
        self.slots = torch.from_numpy(np.ascontiguousarray(wl.slot_mapping)).to(device)
        self.q = wl.q.to(device)
        self.o = torch.empty_like(self.q)
        ws = B.pic_workspace_size(self.cfg, self.host, wl.is_decode)
        self.workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=device)
        self.table = None
        if table_positions:
            half = wl.head_dim // 2
            # float32 entries are (cos, sin) float pairs, bf16 entries one bf16 pair
            shape = (table_positions, half, 2) if wl.dtype == torch.float32 else (table_positions, half)
            self.table = torch.empty(shape, dtype=torch.float32, device=device)
            assert self.table.numel() * 4 == B.pic_rope_table_bytes(self.cfg, table_positions)
            B.pic_rope_table_build(self.cfg, self.table)

    def write(self, stream=None):
        B.pic_kv_write(self.cfg, self.k_pool, self.v_pool, self.k_new, self.v_new, self.slots, stream=stream)

    def attend(self, stream=None):
        fn = B.pic_attn_decode if self.wl.is_decode else B.pic_attn_prefill
        fn(self.cfg, self.host, self.block_tables, self.positions, self.q, self.o, self.k_pool, self.v_pool,
           workspace=self.workspace, table=self.table, stream=stream)
        return self.o
