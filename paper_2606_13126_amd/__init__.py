"""Position-free paged attention for MI355X (gfx950): Python binding of
libpic_attn.so.  See include/pic_attn.h for the C ABI this package wraps."""
from ._binding import (PIC_BF16, PIC_F32, PIC_PDEP, PIC_QUERY, PIC_ROPE_GPTJ, PIC_ROPE_NEOX, PIC_SSEP, HostBatch,
                       PicError, make_config, pic_attn_decode, pic_attn_prefill, pic_kv_write, pic_plan_debug,
                       pic_rope_rotate, pic_rope_table_build, pic_rope_table_bytes, pic_version, pic_workspace_size)

__all__ = ["PIC_BF16", "PIC_F32", "PIC_PDEP", "PIC_QUERY", "PIC_ROPE_GPTJ", "PIC_ROPE_NEOX", "PIC_SSEP",
           "HostBatch", "PicError", "make_config", "pic_attn_decode", "pic_attn_prefill", "pic_kv_write",
           "pic_plan_debug", "pic_rope_rotate", "pic_rope_table_build", "pic_rope_table_bytes", "pic_version",
           "pic_workspace_size"]
