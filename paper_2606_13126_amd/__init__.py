"""Position-free paged attention for MI355X (gfx950): Python binding of
libpic_attn.so.  See include/pic_attn.h and include/pic_cache.h for the C ABI this
package wraps.

The shared library is loaded on first use of a binding name (importing the
package alone does not load it, so ``python -m paper_2606_13126_amd.build`` works
before the library exists); a missing or broken library raises ImportError.
"""
_EXPORTS = ("PIC_BF16", "PIC_F32", "PIC_PDEP", "PIC_QUERY", "PIC_ROPE_GPTJ", "PIC_ROPE_NEOX", "PIC_SSEP",
            "HostBatch", "PicError", "make_config", "pic_attn_decode", "pic_attn_decode_noalloc", "pic_attn_prefill", "pic_kv_write",
            "pic_plan_debug", "pic_plan_shape", "pic_rope_rotate", "pic_rope_table_build", "pic_rope_table_bytes", "pic_version",
            "pic_workspace_size", "pic_sha256", "pic_block_hashes", "pic_spans_from_blocks",
            "pic_block_cache_create", "pic_block_cache_destroy", "pic_block_cache_lookup", "pic_block_cache_insert",
            "pic_block_cache_erase", "pic_block_cache_size")

__all__ = list(_EXPORTS)


def __getattr__(name):
    if name in _EXPORTS:
        from . import _binding
        return getattr(_binding, name)
    raise AttributeError(name)
