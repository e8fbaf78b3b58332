"""CPU fp64 oracle (test infrastructure only; see pic_oracle)."""
from .pic_oracle import (decode, gather, kv_write, prefill, query_tokens, rope, rope_inv_freq,
                         span_windows, visible_pairs)

__all__ = ["decode", "gather", "kv_write", "prefill", "query_tokens", "rope", "rope_inv_freq",
           "span_windows", "visible_pairs"]
