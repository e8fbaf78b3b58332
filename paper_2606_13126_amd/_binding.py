"""ctypes binding of libpic_attn.so: argument marshalling only.

Every function has the name of the C entry point it calls and takes torch
tensors (device memory) and numpy/int arrays (host metadata).  All arithmetic
happens in the HIP library; there is no fallback: if the library is missing the
import of this module raises.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_float, c_int32, c_size_t, c_void_p
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpic_attn.so")

PIC_OK, PIC_EINVAL, PIC_EUNSUPPORTED, PIC_EHIP, PIC_EWORKSPACE = range(5)
PIC_BF16, PIC_F32 = 0, 1
PIC_ROPE_NEOX, PIC_ROPE_GPTJ = 0, 1
PIC_SSEP, PIC_PDEP, PIC_QUERY = 1, 2, 4


class PicError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"pic status {status}: {message}")
        self.status = status


class pic_config(ctypes.Structure):
    _fields_ = [("num_q_heads", c_int32), ("num_kv_heads", c_int32), ("head_dim", c_int32),
                ("block_size", c_int32), ("dtype", c_int32), ("rope_style", c_int32),
                ("rope_theta", c_double), ("softmax_scale", c_float), ("k_prerotated", c_int32),
                ("inv_freq", POINTER(c_double)), ("rotary_dim", c_int32)]


class pic_batch_host(ctypes.Structure):
    _fields_ = [("num_reqs", c_int32), ("seq_lens", POINTER(c_int32)), ("cu_spans", POINTER(c_int32)),
                ("span_start", POINTER(c_int32)), ("span_flags", POINTER(c_int32)),
                ("span_window", POINTER(c_int32))]


class pic_batch_dev(ctypes.Structure):
    _fields_ = [("block_tables", c_void_p), ("max_blocks", c_int32), ("positions", c_void_p)]


class pic_rope_table(ctypes.Structure):
    _fields_ = [("data", c_void_p), ("len", c_int32)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_13126_amd.build`")
_lib = ctypes.CDLL(LIB_PATH)

_P = ctypes.POINTER
_sig = {
    "pic_version": (c_int32, []),
    "pic_last_error": (ctypes.c_char_p, []),
    "pic_rope_table_bytes": (c_int32, [_P(pic_config), c_int32, _P(c_size_t)]),
    "pic_rope_table_build": (c_int32, [_P(pic_config), c_int32, c_void_p, c_void_p]),
    "pic_rope_rotate": (c_int32, [_P(pic_config), _P(pic_rope_table), c_void_p, c_int32, c_int32, c_void_p,
                                  c_void_p]),
    "pic_kv_write": (c_int32, [_P(pic_config), c_void_p, c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_int32,
                               c_void_p]),
    "pic_blocks_gather": (c_int32, [_P(pic_config), c_void_p, c_void_p, c_int32, c_void_p, c_int32, c_void_p,
                                    c_void_p, c_void_p]),
    "pic_blocks_scatter": (c_int32, [_P(pic_config), c_void_p, c_void_p, c_int32, c_void_p, c_int32, c_void_p,
                                     c_void_p, c_void_p]),
    "pic_workspace_size": (c_int32, [_P(pic_config), _P(pic_batch_host), c_int32, _P(c_size_t)]),
    "pic_attn_prefill": (c_int32, [_P(pic_config), _P(pic_batch_host), _P(pic_batch_dev), _P(pic_rope_table),
                                   c_void_p, c_void_p, c_void_p, c_void_p, c_int32, c_void_p, c_size_t, c_void_p]),
    "pic_attn_decode": (c_int32, [_P(pic_config), _P(pic_batch_host), _P(pic_batch_dev), _P(pic_rope_table),
                                  c_void_p, c_void_p, c_void_p, c_void_p, c_int32, c_void_p, c_size_t, c_void_p]),
    "pic_plan_debug": (c_int32, [_P(pic_config), _P(pic_batch_host), c_int32, _P(c_int32), c_int32, _P(c_int32)]),
    "pic_plan_shape": (c_int32, [_P(pic_config), _P(pic_batch_host), c_int32, _P(c_int32)]),
    "pic_attn_decode_noalloc": (c_int32, [_P(pic_config), _P(pic_batch_host), _P(pic_batch_dev), _P(pic_rope_table),
                                          c_void_p, c_void_p, c_void_p, c_void_p, c_int32, c_void_p]),
    # span cache (include/pic_cache.h): host only
    "pic_sha256": (c_int32, [c_void_p, c_size_t, c_void_p]),
    "pic_block_hashes": (c_int32, [c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p]),
    "pic_spans_from_blocks": (c_int32, [c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p, c_void_p, c_int32,
                                        _P(c_int32)]),
    "pic_block_cache_create": (c_int32, [_P(c_void_p)]),
    "pic_block_cache_destroy": (c_int32, [c_void_p]),
    "pic_block_cache_lookup": (c_int32, [c_void_p, c_void_p, c_int32, c_void_p, _P(c_int32)]),
    "pic_block_cache_insert": (c_int32, [c_void_p, c_void_p, c_void_p, c_int32]),
    "pic_block_cache_erase": (c_int32, [c_void_p, c_void_p, c_int32]),
    "pic_block_cache_size": (c_int32, [c_void_p, _P(c_int32)]),
}
for _name, (_res, _args) in _sig.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def _check(status: int) -> None:
    if status != PIC_OK:
        raise PicError(status, _lib.pic_last_error().decode())


def exported_symbols():
    return list(_sig)


def lib():
    return _lib


# ------------------------------------------------------------------------------------
# argument helpers
# ------------------------------------------------------------------------------------

def make_config(num_q_heads, num_kv_heads, head_dim, dtype=PIC_BF16, rope_theta=10000.0,
                rope_style=PIC_ROPE_NEOX, softmax_scale=0.0, k_prerotated=0, block_size=16, inv_freq=None,
                rotary_dim=0) -> pic_config:
    """A pic_config; ``inv_freq`` (rotary_dim/2 floats) is copied and kept alive with it."""
    freq = None if inv_freq is None else np.ascontiguousarray(inv_freq, dtype=np.float64)
    cfg = pic_config(num_q_heads, num_kv_heads, head_dim, block_size, dtype, rope_style, float(rope_theta),
                     float(softmax_scale), int(k_prerotated),
                     None if freq is None else freq.ctypes.data_as(POINTER(c_double)), int(rotary_dim or 0))
    cfg._inv_freq = freq
    return cfg


class HostBatch:
    """Keeps the int32 host arrays of a pic_batch_host alive."""

    def __init__(self, seq_lens, cu_spans, span_start, span_flags, span_window=None):
        self._arrays = [np.ascontiguousarray(a, dtype=np.int32) for a in (seq_lens, cu_spans, span_start, span_flags)]
        self._win = None if span_window is None else np.ascontiguousarray(span_window, dtype=np.int32)
        ptr = lambda a: a.ctypes.data_as(POINTER(c_int32))  # noqa: E731
        self.c = pic_batch_host(len(self._arrays[0]), *[ptr(a) for a in self._arrays],
                                ptr(self._win) if self._win is not None else None)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _dev(block_tables, positions) -> pic_batch_dev:
    return pic_batch_dev(_ptr(block_tables), int(block_tables.shape[1]) if block_tables.dim() == 2 else 0,
                         _ptr(positions))


def _rope(table) -> pic_rope_table:
    if table is None:
        return pic_rope_table(None, 0)
    return pic_rope_table(_ptr(table), int(table.shape[0]))


# ------------------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ------------------------------------------------------------------------------------

def pic_version() -> int:
    return _lib.pic_version()


def pic_rope_table_bytes(cfg: pic_config, num_positions: int) -> int:
    out = c_size_t(0)
    _check(_lib.pic_rope_table_bytes(ctypes.byref(cfg), num_positions, ctypes.byref(out)))
    return out.value


def pic_rope_table_build(cfg: pic_config, table, stream=None) -> None:
    """table: device tensor of pic_rope_table_bytes(cfg, num_positions) bytes whose first
    dimension is num_positions ([n][D/2][2] float32 for PIC_F32, [n][D/2] 4-byte words
    for PIC_BF16)."""
    _check(_lib.pic_rope_table_build(ctypes.byref(cfg), int(table.shape[0]), _ptr(table), _stream(stream)))


def pic_rope_rotate(cfg: pic_config, x, positions, table=None, stream=None) -> None:
    """x: [n][heads][D] tensor rotated in place; positions: int32 [n]."""
    _check(_lib.pic_rope_rotate(ctypes.byref(cfg), ctypes.byref(_rope(table)), _ptr(x), int(x.shape[0]),
                                int(x.shape[1]), _ptr(positions), _stream(stream)))


def pic_kv_write(cfg: pic_config, k_pool, v_pool, k_new, v_new, slot_mapping, stream=None) -> None:
    _check(_lib.pic_kv_write(ctypes.byref(cfg), _ptr(k_pool), _ptr(v_pool), int(k_pool.shape[0]), _ptr(k_new),
                             _ptr(v_new), _ptr(slot_mapping), int(k_new.shape[0]), _stream(stream)))


def pic_blocks_gather(cfg: pic_config, k_pool, v_pool, block_ids, dst_k, dst_v, stream=None) -> None:
    """dst_k[i], dst_v[i] <- pool block block_ids[i]; dst may be pinned host memory."""
    _check(_lib.pic_blocks_gather(ctypes.byref(cfg), _ptr(k_pool), _ptr(v_pool), int(k_pool.shape[0]),
                                  _ptr(block_ids), int(block_ids.shape[0]), _ptr(dst_k), _ptr(dst_v),
                                  _stream(stream)))


def pic_blocks_scatter(cfg: pic_config, k_pool, v_pool, block_ids, src_k, src_v, stream=None) -> None:
    """Pool block block_ids[i] <- src_k[i], src_v[i]; src may be pinned host memory."""
    _check(_lib.pic_blocks_scatter(ctypes.byref(cfg), _ptr(k_pool), _ptr(v_pool), int(k_pool.shape[0]),
                                   _ptr(block_ids), int(block_ids.shape[0]), _ptr(src_k), _ptr(src_v),
                                   _stream(stream)))


def pic_workspace_size(cfg: pic_config, batch: HostBatch, is_decode: bool) -> int:
    out = c_size_t(0)
    _check(_lib.pic_workspace_size(ctypes.byref(cfg), ctypes.byref(batch.c), int(is_decode), ctypes.byref(out)))
    return out.value


def pic_attn_prefill(cfg: pic_config, batch: HostBatch, block_tables, positions, q, o, k_pool, v_pool,
                     workspace=None, table=None, stream=None) -> None:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.pic_attn_prefill(ctypes.byref(cfg), ctypes.byref(batch.c), ctypes.byref(_dev(block_tables, positions)),
                                 ctypes.byref(_rope(table)), _ptr(q), _ptr(o), _ptr(k_pool), _ptr(v_pool),
                                 int(k_pool.shape[0]), _ptr(workspace), ws_bytes, _stream(stream)))


def pic_attn_decode(cfg: pic_config, batch: HostBatch, block_tables, positions, q, o, k_pool, v_pool,
                    workspace=None, table=None, stream=None) -> None:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.pic_attn_decode(ctypes.byref(cfg), ctypes.byref(batch.c), ctypes.byref(_dev(block_tables, positions)),
                                ctypes.byref(_rope(table)), _ptr(q), _ptr(o), _ptr(k_pool), _ptr(v_pool),
                                int(k_pool.shape[0]), _ptr(workspace), ws_bytes, _stream(stream)))


def pic_attn_decode_noalloc(cfg: pic_config, batch: HostBatch, block_tables, positions, q, o, k_pool, v_pool,
                            table=None, stream=None) -> None:
    """pic_attn_decode without a workspace (the library's device scratch holds the partials)."""
    _check(_lib.pic_attn_decode_noalloc(ctypes.byref(cfg), ctypes.byref(batch.c),
                                        ctypes.byref(_dev(block_tables, positions)), ctypes.byref(_rope(table)),
                                        _ptr(q), _ptr(o), _ptr(k_pool), _ptr(v_pool), int(k_pool.shape[0]),
                                        _stream(stream)))


def pic_plan_debug(cfg: pic_config, batch: HostBatch, is_decode: bool) -> np.ndarray:
    n = c_int32(0)
    _check(_lib.pic_plan_debug(ctypes.byref(cfg), ctypes.byref(batch.c), int(is_decode), None, 0, ctypes.byref(n)))
    out = np.zeros((max(n.value, 1), 8), dtype=np.int32)
    _check(_lib.pic_plan_debug(ctypes.byref(cfg), ctypes.byref(batch.c), int(is_decode),
                               out.ctypes.data_as(POINTER(c_int32)), n.value, ctypes.byref(n)))
    return out[: n.value]


def pic_plan_shape(cfg: pic_config, batch: HostBatch, is_decode: bool) -> dict:
    out = (c_int32 * 5)()
    _check(_lib.pic_plan_shape(ctypes.byref(cfg), ctypes.byref(batch.c), int(is_decode), out))
    return {"attention_blocks": out[0], "merge_blocks": out[1], "groups": out[2], "upload_launches": out[3],
            "partial_slots": out[4]}


# ------------------------------------------------------------------------------------
# span cache (host only): block hashes by the rule of Sec. 3.1.1 eq. (1), span
# boundaries from cache hits, and the hash -> block map
# ------------------------------------------------------------------------------------

def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _u8(a) -> np.ndarray:
    return np.ascontiguousarray(np.frombuffer(a, dtype=np.uint8) if isinstance(a, (bytes, bytearray)) else a,
                                dtype=np.uint8)


def pic_sha256(data: bytes) -> bytes:
    buf = np.frombuffer(bytes(data), dtype=np.uint8)
    out = np.zeros(32, dtype=np.uint8)
    _check(_lib.pic_sha256(buf.ctypes.data if len(buf) else None, len(buf), out.ctypes.data))
    return out.tobytes()


def pic_block_hashes(tokens, ssep_token: int, pdep_token: int, seed: bytes) -> np.ndarray:
    """uint8 [len(tokens)//16][32]: the hash of every full block."""
    tok = _i32(tokens)
    sd = _u8(seed)
    if sd.size != 32:
        raise ValueError("seed must be 32 bytes")
    out = np.zeros((len(tok) // 16, 32), dtype=np.uint8)
    _check(_lib.pic_block_hashes(tok.ctypes.data, len(tok), int(ssep_token), int(pdep_token), sd.ctypes.data,
                                 out.ctypes.data))
    return out


def pic_spans_from_blocks(tokens, ssep_token: int, pdep_token: int, hit):
    """(span_start, span_flags) int32 arrays for pic_attn_prefill from per-block hits."""
    tok = _i32(tokens)
    h = np.ascontiguousarray(np.asarray(hit, dtype=bool).astype(np.uint8))
    if h.size != len(tok) // 16:
        raise ValueError("hit needs one entry per full block")
    cap = -(-len(tok) // 16) + 1
    start = np.zeros(cap, dtype=np.int32)
    flags = np.zeros(cap, dtype=np.int32)
    n = c_int32(0)
    _check(_lib.pic_spans_from_blocks(tok.ctypes.data, len(tok), int(ssep_token), int(pdep_token),
                                      h.ctypes.data if h.size else None, start.ctypes.data, flags.ctypes.data, cap,
                                      ctypes.byref(n)))
    return start[: n.value].copy(), flags[: n.value].copy()


def pic_block_cache_create() -> int:
    handle = c_void_p()
    _check(_lib.pic_block_cache_create(ctypes.byref(handle)))
    return handle.value


def pic_block_cache_destroy(cache: int) -> None:
    _check(_lib.pic_block_cache_destroy(cache))


def pic_block_cache_lookup(cache: int, hashes):
    """(block_ids int32 [n] with -1 for a miss, number of hits)."""
    hs = _u8(hashes).reshape(-1, 32)
    ids = np.zeros(len(hs), dtype=np.int32)
    hits = c_int32(0)
    _check(_lib.pic_block_cache_lookup(cache, hs.ctypes.data, len(hs), ids.ctypes.data, ctypes.byref(hits)))
    return ids, hits.value


def pic_block_cache_insert(cache: int, hashes, block_ids) -> None:
    hs = _u8(hashes).reshape(-1, 32)
    ids = _i32(block_ids)
    if len(ids) != len(hs):
        raise ValueError("one block id per hash")
    _check(_lib.pic_block_cache_insert(cache, hs.ctypes.data, ids.ctypes.data, len(hs)))


def pic_block_cache_erase(cache: int, hashes) -> None:
    hs = _u8(hashes).reshape(-1, 32)
    _check(_lib.pic_block_cache_erase(cache, hs.ctypes.data, len(hs)))


def pic_block_cache_size(cache: int) -> int:
    n = c_int32(0)
    _check(_lib.pic_block_cache_size(cache, ctypes.byref(n)))
    return n.value
