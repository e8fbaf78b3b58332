"""C-ABI tests that need no GPU: the library loads, exports what the header
declares, validates arguments before any HIP call, and plans work that covers
every visible (query, key) pair exactly once."""
import ctypes
import os
import re

import numpy as np
import pytest

import workloads as W
from oracle import pic_oracle as O

P = pytest.importorskip("paper_2606_13126_amd")
from paper_2606_13126_amd import _binding as B  # noqa: E402

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = "".join(open(os.path.join(ROOT, "include", h)).read() for h in ("pic_attn.h", "pic_cache.h"))
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pic_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("pic_kv_write", "pic_attn_prefill", "pic_attn_decode", "pic_workspace_size",
                     "pic_blocks_gather", "pic_blocks_scatter"):
        assert required in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(B.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert set(declared_functions()) <= set(B.exported_symbols())


def test_version():
    assert P.pic_version() >= 100


def batch_of(wl):
    return P.HostBatch(wl.seq_lens, wl.cu_spans, wl.span_start, wl.span_flags, wl.span_window)


@pytest.mark.parametrize("kw,status", [
    (dict(num_q_heads=0, num_kv_heads=1, head_dim=64), B.PIC_EINVAL),
    (dict(num_q_heads=6, num_kv_heads=4, head_dim=64), B.PIC_EINVAL),
    (dict(num_q_heads=4, num_kv_heads=1, head_dim=96), B.PIC_EUNSUPPORTED),
    (dict(num_q_heads=4, num_kv_heads=1, head_dim=64, block_size=32), B.PIC_EUNSUPPORTED),
    (dict(num_q_heads=4, num_kv_heads=1, head_dim=64, dtype=7), B.PIC_EUNSUPPORTED),
    (dict(num_q_heads=4, num_kv_heads=1, head_dim=64, rope_theta=-1.0), B.PIC_EINVAL),
    (dict(num_q_heads=4, num_kv_heads=1, head_dim=64, rope_style=5), B.PIC_EINVAL),
    (dict(num_q_heads=4, num_kv_heads=1, head_dim=64, rotary_dim=33, rope_style=1), B.PIC_EINVAL),
    (dict(num_q_heads=4, num_kv_heads=1, head_dim=64, rotary_dim=66, rope_style=1), B.PIC_EINVAL),
    (dict(num_q_heads=4, num_kv_heads=1, head_dim=64, rotary_dim=24), B.PIC_EUNSUPPORTED),
    (dict(num_q_heads=4, num_kv_heads=1, head_dim=64, inv_freq=[1.0] * 31 + [float("nan")]), B.PIC_EINVAL),
    (dict(num_q_heads=4, num_kv_heads=1, head_dim=64, rotary_dim=16, rope_style=1,
          inv_freq=[0.5] * 7 + [float("inf")]), B.PIC_EINVAL),
])
def test_config_validation(kw, status):
    cfg = P.make_config(**kw)
    hb = batch_of(W.tiny_fp32())
    with pytest.raises(P.PicError) as e:
        P.pic_workspace_size(cfg, hb, False)
    assert e.value.status == status


@pytest.mark.parametrize("mut", ["zero_len", "first_span", "order", "both_flags", "bad_bits", "window", "no_span"])
def test_batch_validation(mut):
    seq = np.array([40], np.int32)
    cu = np.array([0, 3], np.int32)
    st = np.array([0, 16, 32], np.int32)
    fl = np.array([W.SSEP, W.SSEP | W.QUERY, W.PDEP | W.QUERY], np.int32)
    win = None
    if mut == "zero_len":
        seq[0] = 0
    elif mut == "first_span":
        st[0] = 1
    elif mut == "order":
        st[2] = 16
    elif mut == "both_flags":
        fl[1] = W.SSEP | W.PDEP
    elif mut == "bad_bits":
        fl[1] = 8
    elif mut == "window":
        win = np.array([-1, 20, -1], np.int32)
    elif mut == "no_span":
        cu = np.array([0, 0], np.int32)
    cfg = P.make_config(4, 1, 64)
    with pytest.raises(P.PicError) as e:
        P.pic_workspace_size(cfg, P.HostBatch(seq, cu, st, fl, win), False)
    assert e.value.status == B.PIC_EINVAL


def test_misaligned_addresses_are_rejected_before_any_hip_call():
    # the kernels move 16-byte chunks (some straight into LDS) and 4-byte words of the
    # int32 arrays: other addresses are refused on the host, nothing is launched
    cfg = P.make_config(4, 1, 64)
    lib = B.lib()
    ok, off8, off2 = ctypes.c_void_p(256), ctypes.c_void_p(264), ctypes.c_void_p(258)

    def refused(rc):
        return rc == B.PIC_EINVAL and "aligned" in lib.pic_last_error().decode()

    assert refused(lib.pic_kv_write(ctypes.byref(cfg), off8, ok, 4, ok, ok, ok, 3, None))
    assert refused(lib.pic_kv_write(ctypes.byref(cfg), ok, ok, 4, ok, off8, ok, 3, None))
    assert refused(lib.pic_kv_write(ctypes.byref(cfg), ok, ok, 4, ok, ok, off2, 3, None))
    assert refused(lib.pic_rope_rotate(ctypes.byref(cfg), None, off8, 5, 2, ok, None))
    assert refused(lib.pic_rope_rotate(ctypes.byref(cfg), None, ok, 5, 2, off2, None))
    assert refused(lib.pic_rope_table_build(ctypes.byref(cfg), 8, off8, None))
    hb = batch_of(W.tiny_fp32())
    for q, o, kp, vp in ((off8, ok, ok, ok), (ok, off8, ok, ok), (ok, ok, off8, ok), (ok, ok, ok, off8)):
        dev = B.pic_batch_dev(256, 16, 256)
        assert refused(lib.pic_attn_prefill(ctypes.byref(cfg), ctypes.byref(hb.c), ctypes.byref(dev), None, q, o, kp,
                                            vp, 16, None, 0, None))
    for bt, pos in ((258, 256), (256, 258)):
        dev = B.pic_batch_dev(bt, 16, pos)
        assert refused(lib.pic_attn_decode(ctypes.byref(cfg), ctypes.byref(hb.c), ctypes.byref(dev), None, ok, ok, ok,
                                           ok, 16, None, 0, None))
    table = B.pic_rope_table(264, 160)
    dev = B.pic_batch_dev(256, 16, 256)
    assert refused(lib.pic_attn_prefill(ctypes.byref(cfg), ctypes.byref(hb.c), ctypes.byref(dev), ctypes.byref(table),
                                        ok, ok, ok, ok, 16, None, 0, None))


def test_errors_before_any_hip_call():
    # invalid calls return before touching the device, so they are safe without a GPU
    cfg = P.make_config(4, 1, 64)
    lib = B.lib()
    fake = ctypes.c_void_p(16)
    assert lib.pic_kv_write(ctypes.byref(cfg), None, fake, 4, fake, fake, fake, 3, None) == B.PIC_EINVAL
    assert lib.pic_kv_write(ctypes.byref(P.make_config(4, 3, 64)), fake, fake, 4, fake, fake, fake, 3,
                            None) == B.PIC_EINVAL
    assert lib.pic_rope_rotate(ctypes.byref(cfg), None, None, 5, 2, fake, None) == B.PIC_EINVAL
    # block offload: NULL buffers, negative counts, empty pool, oversized n, bad config
    assert lib.pic_blocks_gather(ctypes.byref(cfg), fake, fake, 4, fake, 3, None, fake, None) == B.PIC_EINVAL
    assert lib.pic_blocks_scatter(ctypes.byref(cfg), fake, fake, 4, None, 3, fake, fake, None) == B.PIC_EINVAL
    assert lib.pic_blocks_gather(ctypes.byref(cfg), fake, fake, 4, fake, -1, fake, fake, None) == B.PIC_EINVAL
    assert lib.pic_blocks_gather(ctypes.byref(cfg), fake, fake, 0, fake, 2, fake, fake, None) == B.PIC_EINVAL
    assert lib.pic_blocks_scatter(ctypes.byref(cfg), fake, fake, 4, fake, 1 << 24, fake, fake, None) == B.PIC_EINVAL
    assert lib.pic_blocks_gather(ctypes.byref(P.make_config(4, 3, 64)), fake, fake, 4, fake, 2, fake, fake,
                                 None) == B.PIC_EINVAL
    assert lib.pic_kv_write(ctypes.byref(cfg), fake, fake, 4, fake, fake, fake, 1 << 24, None) == B.PIC_EINVAL
    # nothing to move: success without a launch
    assert lib.pic_blocks_gather(ctypes.byref(cfg), None, None, 0, None, 0, None, None, None) == B.PIC_OK
    wl = W.tiny_fp32()
    hb = batch_of(wl)
    dev = B.pic_batch_dev(16, 1, 16)   # max_blocks 1 < 10 blocks of the request
    rc = lib.pic_attn_prefill(ctypes.byref(cfg), ctypes.byref(hb.c), ctypes.byref(dev), None, fake, fake, fake,
                              fake, 16, None, 0, None)
    assert rc == B.PIC_EINVAL and "max_blocks" in lib.pic_last_error().decode()
    # the bf16 8B RAG tail needs split-KV partials: a missing workspace is reported, nothing launched
    wl1 = W.llama3_8b_rag()
    cfg1 = P.make_config(32, 8, 128, rope_theta=5e5)
    dev1 = B.pic_batch_dev(16, 512, 16)
    rc = lib.pic_attn_prefill(ctypes.byref(cfg1), ctypes.byref(batch_of(wl1).c), ctypes.byref(dev1), None, fake,
                              fake, fake, fake, 512, None, 0, None)
    assert rc == B.PIC_EWORKSPACE


def windows_of(wl, r):
    sl = slice(wl.cu_spans[r], wl.cu_spans[r + 1])
    return O.span_windows(wl.span_start[sl], wl.span_flags[sl], int(wl.seq_lens[r]),
                          None if wl.span_window is None else wl.span_window[sl])


def check_exact_cover(wl, dtype, is_decode):
    """Every (request, kv head, query row) gets key intervals that tile [w(t), t]."""
    cfg = P.make_config(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, dtype=dtype)
    items = P.pic_plan_debug(cfg, batch_of(wl), is_decode)
    G = wl.num_q_heads // wl.num_kv_heads
    got = {}
    for req, kvh, rl, rh, kl, kh, tok0, slot in items:
        for row in range(rl, rh):
            t = tok0 + row // G
            hi = min(kh, t + 1)
            if kl < hi:
                got.setdefault((req, kvh, tok0, row), []).append((kl, hi))
    n_rows = 0
    for r in range(wl.num_reqs):
        w = windows_of(wl, r)
        L = int(wl.seq_lens[r])
        sl = slice(wl.cu_spans[r], wl.cu_spans[r + 1])
        if is_decode:
            spans = [(L - 1, L)]
        else:
            ss, sf = wl.span_start[sl], wl.span_flags[sl]
            spans = [(int(ss[k]), int(ss[k + 1]) if k + 1 < len(ss) else L) for k in range(len(ss)) if sf[k] & W.QUERY]
        for b, e in spans:
            for kvh in range(wl.num_kv_heads):
                for row in range((e - b) * G):
                    t = b + row // G
                    iv = sorted(got.pop((r, kvh, b, row)))
                    assert iv[0][0] == w[t] and iv[-1][1] == t + 1, (r, kvh, row, iv)
                    for (a0, a1), (b0, b1) in zip(iv, iv[1:]):
                        assert a1 == b0
                    n_rows += 1
    assert not got, "plan covers rows that are not queries"
    return n_rows


@pytest.mark.parametrize("dtype", [B.PIC_BF16, B.PIC_F32])
@pytest.mark.parametrize("case", ["c0", "c0tail", "unaligned", "chain", "multi"])
def test_plan_exact_cover_small(case, dtype):
    S, Pd, Q, Sp = W.SSEP, W.PDEP, W.QUERY, W.Span
    if case == "c0":
        wl = W.tiny_fp32()
    elif case == "c0tail":
        wl = W.tiny_fp32(tail_only=True)
    elif case == "unaligned":
        wl = W.small_case("u", [[Sp(21, S | Q, fresh=True), Sp(37, S | Q, fresh=True), Sp(11, Pd | Q, fresh=True)]],
                          Hq=8, Hkv=2, D=64)
    elif case == "chain":
        wl = W.small_case("c", [[Sp(10, S), Sp(7, Q, fresh=True), Sp(300, S | Q, fresh=True), Sp(5, Q, fresh=True)]],
                          Hq=4, Hkv=2, D=64)
    else:
        wl = W.small_case("m", [[Sp(16, S, key="a"), Sp(100, Pd | Q, fresh=True)], [Sp(3, Q, fresh=True)],
                                [Sp(16, S, key="a"), Sp(16, S)]], Hq=2, Hkv=2, D=128)
    check_exact_cover(wl, dtype, False)


def test_plan_exact_cover_8b_rag_and_decode():
    assert check_exact_cover(W.llama3_8b_rag(), B.PIC_BF16, False) == 8 * 256 * 4
    dec = W.decode_64req(num_reqs=4)
    assert check_exact_cover(dec, B.PIC_BF16, True) == 4 * 8 * 4


@pytest.mark.parametrize("name", ["concurrent_reuse", "llama3_70b_long"])
def test_plan_pair_count_large(name):
    # every item's key range stays inside its rows' windows, and the pairs add up
    wl = W.make(name)
    G = wl.num_q_heads // wl.num_kv_heads
    cfg = P.make_config(wl.num_q_heads, wl.num_kv_heads, wl.head_dim)
    items = P.pic_plan_debug(cfg, batch_of(wl), False).astype(np.int64)
    total = 0
    for req, kvh, rl, rh, kl, kh, tok0, slot in items:
        rows = np.arange(rl, rh)
        t = tok0 + rows // G
        w = windows_of(wl, int(req))
        assert (kl >= w[t]).all()
        total += np.clip(np.minimum(kh, t + 1) - kl, 0, None).sum()
    pairs = O.visible_pairs(wl.seq_lens, wl.cu_spans, wl.span_start, wl.span_flags)
    assert total == pairs * wl.num_q_heads


@pytest.mark.parametrize("Hq,Hkv,D", [(8, 8, 64), (16, 16, 64), (40, 10, 128), (32, 2, 128), (34, 2, 64)])
def test_plan_exact_cover_decode_shapes(Hq, Hkv, D):
    from tests.cases import decode_case
    wl = decode_case(Hq, Hkv, D, seed=1)
    G = Hq // Hkv
    assert check_exact_cover(wl, B.PIC_BF16, True) == wl.num_reqs * Hkv * G
    # split partial slots are distinct per (split, head group) and dense from 0
    cfg = P.make_config(Hq, Hkv, D)
    items = P.pic_plan_debug(cfg, batch_of(wl), True)
    slots = {}
    for req, kvh, rl, rh, kl, kh, tok0, slot in items:
        if slot >= 0:
            slots.setdefault(int(slot), set()).add((int(req), int(kl), int(kvh) // 8 if G <= 16 else int(kvh)))
    for s, owners in slots.items():
        assert len({(r, k) for r, k, _ in owners}) == 1, (s, owners)
    if slots:
        assert sorted(slots) == list(range(len(slots)))


@pytest.mark.parametrize("dtype", [B.PIC_BF16, B.PIC_F32])
def test_plan_exact_cover_explicit_windows(dtype):
    from tests.cases import windows_decode_case, windows_prefill_case
    wl = windows_prefill_case()
    assert check_exact_cover(wl, dtype, False) == (16 + 16 + 40 + 37) * 8
    assert check_exact_cover(windows_decode_case(), dtype, True) == 2 * 32


# ---- batches with more groups than the kernel arguments hold ----------------------------

@pytest.mark.parametrize("dtype", [B.PIC_BF16, B.PIC_F32])
def test_plan_exact_cover_many_spans(dtype):
    from tests.cases import many_spans_prefill
    wl = many_spans_prefill()
    n = check_exact_cover(wl, dtype, False)
    assert n == wl.q.shape[0] * wl.num_q_heads
    cfg = P.make_config(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, dtype=dtype)
    shape = P.pic_plan_shape(cfg, batch_of(wl), False)
    assert shape["groups"] == 82 and shape["upload_launches"] == 2
    if dtype == B.PIC_BF16:
        assert shape["merge_blocks"] > 0 and shape["partial_slots"] > 0   # the long tails are split
    # the workspace holds the group table and block maps besides the partials
    ws = P.pic_workspace_size(cfg, batch_of(wl), False)
    parts = shape["partial_slots"] * 256 * (wl.head_dim + 2) * 4
    assert ws >= parts + 82 * 48 + 4 * (shape["attention_blocks"] + shape["merge_blocks"])


def test_plan_exact_cover_short_causal_spans():
    from tests.cases import short_causal_spans_prefill
    wl = short_causal_spans_prefill()
    n = check_exact_cover(wl, B.PIC_BF16, False)
    assert n == wl.q.shape[0] * wl.num_q_heads
    cfg = P.make_config(wl.num_q_heads, wl.num_kv_heads, wl.head_dim)
    shape = P.pic_plan_shape(cfg, batch_of(wl), False)
    assert shape["groups"] == 122 and shape["upload_launches"] == 2
    # one attention block per (row tile, KV head, key split), padded to 8 per group
    assert shape["attention_blocks"] >= len(P.pic_plan_debug(cfg, batch_of(wl), False)) == 2744


@pytest.mark.parametrize("Hq,Hkv,D", [(32, 8, 128), (34, 2, 64)])
def test_plan_exact_cover_many_requests_decode(Hq, Hkv, D):
    from tests.cases import many_requests_decode
    wl = many_requests_decode(Hq=Hq, Hkv=Hkv, D=D)
    assert check_exact_cover(wl, B.PIC_BF16, True) == 256 * Hq
    cfg = P.make_config(Hq, Hkv, D)
    shape = P.pic_plan_shape(cfg, batch_of(wl), True)
    assert shape["groups"] == 256 and shape["upload_launches"] == 4


def test_decode_256_requests_is_one_launch_filling_the_chip():
    # 256 requests of 8193 keys: one attention launch of at least 256 workgroups (one
    # per request and head group), not a series of launches over slices of the batch
    wl = W.decode_64req(num_reqs=256, num_spans=4, span_len=512)
    cfg = P.make_config(32, 8, 128)
    shape = P.pic_plan_shape(cfg, batch_of(wl), True)
    assert shape["groups"] == 256 and shape["attention_blocks"] >= 256
    assert shape["upload_launches"] == 4


def test_noalloc_decode_refuses_batches_beyond_its_scratch():
    # 255 requests of 4097 keys: 2 key splits each (510 partial slots), more than the
    # no-allocation entry point's 64 MiB of scratch.  Refused on the host with
    # PIC_EWORKSPACE before any HIP call (the pointers are never dereferenced).
    lib = B.lib()
    R, L = 255, 4097
    seq = np.full(R, L, np.int32)
    cu = np.arange(R + 1, dtype=np.int32)
    hb = B.HostBatch(seq, cu, np.zeros(R, np.int32), np.full(R, W.PDEP, np.int32))
    cfg = P.make_config(32, 8, 128, rope_theta=5e5)
    need = P.pic_workspace_size(cfg, hb, True)
    assert need > 64 << 20
    fake = 16
    dev = B.pic_batch_dev(fake, (L + 15) // 16, fake)
    rc = lib.pic_attn_decode_noalloc(ctypes.byref(cfg), ctypes.byref(hb.c), ctypes.byref(dev), None, fake, fake, fake,
                                     fake, 16, None)
    assert rc == B.PIC_EWORKSPACE
    msg = lib.pic_last_error().decode()
    assert "scratch" in msg and str(need) in msg
