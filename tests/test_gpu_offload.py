"""GPU: moving cache blocks out of the pool and back (Sec. 3.2.3).  The blocks hold
unrotated keys, so after a round trip through pinned host memory they may come back
under new block ids and be read at new logical positions with nothing but the block
table and the positions changed."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import pic_oracle as O
from oracle import workload_oracle as WO
from tests.gpu_util import assert_close, gpu_run, say, to_np

pytestmark = pytest.mark.gpu

S, Pd, Q, Sp = W.SSEP, W.PDEP, W.QUERY, W.Span


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_13126_amd  # noqa: F401  (fails loudly if the library is missing)


def int_view(t):
    return t.view(torch.int32 if t.dtype == torch.float32 else torch.int16)


def shared_span_case(dtype):
    # one cached span at two different offsets in two requests, with fresh tails
    reqs = [[Sp(48, S, key="a"), Sp(32, S, key="b"), Sp(29, Pd | Q, fresh=True)],
            [Sp(32, S, key="b"), Sp(16, S | Q, fresh=True), Sp(48, S, key="a"), Sp(7, Pd | Q, fresh=True)]]
    return W.small_case("offload", reqs, Hq=8, Hkv=2, D=128, theta=5e5, dtype=dtype, seed=41, value_scale=0.5)


def relocate(wl, db, shift, pinned=True):
    """Gather every used block to host memory, scatter it back under new ids into a
    fresh pool of garbage, and point the batch at the new pool, with positions moved
    by ``shift``.  Returns the oracle-side relocated pools and new block table."""
    from paper_2606_13126_amd import _binding as B
    used = np.unique(wl.block_tables[wl.block_tables >= 0]).astype(np.int32)
    n = len(used)
    page = tuple(db.k_pool.shape[1:])
    say(f"[gpu] offload {wl.name}: {n} blocks of {page} {wl.dtype}, pinned={pinned}, shift={shift}")
    ids = torch.from_numpy(used).cuda()
    dev = "cpu" if pinned else "cuda"
    host_k = torch.empty((n,) + page, dtype=db.k_pool.dtype, device=dev, pin_memory=pinned)
    host_v = torch.empty((n,) + page, dtype=db.v_pool.dtype, device=dev, pin_memory=pinned)
    B.pic_blocks_gather(db.cfg, db.k_pool, db.v_pool, ids, host_k, host_v)
    torch.cuda.synchronize()
    kr = O.blocks_gather(int_view(db.k_pool.cpu()).numpy(), used)
    vr = O.blocks_gather(int_view(db.v_pool.cpu()).numpy(), used)
    assert np.array_equal(int_view(host_k.cpu()).numpy(), kr)
    assert np.array_equal(int_view(host_v.cpu()).numpy(), vr)

    nb2 = db.k_pool.shape[0] + 9
    rng = np.random.default_rng(5)
    new_ids = rng.permutation(nb2)[:n].astype(np.int32)
    k2 = (torch.randn((nb2,) + page, device="cuda") * 100).to(db.k_pool.dtype)
    v2 = (torch.randn((nb2,) + page, device="cuda") * 100).to(db.v_pool.dtype)
    k_keep, v_keep = k2.clone(), v2.clone()
    B.pic_blocks_scatter(db.cfg, k2, v2, torch.from_numpy(new_ids).cuda(), host_k, host_v)
    torch.cuda.synchronize()
    want_k = int_view(k_keep.cpu()).numpy().copy()
    want_v = int_view(v_keep.cpu()).numpy().copy()
    O.blocks_scatter(want_k, new_ids, kr)
    O.blocks_scatter(want_v, new_ids, vr)
    assert np.array_equal(int_view(k2.cpu()).numpy(), want_k)
    assert np.array_equal(int_view(v2.cpu()).numpy(), want_v)

    remap = np.full(db.k_pool.shape[0], -1, dtype=np.int64)
    remap[used] = new_ids
    bt = np.where(wl.block_tables >= 0, remap[np.maximum(wl.block_tables, 0)], -1).astype(np.int32)
    db.k_pool, db.v_pool = k2, v2
    db.block_tables = torch.from_numpy(bt).cuda()
    if shift:
        pos = wl.positions.astype(np.int64) + shift
        db.positions = torch.from_numpy(pos.astype(np.int32)).cuda()
        if db.table is not None:
            db.table = torch.empty((int(pos.max()) + 1, wl.head_dim // 2, 2), dtype=torch.float32, device="cuda")
            B.pic_rope_table_build(db.cfg, db.table)

    # the oracle's own pools, relocated by the oracle's copies
    k, v = WO.pools_after_write(wl)
    ko = np.zeros((nb2,) + k.shape[1:])
    vo = np.zeros((nb2,) + v.shape[1:])
    O.blocks_scatter(ko, new_ids, O.blocks_gather(k, used))
    O.blocks_scatter(vo, new_ids, O.blocks_gather(v, used))
    wl.block_tables = bt
    if shift:
        wl.positions = (wl.positions.astype(np.int64) + shift).astype(np.int32)
    return ko, vo


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("shift", [0, 3000])
def test_round_trip_new_ids_new_positions(dtype, shift):
    wl = shared_span_case(dtype)
    db = gpu_run(wl)
    o0 = db.o.clone()
    ko, vo = relocate(wl, db, shift)
    db.attend()
    torch.cuda.synchronize()
    if shift == 0:
        # same data, same plan, same positions: the output is bit-identical
        assert torch.equal(int_view(db.o), int_view(o0))
    assert_close(to_np(db.o), WO.run(wl, pools=(ko, vo)), wl.dtype, f"offload shift={shift}")


def test_round_trip_device_buffer_and_decode():
    wl = W.decode_64req(num_reqs=4, num_spans=3, span_len=64)
    db = gpu_run(wl)
    ko, vo = relocate(wl, db, 1234, pinned=False)
    db.attend()
    torch.cuda.synchronize()
    assert_close(to_np(db.o), WO.run(wl, pools=(ko, vo)), wl.dtype, "offload decode")


def test_round_trip_8b_rag_sampled_rows():
    # the 8B RAG batch: every cached block leaves and comes back under new ids
    wl = W.llama3_8b_rag()
    db = gpu_run(wl)
    o0 = db.o.clone()
    ko, vo = relocate(wl, db, 0)
    db.attend()
    torch.cuda.synchronize()
    assert torch.equal(int_view(db.o), int_view(o0))
    rows = np.random.default_rng(2).choice(wl.q.shape[0], 32, replace=False)
    assert_close(to_np(db.o)[rows], WO.run(wl, rows=rows, pools=(ko, vo)), wl.dtype, "offload 8B RAG")


def test_pageable_host_memory_is_rejected():
    from paper_2606_13126_amd import _binding as B
    wl = shared_span_case(torch.bfloat16)
    db = gpu_run(wl)
    ids = torch.zeros(2, dtype=torch.int32, device="cuda")
    pageable = torch.empty((2,) + tuple(db.k_pool.shape[1:]), dtype=db.k_pool.dtype)
    say("[gpu] offload: pageable destination (host-side rejection)")
    with pytest.raises(B.PicError) as e:
        B.pic_blocks_gather(db.cfg, db.k_pool, db.v_pool, ids, pageable, pageable)
    assert e.value.status == B.PIC_EINVAL and "pinned" in str(e.value)
    torch.cuda.synchronize()
    # the library still works afterwards
    db.attend()
    torch.cuda.synchronize()
    assert torch.isfinite(db.o.float()).all()


def test_misaligned_buffer_is_rejected():
    # the copies move 16-byte chunks: a buffer starting 2 bytes into an allocation is
    # refused on the host, before any launch
    from paper_2606_13126_amd import _binding as B
    wl = shared_span_case(torch.bfloat16)
    db = gpu_run(wl)
    ids = torch.zeros(1, dtype=torch.int32, device="cuda")
    flat = torch.empty(db.k_pool[0].numel() + 8, dtype=db.k_pool.dtype, device="cuda")
    dst = flat[1:1 + db.k_pool[0].numel()].view((1,) + tuple(db.k_pool.shape[1:]))
    say("[gpu] offload: misaligned destination (host-side rejection)")
    with pytest.raises(B.PicError) as e:
        B.pic_blocks_gather(db.cfg, db.k_pool, db.v_pool, ids, dst, dst)
    assert e.value.status == B.PIC_EINVAL and "aligned" in str(e.value)
    # the same buffer aligned works, and empty requests are no-ops
    B.pic_blocks_gather(db.cfg, db.k_pool, db.v_pool, ids[:0], dst, dst)
    ok = flat[8:8 + db.k_pool[0].numel()].view((1,) + tuple(db.k_pool.shape[1:]))
    B.pic_blocks_gather(db.cfg, db.k_pool, db.v_pool, ids, ok, ok)
    torch.cuda.synchronize()
    assert torch.equal(ok.cpu().view(torch.int16), db.v_pool[0:1].cpu().view(torch.int16))
