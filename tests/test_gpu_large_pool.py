"""GPU: K/V pools of more than 2^32 bytes each.  The batch's blocks are moved to ids
near the top of such a pool, so that every kernel that touches the pool (the
prefill and decode gathers, kv_write, the block copies) forms byte offsets past
4 GiB; the results must equal those of the same batch in its small pool bit for
bit (same data, same plan, same arithmetic)."""
import numpy as np
import pytest
import torch

import workloads as W
from tests.gpu_util import gpu_run, say

pytestmark = pytest.mark.gpu

# 140,000 blocks x 8 KV heads x 16 rows x 128 dims x 2 bytes = 4.59 GB per pool
BIG_BLOCKS = 140_000


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_13126_amd  # noqa: F401  (fails loudly if the library is missing)


def int_view(t):
    return t.view(torch.int32 if t.dtype == torch.float32 else torch.int16)


def move_to_big_pools(wl, db):
    """Copy the batch's blocks (fresh rows excluded) to high ids of two big pools;
    point the batch and its fresh-row slots there.  Returns those slots."""
    used = np.unique(wl.block_tables[wl.block_tables >= 0]).astype(np.int64)
    page = tuple(db.k_pool.shape[1:])
    big = BIG_BLOCKS * int(np.prod(page)) * db.k_pool.element_size()
    assert big > 2 ** 32, big
    new_ids = BIG_BLOCKS - 1 - 3 * np.arange(len(used), dtype=np.int64)
    assert new_ids.min() > 0
    say(f"[gpu] large pool {wl.name}: {len(used)} blocks to ids {new_ids.min()}..{new_ids.max()} "
        f"of {BIG_BLOCKS} ({big / 2 ** 30:.2f} GiB per pool)")
    kb = torch.empty((BIG_BLOCKS,) + page, dtype=db.k_pool.dtype, device="cuda")
    vb = torch.empty((BIG_BLOCKS,) + page, dtype=db.v_pool.dtype, device="cuda")
    src, dst = torch.from_numpy(used).cuda(), torch.from_numpy(new_ids).cuda()
    kb[dst] = db.k_pool[src]
    vb[dst] = db.v_pool[src]
    remap = np.full(db.k_pool.shape[0], -1, dtype=np.int64)
    remap[used] = new_ids
    # the fresh rows are written again, by kv_write, into garbage
    slots = wl.slot_mapping.astype(np.int64)
    ok = slots >= 0
    new_slots = np.where(ok, remap[np.maximum(slots, 0) // 16] * 16 + np.maximum(slots, 0) % 16, -1)
    fresh = torch.from_numpy(new_slots[ok]).cuda()
    db.k_pool, db.v_pool = kb, vb
    db.block_tables = torch.from_numpy(np.where(wl.block_tables >= 0, remap[np.maximum(wl.block_tables, 0)],
                                                -1).astype(np.int32)).cuda()
    db.slots = torch.from_numpy(new_slots.astype(np.int32)).cuda()
    return fresh


def scramble_fresh_rows(db, fresh):
    # overwrite the fresh rows' places in the big pools with garbage first
    page = tuple(db.k_pool.shape[1:])
    blk, off = fresh // 16, fresh % 16
    db.k_pool[blk, :, off, :] = (torch.randn((len(fresh), page[0], page[2]), device="cuda") * 100).to(db.k_pool.dtype)
    db.v_pool[blk, :, off, :] = (torch.randn((len(fresh), page[0], page[2]), device="cuda") * 100).to(db.v_pool.dtype)


def check_same_result(wl):
    db = gpu_run(wl)
    o0 = db.o.clone()
    fresh = move_to_big_pools(wl, db)
    scramble_fresh_rows(db, fresh)
    db.write()
    db.o.zero_()
    db.attend()
    torch.cuda.synchronize()
    assert torch.equal(int_view(db.o), int_view(o0))
    return db


def test_prefill_8b_rag_in_pools_past_4gib():
    check_same_result(W.llama3_8b_rag())


def test_decode_in_pools_past_4gib():
    check_same_result(W.decode_64req(num_reqs=4, num_spans=3, span_len=64))


def test_block_copies_past_4gib():
    from paper_2606_13126_amd import _binding as B
    db = check_same_result(W.decode_64req(num_reqs=2, num_spans=2, span_len=64))
    ids = torch.unique(db.block_tables[db.block_tables >= 0]).to(torch.int32)
    n = len(ids)
    page = tuple(db.k_pool.shape[1:])
    host_k = torch.empty((n,) + page, dtype=db.k_pool.dtype, pin_memory=True)
    host_v = torch.empty((n,) + page, dtype=db.v_pool.dtype, pin_memory=True)
    say(f"[gpu] large pool: gather {n} blocks from ids up to {int(ids.max())}")
    B.pic_blocks_gather(db.cfg, db.k_pool, db.v_pool, ids, host_k, host_v)
    torch.cuda.synchronize()
    idx = ids.to(torch.int64)
    assert torch.equal(int_view(host_k), int_view(db.k_pool[idx].cpu()))
    assert torch.equal(int_view(host_v), int_view(db.v_pool[idx].cpu()))
    # and back, under other high ids
    back = (BIG_BLOCKS - 2 - 3 * torch.arange(n, device="cuda")).to(torch.int32)
    B.pic_blocks_scatter(db.cfg, db.k_pool, db.v_pool, back, host_k, host_v)
    torch.cuda.synchronize()
    assert torch.equal(int_view(db.k_pool[back.to(torch.int64)].cpu()), int_view(host_k))
    assert torch.equal(int_view(db.v_pool[back.to(torch.int64)].cpu()), int_view(host_v))
