"""The entry point that allocates nothing (pic_attn_decode_noalloc) against
pic_attn_decode with a caller workspace: same kernels, so the outputs must agree
bit for bit, on two calls in a row (the second with a smaller batch that reuses the
library's scratch), and both within the oracle tolerance."""
import ctypes

import numpy as np
import pytest
import torch

import workloads as W
from oracle import workload_oracle as WO
from tests.cases import many_requests_decode
from tests.gpu_util import assert_close, say, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_13126_amd  # noqa: F401  (fails loudly if the library is missing)


def _noalloc(db):
    """Call the C entry point through ctypes with the batch of a DeviceBatch."""
    from paper_2606_13126_amd import _binding as B
    lib = B.lib()
    dev = B._dev(db.block_tables, db.positions)
    rope = B._rope(db.table)
    rc = lib.pic_attn_decode_noalloc(ctypes.byref(db.cfg), ctypes.byref(db.host.c), ctypes.byref(dev),
                                     ctypes.byref(rope), db.q.data_ptr(), db.o.data_ptr(), db.k_pool.data_ptr(),
                                     db.v_pool.data_ptr(), int(db.k_pool.shape[0]),
                                     torch.cuda.current_stream().cuda_stream)
    assert rc == B.PIC_OK, lib.pic_last_error().decode()


def _case(wl):
    from paper_2606_13126_amd.runner import DeviceBatch
    db = DeviceBatch(wl, table_positions=int(wl.positions.max()) + 1)
    db.write()
    db.attend()                     # pic_attn_decode with its own workspace
    torch.cuda.synchronize()
    ref = db.o.clone()
    db.o.fill_(float("nan"))
    _noalloc(db)
    torch.cuda.synchronize()
    return db, ref


def test_noalloc_decode_matches_workspace_decode_two_calls():
    # first call: 64 requests of 8193 keys (4 key splits each: the scratch holds the
    # split partials); second call: a smaller batch of 256 short requests, whose group
    # table also goes through the scratch, reading what the first call left there
    first = W.decode_64req()
    second = many_requests_decode(num_reqs=96)
    for wl in (first, second):
        say(f"[gpu] noalloc decode {wl.name}: {wl.num_reqs} requests, {int(wl.seq_lens.sum())} keys")
        db, ref = _case(wl)
        assert torch.equal(db.o.view(torch.int16), ref.view(torch.int16)), wl.name
        assert_close(to_np(db.o), WO.run(wl), wl.dtype, f"noalloc {wl.name} vs oracle")
        del db
        torch.cuda.empty_cache()


def test_noalloc_decode_narrow_workgroups():
    # models with one or two KV heads decode with 2- and 4-wave workgroups (three or
    # two per CU, more key splits): the scratch holds their partials too
    for hq, hkv in ((32, 1), (64, 2)):
        wl = many_requests_decode(num_reqs=64, Hq=hq, Hkv=hkv, D=128)
        say(f"[gpu] noalloc decode Hq={hq} Hkv={hkv}: {wl.num_reqs} requests, {int(wl.seq_lens.sum())} keys")
        db, ref = _case(wl)
        assert torch.equal(db.o.view(torch.int16), ref.view(torch.int16)), (hq, hkv)
        assert_close(to_np(db.o), WO.run(wl), wl.dtype, f"noalloc Hq={hq} Hkv={hkv} vs oracle")
        del db
        torch.cuda.empty_cache()
