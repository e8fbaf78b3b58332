"""Prefill spans once, reuse them at any offset (Sec. 3.1.1 eq. (1), Sec. 3.2,
Sec. 3.3.1): a RAG session in which a first prompt prefills three documents and
a second prompt places two of them at new offsets behind a longer system prompt.

CPU: with the hash rule and span builder of the oracle, the second prompt's
computed rows equal those of recomputing the whole prompt from scratch (the
position-free pool makes a cached SSEP span valid at any offset).
GPU: the same session through the native span cache and the kernels matches the
oracle on every computed row, and reads the documents from the cache.
"""
import numpy as np
import pytest
import torch

from oracle import block_hash as BH
from oracle import pic_oracle as O
from tests.span_reuse import PDEP_TOK, SEED, SSEP_TOK, plan_prompt, rag_prompt, rand_tokens

Hq, Hkv, D, THETA = 8, 2, 128, 5e5


def prompts():
    rng = np.random.default_rng(11)
    docs = [rand_tokens(rng, n) for n in (100, 75, 130)]
    p1 = rag_prompt(rng, docs, system_len=32, task_len=40)
    p2 = rag_prompt(rng, [docs[2], docs[0], rand_tokens(rng, 50)], system_len=56, task_len=33)
    return p1, p2


class OracleSession:
    """The session with the oracle's hash rule, a dict as the cache and a numpy pool."""

    def __init__(self, num_blocks, dtype):
        self.cache = {}
        self.next = 0
        self.dtype = dtype
        self.k = np.zeros((num_blocks, Hkv, 16, D))
        self.v = np.zeros((num_blocks, Hkv, 16, D))

    def alloc(self):
        self.next += 1
        return self.next - 1

    def run(self, tokens, use_cache=True):
        hashes = BH.block_hashes(tokens, SSEP_TOK, PDEP_TOK, SEED)
        ids = [self.cache.get(h, -1) if use_cache else -1 for h in hashes]
        step = plan_prompt(tokens, [np.frombuffer(h, np.uint8) for h in hashes], ids,
                           lambda t, hit: BH.spans_from_blocks(t, SSEP_TOK, PDEP_TOK, hit), self.alloc,
                           Hq, Hkv, D, self.dtype)
        O.kv_write(self.k, self.v, step.k_new.double().numpy(), step.v_new.double().numpy(), step.slots)
        L = len(tokens)
        out = O.prefill(step.q.double().numpy(), self.k, self.v, step.table[None, :], np.arange(L), [L], [0, len(step.span_start)],
                        step.span_start, step.span_flags, Hkv, THETA)
        for b, h in enumerate(hashes):
            self.cache.setdefault(h, int(step.table[b]))
        return step, out


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_oracle_reuse_equals_recompute(dtype):
    p1, p2 = prompts()
    s = OracleSession(200, dtype)
    first, _ = s.run(p1)
    assert first.n_hits == 0
    step, out = s.run(p2)
    scratch, out_scratch = s.run(p2, use_cache=False)
    # the documents hit: only the system prompt, the new document and the task are computed
    assert step.n_hits == (131 + 15) // 16 + (101 + 15) // 16
    assert len(step.fresh) < len(scratch.fresh)
    rows = np.searchsorted(scratch.fresh, step.fresh)
    assert np.array_equal(scratch.fresh[rows], step.fresh)
    np.testing.assert_allclose(out, out_scratch[rows], rtol=0, atol=1e-12)


@pytest.mark.gpu
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_gpu_rag_session_reuses_spans_at_new_offsets(dtype):
    from paper_2606_13126_amd import _binding as B
    from tests.gpu_util import assert_close, say

    say(f"span reuse session dtype={dtype}")
    p1, p2 = prompts()
    nblocks = 200
    dev = "cuda"
    k_pool = torch.zeros((nblocks, Hkv, 16, D), dtype=dtype, device=dev)
    v_pool = torch.zeros_like(k_pool)
    cfg = B.make_config(Hq, Hkv, D, dtype=B.PIC_F32 if dtype == torch.float32 else B.PIC_BF16, rope_theta=THETA)
    cache = B.pic_block_cache_create()
    oracle = OracleSession(nblocks, dtype)
    nxt = [0]

    def alloc():
        nxt[0] += 1
        return nxt[0] - 1

    try:
        for i, tokens in enumerate((p1, p2)):
            hashes = B.pic_block_hashes(tokens, SSEP_TOK, PDEP_TOK, SEED)
            ids, n_hits = B.pic_block_cache_lookup(cache, hashes)
            step = plan_prompt(tokens, hashes, ids,
                               lambda t, hit: B.pic_spans_from_blocks(t, SSEP_TOK, PDEP_TOK, hit), alloc,
                               Hq, Hkv, D, dtype)
            # the oracle session takes the same decisions from its own hash rule
            o_step, ref = oracle.run(tokens)
            assert np.array_equal(o_step.span_start, step.span_start)
            assert np.array_equal(o_step.span_flags, step.span_flags)
            assert np.array_equal(o_step.table, step.table)
            L = len(tokens)
            host = B.HostBatch([L], [0, len(step.span_start)], step.span_start, step.span_flags)
            bt = torch.from_numpy(step.table[None, :].copy()).to(dev)
            pos = torch.arange(L, dtype=torch.int32, device=dev)
            B.pic_kv_write(cfg, k_pool, v_pool, step.k_new.to(dev), step.v_new.to(dev),
                           torch.from_numpy(step.slots).to(dev))
            q = step.q.to(dev)
            o = torch.empty_like(q)
            ws = B.pic_workspace_size(cfg, host, False)
            work = torch.empty(max(ws, 1), dtype=torch.uint8, device=dev)
            B.pic_attn_prefill(cfg, host, bt, pos, q, o, k_pool, v_pool, workspace=work)
            torch.cuda.synchronize()
            assert_close(o.double().cpu().numpy(), ref, dtype, f"prompt {i}")
            B.pic_block_cache_insert(cache, hashes, step.table[: len(hashes)])
            if i == 1:
                assert n_hits == step.n_hits > 0
    finally:
        B.pic_block_cache_destroy(cache)
