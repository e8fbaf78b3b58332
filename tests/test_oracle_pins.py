"""Pins for the fp64 oracle: what the paper and the mathematics fix, checked
without trusting the oracle itself (CPU only)."""
import math

import numpy as np
import pytest
import torch

import workloads as W
from oracle import pic_oracle as O
from oracle import workload_oracle as WO
from tests import brute

RNG = np.random.default_rng(7)


def oracle_of(wl, style="neox", rows=None):
    return WO.run(wl, rows=rows, style=style)


def brute_of(wl, style="neox"):
    k, v = WO.pools_after_write(wl)
    scale = wl.softmax_scale or 1.0 / math.sqrt(wl.head_dim)
    return brute.attention(wl.q.double().numpy(), k, v, wl.block_tables, wl.positions, wl.seq_lens,
                           wl.cu_spans, wl.span_start, wl.span_flags, wl.num_kv_heads, wl.rope_theta,
                           scale, style, decode=wl.is_decode)


S, P, Q = W.SSEP, W.PDEP, W.QUERY
Sp = W.Span

# A spread of tiny span structures: SSEP / PDEP / unflagged continuation, unaligned
# boundaries, cached and fresh spans, shared spans across requests, GQA.
TINY = {
    "ssep_pdep": [[Sp(16, S | Q, fresh=True), Sp(16, S | Q, fresh=True), Sp(8, P | Q, fresh=True)]],
    "unflagged_chain": [[Sp(10, S), Sp(7, Q), Sp(9, S | Q, fresh=True), Sp(5, Q, fresh=True)]],
    "first_unflagged": [[Sp(12, Q, fresh=True), Sp(9, S | Q, fresh=True), Sp(6, P | Q, fresh=True)]],
    "cached_then_tail": [[Sp(16, S, key="a"), Sp(32, S, key="b"), Sp(11, P | Q, fresh=True)]],
    "shared_two_reqs": [[Sp(16, S, key="a"), Sp(16, S, key="b"), Sp(5, P | Q, fresh=True)],
                        [Sp(16, S, key="b"), Sp(16, S, key="a"), Sp(3, P | Q, fresh=True)]],
}


@pytest.mark.parametrize("name", sorted(TINY))
@pytest.mark.parametrize("style", ["neox", "gptj"])
def test_oracle_equals_bruteforce(name, style):
    wl = W.small_case(name, TINY[name], Hq=4, Hkv=2, D=8, theta=10.0, seed=11)
    # arbitrary (non-monotone) positions: causality must not depend on them
    wl.positions = np.asarray(RNG.integers(-50, 50, size=wl.positions.shape), dtype=np.int32)
    o = oracle_of(wl, style)
    b = brute_of(wl, style)
    assert o.shape == b.shape
    assert np.max(np.abs(o - b)) <= 1e-12


def test_oracle_equals_bruteforce_decode():
    reqs = [[Sp(16, S, key="a"), Sp(16, S, key="b"), Sp(1, P, fresh=True)],
            [Sp(16, S, key="b"), Sp(7, S), Sp(1, 0, fresh=True)]]
    wl = W.small_case("dec", reqs, Hq=6, Hkv=3, D=8, theta=100.0, seed=5, decode=True)
    assert np.max(np.abs(oracle_of(wl) - brute_of(wl))) <= 1e-12


# ---- RoPE ---------------------------------------------------------------------------

def test_rope_identity_at_zero():
    x = RNG.standard_normal((5, 3, 16))
    for style in ("neox", "gptj"):
        assert np.array_equal(O.rope(x, np.zeros((5, 3), dtype=np.int64), 1e4, style), x)


def test_rope_preserves_pair_norms():
    x = RNG.standard_normal((7, 32))
    p = RNG.integers(-10**5, 10**5, size=7)
    y = O.rope(x, p, 5e5, "neox")
    n0 = x[:, :16] ** 2 + x[:, 16:] ** 2
    n1 = y[:, :16] ** 2 + y[:, 16:] ** 2
    assert np.max(np.abs(n0 - n1)) <= 1e-12


def test_rope_composes():
    x = RNG.standard_normal((4, 16))
    a = np.array([3, -8, 1000, 77])
    b = np.array([5, 2, -999, 123456])
    for style in ("neox", "gptj"):
        lhs = O.rope(O.rope(x, b, 1e4, style), a, 1e4, style)
        rhs = O.rope(x, a + b, 1e4, style)
        assert np.max(np.abs(lhs - rhs)) <= 1e-9


def test_rope_matches_complex_exponential():
    x = RNG.standard_normal((6, 64))
    p = RNG.integers(0, 40000, size=6)
    # the two routes to omega_i (power vs exp/log) may differ by an ulp, which turns
    # into an angle error of about p * 2^-52 rad
    bound = 4 * 2.0 ** -52 * p.max() * np.abs(x).max() + 1e-14
    for style in ("neox", "gptj"):
        assert np.max(np.abs(O.rope(x, p, 5e5, style) - brute.rotate_abs(x, p, 5e5, style))) <= bound


def test_rope_closed_form_first_pair():
    # omega_0 = theta^0 = 1 for every theta: e_0 at position p turns to (cos p, sin p)
    # in the slots (0, D/2) for NeoX and (0, 1) for GPT-J; the last pair turns by
    # p * theta^(-(D-2)/D).
    D, theta = 8, 1e4
    x = np.zeros(D); x[0] = 1.0
    y = O.rope(x, np.array(3), theta, "neox")
    assert y[0] == pytest.approx(math.cos(3.0), abs=1e-15)
    assert y[D // 2] == pytest.approx(math.sin(3.0), abs=1e-15)
    y = O.rope(x, np.array(3), theta, "gptj")
    assert (y[0], y[1]) == (pytest.approx(math.cos(3.0), abs=1e-15), pytest.approx(math.sin(3.0), abs=1e-15))
    x = np.zeros(D); x[D // 2 - 1] = 1.0
    y = O.rope(x, np.array(1000), theta, "neox")
    ang = 1000 * theta ** (-(D - 2) / D)
    assert y[D // 2 - 1] == pytest.approx(math.cos(ang), abs=1e-13)
    assert y[D - 1] == pytest.approx(math.sin(ang), abs=1e-13)


# ---- RoPE variants: explicit frequencies and partial rotary width ------------------

def test_rope_default_frequencies_through_override():
    x = RNG.standard_normal((5, 3, 64))
    pos = RNG.integers(-5000, 5000, size=(5, 3))
    assert np.array_equal(O.rope(x, pos, 5e5), O.rope(x, pos, 5e5, inv_freq=O.rope_inv_freq(64, 5e5)))


@pytest.mark.parametrize("style", ["neox", "gptj"])
def test_rope_scaled_frequencies_are_scaled_positions(style):
    # frequencies c * omega turn position p as far as the plain frequencies turn c * p
    # (position interpolation with c = 1/4 is the same statement read backwards)
    x = RNG.standard_normal((7, 128))
    pos = RNG.integers(0, 9000, size=7)
    om = O.rope_inv_freq(128, 1e4)
    assert np.allclose(O.rope(x, pos, 1e4, style, inv_freq=3.0 * om), O.rope(x, 3 * pos, 1e4, style), atol=1e-9)
    assert np.allclose(O.rope(x, 4 * pos, 1e4, style, inv_freq=om / 4.0), O.rope(x, pos, 1e4, style), atol=1e-9)


def test_rope_partial_gptj_closed_form():
    # R = 4 of D = 10: pairs (0,1) at omega_0 = 1 and (2,3) at theta^(-1/2); 4..9 pass
    x = RNG.standard_normal(10)
    p, theta = 7, 100.0
    y = O.rope(x, np.array(p), theta, "gptj", rotary_dim=4)
    for (a, b), om in (((0, 1), 1.0), ((2, 3), theta ** -0.5)):
        c, s = math.cos(p * om), math.sin(p * om)
        assert abs(y[a] - (x[a] * c - x[b] * s)) < 1e-13 and abs(y[b] - (x[b] * c + x[a] * s)) < 1e-13
    assert np.array_equal(y[4:], x[4:])


def test_rope_partial_neox_closed_form():
    # R = 4 of D = 10, NeoX: element i pairs with i + R/2, so (0,2) and (1,3)
    x = RNG.standard_normal(10)
    p, theta = 5, 100.0
    y = O.rope(x, np.array(p), theta, "neox", rotary_dim=4)
    for (a, b), om in (((0, 2), 1.0), ((1, 3), theta ** -0.5)):
        c, s = math.cos(p * om), math.sin(p * om)
        assert abs(y[a] - (x[a] * c - x[b] * s)) < 1e-13 and abs(y[b] - (x[b] * c + x[a] * s)) < 1e-13
    assert np.array_equal(y[4:], x[4:])


@pytest.mark.parametrize("style", ["neox", "gptj"])
def test_rope_partial_is_full_rope_of_the_prefix(style):
    x = RNG.standard_normal((6, 64))
    pos = RNG.integers(0, 4000, size=6)
    y = O.rope(x, pos, 1e4, style, rotary_dim=32)
    assert np.allclose(y[:, :32], O.rope(x[:, :32], pos, 1e4, style), atol=1e-12)
    assert np.array_equal(y[:, 32:], x[:, 32:])


def test_variant_attention_is_shift_invariant():
    # any frequencies and a partial width keep scores relative: a shifted request
    # attends the same way
    wl = W.tiny_fp32()
    wl.rotary_dim = 48
    wl.rope_inv_freq = np.linspace(1.0, 1e-3, 24) * 0.9
    o0 = WO.run(wl, style="gptj")
    wl.positions = wl.positions + np.int32(4321)
    assert np.max(np.abs(o0 - WO.run(wl, style="gptj"))) <= 1e-9
    # and it is not the plain rotation
    wl.rotary_dim, wl.rope_inv_freq = None, None
    assert np.max(np.abs(o0 - WO.run(wl, style="gptj"))) > 1e-3


def test_rope_relative():
    # (R_a q)^T (R_b k) depends on a - b only
    q, k = RNG.standard_normal(32), RNG.standard_normal(32)
    d0 = O.rope(q, np.array(10), 5e5) @ O.rope(k, np.array(3), 5e5)
    d1 = O.rope(q, np.array(100010), 5e5) @ O.rope(k, np.array(100003), 5e5)
    assert abs(d0 - d1) <= 1e-9


# ---- closed-form attention ----------------------------------------------------------

def test_closed_form_two_dims():
    # D = 2, one pair, omega_0 = 1, q = k = e_0 at positions = sequence index, scale 1:
    # score(t, j) = cos(t - j), so O_t = sum_j e^{cos(t-j)} v_j / sum_j e^{cos(t-j)}.
    reqs = [[Sp(3, S | Q, fresh=True), Sp(3, P | Q, fresh=True)]]
    wl = W.small_case("cf", reqs, Hq=1, Hkv=1, D=2, theta=7.0, seed=1, poison=False)
    wl.softmax_scale = 1.0
    wl.q[:] = torch.tensor([1.0, 0.0])
    wl.k_new[:] = torch.tensor([1.0, 0.0])
    vals = torch.tensor([[float(j), 1.0 - j] for j in range(6)])
    wl.v_new[:] = vals[:, None, :]
    o = oracle_of(wl)[:, 0, :]
    for t in range(6):
        js = range(0, t + 1)  # the SSEP span [0,3) starts at 0 and the PDEP tail sees all
        wts = [math.exp(math.cos(t - j)) for j in js]
        exp = sum(wv * vals[j].double().numpy() for wv, j in zip(wts, js)) / sum(wts)
        assert np.max(np.abs(o[t] - exp)) <= 1e-14


def test_first_token_of_ssep_span_returns_its_value():
    wl = W.tiny_fp32()
    o = oracle_of(wl)
    k, v = WO.pools_after_write(wl)
    # q rows are the 160 tokens in order; tokens 0 and 64 each see only themselves
    for t in (0, 64):
        blk = wl.block_tables[0][t // 16]
        assert np.array_equal(o[t, :, :], np.broadcast_to(v[blk, 0, t % 16, :], o[t].shape))


def test_identical_keys_give_mean_of_visible_values():
    reqs = [[Sp(20, S | Q, fresh=True), Sp(13, S | Q, fresh=True), Sp(9, P | Q, fresh=True)]]
    wl = W.small_case("ik", reqs, Hq=2, Hkv=1, D=8, seed=3)
    # identical unrotated keys at one shared logical position rotate identically, so
    # every visible key scores the same; the window still follows sequence indices
    wl.k_new[:] = wl.k_new[0:1]
    wl.positions[:] = 5
    o = oracle_of(wl)
    vv = wl.v_new.double().numpy()[:, 0, :]
    for t in range(42):
        lo = 0 if t >= 33 else (20 if t >= 20 else 0)
        assert np.max(np.abs(o[t, 0] - vv[lo:t + 1].mean(axis=0))) <= 1e-12


# ---- causal special case (torch SDPA in fp64 as an outside reference) ----------------

@pytest.mark.parametrize("flag", [0, P])
def test_contiguous_single_span_is_causal_attention(flag):
    L, H, D = 37, 2, 16
    wl = W.small_case("causal", [[Sp(L, flag | Q, fresh=True)]], Hq=H, Hkv=H, D=D, theta=1e4, seed=9)
    o = oracle_of(wl)
    q = brute.rotate_abs(wl.q.double().numpy(), np.arange(L)[:, None], 1e4, "neox")
    k = brute.rotate_abs(wl.k_new.double().numpy(), np.arange(L)[:, None], 1e4, "neox")
    v = wl.v_new.double().numpy()
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).transpose(0, 1), torch.from_numpy(k).transpose(0, 1),
        torch.from_numpy(v).transpose(0, 1), is_causal=True).transpose(0, 1).numpy()
    assert np.max(np.abs(o - ref)) <= 1e-12


def test_cached_prefix_then_tail_is_bottom_right_causal():
    # unflagged continuation of a cached prefix: the tail sees every earlier token;
    # torch's is_causal is top-left aligned for Lq != Lk, so pass the mask explicitly
    Lc, Lt, H, D = 32, 9, 2, 8
    wl = W.small_case("tail", [[Sp(Lc, 0, key="c"), Sp(Lt, Q, fresh=True)]], Hq=H, Hkv=H, D=D, seed=4)
    o = oracle_of(wl)
    k_pool, v_pool = WO.pools_after_write(wl)
    L = Lc + Lt
    kk = np.array([[brute.page_row(k_pool, wl.block_tables[0], n, g) for g in range(H)] for n in range(L)])
    vv = np.array([[brute.page_row(v_pool, wl.block_tables[0], n, g) for g in range(H)] for n in range(L)])
    q = brute.rotate_abs(wl.q.double().numpy(), np.arange(Lc, L)[:, None], 1e4, "neox")
    k = brute.rotate_abs(kk, np.arange(L)[:, None], 1e4, "neox")
    mask = torch.from_numpy(np.arange(L)[None, :] <= np.arange(Lc, L)[:, None])
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).transpose(0, 1), torch.from_numpy(k).transpose(0, 1),
        torch.from_numpy(vv).transpose(0, 1), attn_mask=mask).transpose(0, 1).numpy()
    assert np.max(np.abs(o - ref)) <= 1e-12


# ---- invariances --------------------------------------------------------------------

@pytest.mark.parametrize("shift", [1, -37, 1000, 65536, 100003])
def test_shift_invariance(shift):
    wl = W.tiny_fp32()
    o0 = oracle_of(wl)
    wl.positions = wl.positions + np.int32(shift)
    o1 = oracle_of(wl)
    assert np.max(np.abs(o0 - o1)) <= 1e-9


def test_block_permutation_invariance():
    wl = W.tiny_fp32()
    o0 = oracle_of(wl)
    perm = RNG.permutation(wl.num_blocks)           # new id of old block b is perm[b]
    inv = np.argsort(perm)
    wl.k_pool = wl.k_pool[torch.from_numpy(inv)]
    wl.v_pool = wl.v_pool[torch.from_numpy(inv)]
    wl.block_tables = np.where(wl.block_tables >= 0, perm[wl.block_tables], -1).astype(np.int32)
    wl.slot_mapping = (perm[wl.slot_mapping // 16] * 16 + wl.slot_mapping % 16).astype(np.int32)
    assert np.array_equal(o0, oracle_of(wl))


def test_fresh_ssep_span_equals_its_own_request():
    # Sec. 3.3.1: a detached span computed inside a combined request equals the span
    # prefilled as a request of its own
    full = W.small_case("comb", [[Sp(24, S | Q, fresh=True), Sp(21, S | Q, fresh=True)]],
                        Hq=2, Hkv=1, D=8, seed=8)
    alone = W.small_case("alone", [[Sp(21, S | Q, fresh=True)]], Hq=2, Hkv=1, D=8, seed=8)
    alone.q = full.q[24:].clone()
    alone.k_new = full.k_new[24:].clone()
    alone.v_new = full.v_new[24:].clone()
    alone.positions = full.positions[24:].copy()
    assert np.max(np.abs(oracle_of(full)[24:] - oracle_of(alone))) <= 1e-13


def test_concurrent_reuse_equals_requests_alone():
    # the same physical blocks at different offsets in two requests (Sec. 3.2.1)
    reqs = [[Sp(16, S, key="a"), Sp(32, S, key="b"), Sp(6, P | Q, fresh=True)],
            [Sp(32, S, key="b"), Sp(16, S, key="a"), Sp(4, P | Q, fresh=True)]]
    both = W.small_case("both", reqs, Hq=4, Hkv=2, D=8, seed=12)
    ob = oracle_of(both)
    k, v = WO.pools_after_write(both)
    off = both.seq_offsets
    row = 0
    for r in range(2):
        sl = slice(both.cu_spans[r], both.cu_spans[r + 1])
        nq = int(np.sum([s.length for s in reqs[r] if s.flags & Q]))
        o = O.prefill(both.q[row:row + nq].double().numpy(), k, v, both.block_tables[r:r + 1],
                      both.positions[off[r]:off[r + 1]], both.seq_lens[r:r + 1],
                      np.array([0, sl.stop - sl.start]), both.span_start[sl], both.span_flags[sl],
                      both.num_kv_heads, both.rope_theta)
        assert np.array_equal(o, ob[row:row + nq])
        row += nq


def test_duplicate_block_in_one_request():
    # the same cached span twice in one prompt (Sec. 4.3 double-free case): block ids
    # repeat in the table, and the result equals a layout with two separate copies
    dup = W.small_case("dup", [[Sp(16, S, key="a"), Sp(16, S, key="a"), Sp(5, P | Q, fresh=True)]],
                       Hq=2, Hkv=1, D=8, seed=21)
    assert dup.block_tables[0][0] == dup.block_tables[0][1]
    sep = W.small_case("sep", [[Sp(16, S, key="a"), Sp(16, S, key="b"), Sp(5, P | Q, fresh=True)]],
                       Hq=2, Hkv=1, D=8, seed=21)
    sep.q, sep.k_new, sep.v_new = dup.q, dup.k_new, dup.v_new
    a = dup.block_tables[0][0]
    b = sep.block_tables[0][1]
    sep.k_pool[b] = dup.k_pool[a]
    sep.v_pool[b] = dup.v_pool[a]
    sa = sep.block_tables[0][0]
    sep.k_pool[sa] = dup.k_pool[a]
    sep.v_pool[sa] = dup.v_pool[a]
    assert np.max(np.abs(oracle_of(dup) - oracle_of(sep))) <= 1e-15


def test_decode_equals_prefill_of_last_token():
    dec = W.small_case("d", [[Sp(16, S, key="a"), Sp(23, S), Sp(1, P, fresh=True)]], Hq=4, Hkv=2, D=8,
                       seed=30, decode=True)
    od = oracle_of(dec)
    pre = W.small_case("p", [[Sp(16, S, key="a"), Sp(23, S), Sp(1, P | Q, fresh=True)]], Hq=4, Hkv=2,
                       D=8, seed=30)
    assert np.array_equal(pre.block_tables, dec.block_tables)
    pre.q, pre.k_new, pre.v_new = dec.q, dec.k_new, dec.v_new
    pre.k_pool, pre.v_pool = dec.k_pool, dec.v_pool
    assert np.max(np.abs(od - oracle_of(pre))) <= 1e-15


def test_kv_write_scatter():
    kp = np.full((4, 2, 16, 3), -1, dtype=np.int16)
    vp = kp.copy()
    kn = np.arange(3 * 2 * 3, dtype=np.int16).reshape(3, 2, 3)
    O.kv_write(kp, vp, kn, kn + 100, [17, -5, 63])
    assert np.array_equal(kp[1, :, 1, :], kn[0]) and np.array_equal(vp[3, :, 15, :], kn[2] + 100)
    assert (kp == -1).sum() == kp.size - 2 * 2 * 3


# ---- block offload (Sec. 3.2.3) -------------------------------------------------------

def test_blocks_gather_scatter_index_order():
    # every element of a tiny pool encodes its own (block, head, offset, dim): a swapped
    # or transposed index in the copies shows up as a wrong code
    nb, hkv, d = 6, 3, 5
    b, h, o, e = np.meshgrid(np.arange(nb), np.arange(hkv), np.arange(16), np.arange(d), indexing="ij")
    pool = (b * 10000 + h * 1000 + o * 10 + e).astype(np.int32)
    ids = [4, 0, 4, 2]
    out = O.blocks_gather(pool, ids)
    assert out.shape == (4, hkv, 16, d)
    for i, bi in enumerate(ids):
        for hh in range(hkv):
            for oo in range(16):
                for ee in range(d):
                    assert out[i, hh, oo, ee] == bi * 10000 + hh * 1000 + oo * 10 + ee
    dst = np.full_like(pool, -1)
    O.blocks_scatter(dst, [5, 1, 3], out[[0, 1, 3]])
    assert np.array_equal(dst[5], pool[4]) and np.array_equal(dst[1], pool[0]) and np.array_equal(dst[3], pool[2])
    assert (dst[[0, 2, 4]] == -1).all()


def test_offload_and_reload_under_new_ids_keeps_outputs():
    # Sec. 3.2.3: blocks leave the pool (here to a bf16-width byte buffer standing in for
    # host memory), come back under different ids into a pool whose other blocks hold
    # garbage, and the block table is the only thing updated: outputs are unchanged
    wl = W.tiny_fp32()
    k, v = WO.pools_after_write(wl)
    o0 = oracle_of(wl)
    used = np.unique(wl.block_tables[wl.block_tables >= 0])
    host_k = O.blocks_gather(k, used).tobytes()
    host_v = O.blocks_gather(v, used).tobytes()
    nb = k.shape[0] + 7
    new_ids = RNG.permutation(nb)[:len(used)]
    k2 = RNG.standard_normal((nb,) + k.shape[1:])
    v2 = RNG.standard_normal((nb,) + v.shape[1:])
    shape = (len(used),) + k.shape[1:]
    O.blocks_scatter(k2, new_ids, np.frombuffer(host_k, dtype=k.dtype).reshape(shape))
    O.blocks_scatter(v2, new_ids, np.frombuffer(host_v, dtype=v.dtype).reshape(shape))
    remap = np.full(k.shape[0], -1, dtype=np.int64)
    remap[used] = new_ids
    wl.block_tables = np.where(wl.block_tables >= 0, remap[np.maximum(wl.block_tables, 0)], -1).astype(np.int32)
    assert np.array_equal(o0, WO.run(wl, pools=(k2, v2)))


def test_span_windows_rule():
    w = O.span_windows([0, 5, 9, 14, 20], [S, 0, P, 0, S], 25)
    assert list(w) == [0] * 5 + [0] * 4 + [0] * 5 + [0] * 6 + [20] * 5
    w = O.span_windows([0, 4, 9, 12], [0, S, 0, S], 15)
    assert list(w) == [0] * 4 + [4] * 5 + [4] * 3 + [12] * 3
    w = O.span_windows([0, 4], [S, 0], 8, span_window=[-1, 2])
    assert list(w) == [0] * 4 + [2] * 4


# ---- planted mistakes: the pins above must catch each of them ------------------------

def _mut_sign(orig):
    def f(x, pos, theta, style="neox", **kw):
        return orig(x, -np.asarray(pos), theta, style, **kw)
    return f


def _mut_pairing(orig):
    def f(x, pos, theta, style="neox", **kw):
        return orig(x, pos, theta, "gptj" if style == "neox" else "neox", **kw)
    return f


def _mut_freq(orig):
    def f(head_dim, theta):
        i = np.arange(head_dim // 2, dtype=np.float64)
        return np.power(float(theta), -i / head_dim)      # dropped factor 2
    return f


def _mut_window(orig):
    def f(*a, **k):
        w = orig(*a, **k)
        return np.where(w > 0, w + 1, w)                   # SSEP start off by one
    return f


def _mut_scale(orig):
    return lambda head_dim, s: 1.0


def _mut_gather(orig):
    def f(pool, block_row, n_tokens, kv_head):
        return orig(pool, block_row[::-1] if block_row.shape[0] > 1 else block_row, n_tokens, kv_head)
    return f


@pytest.mark.parametrize("target,mut", [("rope", _mut_sign), ("rope", _mut_pairing),
                                        ("rope_inv_freq", _mut_freq), ("span_windows", _mut_window),
                                        ("_scale", _mut_scale), ("gather", _mut_gather)])
def test_planted_mistake_is_caught(monkeypatch, target, mut):
    wl = W.small_case("m", TINY["unflagged_chain"], Hq=4, Hkv=2, D=8, theta=10.0, seed=11)
    wl.positions = np.asarray(RNG.integers(-50, 50, size=wl.positions.shape), dtype=np.int32)
    b = brute_of(wl)
    monkeypatch.setattr(O, target, mut(getattr(O, target)))
    with np.errstate(all="ignore"):
        o = oracle_of(wl)
    assert not np.max(np.abs(o - b)) <= 1e-6   # NaN (an emptied window) counts as caught


def test_planted_gqa_map_is_caught(monkeypatch):
    wl = W.small_case("g", TINY["ssep_pdep"], Hq=4, Hkv=2, D=8, seed=2)
    b = brute_of(wl)
    orig = O._attend_request

    def swapped(q_rows, *a, **k):
        T, Hq, D = q_rows.shape
        perm = np.arange(Hq).reshape(2, -1).T.reshape(-1)  # h -> head-interleaved map
        return orig(q_rows[:, perm], *a, **k)[:, np.argsort(perm)]
    monkeypatch.setattr(O, "_attend_request", swapped)
    assert not np.max(np.abs(oracle_of(wl) - b)) <= 1e-6


def test_config_work_counts():
    # visible-pair counts of the five workloads (4*D*Hq*P flops for prefill)
    assert O.visible_pairs(*[getattr(W.tiny_fp32(), a) for a in ("seq_lens", "cu_spans", "span_start",
                                                                 "span_flags")]) == 8784
    wl = W.tiny_fp32(tail_only=True)
    assert O.visible_pairs(wl.seq_lens, wl.cu_spans, wl.span_start, wl.span_flags) == 4624
    wl = W.llama3_8b_rag()
    assert O.visible_pairs(wl.seq_lens, wl.cu_spans, wl.span_start, wl.span_flags) == 1343616


def test_stored_oracle_fixture():
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "oracle_tiny_fp32.json")
    with open(path) as f:
        fx = json.load(f)
    for name, wl in (("tiny_fp32_prefill", W.tiny_fp32()), ("tiny_fp32_prefill_tail", W.tiny_fp32(tail_only=True))):
        o = oracle_of(wl)
        ref = fx[name]
        assert list(o.shape) == ref["shape"]
        got = np.array([o[tuple(i)] for i in ref["index"]])
        assert np.max(np.abs(got - np.array(ref["value"]))) <= 1e-12
        assert abs(o.sum() - ref["sum"]) <= 1e-9


# ---- generalised windows (explicit per-span window starts) --------------------------

def test_explicit_windows_equal_flag_windows():
    # windows given explicitly reproduce the flag-derived ones exactly
    reqs = [[Sp(10, S), Sp(7, Q, fresh=True), Sp(12, S | Q, fresh=True), Sp(5, P | Q, fresh=True)],
            [Sp(16, S, key="a"), Sp(9, Q, fresh=True)]]
    wl = W.small_case("flags", reqs, Hq=4, Hkv=2, D=8, theta=50.0, seed=21)
    ref = oracle_of(wl)
    win = []
    for r in range(wl.num_reqs):
        sl = slice(wl.cu_spans[r], wl.cu_spans[r + 1])
        w_tok = O.span_windows(wl.span_start[sl], wl.span_flags[sl], int(wl.seq_lens[r]))
        win += [int(w_tok[b]) for b in wl.span_start[sl]]
    wl.span_window = np.array(win, dtype=np.int32)
    wl.span_flags = wl.span_flags & Q          # flags no longer carry the windows
    assert np.array_equal(oracle_of(wl), ref)


def test_nback_window_equals_subrequest():
    # a query span whose window starts at the previous document (one-back) sees
    # exactly what the same tokens see as a request made of those two documents
    # (without the explicit window the unflagged middle document would keep the first
    # document's window and the query span would see all 32 tokens)
    full = W.small_case("nb", [[Sp(12, S), Sp(11, 0), Sp(9, Q, fresh=True)]], Hq=4, Hkv=2, D=8, seed=22)
    full.span_window = np.array([-1, -1, 12], dtype=np.int32)
    sub = W.small_case("sub", [[Sp(11, S), Sp(9, Q, fresh=True)]], Hq=4, Hkv=2, D=8, seed=22)
    k, v = WO.pools_after_write(full)
    blk = full.block_tables[0]
    # copy tokens 12..31 of the full request into the sub-request's pool slots
    ks, vs = WO.pools_after_write(sub)
    for n in range(20):
        src = 12 + n
        ks[sub.block_tables[0][n // 16], :, n % 16] = k[blk[src // 16], :, src % 16]
        vs[sub.block_tables[0][n // 16], :, n % 16] = v[blk[src // 16], :, src % 16]
    sub.positions = full.positions[12:32].copy()
    sub.q = full.q.clone()
    o_sub = WO.run(sub, pools=(ks, vs))
    assert np.max(np.abs(oracle_of(full) - o_sub)) <= 1e-13


def test_planted_ignored_window_override_is_caught(monkeypatch):
    orig = O.span_windows
    monkeypatch.setattr(O, "span_windows", lambda a, b, c, span_window=None: orig(a, b, c, None))
    with pytest.raises(AssertionError):
        test_nback_window_equals_subrequest()


# ---- row / request subsets ------------------------------------------------------------
# The GPU parity tests of the largest workloads ask the oracle for a subset of the query
# rows (prefill) or requests (decode).  The subset branch selects, reorders and scatters
# rows, so it is pinned directly against the brute force, in the order asked for.

def test_prefill_row_subset_equals_bruteforce_rows():
    reqs = TINY["shared_two_reqs"] + [[Sp(9, S | Q, fresh=True), Sp(7, Q, fresh=True), Sp(4, P | Q, fresh=True)]]
    wl = W.small_case("subset", reqs, Hq=4, Hkv=2, D=8, theta=10.0, seed=21)
    b = brute_of(wl)
    n = b.shape[0]
    for rows in (np.array([n - 1, 0, 5, 3]),                      # unsorted, both ends
                 np.array([7, 6, 5, 4]),                           # descending inside request 1
                 RNG.permutation(n)[: n // 2],                     # random half, any order
                 np.arange(n)[::-1]):                              # every row, reversed
        got = oracle_of(wl, rows=rows)
        assert got.shape == (len(rows),) + b.shape[1:]
        assert np.max(np.abs(got - b[rows])) <= 1e-12, rows


def test_decode_request_subset_equals_bruteforce_requests():
    reqs = [[Sp(16, S, key="a"), Sp(16, S, key="b"), Sp(1, P, fresh=True)],
            [Sp(16, S, key="b"), Sp(7, S), Sp(1, 0, fresh=True)],
            [Sp(5, P), Sp(1, S, fresh=True)],
            [Sp(16, S, key="a"), Sp(3, 0, fresh=True)]]
    wl = W.small_case("dec_subset", reqs, Hq=6, Hkv=3, D=8, theta=100.0, seed=6, decode=True)
    b = brute_of(wl)
    for sel in ([3, 0], [2], [1, 3, 0, 2], [0, 1, 2, 3]):
        got = oracle_of(wl, rows=sel)
        assert got.shape == (len(sel),) + b.shape[1:]
        assert np.max(np.abs(got - b[sel])) <= 1e-12, sel


def test_planted_subset_misorder_is_caught():
    # a subset branch that returned rows in sorted order instead of the order asked
    # for would fail the pins above: check that such a mistake is visible
    wl = W.small_case("subset_mut", TINY["ssep_pdep"], Hq=4, Hkv=2, D=8, theta=10.0, seed=22)
    b = brute_of(wl)
    rows = np.array([30, 2, 17])
    wrong = oracle_of(wl, rows=np.sort(rows))
    assert np.max(np.abs(wrong - b[rows])) > 1e-3
