"""The block-hash rule (Sec. 3.1.1, eq. (1)) and the span reuse decision.

Oracle pins: published SHA-256 test vectors for H, and properties the rule fixes
whatever its encoding (SSEP blocks hash the same at any offset, chaining
propagates a change until the next SSEP block, PDEP blocks see the whole prefix,
markers act only as a block's first token, the seed enters every hash); for the
reuse decision, the attention windows that the resulting spans give equal the
windows of the markers alone, for every pattern of hits.  Then the native span
cache matches the oracle bit for bit.
"""
import hashlib

import numpy as np
import pytest

from oracle import block_hash as BH
from oracle import pic_oracle as O
from workloads import PDEP, QUERY, SSEP

from tests.span_reuse import PDEP_TOK, SEED, SSEP_TOK, rag_prompt, rand_tokens


# ------------------------------------------------------------------------------------
# H: SHA-256 (FIPS 180-2 appendix B examples)
# ------------------------------------------------------------------------------------

FIPS_VECTORS = [
    (b"abc", "ba7816bf8f01cfea414140de5dae2223b00361a396177a9cb410ff61f20015ad"),
    (b"abcdbcdecdefdefgefghfghighijhijkijkljklmklmnlmnomnopnopq",
     "248d6a61d20638b8e5c026930c3e6039a33ce45964ff2167f6ecedd419db06c1"),
    (b"", "e3b0c44298fc1c149afbf4c8996fb92427ae41e4649b934ca495991b7852b855"),
]


@pytest.mark.parametrize("msg,digest", FIPS_VECTORS)
def test_oracle_hash_is_sha256(msg, digest):
    assert hashlib.sha256(msg).hexdigest() == digest


# ------------------------------------------------------------------------------------
# eq. (1) properties of the oracle
# ------------------------------------------------------------------------------------

def check_ssep_offset_invariance(block_hashes):
    rng = np.random.default_rng(1)
    doc = [SSEP_TOK] + list(rand_tokens(rng, 47))  # 3 blocks
    a = block_hashes(list(rand_tokens(rng, 32)) + doc, SSEP_TOK, PDEP_TOK, SEED)
    b = block_hashes(list(rand_tokens(rng, 80)) + doc, SSEP_TOK, PDEP_TOK, SEED)
    c = block_hashes(doc, SSEP_TOK, PDEP_TOK, SEED)
    assert a[2:] == b[5:] == c
    # ... and unlike the same tokens without the marker, which chain through the prefix
    d = block_hashes(list(rand_tokens(rng, 32)) + [7] + doc[1:], SSEP_TOK, PDEP_TOK, SEED)
    assert d[2] != a[2]


def check_chain_until_next_ssep(block_hashes):
    rng = np.random.default_rng(2)
    toks = list(rand_tokens(rng, 64)) + [SSEP_TOK] + list(rand_tokens(rng, 63))  # 8 blocks, SSEP at block 4
    base = block_hashes(toks, SSEP_TOK, PDEP_TOK, SEED)
    assert len(set(base)) == 8
    changed = list(toks)
    changed[16 + 5] += 1  # a token of block 1
    h = block_hashes(changed, SSEP_TOK, PDEP_TOK, SEED)
    assert h[0] == base[0]
    assert all(h[i] != base[i] for i in (1, 2, 3))
    assert h[4:] == base[4:]


def check_pdep_sees_whole_prefix(block_hashes):
    rng = np.random.default_rng(3)
    head = list(rand_tokens(rng, 16)) + [SSEP_TOK] + list(rand_tokens(rng, 31))  # blocks 0..2, SSEP at 1
    task = [PDEP_TOK] + list(rand_tokens(rng, 31))  # blocks 3, 4
    base = block_hashes(head + task, SSEP_TOK, PDEP_TOK, SEED)
    for pos in (0, 15, 20, 40):  # a change before the SSEP block, and inside the SSEP span
        ch = head + task
        ch[pos] += 3
        h = block_hashes(ch, SSEP_TOK, PDEP_TOK, SEED)
        assert h[3] != base[3] and h[4] != base[4]
        blk = pos // 16
        assert h[:blk] == base[:blk] and h[blk] != base[blk]
        if blk == 0:
            assert h[1:3] == base[1:3]  # the SSEP chain ignores what precedes it
    # the same task block after an identical prefix hashes alike
    assert block_hashes(head + task, SSEP_TOK, PDEP_TOK, SEED) == base
    # and unlike the same task with another seed-reset structure before it
    other = head[:16] + [7] + head[17:] + task
    assert block_hashes(other, SSEP_TOK, PDEP_TOK, SEED)[3] != base[3]


def check_markers_only_at_block_starts(block_hashes):
    rng = np.random.default_rng(4)
    pre_a, pre_b = list(rand_tokens(rng, 16)), list(rand_tokens(rng, 16))
    mid = list(rand_tokens(rng, 3)) + [SSEP_TOK] + list(rand_tokens(rng, 12))
    a = block_hashes(pre_a + mid, SSEP_TOK, PDEP_TOK, SEED)
    b = block_hashes(pre_b + mid, SSEP_TOK, PDEP_TOK, SEED)
    assert a[1] != b[1]  # an SSEP token inside a block does not detach the block
    mid_p = list(rand_tokens(rng, 5)) + [PDEP_TOK] + list(rand_tokens(rng, 10))
    x = list(rand_tokens(rng, 16)) + [SSEP_TOK] + list(rand_tokens(rng, 15)) + mid_p
    y = [t + 1 for t in x[:16]] + x[16:]
    hx, hy = block_hashes(x, SSEP_TOK, PDEP_TOK, SEED), block_hashes(y, SSEP_TOK, PDEP_TOK, SEED)
    assert hx[2] == hy[2]  # a PDEP token inside a block does not pull in the prefix


PROPERTIES = [check_ssep_offset_invariance, check_chain_until_next_ssep, check_pdep_sees_whole_prefix,
              check_markers_only_at_block_starts]


@pytest.mark.parametrize("prop", PROPERTIES, ids=lambda f: f.__name__)
def test_oracle_hash_rule_properties(prop):
    prop(BH.block_hashes)


def _planted(kind):
    """eq. (1) with one planted mistake (for checking that the properties catch it)."""
    def H(chain, toks):
        return hashlib.sha256(chain + np.asarray(toks, dtype="<i4").tobytes()).digest()

    def fn(tokens, ssep, pdep, seed):
        toks = [int(t) for t in tokens]
        out, prev = [], seed
        for i in range(len(toks) // 16):
            x = toks[16 * i:16 * i + 16]
            marker = {ssep: "s", pdep: "p"}.get(x[0]) if kind != "marker_anywhere" else \
                ("s" if ssep in x else "p" if pdep in x else None)
            if marker == "s":
                h = H(prev if kind == "ssep_keeps_chain" else seed, x)
            elif marker == "p":
                h = H(prev, x) if kind == "pdep_as_chain" else H(seed, toks[16 * i:16 * i + 16]) \
                    if kind == "pdep_block_only" else H(seed, toks[:16 * i + 16])
            else:
                h = H(seed, x) if kind == "no_chain" else H(prev, x)
            out.append(h)
            prev = h
        return out
    return fn


@pytest.mark.parametrize("kind", ["ssep_keeps_chain", "pdep_as_chain", "pdep_block_only", "no_chain",
                                  "marker_anywhere"])
def test_planted_hash_rule_mistakes_are_caught(kind):
    failed = 0
    for prop in PROPERTIES:
        try:
            prop(_planted(kind))
        except AssertionError:
            failed += 1
    assert failed > 0, kind


def test_planted_harness_without_mistake_passes():
    for prop in PROPERTIES:
        prop(_planted("none"))


def test_seed_enters_every_hash_and_partial_blocks_are_not_hashed():
    rng = np.random.default_rng(5)
    toks = rag_prompt(rng, [rand_tokens(rng, 40), rand_tokens(rng, 20)])
    a = BH.block_hashes(toks, SSEP_TOK, PDEP_TOK, SEED)
    b = BH.block_hashes(toks, SSEP_TOK, PDEP_TOK, bytes(32))
    assert len(a) == len(toks) // 16
    assert all(x != y for x, y in zip(a, b))
    assert BH.block_hashes(toks[:15], SSEP_TOK, PDEP_TOK, SEED) == []


# ------------------------------------------------------------------------------------
# reuse decision of the oracle
# ------------------------------------------------------------------------------------

def random_marked_stream(rng, n):
    toks = rand_tokens(rng, n)
    for b in range(-(-n // 16)):
        r = rng.random()
        if r < 0.25:
            toks[16 * b] = SSEP_TOK
        elif r < 0.35:
            toks[16 * b] = PDEP_TOK
        if rng.random() < 0.2 and 16 * b + 15 < n:  # markers inside blocks are ordinary tokens
            toks[16 * b + rng.integers(1, 16)] = SSEP_TOK if rng.random() < 0.5 else PDEP_TOK
    return toks


@pytest.mark.parametrize("seed", range(6))
def test_spans_keep_the_marker_windows_for_any_hits(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 300))
    toks = random_marked_stream(rng, n)
    want = BH.token_windows(toks, SSEP_TOK, PDEP_TOK)
    for trial in range(8):
        hits = rng.random(n // 16) < (trial / 7)
        starts, flags = BH.spans_from_blocks(toks, SSEP_TOK, PDEP_TOK, hits)
        assert starts[0] == 0 and all(s % 16 == 0 for s in starts)
        assert np.array_equal(O.span_windows(starts, flags, n), want)
        # computed tokens = tokens of missed full blocks + the partial tail block
        computed = np.zeros(n, dtype=bool)
        for b in range(-(-n // 16)):
            if b >= n // 16 or not hits[b]:
                computed[16 * b:16 * (b + 1)] = True
        assert np.array_equal(O.query_tokens(starts, flags, n), np.flatnonzero(computed))
        # every marker block opens a span carrying its flag
        for b in range(-(-n // 16)):
            m = BH.marker_of_block(toks, b, SSEP_TOK, PDEP_TOK)
            if m:
                k = starts.index(16 * b)
                assert flags[k] & (SSEP | PDEP) == m


def test_rag_second_prompt_reuses_documents_and_recomputes_the_task():
    rng = np.random.default_rng(7)
    docs = [rand_tokens(rng, 60), rand_tokens(rng, 45), rand_tokens(rng, 90)]
    first = rag_prompt(rng, docs)
    cached = set(BH.block_hashes(first, SSEP_TOK, PDEP_TOK, SEED))
    second = rag_prompt(rng, [docs[2], docs[0], rand_tokens(rng, 30)], system_len=48)
    h = BH.block_hashes(second, SSEP_TOK, PDEP_TOK, SEED)
    hits = [x in cached for x in h]
    starts, flags = BH.spans_from_blocks(second, SSEP_TOK, PDEP_TOK, hits)
    # system prompt (different length) misses; doc 2 and doc 0 hit at new offsets; the
    # new doc and the PDEP task miss
    assert [f & ~QUERY for f in flags] == [0, SSEP, SSEP, SSEP, PDEP]
    assert [bool(f & QUERY) for f in flags] == [True, False, False, True, True]


# ------------------------------------------------------------------------------------
# native span cache == oracle
# ------------------------------------------------------------------------------------

B = pytest.importorskip("paper_2606_13126_amd._binding")


@pytest.mark.parametrize("n", [0, 1, 3, 55, 56, 63, 64, 65, 119, 120, 128, 1000, 4096 + 7])
def test_native_sha256_matches(n):
    rng = np.random.default_rng(n)
    data = rng.integers(0, 256, size=n, dtype=np.uint8).tobytes()
    assert B.pic_sha256(data) == hashlib.sha256(data).digest()


@pytest.mark.parametrize("msg,digest", FIPS_VECTORS)
def test_native_sha256_vectors(msg, digest):
    assert B.pic_sha256(msg).hex() == digest


@pytest.mark.parametrize("seed", range(8))
def test_native_block_hashes_match_oracle(seed):
    rng = np.random.default_rng(100 + seed)
    n = [0, 15, 16, 17, 300, 1023, 1024, 5000][seed]
    toks = random_marked_stream(rng, n) if n else np.zeros(0, dtype=np.int64)
    if seed == 3:
        toks[::16] = PDEP_TOK  # every block a PDEP block (quadratic prefix in the oracle)
    sd = rng.integers(0, 256, 32, dtype=np.uint8).tobytes()
    got = B.pic_block_hashes(toks, SSEP_TOK, PDEP_TOK, sd)
    want = BH.block_hashes(toks, SSEP_TOK, PDEP_TOK, sd)
    assert got.shape == (n // 16, 32)
    assert [bytes(r) for r in got] == want


def test_native_block_hashes_negative_token_ids():
    toks = np.array([-1, 2**31 - 1, -2**31] + [9] * 29, dtype=np.int64)
    got = B.pic_block_hashes(toks, -1, 3, SEED)
    assert [bytes(r) for r in got] == BH.block_hashes(toks, -1, 3, SEED)


@pytest.mark.parametrize("seed", range(10))
def test_native_spans_match_oracle(seed):
    rng = np.random.default_rng(200 + seed)
    n = int(rng.integers(1, 400))
    toks = random_marked_stream(rng, n)
    hits = rng.random(n // 16) < rng.random()
    got = B.pic_spans_from_blocks(toks, SSEP_TOK, PDEP_TOK, hits)
    want = BH.spans_from_blocks(toks, SSEP_TOK, PDEP_TOK, hits)
    assert got[0].tolist() == want[0] and got[1].tolist() == want[1]


def test_native_argument_errors():
    with pytest.raises(B.PicError):
        B.pic_block_hashes(np.zeros(32), 1, 1, SEED)
    with pytest.raises(B.PicError):
        B.pic_spans_from_blocks(np.zeros(0), 1, 2, [])
    cap_short = B._lib.pic_spans_from_blocks
    toks = np.zeros(64, dtype=np.int32)
    toks[::16] = 1
    hit = np.zeros(4, dtype=np.uint8)
    st = np.zeros(2, dtype=np.int32)
    import ctypes
    n = ctypes.c_int32(0)
    assert cap_short(toks.ctypes.data, 64, 1, 2, hit.ctypes.data, st.ctypes.data, st.ctypes.data, 2,
                     ctypes.byref(n)) == B.PIC_EINVAL
    assert n.value == 4


def test_native_block_cache_roundtrip():
    rng = np.random.default_rng(9)
    c = B.pic_block_cache_create()
    try:
        first = rag_prompt(rng, [rand_tokens(rng, 70), rand_tokens(rng, 33)])
        h1 = B.pic_block_hashes(first, SSEP_TOK, PDEP_TOK, SEED)
        ids, hits = B.pic_block_cache_lookup(c, h1)
        assert hits == 0 and (ids == -1).all()
        B.pic_block_cache_insert(c, h1, np.arange(len(h1)) + 100)
        assert B.pic_block_cache_size(c) == len(set(bytes(r) for r in h1))
        ids, hits = B.pic_block_cache_lookup(c, h1)
        assert hits == len(h1) and ids.tolist() == list(range(100, 100 + len(h1)))
        B.pic_block_cache_insert(c, h1[:1], [7])  # an existing hash keeps its block
        assert B.pic_block_cache_lookup(c, h1[:1])[0][0] == 100
        B.pic_block_cache_erase(c, h1[:2])
        ids, hits = B.pic_block_cache_lookup(c, h1)
        assert hits == len(h1) - 2 and ids[0] == -1 and ids[1] == -1
    finally:
        B.pic_block_cache_destroy(c)
