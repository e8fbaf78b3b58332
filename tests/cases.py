"""Hand-shaped workloads shared by the plan tests (CPU) and the parity tests (GPU)."""
import numpy as np
import torch

import workloads as W

S, Pd, Q, Sp = W.SSEP, W.PDEP, W.QUERY, W.Span


def decode_case(Hq, Hkv, D, seed, offsets=(0, 5, 100000, -37, 70000)):
    """Decode batch covering the window rules and split shapes of one-query attention:
    a 1-token request, an unaligned SSEP window, a continuation span inheriting its
    window, a PDEP query over a shared span, and a long context that is split."""
    reqs = [[Sp(1, Pd, fresh=True)],
            [Sp(37, S), Sp(5, S, fresh=True)],
            [Sp(16, S, key="a"), Sp(300, S), Sp(29, 0, fresh=True)],
            [Sp(64, S, key="b"), Sp(16, S, key="a"), Sp(200, Pd, fresh=True)],
            [Sp(1000, Pd), Sp(1, Pd, fresh=True)]]
    return W.small_case(f"decode_h{Hq}_{Hkv}_d{D}", reqs, Hq=Hq, Hkv=Hkv, D=D, theta=5e5, dtype=torch.bfloat16,
                        seed=seed, value_scale=0.5, decode=True, position_offsets=list(offsets))


def windows_prefill_case(dtype=torch.bfloat16):
    """Explicit per-span window starts: EPIC/LegoLink-style recomputed document heads
    that attend to everything before them (window 0) followed by cached document
    bodies that keep their own document's start, and (request 1) a one-back query
    span whose window is the start of the previous document."""
    reqs = [[Sp(48, S, key="d0"), Sp(16, Q, fresh=True), Sp(32, 0, key="d1b"), Sp(16, Q, fresh=True),
             Sp(64, 0, key="d2b"), Sp(40, Pd | Q, fresh=True)],
            [Sp(32, S, key="d1b"), Sp(48, S, key="d0"), Sp(37, Q, fresh=True)]]
    wl = W.small_case("gen_windows", reqs, Hq=8, Hkv=2, D=128, theta=5e5, dtype=dtype, seed=41, value_scale=0.5)
    wl.span_window = np.array([-1, 0, 64, 0, 112, -1, -1, -1, 32], dtype=np.int32)
    return wl


def windows_decode_case():
    """Decode with explicit windows: one document back, and an unaligned start."""
    reqs = [[Sp(64, S, key="a"), Sp(48, S, key="b"), Sp(80, S), Sp(1, 0, fresh=True)],
            [Sp(48, S, key="b"), Sp(64, S, key="a"), Sp(300, S), Sp(1, 0, fresh=True)]]
    wl = W.small_case("gen_windows_dec", reqs, Hq=32, Hkv=8, D=128, theta=5e5, dtype=torch.bfloat16, seed=42,
                      value_scale=0.5, decode=True)
    wl.span_window = np.array([-1, -1, -1, 64, -1, -1, 48, 37], dtype=np.int32)
    return wl


def llama3_inv_freq(head_dim, theta, factor=8.0, low_freq_factor=1.0, high_freq_factor=4.0, original_max=8192):
    """Band-scaled RoPE frequencies of the Llama 3.1 family: wavelengths shorter than
    original_max / high_freq_factor keep their frequency, longer than
    original_max / low_freq_factor are slowed by ``factor``, and the band between
    interpolates linearly in original_max / wavelength."""
    om = 1.0 / np.power(float(theta), np.arange(0, head_dim, 2, dtype=np.float64) / head_dim)
    wavelen = 2.0 * np.pi / om
    smooth = (original_max / wavelen - low_freq_factor) / (high_freq_factor - low_freq_factor)
    mid = (1.0 - smooth) * om / factor + smooth * om
    out = np.where(wavelen < original_max / high_freq_factor, om,
                   np.where(wavelen > original_max / low_freq_factor, om / factor, mid))
    return out


def rope_variant_case(dtype, D=128, rotary_dim=None, inv_freq=None, decode=False, seed=51):
    """Prefill (or decode) batch with long positions for the RoPE-variant tests."""
    if decode:
        reqs = [[Sp(64, S, key="a"), Sp(300, S), Sp(1, Pd, fresh=True)],
                [Sp(48, S, key="b"), Sp(64, S, key="a"), Sp(1, 0, fresh=True)]]
    else:
        reqs = [[Sp(64, S, key="a"), Sp(200, S | Q, fresh=True), Sp(45, Pd | Q, fresh=True)],
                [Sp(48, S, key="b"), Sp(64, S, key="a"), Sp(33, Pd | Q, fresh=True)]]
    wl = W.small_case(f"rope_variant_d{D}_r{rotary_dim}", reqs, Hq=8, Hkv=2, D=D, theta=5e5, dtype=dtype,
                      seed=seed, value_scale=0.5, decode=decode, position_offsets=[60000, 123])
    wl.rotary_dim = rotary_dim
    wl.rope_inv_freq = inv_freq
    return wl


def many_spans_prefill(dtype=torch.bfloat16, seed=60):
    """More query spans than the kernel arguments hold (82 groups, so the group table
    goes through the workspace in two upload launches): 26 requests of three query
    spans over a shared cached prefix, and 4 requests whose query tail sees 1024
    cached keys (long enough to be split, so the split merge reads the table too)."""
    rng = np.random.default_rng(seed)
    reqs = []
    for r in range(26):
        n1, n2, n3 = (int(x) for x in rng.integers(1, 70, size=3))
        reqs.append([Sp(32, S, key="pre"), Sp(n1, S | Q, fresh=True), Sp(n2, Q, fresh=True),
                     Sp(n3, Pd | Q, fresh=True)])
    for r in range(4):
        reqs.append([Sp(1024, S, key="long"), Sp(int(rng.integers(20, 90)), Pd | Q, fresh=True)])
    return W.small_case("many_spans", reqs, Hq=8, Hkv=2, D=128, theta=5e5, dtype=dtype, seed=seed,
                        value_scale=0.5)


def short_causal_spans_prefill(D=128, seed=62, cycles=24):
    """Many short causal query spans, the shape of a prefill whose fresh documents are
    short: fresh SSEP spans of 100, 64, 33, 160 and 7 tokens (4, 2, 2, 5 and 1 row
    tiles of 8 heads, the last ones partial) in one request, 2,744 row-tile items
    and 122 groups (the group table goes through the workspace); a second request
    whose query span continues a cached span (window > 0); and a short PDEP tail
    that sees every key (split)."""
    lens = [100, 64, 33, 160, 7] * cycles
    reqs = [[Sp(n, S | Q, fresh=True) for n in lens] + [Sp(16, Pd | Q, fresh=True)],
            [Sp(64, S, key="pre"), Sp(48, S), Sp(37, Q, fresh=True)]]
    return W.small_case(f"short_causal_spans_d{D}", reqs, Hq=64, Hkv=8, D=D, theta=5e5, dtype=torch.bfloat16,
                        seed=seed, value_scale=0.5)


def long_context_decode(seed=81, num_reqs=2, num_spans=256, span_len=512):
    """131,073-key decode: each request holds the same 256 SSEP spans of 512 tokens in
    its own order, plus the new token (splits of thousands of keys per request)."""
    rng = np.random.default_rng(seed)
    reqs = [[Sp(span_len, S, key=("d", int(i))) for i in rng.permutation(num_spans)] + [Sp(1, Pd, fresh=True)]
            for _ in range(num_reqs)]
    nb = num_spans * span_len // 16 + num_reqs + 16
    return W.build("long_context_decode", reqs, num_q_heads=32, num_kv_heads=8, head_dim=128, rope_theta=5e5,
                   dtype=torch.bfloat16, seed=seed, value_scale=0.5, num_blocks=nb, decode=True, poison=False)


def long_context_prefill(seed=82, num_spans=256, span_len=512, tail=40, dtype=torch.bfloat16):
    """A 40-token PDEP query tail over 131,072 cached keys (256 SSEP spans)."""
    reqs = [[Sp(span_len, S, key=("d", i)) for i in range(num_spans)] + [Sp(tail, Pd | Q, fresh=True)]]
    nb = (num_spans * span_len + tail) // 16 + 16
    return W.build("long_context_prefill", reqs, num_q_heads=8, num_kv_heads=2, head_dim=128, rope_theta=5e5,
                   dtype=dtype, seed=seed, value_scale=0.5, num_blocks=nb, poison=False)


def many_requests_decode(num_reqs=256, Hq=32, Hkv=8, D=128, seed=61):
    """256 decode requests of 1 to ~600 tokens (more groups than the kernel
    arguments hold; the longer ones are split, the shorter are not)."""
    rng = np.random.default_rng(seed)
    reqs = []
    for r in range(num_reqs):
        kind = r % 4
        if kind == 0:
            spans = [Sp(int(rng.integers(1, 40)), Pd, fresh=True)]
        elif kind == 1:
            spans = [Sp(64, S, key="a"), Sp(int(rng.integers(1, 200)), S), Sp(1, 0, fresh=True)]
        elif kind == 2:
            spans = [Sp(128, S, key="b"), Sp(64, S, key="a"), Sp(int(rng.integers(100, 400)), Pd), Sp(1, Pd, fresh=True)]
        else:
            spans = [Sp(int(rng.integers(16, 80)), S), Sp(1, S, fresh=True)]
        reqs.append(spans)
    return W.small_case("many_requests_decode", reqs, Hq=Hq, Hkv=Hkv, D=D, theta=5e5, dtype=torch.bfloat16,
                        seed=seed, value_scale=0.5, decode=True,
                        position_offsets=[int(x) for x in rng.integers(0, 5000, size=num_reqs)])


# ---- peaked scores: the running maximum of the online softmax must move -------------------

LOG2E = 1.4426950408889634
PEAK_SCALE = 0.125 / LOG2E   # softmax scale whose log2-domain factor is 1/8 exactly


def plant_rising_keys(wl, every=64, offset=37, q_val=4.0, a_max=250.0):
    """Make later keys dominate: every `every`-th key (sequence index = offset mod
    `every`) of every request gets amplitude A(j) = 16 .. a_max, growing with its
    sequence index j, on the lowest-frequency RoPE pair (NeoX dims D/2-1 and D-1,
    which turn by less than a milliradian over these positions), and every query
    gets q_val on the same pair.  With softmax_scale = PEAK_SCALE a planted key's
    score is q_val * A / 8 in log2 units plus the small random part of the other
    dims, so along the sequence the row maximum rises by several times the kernels'
    rescale threshold and the output is a mix of the last few planted values (O(1)
    entries).  Values are exact in bf16 (even integers below 256)."""
    D = wl.head_dim
    lo, hi = D // 2 - 1, D - 1
    fresh_row = {(int(r), int(t)): i for i, (r, t) in enumerate(wl.info["fresh_tokens"])}
    for r in range(wl.num_reqs):
        L = int(wl.seq_lens[r])
        for j in range(offset, L, every):
            a = float(2 * round((16.0 + (a_max - 16.0) * j / max(L - 1, 1)) / 2))
            if (r, j) in fresh_row:
                i = fresh_row[(r, j)]
                wl.k_new[i, :, lo] = a
                wl.k_new[i, :, hi] = 0.0
            else:
                b = int(wl.block_tables[r, j // 16])
                wl.k_pool[b, :, j % 16, lo] = a
                wl.k_pool[b, :, j % 16, hi] = 0.0
    wl.q[:, :, lo] = q_val
    wl.q[:, :, hi] = 0.0
    wl.softmax_scale = PEAK_SCALE
    return wl


def rise_of_max(wl, rows=None):
    """Premise check in fp64 (oracle RoPE): for each query row t and head h, the
    maximum log2-domain score over its visible keys after the first 64 minus the
    maximum over the first 64 (NaN for rows seeing at most 64 keys).  A value above 8
    means the kernels' running maximum has to move after their first key tile."""
    import math
    from oracle import pic_oracle as O
    from oracle import workload_oracle as WO
    k, _ = WO.pools_after_write(wl)
    q = wl.q.double().numpy()
    G = wl.num_q_heads // wl.num_kv_heads
    scale = (wl.softmax_scale or 1.0 / math.sqrt(wl.head_dim)) * LOG2E
    out = []
    row = 0
    for r in range(wl.num_reqs):
        L = int(wl.seq_lens[r])
        sl = slice(wl.cu_spans[r], wl.cu_spans[r + 1])
        w = O.span_windows(wl.span_start[sl], wl.span_flags[sl], L, None)
        qi = np.array([L - 1]) if wl.is_decode else O.query_tokens(wl.span_start[sl], wl.span_flags[sl], L)
        pos = wl.positions[wl.seq_offsets[r]:wl.seq_offsets[r] + L].astype(np.int64)
        n = np.arange(L)
        K = O.rope(k[wl.block_tables[r][n // 16], :, n % 16, :], pos[:, None], wl.rope_theta)
        sel = np.arange(len(qi)) if rows is None else np.array([i for i in range(len(qi)) if row + i in rows], int)
        if len(sel):
            t = qi[sel]
            lo, first_end = w[t], w[t] + 64
            j = np.arange(L)[None, :]
            early = (j >= lo[:, None]) & (j < first_end[:, None]) & (j <= t[:, None])
            late = (j >= first_end[:, None]) & (j <= t[:, None])
            qr = O.rope(q[row + sel], pos[t][:, None], wl.rope_theta)       # [n][Hq][D]
            for h in range(wl.num_q_heads):
                s = qr[:, h, :] @ K[:, h // G, :].T * scale                 # [n][L]
                m1 = np.where(early, s, -np.inf).max(axis=1)
                m2 = np.where(late, s, -np.inf).max(axis=1)
                out.append(np.where(np.isfinite(m2), m2 - m1, np.nan))
        row += len(qi)
    return np.concatenate(out) if out else np.array([])
