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
