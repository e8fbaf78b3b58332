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
