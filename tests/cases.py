"""Hand-shaped workloads shared by the plan tests (CPU) and the parity tests (GPU)."""
import torch

import workloads as W

S, Pd, Sp = W.SSEP, W.PDEP, W.Span


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
