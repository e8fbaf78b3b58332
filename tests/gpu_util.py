"""Helpers of the GPU parity tests: run the library on a workload, compare with
the fp64 oracle at the stated tolerances."""
import math
import sys

import numpy as np
import torch

from oracle import workload_oracle as WO

# bf16 inputs with fp32 accumulation: max-abs and relative L2; fp32 inputs: max-abs
BF16_MAX_ABS, BF16_REL_L2 = 2e-2, 5e-3
F32_MAX_ABS = 1e-4

# every comparison of the session: (what, max_abs, rel_l2, max |reference|), printed
# as a table at the end of the run (tests/conftest.py)
RECORDS = []


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def gpu_run(wl, rope_style=0, table=True, k_prerotated=False, table_len=None):
    from paper_2606_13126_amd.runner import DeviceBatch
    n_tab = None
    if table:
        n_tab = table_len if table_len is not None else int(max(1, int(wl.positions.max()) + 1))
    db = DeviceBatch(wl, rope_style=rope_style, table_positions=n_tab, k_prerotated=k_prerotated)
    db.write()
    db.attend()
    torch.cuda.synchronize()
    return db


def to_np(t):
    return t.detach().to(torch.float64).cpu().numpy()


def errors(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = got - ref
    max_abs = float(np.max(np.abs(d))) if d.size else 0.0
    rel = float(np.linalg.norm(d) / max(np.linalg.norm(ref), 1e-300)) if d.size else 0.0
    return max_abs, rel


def assert_close(got, ref, dtype, what=""):
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    max_abs, rel = errors(got, ref)
    peak = float(np.max(np.abs(ref))) if np.size(ref) else 0.0
    RECORDS.append((what, max_abs, rel, peak, "fp32" if dtype == torch.float32 else "bf16"))
    say(f"  {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e} max|ref|={peak:.3g}")
    if dtype == torch.float32:
        assert max_abs <= F32_MAX_ABS, (what, max_abs)
    else:
        assert max_abs <= BF16_MAX_ABS and rel <= BF16_REL_L2, (what, max_abs, rel)
    return max_abs, rel
