"""Write the stored oracle fixtures of tests/golden/ (calls only oracle/ and the
seeded input generator).  Run from the repository root:

    python -m tests.golden.make_golden
"""
import json
import os

import numpy as np

import workloads as W
from oracle import workload_oracle as WO

HERE = os.path.dirname(os.path.abspath(__file__))


def sample_indices(shape, n, seed):
    rng = np.random.default_rng(seed)
    return [[int(rng.integers(0, d)) for d in shape] for _ in range(n)]


def main():
    fixtures = {}
    for name, wl in (("tiny_fp32_prefill", W.tiny_fp32()), ("tiny_fp32_prefill_tail", W.tiny_fp32(tail_only=True))):
        o = WO.run(wl)
        idx = sample_indices(o.shape, 48, 99)
        fixtures[name] = {"shape": list(o.shape), "index": idx,
                          "value": [float(o[tuple(i)]) for i in idx],
                          "sum": float(o.sum()), "sum_abs": float(np.abs(o).sum())}
    with open(os.path.join(HERE, "oracle_tiny_fp32.json"), "w") as f:
        json.dump(fixtures, f, indent=1)
        f.write("\n")


if __name__ == "__main__":
    main()
