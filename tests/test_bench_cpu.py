"""The measurement contract of bench.py, checked on the CPU: algorithmic work and
bytes against independent counts, the one-GPU refusal, and the traffic figure's
source check."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
import workloads as W
from oracle import pic_oracle as O
from tests.cases import windows_prefill_case

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def oracle_flops(wl):
    p = O.visible_pairs(wl.seq_lens, wl.cu_spans, wl.span_start, wl.span_flags, wl.is_decode, wl.span_window)
    return 4.0 * wl.head_dim * wl.num_q_heads * p


def test_flops_of_the_8b_rag_tail():
    # 1,343,616 visible (query, key) pairs: 256 tail tokens of a PDEP span after
    # 5120 cached tokens see 5121..5376 keys each
    wl = W.llama3_8b_rag()
    pairs = sum(5120 + t + 1 for t in range(256))
    assert pairs == 1343616
    assert bench.flops_of(wl) == 4.0 * 128 * 32 * pairs == oracle_flops(wl)


@pytest.mark.parametrize("make", [W.tiny_fp32, lambda: W.decode_64req(num_reqs=4, num_spans=3, span_len=64),
                                  windows_prefill_case, lambda: W.concurrent_reuse(num_reqs=4, pool_spans=6, per_req=3,
                                                                          span_len=256, tail=64)])
def test_flops_of_matches_the_oracle_pair_count(make):
    wl = make()
    assert bench.flops_of(wl) == oracle_flops(wl)


def test_decode_bytes():
    wl = W.decode_64req()
    # 64 requests x 8193 keys x 8 heads x 128 dims x (K + V) x 2 bytes, plus q/o,
    # positions and block tables
    kv = 64 * 8193 * 8 * 128 * 2 * 2
    assert abs(bench.decode_bytes(wl) - kv) / kv < 0.01
    assert abs(bench.decode_bytes(wl) - 2.151e9) / 2.151e9 < 0.005


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2", "--no-cpu"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_flops_and_row_pairs_of_the_70b_long_prefill():
    # 32 fresh SSEP spans of 512 tokens (each token t of a span sees t+1 keys of its
    # own span) and a 512-token PDEP tail after 32,768 tokens: 21,111,040 pairs
    wl = W.llama3_70b_long()
    fresh = 32 * sum(range(1, 513))
    tail = sum(32768 + t + 1 for t in range(512))
    assert fresh == 4202496 and tail == 16908544
    assert bench.flops_of(wl) == 4.0 * 128 * 64 * (fresh + tail) == oracle_flops(wl)
    rp = bench.row_pairs(wl)
    assert rp.shape == (wl.q.shape[0],) and int(rp.sum()) == fresh + tail


def test_unique_kv_bytes_shared_and_unshared_decode():
    page = 8 * 16 * 128 * 2 * 2
    assert bench.unique_kv_bytes(W.decode_64req()) == (16 * 32 + 64) * page    # 16 shared spans + 64 private blocks
    un = W.decode_64req(num_reqs=8, num_spans=4, shared=False)
    assert bench.unique_kv_bytes(un) == 8 * (4 * 32 + 1) * page


def test_traffic_is_reported_only_for_the_measured_sources(monkeypatch):
    if not os.path.exists(bench.TRAFFIC_FILE):
        assert bench.measured_traffic() is None
        pytest.skip("no counter summary for the headline workload yet")
    with open(bench.TRAFFIC_FILE) as f:
        t = json.load(f)
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: t["source_hash"])
    assert bench.measured_traffic() == t["bytes_per_call"]
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0" * 16)
    assert bench.measured_traffic() is None
