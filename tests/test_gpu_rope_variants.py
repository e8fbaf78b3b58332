"""GPU parity of the RoPE variants: explicit (scaled) frequencies and a partial
rotary width, through the fused prefill and decode kernels, the cos/sin table and
the conventional rotation of the pre-rotated comparison path."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import pic_oracle as O
from oracle import workload_oracle as WO
from tests.cases import llama3_inv_freq, rope_variant_case
from tests.gpu_util import assert_close, gpu_run, say, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_13126_amd  # noqa: F401  (fails loudly if the library is missing)


def run_check(wl, style, table):
    say(f"[gpu] {wl.name}: dtype={wl.dtype} style={style} table={table} R={wl.rotary_dim} "
        f"inv_freq={'set' if wl.rope_inv_freq is not None else 'theta'}")
    db = gpu_run(wl, rope_style=style, table=table)
    ref = WO.run(wl, style="neox" if style == 0 else "gptj")
    return assert_close(to_np(db.o), ref, wl.dtype, wl.name)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("style", [0, 1])
@pytest.mark.parametrize("table", [True, False])
def test_scaled_frequencies_prefill(dtype, style, table):
    wl = rope_variant_case(dtype, inv_freq=llama3_inv_freq(128, 5e5))
    run_check(wl, style, table)


@pytest.mark.parametrize("D,R", [(128, 64), (64, 32), (128, 2), (64, 62)])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_partial_rotary_gptj_prefill(D, R, dtype):
    run_check(rope_variant_case(dtype, D=D, rotary_dim=R), 1, True)


@pytest.mark.parametrize("D,R", [(128, 32), (128, 96), (64, 16), (64, 48), (128, 16)])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_partial_rotary_neox_prefill(D, R, dtype):
    run_check(rope_variant_case(dtype, D=D, rotary_dim=R), 0, True)


def test_partial_rotary_neox_computed_cossin_decode():
    freq = llama3_inv_freq(32, 1e4)
    run_check(rope_variant_case(torch.bfloat16, rotary_dim=32, inv_freq=freq, decode=True), 0, False)
    run_check(rope_variant_case(torch.bfloat16, rotary_dim=64, decode=True), 0, True)


def test_partial_rotary_with_scaled_frequencies_computed_cossin():
    wl = rope_variant_case(torch.bfloat16, rotary_dim=64, inv_freq=llama3_inv_freq(64, 1e4) * 1.7)
    run_check(wl, 1, False)


@pytest.mark.parametrize("style,R,table", [(0, None, True), (1, 64, True), (1, 96, False), (0, 64, True)])
def test_variants_decode(style, R, table):
    freq = llama3_inv_freq(R or 128, 5e5)
    run_check(rope_variant_case(torch.bfloat16, rotary_dim=R, inv_freq=freq, decode=True), style, table)


def test_variant_table_entries():
    # pairs past the rotary width hold cos 1, sin 0 exactly; the others follow the
    # given frequencies
    import paper_2606_13126_amd as P
    n, D, R = 5000, 128, 48
    freq = llama3_inv_freq(R, 5e5)
    cfg = P.make_config(8, 8, D, dtype=P.PIC_F32, rope_style=P.PIC_ROPE_GPTJ, rotary_dim=R, inv_freq=freq)
    tab = torch.empty((n, D // 2, 2), dtype=torch.float32, device="cuda")
    P.pic_rope_table_build(cfg, tab)
    got = tab.cpu().double().numpy()
    p = np.arange(n, dtype=np.float64)[:, None] * freq[None, :]
    assert np.max(np.abs(got[:, :R // 2, 0] - np.cos(p))) <= 1e-7
    assert np.max(np.abs(got[:, :R // 2, 1] - np.sin(p))) <= 1e-7
    assert (got[:, R // 2:, 0] == 1.0).all() and (got[:, R // 2:, 1] == 0.0).all()


@pytest.mark.parametrize("style", [0, 1])
def test_variant_prerotated_equals_fused(style):
    # the conventional rotation (pic_rope_rotate) with the same variant, applied to
    # every stored key and to the queries, gives the fused result
    import paper_2606_13126_amd as P
    from paper_2606_13126_amd.runner import DeviceBatch
    Sp, S, Pd, Q = W.Span, W.SSEP, W.PDEP, W.QUERY
    wl = W.small_case("variant_pre", [[Sp(64, S, key="a"), Sp(200, S | Q, fresh=True), Sp(45, Pd | Q, fresh=True)]],
                      Hq=8, Hkv=2, D=128, theta=5e5, dtype=torch.bfloat16, seed=52, value_scale=0.5,
                      position_offsets=[60000])
    wl.rotary_dim, wl.rope_inv_freq = 96, llama3_inv_freq(96, 5e5)
    fused = gpu_run(wl, rope_style=style)
    ctl = DeviceBatch(wl, k_prerotated=True, rope_style=style, table_positions=int(wl.positions.max()) + 1)
    ctl.write()
    # one request: rotate every stored key once, at its position
    kp = ctl.k_pool.permute(0, 2, 1, 3).reshape(-1, wl.num_kv_heads, wl.head_dim)
    off = wl.seq_offsets
    L = int(wl.seq_lens[0])
    n = torch.arange(L)
    slots = (torch.from_numpy(wl.block_tables[0].astype(np.int64))[n // 16] * 16 + n % 16).cuda()
    rows = kp[slots].contiguous()
    P.pic_rope_rotate(ctl.cfg, rows, torch.from_numpy(wl.positions[:L]).cuda(), table=ctl.table)
    kp[slots] = rows
    ctl.k_pool = kp.reshape(-1, 16, wl.num_kv_heads, wl.head_dim).permute(0, 2, 1, 3).contiguous()
    qtok = wl.q_tokens
    qpos = np.array([wl.positions[off[r] + t] for r, t in qtok], dtype=np.int32)
    P.pic_rope_rotate(ctl.cfg, ctl.q, torch.from_numpy(qpos).cuda(), table=ctl.table)
    ctl.attend()
    torch.cuda.synchronize()
    assert_close(to_np(ctl.o), to_np(fused.o), wl.dtype, "pre-rotated variant vs fused")
    assert_close(to_np(fused.o), WO.run(wl, style="gptj" if style else "neox"), wl.dtype, "fused variant vs oracle")
