"""GPU parity: libpic_attn against the fp64 oracle on the same seeded inputs."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import pic_oracle as O
from oracle import workload_oracle as WO
from tests.cases import (decode_case, long_context_decode, long_context_prefill, many_requests_decode,
                         many_spans_prefill, plant_rising_keys, rise_of_max, short_causal_spans_prefill,
                         windows_decode_case, windows_prefill_case)
from tests.gpu_util import assert_close, gpu_run, say, to_np

pytestmark = pytest.mark.gpu

S, Pd, Q, Sp = W.SSEP, W.PDEP, W.QUERY, W.Span


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_13126_amd  # noqa: F401  (fails loudly if the library is missing)


def check(wl, style=0, table=True, rows=None, what=None):
    what = what or wl.name
    say(f"[gpu] {what}: shape q={tuple(wl.q.shape)} dtype={wl.dtype} style={style} table={table}")
    db = gpu_run(wl, rope_style=style, table=table)
    got = to_np(db.o)
    ref = WO.run(wl, rows=rows, style="neox" if style == 0 else "gptj")
    if rows is not None:
        got = got[rows]
    return assert_close(got, ref, wl.dtype, what)


@pytest.mark.parametrize("tail_only", [False, True])
@pytest.mark.parametrize("table", [True, False])
def test_tiny_fp32(tail_only, table):
    check(W.tiny_fp32(tail_only=tail_only), table=table)


def test_kv_write_bit_exact():
    for wl in (W.tiny_fp32(), W.llama3_8b_rag()):
        db = gpu_run(wl)
        k_ref, v_ref = wl.k_pool.clone(), wl.v_pool.clone()
        iv = torch.int32 if wl.dtype == torch.float32 else torch.int16
        kr, vr = k_ref.view(iv).numpy(), v_ref.view(iv).numpy()
        O.kv_write(kr, vr, wl.k_new.view(iv).numpy(), wl.v_new.view(iv).numpy(), wl.slot_mapping)
        assert np.array_equal(db.k_pool.cpu().view(iv).numpy(), kr)
        assert np.array_equal(db.v_pool.cpu().view(iv).numpy(), vr)


@pytest.mark.parametrize("table", [True, False])
def test_llama3_8b_rag_bf16(table):
    check(W.llama3_8b_rag(), table=table)


def test_concurrent_reuse_bf16():
    check(W.concurrent_reuse())


def test_decode_64req_bf16():
    check(W.decode_64req())


def test_llama3_70b_long_all_rows():
    # the largest workload, every one of its 16,896 query tokens x 64 heads
    check(W.llama3_70b_long())


@pytest.mark.parametrize("style", [0, 1])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_unaligned_spans_gqa(style, dtype):
    wl = W.small_case("unaligned", [[Sp(21, S | Q, fresh=True), Sp(37, Q, fresh=True), Sp(300, S | Q, fresh=True),
                                     Sp(11, Pd | Q, fresh=True)]], Hq=8, Hkv=2, D=128, theta=1e4, dtype=dtype,
                      seed=5, value_scale=0.5)
    check(wl, style=style)


@pytest.mark.parametrize("Hq,Hkv,D,style", [
    (12, 4, 128, 0),    # G = 3: 256-row tiles end inside a token's heads
    (14, 2, 64, 1),     # G = 7
    (24, 2, 128, 1),    # G = 12
    (48, 3, 64, 0),     # G = 16, three KV heads (no XCD grouping of KV heads)
])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_prefill_query_groups_straddling_row_tiles(Hq, Hkv, D, style, dtype):
    # query rows are (token, head) pairs; with G not dividing the 256-row tile the
    # heads of one token are split between two workgroups
    reqs = [[Sp(48, S, key="a"), Sp(100, S | Q, fresh=True), Sp(61, Pd | Q, fresh=True)],
            [Sp(48, S, key="a"), Sp(23, Pd | Q, fresh=True)]]
    wl = W.small_case("groups", reqs, Hq=Hq, Hkv=Hkv, D=D, theta=1e4, dtype=dtype, seed=40 + Hq, value_scale=0.5)
    check(wl, style=style)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_mha_d64_multi_request(dtype):
    reqs = [[Sp(64, S, key="a"), Sp(48, S, key="b"), Sp(70, Pd | Q, fresh=True)],
            [Sp(48, S, key="b"), Sp(64, S, key="a"), Sp(5, Pd | Q, fresh=True)],
            [Sp(32, S, key="c")] + [Sp(16, S | Q, fresh=True)],
            [Sp(9, S, key=None), Sp(40, Q, fresh=True)]]
    wl = W.small_case("mha", reqs, Hq=4, Hkv=4, D=64, theta=1e4, dtype=dtype, seed=6, value_scale=0.5)
    check(wl)


def test_zero_query_request_and_empty_batch():
    reqs = [[Sp(32, S, key="a")], [Sp(32, S, key="a"), Sp(17, Pd | Q, fresh=True)], [Sp(16, S)]]
    wl = W.small_case("zq", reqs, Hq=8, Hkv=2, D=128, dtype=torch.bfloat16, seed=7, value_scale=0.5)
    check(wl)


def test_first_token_of_ssep_span_is_its_value():
    wl = W.small_case("first", [[Sp(32, S | Q, fresh=True), Sp(48, S | Q, fresh=True)]], Hq=4, Hkv=1, D=128,
                      dtype=torch.bfloat16, seed=8, value_scale=0.5)
    db = gpu_run(wl)
    o = db.o.cpu()
    for t in (0, 32):
        assert torch.equal(o[t], wl.v_new[t, 0].expand(4, 128)), t


def test_excluded_blocks_are_never_read():
    # span 1 is detached (SSEP) from span 0, whose blocks hold NaN: output must be finite
    wl = W.small_case("poison", [[Sp(64, S, key="a"), Sp(96, S | Q, fresh=True), Sp(32, S | Q, fresh=True)]],
                      Hq=8, Hkv=2, D=128, dtype=torch.bfloat16, seed=9, value_scale=0.5)
    for b in wl.block_tables[0][:4]:
        wl.k_pool[b] = float("nan")
        wl.v_pool[b] = float("nan")
    check(wl, what="poisoned excluded span")


def test_duplicate_block_in_one_request():
    wl = W.small_case("dup", [[Sp(64, S, key="a"), Sp(64, S, key="a"), Sp(40, Pd | Q, fresh=True)]], Hq=8, Hkv=2,
                      D=128, dtype=torch.bfloat16, seed=10, value_scale=0.5)
    assert wl.block_tables[0][0] == wl.block_tables[0][4]
    check(wl)


def test_shift_invariance_bf16():
    wl = W.small_case("shift", [[Sp(128, S, key="a"), Sp(200, S | Q, fresh=True), Sp(64, Pd | Q, fresh=True)]],
                      Hq=8, Hkv=2, D=128, theta=5e5, dtype=torch.bfloat16, seed=11, value_scale=0.5)
    base = to_np(gpu_run(wl).o)
    for shift in (1000, 65536, -37):
        wl.positions = (wl.positions.astype(np.int64) + shift).astype(np.int32)
        got = to_np(gpu_run(wl).o)    # table for non-negative positions, computed otherwise
        assert_close(got, base, wl.dtype, f"shift {shift} vs unshifted")
        wl.positions = (wl.positions.astype(np.int64) - shift).astype(np.int32)
    ref = WO.run(wl)
    assert_close(base, ref, wl.dtype, "unshifted vs oracle")


@pytest.mark.parametrize("Hq,Hkv", [(32, 1), (64, 2), (32, 8)])
def test_decode_shift_invariance_full_size(Hq, Hkv):
    # 64 requests x 8,193 keys through the 2-, 4- and 8-wave decode workgroups: adding
    # a constant to every position leaves the scores unchanged (relative positions),
    # so the outputs agree to bf16 rounding; checked where the fp64 oracle would be slow
    reqs = [[Sp(8192, S, key=("d", r)), Sp(1, Pd, fresh=True)] for r in range(64)]
    wl = W.build("decode_shift", reqs, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=128, rope_theta=5e5,
                 dtype=torch.bfloat16, seed=71, value_scale=0.5, num_blocks=64 * 514 + 16, decode=True, poison=False)
    say(f"[gpu] decode shift invariance Hq={Hq} Hkv={Hkv}: {wl.num_reqs} requests x {int(wl.seq_lens[0])} keys")
    base = to_np(gpu_run(wl).o)
    wl.positions = (wl.positions.astype(np.int64) + 4321).astype(np.int32)
    got = to_np(gpu_run(wl).o)
    assert_close(got, base, wl.dtype, f"decode Hq={Hq} Hkv={Hkv} shift 4321 vs unshifted")


@pytest.mark.parametrize("decode", [False, True])
def test_positions_at_the_int32_limits(decode):
    # logical positions next to 2^31 - 1 and -2^31: the angle is an exact fixed-point
    # phase, so attention matches the oracle there (cos/sin computed in the kernel;
    # the table covers only [0, 1000))
    if decode:
        wl = W.small_case("lim_dec", [[Sp(64, S, key="a"), Sp(300, S), Sp(1, Pd, fresh=True)],
                                      [Sp(64, S, key="a"), Sp(1, Pd, fresh=True)]], Hq=8, Hkv=2, D=128, theta=5e5,
                          dtype=torch.bfloat16, seed=13, value_scale=0.5, decode=True,
                          position_offsets=[2**31 - 400, -2**31])
    else:
        wl = W.small_case("lim", [[Sp(64, S, key="a"), Sp(300, S | Q, fresh=True), Sp(29, Pd | Q, fresh=True)],
                                  [Sp(64, S, key="a"), Sp(37, Pd | Q, fresh=True)]], Hq=8, Hkv=2, D=128, theta=5e5,
                          dtype=torch.bfloat16, seed=13, value_scale=0.5, position_offsets=[2**31 - 400, -2**31])
    assert int(wl.positions.max()) >= 2**31 - 64 and int(wl.positions.min()) == -2**31
    say(f"[gpu] int32-limit positions, decode={decode}")
    got = to_np(gpu_run(wl, table_len=1000).o)
    assert_close(got, WO.run(wl), wl.dtype, f"int32-limit positions decode={decode}")


def test_concurrent_reuse_equals_alone():
    wl = W.concurrent_reuse(num_reqs=4, pool_spans=6, per_req=3, span_len=256, tail=64)
    full = to_np(gpu_run(wl).o)
    row = 0
    for r in range(wl.num_reqs):
        sl = slice(wl.cu_spans[r], wl.cu_spans[r + 1])
        nq = 64
        one = W.Workload(**{**wl.__dict__})
        one.seq_lens = wl.seq_lens[r:r + 1]
        one.cu_spans = np.array([0, sl.stop - sl.start], np.int32)
        one.span_start, one.span_flags = wl.span_start[sl], wl.span_flags[sl]
        one.block_tables = wl.block_tables[r:r + 1]
        off = wl.seq_offsets
        one.positions = wl.positions[off[r]:off[r + 1]]
        one.q = wl.q[row:row + nq]
        one.k_new, one.v_new = wl.k_new[row:row + nq], wl.v_new[row:row + nq]
        one.slot_mapping = wl.slot_mapping[row:row + nq]
        alone = to_np(gpu_run(one).o)
        assert_close(alone, full[row:row + nq], wl.dtype, f"request {r} alone vs batched")
        row += nq


def test_decode_equals_prefill_of_last_token():
    dec = W.decode_64req(num_reqs=3, num_spans=4, span_len=128)
    od = to_np(gpu_run(dec).o)
    pre = W.Workload(**{**dec.__dict__})
    pre.is_decode = False
    pre.span_flags = dec.span_flags.copy()
    last = dec.cu_spans[1:] - 1
    pre.span_flags[last] |= W.QUERY
    op = to_np(gpu_run(pre).o)
    assert_close(od, op, dec.dtype, "decode vs prefill of the last token")
    assert_close(od, WO.run(dec), dec.dtype, "decode vs oracle")


def test_fused_rope_equals_prerotated_baseline():
    # Sec. 3.2.1: rotating inside attention equals attention over pre-rotated keys
    import paper_2606_13126_amd as P
    from paper_2606_13126_amd.runner import DeviceBatch
    wl = W.small_case("pre", [[Sp(128, S, key="a"), Sp(256, S | Q, fresh=True), Sp(100, Pd | Q, fresh=True)]],
                      Hq=8, Hkv=2, D=128, theta=5e5, dtype=torch.bfloat16, seed=12, value_scale=0.5)
    fused = gpu_run(wl)
    ctl = DeviceBatch(wl, k_prerotated=True, table_positions=int(wl.positions.max()) + 1)
    ctl.write()
    # rotate every stored key at its position (all slots of the request) and the queries
    L = int(wl.seq_lens[0])
    n = torch.arange(L)
    slots = (torch.from_numpy(wl.block_tables[0].astype(np.int64))[n // 16] * 16 + n % 16)
    pos = torch.from_numpy(wl.positions[:L]).cuda()
    kp = ctl.k_pool.permute(0, 2, 1, 3).reshape(-1, wl.num_kv_heads, wl.head_dim)
    rows = kp[slots.cuda()].contiguous()
    P.pic_rope_rotate(ctl.cfg, rows, pos, table=ctl.table)
    kp[slots.cuda()] = rows
    ctl.k_pool = kp.reshape(-1, 16, wl.num_kv_heads, wl.head_dim).permute(0, 2, 1, 3).contiguous()
    qpos = torch.from_numpy(wl.q_tokens[:, 1].astype(np.int32)).cuda()
    qpos = pos[qpos.long()].contiguous()
    P.pic_rope_rotate(ctl.cfg, ctl.q, qpos, table=ctl.table)
    ctl.attend()
    torch.cuda.synchronize()
    assert_close(to_np(ctl.o), to_np(fused.o), wl.dtype, "pre-rotated baseline vs fused")
    assert_close(to_np(fused.o), WO.run(wl), wl.dtype, "fused vs oracle")


def test_rope_table_accuracy():
    # float32 tables: (cos, sin) within float32 rounding of the fp64 values; bf16
    # tables: (cos, sin) equal to those values rounded to bf16
    import paper_2606_13126_amd as P
    n = 40000
    p = np.arange(n, dtype=np.float64)[:, None] * O.rope_inv_freq(128, 5e5)[None, :]
    cfg = P.make_config(8, 8, 128, rope_theta=5e5, dtype=P.PIC_F32)
    tab = torch.empty((n, 64, 2), dtype=torch.float32, device="cuda")
    P.pic_rope_table_build(cfg, tab)
    got = tab.cpu().double().numpy()
    assert np.max(np.abs(got[..., 0] - np.cos(p))) <= 1e-7
    assert np.max(np.abs(got[..., 1] - np.sin(p))) <= 1e-7
    cfg = P.make_config(8, 8, 128, rope_theta=5e5, dtype=P.PIC_BF16)
    assert P.pic_rope_table_bytes(cfg, n) == n * 64 * 4
    tab = torch.empty((n, 64), dtype=torch.float32, device="cuda")
    P.pic_rope_table_build(cfg, tab)
    got = tab.cpu().view(torch.bfloat16).double().numpy().reshape(n, 64, 2)   # (cos, sin)
    # values are the fp64 cos/sin rounded to bf16 (the device's fp64 sin may differ
    # from numpy's by an ulp, which can flip a rounding: 1 bf16 ulp)
    for k, ref in ((0, np.cos(p)), (1, np.sin(p))):
        ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-30))) - 7)
        assert np.all(np.abs(got[..., k] - ref) <= ulp)


@pytest.mark.parametrize("Hq,Hkv,D,style,table_len", [
    (8, 8, 64, 0, None),        # MHA, one full group of 8 KV heads
    (16, 16, 64, 1, 0),         # MHA, two head groups, computed cos/sin only
    (40, 10, 128, 0, 2000),     # G = 4, a partial second head group, table + computed
    (32, 2, 128, 1, None),      # G = 16, the widest query group of one MFMA tile (2-wave workgroups)
    (34, 2, 64, 0, None),       # G = 17: two waves per KV head, the second with one query (4-wave workgroups)
    (32, 1, 128, 0, None),      # G = 32 (MQA): two full column blocks, 2-wave workgroups
    (16, 1, 64, 1, 0),          # one KV head, G = 16: 2-wave workgroups, 4 stages, computed cos/sin
    (8, 1, 128, 0, 0),          # one KV head, G = 8: 2-wave workgroups, 2 stages, computed cos/sin
    (28, 4, 128, 1, None),      # four KV heads, G = 7: 4-wave workgroups
    (64, 1, 128, 0, 0),         # one KV head, G = 64: one 4-wave workgroup per head, computed cos/sin
    (15, 3, 128, 0, None),      # three KV heads, G = 5: 4-wave workgroups with an idle head slot
    (1, 1, 64, 1, None),        # one query head: a 2-wave workgroup with an idle head slot
    (48, 1, 64, 1, 0),          # G = 48: four waves per KV head, the last without queries (4-wave workgroups)
    (128, 2, 128, 0, 2000),     # G = 64: four full column blocks, two KV heads per workgroup
    (130, 2, 64, 0, None),      # G = 65: past the decode kernel, the prefill kernel takes it
])
def test_decode_head_groups_and_windows(Hq, Hkv, D, style, table_len):
    wl = decode_case(Hq, Hkv, D, seed=20 + Hq)
    say(f"[gpu] decode Hq={Hq} Hkv={Hkv} D={D} style={style} table_len={table_len}")
    db = gpu_run(wl, rope_style=style, table=table_len != 0, table_len=table_len or None)
    assert_close(to_np(db.o), WO.run(wl, style="neox" if style == 0 else "gptj"), wl.dtype, wl.name)


def test_decode_prerotated_equals_fused():
    # the k_prerotated variant of the decode kernel (the RoPE-cost baseline) gives
    # the fused result when K and q are rotated beforehand (private spans only)
    import paper_2606_13126_amd as P
    from paper_2606_13126_amd.runner import DeviceBatch
    reqs = [[Sp(37, S), Sp(5, S, fresh=True)], [Sp(333, Pd), Sp(1, Pd, fresh=True)], [Sp(64, S), Sp(9, 0, fresh=True)]]
    wl = W.small_case("decode_pre", reqs, Hq=32, Hkv=8, D=128, theta=5e5, dtype=torch.bfloat16, seed=31,
                      value_scale=0.5, decode=True, position_offsets=[3, 900, 17])
    fused = gpu_run(wl)
    ctl = DeviceBatch(wl, k_prerotated=True, table_positions=int(wl.positions.max()) + 1)
    ctl.write()
    kp = ctl.k_pool.permute(0, 2, 1, 3).reshape(-1, wl.num_kv_heads, wl.head_dim)
    off = wl.seq_offsets
    qpos = []
    for r in range(wl.num_reqs):
        L = int(wl.seq_lens[r])
        n = torch.arange(L)
        slots = (torch.from_numpy(wl.block_tables[r].astype(np.int64))[n // 16] * 16 + n % 16).cuda()
        pos = torch.from_numpy(wl.positions[off[r]:off[r + 1]]).cuda()
        rows = kp[slots].contiguous()
        P.pic_rope_rotate(ctl.cfg, rows, pos, table=ctl.table)
        kp[slots] = rows
        qpos.append(int(wl.positions[off[r] + L - 1]))
    ctl.k_pool = kp.reshape(-1, 16, wl.num_kv_heads, wl.head_dim).permute(0, 2, 1, 3).contiguous()
    P.pic_rope_rotate(ctl.cfg, ctl.q, torch.tensor(qpos, dtype=torch.int32, device="cuda"), table=ctl.table)
    ctl.attend()
    torch.cuda.synchronize()
    assert_close(to_np(ctl.o), to_np(fused.o), wl.dtype, "pre-rotated decode vs fused")
    assert_close(to_np(fused.o), WO.run(wl), wl.dtype, "fused decode vs oracle")


@pytest.mark.parametrize("style,table", [(0, True), (1, False)])
def test_decode_fp32(style, table):
    # fp32 decode runs the fp32 kernel (one wave per query and head): max-abs 1e-4
    wl = decode_case(8, 2, 128, seed=17)
    wl.dtype = torch.float32
    for name in ("q", "k_pool", "v_pool", "k_new", "v_new"):
        setattr(wl, name, getattr(wl, name).float())
    check(wl, style=style, table=table, what=f"fp32 decode style={style} table={table}")


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_generalised_windows_prefill(dtype):
    check(windows_prefill_case(dtype), what=f"generalised windows {dtype}")


def test_generalised_windows_decode():
    check(windows_decode_case(), what="generalised windows decode")


# ---- more groups than the kernel arguments hold: the group table goes through the
# workspace (written by plan-upload launches), one attention and one merge launch ----

def shape_of(wl, dtype=None):
    import paper_2606_13126_amd as P
    from paper_2606_13126_amd.runner import config_of
    cfg = config_of(wl)
    return P.pic_plan_shape(cfg, P.HostBatch(wl.seq_lens, wl.cu_spans, wl.span_start, wl.span_flags,
                                             wl.span_window), wl.is_decode)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_many_query_spans_prefill(dtype):
    wl = many_spans_prefill(dtype)
    sh = shape_of(wl)
    say(f"[gpu] many spans {dtype}: {sh}")
    assert sh["groups"] == 82 and sh["upload_launches"] == 2
    if dtype == torch.bfloat16:
        assert sh["merge_blocks"] > 0
    check(wl, what=f"82 query spans {dtype}")


@pytest.mark.parametrize("D", [128, 64])
def test_short_causal_spans_prefill(D):
    # 2,744 short causal row-tile items (ragged last row tiles, idle waves), a window
    # > 0, 122 groups through the workspace table: RoPE from the table and computed,
    # and the pre-rotated kernel with every position 0 (the rotation is the identity)
    from paper_2606_13126_amd.runner import DeviceBatch
    wl = short_causal_spans_prefill(D=D)
    sh = shape_of(wl)
    say(f"[gpu] short causal spans D={D}: {sh}")
    assert sh["groups"] == 122
    ref = WO.run(wl)
    for table in (True, False):
        assert_close(to_np(gpu_run(wl, table=table).o), ref, wl.dtype, f"short causal spans D={D} table={table}")
    wl.positions = np.zeros_like(wl.positions)
    ref0 = WO.run(wl)
    ctl = DeviceBatch(wl, k_prerotated=True, table_positions=None)
    ctl.write()
    ctl.attend()
    torch.cuda.synchronize()
    assert_close(to_np(ctl.o), ref0, wl.dtype, f"short causal spans D={D} pre-rotated kernel, positions 0")


@pytest.mark.parametrize("case", ["decode", "decode_gptj", "prefill", "prefill_fp32"])
def test_long_context(case):
    # 131K-key contexts: decode of 2 requests holding 256 shared spans in their own
    # orders, and a 40-token query tail over 131,072 cached keys (many key splits);
    # RoPE from the table and computed.  (No peaked variant here: at these positions
    # the planted keys' pair has turned by up to 0.3 rad, its rotated values are no
    # longer exact in bf16, and scores of ~100 log2 units carry bf16 rounding errors
    # of ~0.3 units, which the softmax turns into errors far past the tolerance.)
    if case.startswith("decode"):
        wl = long_context_decode()
    else:
        wl = long_context_prefill(dtype=torch.float32 if case == "prefill_fp32" else torch.bfloat16)
    style = 1 if case == "decode_gptj" else 0
    say(f"[gpu] long context {case}: {int(wl.seq_lens.max())} keys, {shape_of(wl)}")
    ref = WO.run(wl, style="gptj" if style else "neox")
    for table in (True, False):
        assert_close(to_np(gpu_run(wl, rope_style=style, table=table).o), ref, wl.dtype,
                     f"long context {case} table={table}")


@pytest.mark.parametrize("Hq,Hkv,D,style", [(32, 8, 128, 0), (34, 2, 64, 1), (32, 1, 128, 0)])
def test_many_requests_decode(Hq, Hkv, D, style):
    wl = many_requests_decode(Hq=Hq, Hkv=Hkv, D=D)
    sh = shape_of(wl)
    say(f"[gpu] 256-request decode Hq={Hq} Hkv={Hkv} D={D}: {sh}")
    assert sh["groups"] == 256 and sh["upload_launches"] == 4
    check(wl, style=style, what=f"256-request decode Hq={Hq} D={D}")


def test_many_requests_decode_fp32():
    wl = many_requests_decode(Hq=8, Hkv=2, D=128)
    wl.dtype = torch.float32
    for name in ("q", "k_pool", "v_pool", "k_new", "v_new"):
        setattr(wl, name, getattr(wl, name).float())
    check(wl, what="256-request decode fp32")


# ---- peaked scores: keys whose alignment with the queries grows along the sequence, so
# the online softmax's running maximum rises by far more than its rescale threshold
# after the first key tile, in unsplit and split prefill, decode and the fp32 path ----

def check_peaked(wl, expect_split, min_frac, style=0, rows=None):
    plant_rising_keys(wl)
    rise = rise_of_max(wl, rows=None if rows is None else set(int(x) for x in rows))
    frac = float(np.nanmean(rise > 8)) if np.any(~np.isnan(rise)) else 0.0
    sh = shape_of(wl)
    say(f"[gpu] peaked {wl.name}: rows whose max rises by >8 (log2) after the first tile: {frac:.2f}, "
        f"largest rise {np.nanmax(rise):.1f}; plan {sh}")
    assert frac >= min_frac, frac
    if expect_split is not None and wl.dtype == torch.bfloat16:
        assert (sh["partial_slots"] > 0) == expect_split, sh
    max_abs, _ = check(wl, style=style, rows=rows, what=f"peaked {wl.name}")
    return max_abs


def test_peaked_prefill_unsplit():
    # 16 requests x 2 row tiles x 8 KV heads fill the chip without key splits
    check_peaked(W.concurrent_reuse(), expect_split=False, min_frac=0.9)


def test_peaked_prefill_split_small():
    wl = W.small_case("peak_small", [[Sp(64, S, key="a"), Sp(300, S | Q, fresh=True), Sp(200, Pd | Q, fresh=True)]],
                      Hq=4, Hkv=2, D=128, theta=5e5, dtype=torch.bfloat16, seed=3, value_scale=0.5)
    check_peaked(wl, expect_split=True, min_frac=0.5)


def test_peaked_llama3_8b_rag_split():
    # 8 key splits per row tile: every split's running maximum moves, and the merge
    # combines splits whose maxima differ by up to ~100 (log2)
    check_peaked(W.llama3_8b_rag(), expect_split=True, min_frac=0.9)


def test_peaked_decode():
    check_peaked(W.decode_64req(num_reqs=16), expect_split=True, min_frac=0.8)


def test_peaked_decode_mixed_windows():
    check_peaked(decode_case(32, 8, 128, seed=71), expect_split=None, min_frac=0.4)


def test_peaked_tiny_fp32():
    check_peaked(W.tiny_fp32(), expect_split=None, min_frac=0.15)


def test_peaked_decode_fp32():
    wl = decode_case(8, 2, 128, seed=72)
    wl.dtype = torch.float32
    for name in ("q", "k_pool", "v_pool", "k_new", "v_new"):
        setattr(wl, name, getattr(wl, name).float())
    check_peaked(wl, expect_split=None, min_frac=0.4)
