"""One-launch mixed step (FLEX_MODE_FUSED) on the GPU, through the C ABI.

The fused launch runs the same per-row arithmetic as the two-launch path, so
under one plan its outputs must be bit-identical to SERIAL mode; it is also
held to the fp64 oracle. Shapes cover two decode ranges per work-group
(Hkv <= 4), one (5..8 KV heads), a prefill column count that does not divide
8 (round-robin placement), pages of 16 and 64, head dims 64 and 128,
split decode sequences, a phase with no work, and the full mixed workload.
"""
import numpy as np
import pytest
import torch

import oracle.attention as OA
from paper_2606_04415_amd import flexattn as F
from paper_2606_04415_amd.workloads import WORKLOADS, make_batch

from gpu_common import check_close, custom_batch, device_inputs, log, run

pytestmark = pytest.mark.gpu

QW = WORKLOADS["decode"]     # Qwen2.5-7B geometry: 28 query heads, 4 KV heads, d 128, page 16


def oracle_full(b):
    w = b.workload
    return OA.paged_attention(b.q, b.k_cache, b.v_cache, b.block_table, b.seq_lens, b.query_start_loc,
                              w.sm_scale, num_kv_heads=w.num_kv_heads, page_size=w.page_size,
                              head_dim_v=w.head_dim_v, v_aliases_k=w.v_aliases_k)


def fused_vs_serial(b, opts=None, oracle=True, what=""):
    d = device_inputs(b)
    o_s, l_s, pa = run(b, d=d, opts=opts)
    assert pa.plan.info["n_fused_wgs"] > 0
    o_f, l_f, _ = run(b, d=d, pa=pa, mode=F.FLEX_MODE_FUSED)
    o_f2, l_f2, _ = run(b, d=d, pa=pa, mode=F.FLEX_MODE_FUSED)
    assert torch.equal(o_s.view(torch.int16), o_f.view(torch.int16)), f"{what}: fused != serial"
    assert torch.equal(l_s, l_f), f"{what}: fused lse != serial"
    assert torch.equal(o_f.view(torch.int16), o_f2.view(torch.int16)) and torch.equal(l_f, l_f2)
    if oracle:
        ref_o, ref_l = oracle_full(b)
        rows = ~np.isnan(ref_l[:, 0])
        check_close(o_f, ref_o, f"{what} fused out", rows)
        check_close(l_f, ref_l, f"{what} fused lse", rows)
    return pa


@pytest.mark.parametrize("wgpc", [1, 4])
def test_fused_qwen_ragged(wgpc):
    ns = [1, 1, 1, 1, 1, 1, 1, 0, 200, 100, 2, 129, 1, 33]
    ls = [1, 15, 16, 17, 129, 1000, 4095, 7, 200, 300, 5, 129, 33, 2000]
    b = custom_batch(QW, ns, ls, seed=21)
    log(f"fused 28/4 d128 page16, wg_per_cu={wgpc}, ragged prefill + split decodes")
    pa = fused_vs_serial(b, F.make_opts(min_split_tokens=16, wg_per_cu=wgpc), what=f"qwen-wgpc{wgpc}")
    assert pa.plan.info["n_split_seqs"] > 0


def test_fused_one_range_per_wg_and_round_robin_columns():
    # 40/5: G = 8, five KV heads -> one decode range per work-group; five
    # prefill columns do not divide 8 -> entries placed round-robin
    ns, ls = [1, 70, 1, 1, 130, 1], [63, 70, 2000, 700, 400, 5]
    b = custom_batch(QW, ns, ls, seed=22, num_q_heads=40, num_kv_heads=5, head_dim_qk=64, head_dim_v=64,
                     sm_scale=0.125)
    log("fused 40/5 d64 page16")
    fused_vs_serial(b, F.make_opts(min_split_tokens=64), what="40/5")


def test_fused_group16_page64():
    # 48/3: G = 16 -> two prefill work-groups per KV head (6 columns)
    ns, ls = [1, 90, 1, 1, 3], [300, 90, 1500, 64, 3]
    b = custom_batch(QW, ns, ls, seed=23, num_q_heads=48, num_kv_heads=3, page_size=64, sm_scale=0.09)
    log("fused 48/3 d128 page64")
    fused_vs_serial(b, F.make_opts(min_split_tokens=64, wg_per_cu=2), what="48/3")


@pytest.mark.parametrize("ns,ls", [([1, 1, 1], [500, 17, 3000]), ([64, 40], [64, 100])])
def test_fused_single_phase(ns, ls):
    b = custom_batch(QW, ns, ls, seed=24)
    log(f"fused with one phase only: n={ns}")
    fused_vs_serial(b, F.make_opts(min_split_tokens=16), what="one-phase")


def test_fused_unsupported_shape_is_an_error():
    b = make_batch(WORKLOADS["tiny"], seed=0)   # 4 query heads per KV head: no one-launch form
    d = device_inputs(b)
    _, _, pa = run(b, d=d)
    assert pa.plan.info["n_fused_wgs"] == 0
    out, lse = pa.alloc_out(d["q"])
    args = pa.args(d["q"], d["k_cache"], d["v_cache"], d["block_table"], d["seq_lens"], d["query_start_loc"],
                   out, lse)
    with pytest.raises(F.FlexAttnError) as e:
        F.flex_attn_mixed(pa.plan, args, F.FLEX_MODE_FUSED)
    assert e.value.status == F.FLEX_ERR_UNSUPPORTED


def test_fused_full_mixed_workload():
    w = WORKLOADS["mixed"]
    log("mixed: full-size batch, fused vs serial bitwise, sampled oracle rows")
    b = make_batch(w, seed=0)
    d = device_inputs(b)
    opts = F.make_opts(wg_per_cu=4)
    o_s, l_s, pa = run(b, d=d, opts=opts)
    o_f, l_f, _ = run(b, d=d, pa=pa, mode=F.FLEX_MODE_FUSED)
    assert torch.equal(o_s.view(torch.int16), o_f.view(torch.int16))
    assert torch.equal(l_s, l_f)
    qsl, ls = b.query_start_loc.tolist(), b.seq_lens.tolist()
    picks = [(0, r) for r in (0, 1, 31, 32, 1000, 2047)] + [(s, 0) for s in (1, 2, 64, 128)]
    ref_o, ref_l = OA.attention_rows(b.q, b.k_cache, b.v_cache, b.block_table, b.seq_lens, b.query_start_loc,
                                     w.sm_scale, picks, num_kv_heads=w.num_kv_heads, page_size=w.page_size,
                                     head_dim_v=w.head_dim_v, v_aliases_k=w.v_aliases_k)
    idx = [qsl[s] + i for s, i in picks]
    check_close(o_f[idx], ref_o, "mixed fused sampled out")
    check_close(l_f[idx], ref_l, "mixed fused sampled lse")
