"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Small batches (several tiles, ragged tails, split decode sequences) and the
decode, prefill and mixed workloads at full size are compared in full: every
output and log-sum-exp element, with the mean-error clause taken over the
whole tensor. The latent workloads at full size are compared on every decode
row and every 4th prefill row (all heads): their prefill chunk alone is
about 2.3 TFLOP of fp64 work for the oracle. Unused pages hold NaN and tail
slots hold +/-1e4 (see workloads.make_batch), so a wrong page index or an
unmasked tail read breaks parity.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle.attention as OA
from paper_2606_04415_amd import flexattn as F
from paper_2606_04415_amd.workloads import WORKLOADS, make_batch

from gpu_common import check_close, custom_batch, device_inputs, log, run

pytestmark = pytest.mark.gpu

QW = WORKLOADS["decode"]     # Qwen2.5-7B geometry
TINY = WORKLOADS["tiny"]
MLA = WORKLOADS["mla"]


def oracle_full(b):
    w = b.workload
    return OA.paged_attention(b.q, b.k_cache, b.v_cache, b.block_table, b.seq_lens, b.query_start_loc,
                              w.sm_scale, num_kv_heads=w.num_kv_heads, page_size=w.page_size,
                              head_dim_v=w.head_dim_v, v_aliases_k=w.v_aliases_k)


def full_check(b, opts=None, what=""):
    out, lse, _ = run(b, opts=opts)
    ref_o, ref_l = oracle_full(b)
    rows = ~np.isnan(ref_l[:, 0])
    check_close(out, ref_o, f"{what} out", rows)
    check_close(lse, ref_l, f"{what} lse", rows)
    return out, lse


def test_tiny_workload_full():
    log("tiny mixed workload (2 prompts x 64 + 4 decodes x 128, GQA 4/1, d 64, page 16)")
    b = make_batch(TINY, seed=0)
    full_check(b, what="tiny")


RAGGED_GQA = [
    # (n, L) per sequence: decodes over ragged contexts, chunked and whole prompts, an empty sequence
    ([1, 1, 1, 1, 1, 1, 1, 0, 200, 100, 2, 129, 1], [1, 15, 16, 17, 129, 1000, 4095, 7, 200, 300, 5, 129, 33]),
]


@pytest.mark.parametrize("min_split", [0, 16])
def test_ragged_gqa_d128_page16(min_split):
    ns, ls = RAGGED_GQA[0]
    b = custom_batch(QW, ns, ls, seed=3)
    opts = F.make_opts(min_split_tokens=min_split)
    log(f"ragged GQA 28/4 d128 page16, min_split_tokens={min_split}")
    full_check(b, opts, "ragged-d128")


def test_decode_ranges_cross_many_pieces():
    """48 decodes of 1 to ~300 keys planned for a 32-CU share: each balanced
    range spans many pieces, so a wave changes piece (finishes one, loads the
    next one's Q) between most chunks, and a wave's prefetch often runs past
    the end of its range."""
    ls = [1 + (37 * i) % 300 for i in range(48)]
    b = custom_batch(QW, [1] * 48, ls, seed=8)
    log("48 short decodes, ranges planned for 32 CUs")
    full_check(b, F.make_opts(cus_decode=32, min_split_tokens=16), "many-pieces")


def test_ragged_gqa_d64_page64_group16():
    ns = [1, 1, 1, 70, 1, 130, 3]
    ls = [1, 63, 65, 70, 2000, 400, 3]
    b = custom_batch(QW, ns, ls, seed=4, num_q_heads=32, num_kv_heads=2, head_dim_qk=64, head_dim_v=64,
                     page_size=64, sm_scale=0.125)
    log("ragged GQA 32/2 (group 16) d64 page64")
    full_check(b, F.make_opts(min_split_tokens=64), "ragged-d64")


def test_gqa_bm16_tiles():
    ns, ls = [77, 1, 150], [77, 500, 300]
    b = custom_batch(QW, ns, ls, seed=5)
    log("GQA prefill with 16-row tiles")
    full_check(b, F.make_opts(bm=16), "bm16")


@pytest.mark.parametrize("hq", [64, 128])
def test_ragged_latent(hq):
    ns = [1, 1, 1, 1, 130, 70, 1]
    ls = [1, 63, 65, 3000, 130, 200, 700]
    b = custom_batch(MLA, ns, ls, seed=6, num_q_heads=hq)
    log(f"ragged latent 576/512 page64, {hq} heads, forced splits")
    full_check(b, F.make_opts(min_split_tokens=128), f"latent-h{hq}")


def test_single_key_is_exact():
    """L = 1: the one weight is exactly 1, so out must equal V[0] bit for bit."""
    b = custom_batch(QW, [1, 1], [1, 1], seed=7)
    out, _, _ = run(b)
    for s in range(2):
        page = int(b.block_table[s, 0])
        v0 = b.v_cache[page, 0]                       # [Hkv, d]
        ref = v0.repeat_interleave(QW.num_q_heads // QW.num_kv_heads, 0)
        assert torch.equal(out[s], ref)


@pytest.mark.parametrize("name", ["tiny", "decode", "prefill", "mixed", "mla", "mla_split"])
def test_gather_bit_exact(name):
    """The block-table contract itself: the debug gather's copy of every
    sequence's key (and value) rows equals a host fancy-index gather, bit for
    bit, on every workload (the latent one with its values aliasing the keys).
    The gather uses a plain per-element page lookup; the attention kernels'
    own addressing is pinned by the NaN-poisoned unused pages of every parity
    test and by test_page_permutation_bitwise."""
    w = WORKLOADS[name]
    b = make_batch(w, seed=0)
    d = device_inputs(b)
    pa = F.PagedAttention(F.make_shape(w.num_q_heads, w.num_kv_heads, w.head_dim_qk, w.head_dim_v,
                                       w.page_size, w.sm_scale, w.v_aliases_k), None,
                          b.query_start_loc.tolist(), b.seq_lens.tolist(), b.block_table.shape[1])
    out, _ = pa.alloc_out(d["q"])
    args = pa.args(d["q"], d["k_cache"], d["v_cache"], d["block_table"], d["seq_lens"],
                   d["query_start_loc"], out)
    log(f"{name}: gather every sequence ({len(b.seq_lens)})")
    for s in range(len(b.seq_lens)):
        L = int(b.seq_lens[s])
        ko = torch.empty((L, w.num_kv_heads, w.head_dim_qk), dtype=torch.bfloat16, device="cuda")
        vo = None if w.v_aliases_k else torch.empty((L, w.num_kv_heads, w.head_dim_v), dtype=torch.bfloat16,
                                                    device="cuda")
        F.flex_attn_debug_gather(pa.plan, args, s, L, ko, vo)
        t = torch.arange(L)
        pages = b.block_table[s, t // w.page_size].long()
        kref = b.k_cache[pages, t % w.page_size]
        torch.cuda.synchronize()
        assert torch.equal(ko.cpu().view(torch.int16), kref.view(torch.int16)), f"K of seq {s}"
        if vo is not None:
            vref = b.v_cache[pages, t % w.page_size]
            assert torch.equal(vo.cpu().view(torch.int16), vref.view(torch.int16)), f"V of seq {s}"


def test_page_permutation_bitwise():
    """Same logical batch in two physical page orders: bit-identical outputs."""
    ns, ls = [1, 1, 60, 1], [700, 31, 90, 2000]
    b1 = custom_batch(QW, ns, ls, seed=8)
    b2 = custom_batch(QW, ns, ls, seed=8)
    # re-place b1's logical pages at a new permutation in b2
    rng = torch.Generator().manual_seed(99)
    perm = torch.randperm(b1.k_cache.shape[0], generator=rng)
    b2.k_cache = torch.empty_like(b1.k_cache)
    b2.v_cache = torch.empty_like(b1.v_cache)
    b2.k_cache[perm] = b1.k_cache
    b2.v_cache[perm] = b1.v_cache
    b2.block_table = perm[b1.block_table.long()].to(torch.int32)
    o1, l1, _ = run(b1)
    o2, l2, _ = run(b2)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1, l2)


def test_run_to_run_bitwise():
    ns, ls = RAGGED_GQA[0]
    b = custom_batch(QW, ns, ls, seed=9)
    opts = F.make_opts(min_split_tokens=16)
    o1, l1, pa = run(b, opts=opts)
    d = device_inputs(b)
    o2, l2, _ = run(b, d=d, pa=pa)
    o3, l3, _ = run(b, d=d, pa=pa)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(o2.view(torch.int16), o3.view(torch.int16))
    assert torch.equal(l1, l3)


@pytest.mark.parametrize("split", [(128, 128), (192, 64), (64, 192)])
def test_corun_bitwise_equals_serial(split):
    cp, cd = split
    ns, ls = [300, 1, 1, 1, 1, 120], [900, 1000, 17, 4000, 2500, 120]
    b = custom_batch(QW, ns, ls, seed=10)
    opts = F.make_opts(cus_decode=cd)
    log(f"co-run prefill {cp} CUs / decode {cd} CUs vs serial")
    d = device_inputs(b)
    o_s, l_s, pa = run(b, d=d, opts=opts)
    corun = F.Corun(cp, cd)
    o_c, l_c, _ = run(b, d=d, pa=pa, mode=F.FLEX_MODE_CORUN, corun=corun)
    assert torch.equal(o_s.view(torch.int16), o_c.view(torch.int16))
    assert torch.equal(l_s, l_c)
    ref_o, ref_l = oracle_full(b)
    check_close(o_c, ref_o, "corun out", ~np.isnan(ref_l[:, 0]))
    corun.close()


def workload_run(name, w=None, modes=(F.FLEX_MODE_SERIAL,), split=(128, 128)):
    """Draw the full-size workload, run it in each mode on one plan (the plan
    partitioned for the co-run split when co-run is among the modes), and
    check that every mode's output is bit-identical to the first's."""
    w = w or WORKLOADS[name]
    log(f"{name}: drawing the full-size batch")
    b = make_batch(w, seed=0)
    d = device_inputs(b)
    opts = F.make_opts(cus_decode=split[1]) if F.FLEX_MODE_CORUN in modes else None
    corun = F.Corun(*split) if F.FLEX_MODE_CORUN in modes else None
    outs = []
    pa = None
    for mode in modes:
        out, lse, pa = run(b, d=d, mode=mode, opts=opts, corun=corun, pa=pa)
        log(f"{name}: mode {mode}: plan {pa.plan.info['n_decode_items']} decode items, "
            f"{pa.plan.info['n_prefill_items']} tiles (bm {pa.plan.info['bm']})")
        outs.append((out, lse))
    for out, lse in outs[1:]:
        assert torch.equal(out.view(torch.int16), outs[0][0].view(torch.int16))
        assert torch.equal(lse, outs[0][1])
    if corun is not None:
        corun.close()
    return b, outs[0][0], outs[0][1]


@pytest.mark.parametrize("name", ["decode", "prefill"])
def test_full_workload(name):
    """Every output and lse element of the decode and prefill workloads."""
    b, out, lse = workload_run(name)
    log(f"{name}: fp64 oracle over the whole batch")
    ref_o, ref_l = oracle_full(b)
    check_close(out, ref_o, f"{name} out (all rows)")
    check_close(lse, ref_l, f"{name} lse (all rows)")


def test_full_mixed_all_modes():
    """The mixed step in serial, co-run (128/128) and one-launch form: the three
    outputs bit-identical, and every element against the oracle."""
    b, out, lse = workload_run("mixed", modes=(F.FLEX_MODE_SERIAL, F.FLEX_MODE_CORUN, F.FLEX_MODE_FUSED))
    log("mixed: fp64 oracle over the whole batch")
    ref_o, ref_l = oracle_full(b)
    check_close(out, ref_o, "mixed out (all rows)")
    check_close(lse, ref_l, "mixed lse (all rows)")


def latent_rows_check(name, stride=4):
    """Every decode row and every stride-th prefill row (all heads) of a latent workload."""
    b, out, lse = workload_run(name)
    w = b.workload
    qsl = b.query_start_loc.tolist()
    ls = b.seq_lens.tolist()
    picks = []
    for s in range(len(ls)):
        n = qsl[s + 1] - qsl[s]
        if n == 1 and w.head_dim_qk != 192:
            picks.append((s, 0))
        elif n >= 1:
            picks += [(s, i) for i in range(0, n, stride)] + ([(s, n - 1)] if (n - 1) % stride else [])
    log(f"{name}: fp64 oracle on {len(picks)} rows")
    ref_o, ref_l = OA.attention_rows(b.q, b.k_cache, b.v_cache, b.block_table, b.seq_lens, b.query_start_loc,
                                     w.sm_scale, picks, num_kv_heads=w.num_kv_heads, page_size=w.page_size,
                                     head_dim_v=w.head_dim_v, v_aliases_k=w.v_aliases_k)
    idx = [qsl[s] + i for s, i in picks]
    check_close(out[idx], ref_o, f"{name} out ({len(picks)} rows: every decode row, every {stride}th prefill row)")
    check_close(lse[idx], ref_l, f"{name} lse")


def test_full_latent_rows():
    latent_rows_check("mla")


SPLIT = WORKLOADS["mla_split"]


def test_split_head_latent_prefill_ragged():
    # keys 192, values 128, two query heads per KV head; prefill only: the one-token
    # sequences run as prefill tiles too; ragged 128-token tiles, an empty sequence
    ns, ls = [1, 130, 5, 0, 64, 300], [70, 130, 200, 10, 300, 700]
    b = custom_batch(SPLIT, ns, ls, seed=7, num_q_heads=8, num_kv_heads=4)
    log("split-head latent prefill 8/4 heads, 192/128, page 64, ragged")
    out, lse = full_check(b, what="split-head")
    _, _, pa = run(b)
    assert pa.plan.info["n_decode_items"] == 0 and pa.plan.info["n_prefill_seqs"] == 5


def test_full_split_head_latent_rows():
    latent_rows_check("mla_split")


@pytest.mark.parametrize("mode", ["serial", "corun", "fused"])
def test_batch_without_query_tokens(mode):
    """Every sequence has context but no new token: each mode returns at once
    with an empty output and nothing launched."""
    b = custom_batch(QW, [0, 0, 0], [40, 0, 7], seed=11)
    corun = F.Corun(128, 128) if mode == "corun" else None
    m = {"serial": F.FLEX_MODE_SERIAL, "corun": F.FLEX_MODE_CORUN, "fused": F.FLEX_MODE_FUSED}[mode]
    log(f"batch with no query tokens, mode {mode}")
    out, lse, pa = run(b, mode=m, corun=corun)
    assert out.shape == (0, QW.num_q_heads, QW.head_dim_v) and lse.shape == (0, QW.num_q_heads)
    assert pa.plan.info["n_decode_items"] == 0 and pa.plan.info["n_prefill_items"] == 0
    if corun is not None:
        corun.close()


@pytest.mark.parametrize("bm", [32, 16])
@pytest.mark.parametrize("d", [128, 64])
def test_narrow_group_prefill_tiles(bm, d):
    """Four query heads per KV head (the 4- and 8-wave prefill forms, 32-key
    tiles) over ragged chunks, both head sizes and tile heights."""
    ns, ls = [1, 77, 1, 150, 33], [500, 77, 40, 300, 1000]
    b = custom_batch(QW, ns, ls, seed=12, num_q_heads=16, num_kv_heads=4, head_dim_qk=d, head_dim_v=d,
                     sm_scale=d ** -0.5)
    log(f"narrow GQA 16/4 d{d} page16, bm {bm}")
    full_check(b, F.make_opts(bm=bm), f"narrow-d{d}-bm{bm}")


def test_full_prefill_narrow_group():
    """The 8 x 2048 causal prefill with 16 query heads on the 4 KV heads (the
    narrow-group forms), every element."""
    w = dataclasses.replace(WORKLOADS["prefill"], num_q_heads=16, name="prefill-16/4")
    b, out, lse = workload_run("prefill-16/4", w=w)
    ref_o, ref_l = oracle_full(b)
    check_close(out, ref_o, "prefill-16/4 out (all rows)")
    check_close(lse, ref_l, "prefill-16/4 lse (all rows)")


# Shapes the plan accepts beyond the five workloads: one, two and three query
# heads per KV head, head dim 64 at page 64, the latent layout at page 16;
# every tile height the plan takes, on ragged batches with split decodes.
ACCEPTED = [
    dict(num_q_heads=8, num_kv_heads=8, head_dim_qk=128, head_dim_v=128, page_size=16),   # G = 1
    dict(num_q_heads=8, num_kv_heads=4, head_dim_qk=128, head_dim_v=128, page_size=16),   # G = 2
    dict(num_q_heads=12, num_kv_heads=4, head_dim_qk=64, head_dim_v=64, page_size=16),    # G = 3
    dict(num_q_heads=20, num_kv_heads=4, head_dim_qk=64, head_dim_v=64, page_size=64),    # G = 5, page 64
    dict(num_q_heads=48, num_kv_heads=3, head_dim_qk=128, head_dim_v=128, page_size=64),  # G = 16, 3 KV heads
]


@pytest.mark.parametrize("bm", [0, 16, 32, 128])
@pytest.mark.parametrize("geo", range(len(ACCEPTED)))
def test_accepted_gqa_shapes(geo, bm):
    g = ACCEPTED[geo]
    d = g["head_dim_qk"]
    ns, ls = [1, 77, 1, 150, 33, 1, 2, 0], [500, 77, 40, 300, 1000, 2049, 9, 5]
    b = custom_batch(QW, ns, ls, seed=40 + geo, sm_scale=d ** -0.5, **g)
    log(f"GQA {g['num_q_heads']}/{g['num_kv_heads']} d{d} page {g['page_size']}, bm {bm}")
    full_check(b, F.make_opts(bm=bm, min_split_tokens=64), f"gqa-{geo}-bm{bm}")


@pytest.mark.parametrize("page", [64, 16])
def test_latent_prefill_64_row_tiles(page):
    """Latent prefill on 64-row tiles (four waves over two LDS stages, two
    work-groups per CU) on ragged chunks at both page sizes, with split
    decodes in the same batch."""
    ns, ls = [1, 130, 70, 1, 200, 64], [900, 130, 300, 65, 2000, 64]
    b = custom_batch(MLA, ns, ls, seed=61, page_size=page)
    log(f"latent prefill bm 64, page {page}")
    full_check(b, F.make_opts(bm=64, min_split_tokens=128), f"latent-bm64-p{page}")


@pytest.mark.parametrize("hq", [64, 128])
def test_latent_page16(hq):
    ns, ls = [1, 1, 1, 100, 1, 40], [1, 33, 700, 130, 2000, 40]
    b = custom_batch(MLA, ns, ls, seed=50, num_q_heads=hq, page_size=16)
    log(f"latent 576/512 page 16, {hq} heads, forced splits")
    full_check(b, F.make_opts(min_split_tokens=64), f"latent-p16-h{hq}")
