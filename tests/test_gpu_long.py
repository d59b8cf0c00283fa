"""Long contexts and the largest decode ranges, on the GPU through the C ABI.

Prefill rows and latent decode pieces stage the block table in LDS windows
of 512 entries (8192 keys at page 16, 32768 at page 64) and drain the tile
pipeline at each window's end; decode stages a whole balanced range, up to
8192 pages. These cases cross windows and use one range for the whole batch
(cus_total = 1 in the plan options), against the fp64 oracle.
"""
import numpy as np
import pytest

import oracle.attention as OA
from paper_2606_04415_amd import flexattn as F
from paper_2606_04415_amd.workloads import WORKLOADS

from gpu_common import check_close, custom_batch, log, run

pytestmark = pytest.mark.gpu

QW = WORKLOADS["decode"]
MLA = WORKLOADS["mla"]


def full_check(b, opts, what):
    w = b.workload
    out, lse, pa = run(b, opts=opts)
    ref_o, ref_l = OA.paged_attention(b.q, b.k_cache, b.v_cache, b.block_table, b.seq_lens, b.query_start_loc,
                                      w.sm_scale, num_kv_heads=w.num_kv_heads, page_size=w.page_size,
                                      head_dim_v=w.head_dim_v, v_aliases_k=w.v_aliases_k)
    rows = ~np.isnan(ref_l[:, 0])
    check_close(out, ref_o, f"{what} out", rows)
    check_close(lse, ref_l, f"{what} lse", rows)
    return pa


def test_prefill_across_page_windows():
    # 70 new tokens after 19930 cached ones: 1250 pages, three LDS windows;
    # plus decodes over 20000 and 8193 keys
    ns, ls = [70, 1, 1], [20000, 20000, 8193]
    b = custom_batch(QW, ns, ls, seed=31)
    log("GQA prefill over 20000 keys (3 block-table windows) + long decodes")
    full_check(b, None, "long-prefill")


def test_one_decode_range_for_the_batch():
    # cus_total = 1: a single balanced range holds every decode page
    ns, ls = [1, 1, 1, 1], [30000, 5000, 17, 80]
    pages = sum(-(-L // QW.page_size) for L in ls)      # 1875 + 313 + 2 + 5 = 2195
    b = custom_batch(QW, ns, ls, seed=32)
    log(f"GQA decode, one range of {pages} pages")
    pa = full_check(b, F.make_opts(cus_total=1), "one-range")
    assert pa.plan.info["n_decode_ranges"] == 1 and pa.plan.info["pages_per_split"] == pages


def test_latent_decode_across_page_windows():
    # 40000 keys at page 64: 625 pages, two windows of a latent decode piece
    ns, ls = [1, 1], [40000, 300]
    b = custom_batch(MLA, ns, ls, seed=33)
    log("latent decode over 40000 keys (2 block-table windows), one range")
    pa = full_check(b, F.make_opts(cus_total=1, wg_per_cu=1), "latent-long")
    assert pa.plan.info["n_decode_ranges"] == 1 and pa.plan.info["n_split_seqs"] == 0
