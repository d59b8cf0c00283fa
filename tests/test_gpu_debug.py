"""Debug mode on the GPU (flex_attn_set_debug): the check kernel refuses a
block-table entry outside the pool and device lengths that differ from the
plan's before any attention kernel runs (the output stays as it was), and
passes a good batch, whose result then matches the oracle. Also: a co-run
call whose pair's split differs from the plan's is refused."""
import numpy as np
import pytest
import torch

import oracle.attention as OA
from paper_2606_04415_amd import flexattn as F
from paper_2606_04415_amd.workloads import WORKLOADS

from gpu_common import check_close, custom_batch, device_inputs, log, shape_of

pytestmark = pytest.mark.gpu

QW = WORKLOADS["decode"]


@pytest.fixture
def debug_on():
    prev = F.set_debug(1)
    yield
    F.set_debug(prev)


def setup(seed=70):
    ns, ls = [1, 100, 1, 1], [700, 300, 33, 2000]
    b = custom_batch(QW, ns, ls, seed=seed)
    d = device_inputs(b)
    # the caches are views of the first num_pages pages of larger buffers, so
    # that even an unchecked read of page num_pages stays inside memory
    for key in ("k_cache", "v_cache"):
        t = d[key]
        big = torch.cat([t, torch.zeros((4,) + tuple(t.shape[1:]), dtype=t.dtype, device=t.device)])
        d[key] = big[:t.shape[0]]
    pa = F.PagedAttention(shape_of(b.workload), F.make_opts(min_split_tokens=64), b.query_start_loc.tolist(),
                          b.seq_lens.tolist(), b.block_table.shape[1])
    out, lse = pa.alloc_out(d["q"], True)
    out.fill_(float("nan"))
    return b, d, pa, out, lse


def run_args(pa, d, out, lse, **over):
    t = dict(d)
    t.update(over)
    return pa.args(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["seq_lens"], t["query_start_loc"], out, lse)


@pytest.mark.parametrize("mode", ["decode", "prefill", "mixed", "mixed_static"])
def test_debug_refuses_bad_block_table_entry(debug_on, mode):
    b, d, pa, out, lse = setup()
    bt = d["block_table"].clone()
    bt[3, 5] = b.num_pages          # one past the pool, inside sequence 3's pages
    a = run_args(pa, d, out, lse, block_table=bt)
    fn = {"decode": lambda: F.flex_attn_decode(pa.plan, a), "prefill": lambda: F.flex_attn_prefill(pa.plan, a),
          "mixed": lambda: F.flex_attn_mixed(pa.plan, a, F.FLEX_MODE_SERIAL),
          "mixed_static": lambda: F.flex_attn_mixed_static(pa.plan, a, F.FLEX_MODE_SERIAL)}[mode]
    log(f"debug mode, {mode}: block-table entry past the pool")
    with pytest.raises(F.FlexAttnError) as e:
        fn()
    assert e.value.status == F.FLEX_ERR_INVALID_ARG and "sequence 3" in str(e.value)
    torch.cuda.synchronize()
    assert torch.isnan(out.float()).all()      # nothing was launched


def test_debug_refuses_mismatched_lengths(debug_on):
    b, d, pa, out, lse = setup()
    sl = d["seq_lens"].clone()
    sl[2] += 1
    log("debug mode: device seq_lens differ from the plan's")
    with pytest.raises(F.FlexAttnError) as e:
        F.flex_attn_mixed(pa.plan, run_args(pa, d, out, lse, seq_lens=sl), F.FLEX_MODE_SERIAL)
    assert "seq_lens" in str(e.value) and "sequence 2" in str(e.value)
    qsl = d["query_start_loc"].clone()
    qsl[2] += 1
    with pytest.raises(F.FlexAttnError) as e:
        F.flex_attn_mixed(pa.plan, run_args(pa, d, out, lse, query_start_loc=qsl), F.FLEX_MODE_SERIAL)
    assert "query_start_loc" in str(e.value)
    torch.cuda.synchronize()
    assert torch.isnan(out.float()).all()


def test_debug_passes_a_good_batch(debug_on):
    b, d, pa, out, lse = setup()
    F.flex_attn_mixed(pa.plan, run_args(pa, d, out, lse), F.FLEX_MODE_SERIAL)
    torch.cuda.synchronize()
    w = b.workload
    ref_o, ref_l = OA.paged_attention(b.q, b.k_cache, b.v_cache, b.block_table, b.seq_lens, b.query_start_loc,
                                      w.sm_scale, num_kv_heads=w.num_kv_heads, page_size=w.page_size)
    rows = ~np.isnan(ref_l[:, 0])
    check_close(out.cpu(), ref_o, "debug-mode out", rows)
    check_close(lse.cpu(), ref_l, "debug-mode lse", rows)


def test_corun_split_mismatch_is_refused():
    b, d, pa, out, lse = setup()          # plan partitioned for all CUs
    corun = F.Corun(128, 128)
    s = torch.cuda.Stream()
    with pytest.raises(F.FlexAttnError) as e:
        F.flex_attn_mixed(pa.plan, run_args(pa, d, out, lse), F.FLEX_MODE_CORUN, stream=s.cuda_stream, corun=corun)
    assert e.value.status == F.FLEX_ERR_INVALID_ARG and "partitioned" in str(e.value)
    corun.close()
