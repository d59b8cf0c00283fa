"""The allocation-free entry point (flex_attn_mixed_static) against
flex_attn_mixed, through the C ABI: bit-identical outputs on two calls in a
row, the second on a smaller batch, so the fixed scratch is reused with the
previous call's contents still in it; and the size limit."""
import pytest
import torch

from paper_2606_04415_amd import flexattn as F
from paper_2606_04415_amd.workloads import WORKLOADS

from gpu_common import custom_batch, device_inputs, log, shape_of

pytestmark = pytest.mark.gpu

QW = WORKLOADS["decode"]


def both(b, mode, opts, corun=None):
    w = b.workload
    d = device_inputs(b)
    pa = F.PagedAttention(shape_of(w), opts, b.query_start_loc.tolist(), b.seq_lens.tolist(), b.block_table.shape[1])
    res = []
    for fn in (F.flex_attn_mixed, F.flex_attn_mixed_static):
        out, lse = pa.alloc_out(d["q"], True)
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        args = pa.args(d["q"], d["k_cache"], d["v_cache"], d["block_table"], d["seq_lens"],
                       d["query_start_loc"], out, lse)
        if fn is F.flex_attn_mixed_static:
            args.workspace = None          # ignored by the allocation-free call
            args.workspace_bytes = 0
        fn(pa.plan, args, mode, corun=corun)
        torch.cuda.synchronize()
        res.append((out.cpu(), lse.cpu()))
    return res, pa


@pytest.mark.parametrize("mode", [F.FLEX_MODE_SERIAL, F.FLEX_MODE_CORUN, F.FLEX_MODE_FUSED])
def test_static_equals_workspace_call_twice(mode):
    corun = F.Corun(128, 128) if mode == F.FLEX_MODE_CORUN else None
    opts = F.make_opts(min_split_tokens=64, cus_decode=128 if corun else 0)
    for k, (ns, ls) in enumerate((([1, 1, 1, 300, 1, 1], [3000, 17, 4000, 900, 2500, 129]),
                                  ([1, 40, 1], [700, 40, 1000]))):   # second call: a smaller batch
        b = custom_batch(QW, ns, ls, seed=60 + k)
        (o_ref, l_ref), (o_st, l_st) = both(b, mode, opts, corun)[0]
        log(f"mode {mode} call {k}: {b.total_q} rows, static scratch vs workspace")
        assert torch.equal(o_st.view(torch.int16), o_ref.view(torch.int16))
        assert torch.equal(l_st, l_ref)
    if corun is not None:
        corun.close()


def test_static_rejects_plans_beyond_the_scratch():
    # enough split decode pieces (one page each) that the partials exceed the fixed scratch
    ns, ls = [1] * 4, [10000] * 4
    b = custom_batch(QW, ns, ls, seed=62)
    pa = F.PagedAttention(shape_of(b.workload), F.make_opts(min_split_tokens=16, wg_per_cu=64),
                          b.query_start_loc.tolist(), b.seq_lens.tolist(), b.block_table.shape[1])
    assert pa.plan.info["workspace_bytes"] > F.static_scratch_bytes()
    d = device_inputs(b)
    out, _ = pa.alloc_out(d["q"])
    args = pa.args(d["q"], d["k_cache"], d["v_cache"], d["block_table"], d["seq_lens"], d["query_start_loc"], out)
    with pytest.raises(F.FlexAttnError) as e:
        F.flex_attn_mixed_static(pa.plan, args, F.FLEX_MODE_SERIAL)
    assert e.value.status == F.FLEX_ERR_WORKSPACE
