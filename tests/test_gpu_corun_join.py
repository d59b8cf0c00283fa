"""Co-run steps joined by step counters (short steps) and by events (steps the
plan's work puts at a millisecond or more) on one co-run pair: alternating
the two kinds must neither stall nor change results, so every co-run output
is compared bit for bit with the serial run of the same plan, and the first
of each kind is checked against the fp64 oracle on sampled rows."""
import pytest
import torch

import oracle.attention as OA
from paper_2606_04415_amd import flexattn as F
from paper_2606_04415_amd.workloads import WORKLOADS

from gpu_common import check_close, custom_batch, device_inputs, log, run

QW = WORKLOADS["decode"]
MLA = WORKLOADS["mla"]


def _sampled_oracle(b, out, lse, picks, what):
    w = b.workload
    ref_o, ref_l = OA.attention_rows(b.q, b.k_cache, b.v_cache, b.block_table, b.seq_lens, b.query_start_loc,
                                     w.sm_scale, picks, num_kv_heads=w.num_kv_heads, page_size=w.page_size,
                                     head_dim_v=w.head_dim_v, v_aliases_k=w.v_aliases_k)
    qsl = b.query_start_loc.tolist()
    idx = [qsl[s] + i for s, i in picks]
    check_close(out[idx], ref_o, f"{what} out ({len(picks)} rows)")
    check_close(lse[idx], ref_l, f"{what} lse")


@pytest.mark.gpu
def test_short_and_long_steps_share_a_pair():
    # short: Qwen-shaped step (well under a millisecond on 192/64 CUs);
    # long: latent step with a 4096-token prompt (about 4 ms of prefill on 192 CUs)
    short = custom_batch(QW, [1] * 24 + [256], [700 + 37 * i for i in range(24)] + [1280], seed=70)
    long_ = custom_batch(MLA, [1] * 16 + [4096], [1500 + 211 * i for i in range(16)] + [4096], seed=71)
    pair = F.Corun(192, 64)
    opts = F.make_opts(cus_decode=64)
    plans = {}
    ref = {}
    for name, b in (("short", short), ("long", long_)):
        d = device_inputs(b)
        out, lse, pa = run(b, d=d, mode=F.FLEX_MODE_SERIAL, opts=opts)
        plans[name] = (b, d, pa)
        ref[name] = (out, lse)
        log(f"{name}: serial reference ({pa.plan.info['n_decode_items']} decode items, "
            f"{pa.plan.info['n_prefill_items']} tiles, prefill {pa.plan.info['prefill_flops'] / 1e12:.2f} TFLOP)")
    checked = set()
    for step, name in enumerate(["short", "long", "short", "long", "long", "short"]):
        b, d, pa = plans[name]
        log(f"step {step}: {name} co-run 192/64")
        out, lse, _ = run(b, d=d, mode=F.FLEX_MODE_CORUN, corun=pair, pa=pa)
        assert torch.equal(out.view(torch.int16), ref[name][0].view(torch.int16)), f"step {step} ({name}) out"
        assert torch.equal(lse.view(torch.int32), ref[name][1].view(torch.int32)), f"step {step} ({name}) lse"
        if name not in checked:
            checked.add(name)
            ns = (b.query_start_loc[1:] - b.query_start_loc[:-1]).tolist()
            picks = [(s, 0) for s in range(0, len(ns) - 1, 5)] + [(len(ns) - 1, i) for i in (0, 17, ns[-1] - 1)]
            _sampled_oracle(b, out, lse, picks, f"{name} co-run")
    pair.close()
