"""Helpers for the GPU tests: move a synthetic batch to the device, run the
library on it, and compare with the fp64 oracle under the parity bar
(|gpu - ref| <= 1e-2 * max(1, |ref|) elementwise and mean |gpu - ref| <= 1e-3)."""
import sys

import numpy as np
import torch

from paper_2606_04415_amd import flexattn as F
from paper_2606_04415_amd.workloads import Segment, Workload, make_batch

ATOL_REL = 1e-2
MEAN_TOL = 1e-3


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def shape_of(w: Workload):
    return F.make_shape(w.num_q_heads, w.num_kv_heads, w.head_dim_qk, w.head_dim_v, w.page_size,
                        w.sm_scale, w.v_aliases_k)


def device_inputs(b, dev="cuda"):
    return dict(q=b.q.to(dev), k_cache=b.k_cache.to(dev),
                v_cache=None if b.v_cache is None else b.v_cache.to(dev),
                block_table=b.block_table.to(dev), seq_lens=b.seq_lens.to(dev),
                query_start_loc=b.query_start_loc.to(dev))


def run(b, d=None, mode=F.FLEX_MODE_SERIAL, opts=None, corun=None, with_lse=True, pa=None):
    """Run the batch; returns (out bf16 [T,Hq,dv] cpu, lse fp32 cpu or None, PagedAttention)."""
    w = b.workload
    d = d or device_inputs(b)
    if pa is None:
        pa = F.PagedAttention(shape_of(w), opts, b.query_start_loc.tolist(), b.seq_lens.tolist(),
                              b.block_table.shape[1])
    out, lse = pa.alloc_out(d["q"], with_lse)
    out.fill_(float("nan"))
    if lse is not None:
        lse.fill_(float("nan"))
    args = pa.args(d["q"], d["k_cache"], d["v_cache"], d["block_table"], d["seq_lens"],
                   d["query_start_loc"], out, lse)
    F.flex_attn_mixed(pa.plan, args, mode, corun=corun)
    torch.cuda.synchronize()
    return out.cpu(), (lse.cpu() if lse is not None else None), pa


def check_close(gpu, ref, what, rows=None):
    """Parity bar on rows that exist (rows: boolean mask over the first axis)."""
    g = gpu.to(torch.float64).numpy() if hasattr(gpu, "numpy") else np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    if rows is not None:
        g, r = g[rows], r[rows]
    assert np.isfinite(r).all(), f"{what}: oracle produced non-finite values"
    assert np.isfinite(g).all(), f"{what}: GPU produced non-finite values ({np.sum(~np.isfinite(g))})"
    err = np.abs(g - r)
    bound = ATOL_REL * np.maximum(1.0, np.abs(r))
    worst = float(np.max(err / bound)) if err.size else 0.0
    mean = float(err.mean()) if err.size else 0.0
    log(f"  {what}: max err/bound {worst:.3f}, mean abs err {mean:.2e}, n={err.size}")
    assert (err <= bound).all(), f"{what}: elementwise bound exceeded (worst ratio {worst:.3f})"
    assert mean <= MEAN_TOL, f"{what}: mean abs error {mean:.3e} > {MEAN_TOL}"


def custom(base: Workload, ns, ls, **kw):
    """A workload with the base geometry and explicit per-sequence (n, L)."""
    fields = dict(name=base.name + "-custom", num_q_heads=base.num_q_heads, num_kv_heads=base.num_kv_heads,
                  head_dim_qk=base.head_dim_qk, head_dim_v=base.head_dim_v, page_size=base.page_size,
                  sm_scale=base.sm_scale, v_aliases_k=base.v_aliases_k,
                  segments=tuple(Segment(1, n, (L, L)) for n, L in zip(ns, ls)), num_pages=None)
    fields.update(kw)
    return Workload(**fields)


def custom_batch(base, ns, ls, seed=0, **kw):
    w = custom(base, ns, ls, **kw)
    return make_batch(w, seed=seed, ns=list(ns), ls=list(ls))
