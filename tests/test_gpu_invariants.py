"""Invariants of attention checked on the device, with no oracle involved.

V2: equal scores (q = 0) give the mean of the visible value rows and
    lse = ln(visible keys).
V8: changing keys and values after a row's causal limit leaves that row
    bit-identical (a masked key must contribute exactly nothing).
V3: constant value rows give that constant, whatever the weights.
V7: the decode kernel at position t agrees with the prefill kernel's row t;
V6: a chunk over cached keys agrees with the same rows of a one-shot prompt.
All through the C ABI on ragged grouped-query and latent batches, so the
decode kernel, the split merge and the prefill kernels are all exercised.
"""
import numpy as np
import pytest
import torch

from paper_2606_04415_amd.workloads import WORKLOADS

from gpu_common import ATOL_REL, MEAN_TOL, custom_batch, log, run

pytestmark = pytest.mark.gpu

QW = WORKLOADS["decode"]
MLA = WORKLOADS["mla"]


def visible_mean_v(b, s, i):
    """fp64 mean of the value rows sequence s's query i sees, per KV head."""
    w = b.workload
    n = int(b.query_start_loc[s + 1] - b.query_start_loc[s])
    L = int(b.seq_lens[s])
    lim = L - n + i + 1
    t = torch.arange(lim)
    pages = b.block_table[s, t // w.page_size].long()
    src = b.k_cache if w.v_aliases_k else b.v_cache
    rows = src[pages, t % w.page_size].double()[..., :w.head_dim_v]
    return rows.mean(0), lim


@pytest.mark.parametrize("base", ["decode", "mla"])
def test_equal_scores_give_mean_values(base):
    w = WORKLOADS[base]
    ns, ls = ([1, 1, 40, 1], [500, 17, 300, 3000]) if base == "decode" else ([1, 1, 70], [130, 1500, 200])
    b = custom_batch(w, ns, ls, seed=11)
    b.q.zero_()
    log(f"V2 on device: {base}, q = 0")
    out, lse, _ = run(b)
    G = w.num_q_heads // w.num_kv_heads
    qsl = b.query_start_loc.tolist()
    for s in range(len(ns)):
        for i in sorted({0, ns[s] // 2, ns[s] - 1}):
            mean, lim = visible_mean_v(b, s, i)
            ref = mean.repeat_interleave(G, 0).numpy()          # [Hq, d_v]
            got = out[qsl[s] + i].double().numpy()
            err = np.abs(got - ref)
            assert (err <= ATOL_REL * np.maximum(1.0, np.abs(ref))).all() and err.mean() <= MEAN_TOL, (s, i)
            assert np.allclose(lse[qsl[s] + i].double().numpy(), np.log(lim), atol=1e-4), (s, i)


@pytest.mark.parametrize("base", ["decode", "mla"])
def test_future_keys_do_not_matter(base):
    w = WORKLOADS[base]
    ns, ls = ([1, 130, 1, 64], [900, 130, 33, 500]) if base == "decode" else ([1, 130, 1], [700, 260, 65])
    b1 = custom_batch(w, ns, ls, seed=12, num_pages=None)
    b2 = custom_batch(w, ns, ls, seed=12, num_pages=None)
    # sequence 1 is a prefill chunk; change its keys/values after position c
    s, c = 1, ls[1] - ns[1] + 37
    t = torch.arange(c + 1, ls[1])
    pages = b2.block_table[s, t // w.page_size].long()
    b2.k_cache[pages, t % w.page_size] = -b2.k_cache[pages, t % w.page_size] * 3.0 + 1.0
    if b2.v_cache is not None:
        b2.v_cache[pages, t % w.page_size] = b2.v_cache[pages, t % w.page_size] * 2.0 - 0.5
    log(f"V8 on device: {base}, keys after position {c} of sequence {s} changed")
    o1, l1, _ = run(b1)
    o2, l2, _ = run(b2)
    q0 = int(b1.query_start_loc[s])
    rows = slice(q0, q0 + 38)        # rows whose causal limit is at most c + 1
    assert torch.equal(o1[rows].view(torch.int16), o2[rows].view(torch.int16))
    assert torch.equal(l1[rows], l2[rows])
    # rows of the other sequences are untouched too
    other = torch.ones(o1.shape[0], dtype=torch.bool)
    other[q0:q0 + ns[1]] = False
    assert torch.equal(o1[other].view(torch.int16), o2[other].view(torch.int16))
    # and later rows of the chunk do change
    assert not torch.equal(o1[q0 + 60], o2[q0 + 60])


def close(a, b, what):
    a, b = a.double().numpy(), b.double().numpy()
    err = np.abs(a - b)
    assert (err <= ATOL_REL * np.maximum(1.0, np.abs(b))).all() and err.mean() <= MEAN_TOL, what


@pytest.mark.parametrize("base", ["decode", "mla"])
def test_constant_values_give_that_constant(base):
    # V3: every visible value row equal to c (per KV head) -> out = c whatever the weights
    w = WORKLOADS[base]
    ns, ls = ([1, 1, 70, 1], [700, 9, 300, 2100]) if base == "decode" else ([1, 70, 1], [300, 200, 1500])
    b = custom_batch(w, ns, ls, seed=13)
    c = torch.linspace(-2.0, 2.0, w.num_kv_heads * w.head_dim_v).view(w.num_kv_heads, w.head_dim_v)
    c = c.to(torch.bfloat16)
    if w.v_aliases_k:
        b.k_cache[..., :w.head_dim_v] = c          # V is the first 512 columns of the key row
    else:
        b.v_cache[...] = c
    log(f"V3 on device: {base}, constant value rows")
    out, _, _ = run(b)
    G = w.num_q_heads // w.num_kv_heads
    ref = c.double().repeat_interleave(G, 0)         # [Hq, d_v]
    for r in range(out.shape[0]):
        close(out[r], ref, f"row {r}")


def test_decode_row_equals_prefill_row():
    # V7: the decode kernel at position t and the prefill kernel's row t agree;
    # V6: a chunk on top of cached keys equals the same rows of a one-shot prompt
    w = QW
    ns, ls = [300, 1, 1, 32, 64], [300, 1, 1, 64, 64]
    b = custom_batch(w, ns, ls, seed=14)
    P = w.page_size
    qsl = b.query_start_loc.tolist()
    for s, t in ((1, 137), (2, 255)):              # decodes at positions 137 and 255 of prompt 0
        L = t + 1
        b.seq_lens[s] = L
        npg = -(-L // P)
        b.block_table[s, :npg] = b.block_table[0, :npg]
        b.q[qsl[s]] = b.q[qsl[0] + t]
    # sequence 3: rows 32..63 of the 64-token prompt 4, as a chunk over its first 32 keys
    b.block_table[3] = b.block_table[4]
    b.q[qsl[3]:qsl[3] + 32] = b.q[qsl[4] + 32:qsl[4] + 64]
    log("V7 / V6 on device: decode vs prefill rows, chunked vs one-shot prefill")
    out, lse, _ = run(b)
    close(out[qsl[1]], out[qsl[0] + 137], "decode at 137 vs prefill row 137")
    close(out[qsl[2]], out[qsl[0] + 255], "decode at 255 vs prefill row 255")
    assert np.allclose(lse[qsl[1]].numpy(), lse[qsl[0] + 137].numpy(), atol=1e-3)
    close(out[qsl[3]:qsl[3] + 32], out[qsl[4] + 32:qsl[4] + 64], "chunk vs one-shot")
    assert np.allclose(lse[qsl[3]:qsl[3] + 32].numpy(), lse[qsl[4] + 32:qsl[4] + 64].numpy(), atol=1e-3)
