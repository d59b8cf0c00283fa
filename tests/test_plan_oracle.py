"""Invariants of the plan re-derivation (oracle/plan.py), CPU only.

These pin the integer plan contract by properties that hold for any batch:
decode pieces tile [0, L) exactly with page-aligned, non-empty ranges in
consecutive workspace slots, and the balanced ranges hold floor or ceil of
T / R pages each; prefill tiles tile [0, n) with the right causal key end;
the tile list is ordered longest-first; counts agree with the header.
"""
import random

import pytest

from oracle import plan as OP


def shape(mla=False, Hq=28, Hkv=4, d=128, P=16):
    if mla:
        return OP.Shape(128, 1, 576, 512, 64, 1 / 192 ** 0.5, 1)
    return OP.Shape(Hq, Hkv, d, d, P, d ** -0.5, 0)


def random_batch(rng, P, n_dec, n_pre, Lmax=9000):
    ns, ls = [], []
    for _ in range(n_dec + n_pre):
        if rng.random() < n_dec / max(1, n_dec + n_pre):
            L = rng.randint(1, Lmax)
            ns.append(1)
        else:
            L = rng.randint(2, Lmax)
            ns.append(rng.randint(2, L))
        ls.append(L)
    if rng.random() < 0.3:
        ns.append(0)
        ls.append(rng.randint(0, 100))
    qsl = [0]
    for n in ns:
        qsl.append(qsl[-1] + n)
    maxp = max([1] + [-(-L // P) for L in ls])
    return qsl, ls, maxp


def check_invariants(sh, opts, qsl, ls, maxp):
    r = OP.build_plan(sh, opts, qsl, ls, maxp)
    assert r.status == OP.OK
    b = r.blob
    P = sh.page_size
    o = opts or OP.Opts()
    assert b[0] == OP.MAGIC and b[15] == len(b) and b[9] == OP.HEADER
    nd, npf, R, off_r = b[3], b[4], b[16], b[17]
    dec_items = [b[b[9] + 8 * i:b[9] + 8 * i + 8] for i in range(nd)]
    pre_items = [b[b[10] + 8 * i:b[10] + 8 * i + 8] for i in range(npf)]
    ranges = b[off_r:off_r + R + 1]
    order = b[b[18]:b[18] + nd]
    assert off_r == b[9] + 8 * nd and b[18] == off_r + R + 1 and b[19] == b[18] + nd
    merge = b[b[19]:b[10]]
    assert merge == [i for i, it in enumerate(dec_items) if it[1] == 0 and it[2] > 1]
    assert len(merge) == r.info["n_split_seqs"]
    assert sorted(order) == list(range(nd))
    keys = [(-(dec_items[i][4] - dec_items[i][3]), i) for i in order]
    assert keys == sorted(keys)                       # longest first, ties by slot
    B = len(ls)
    dec = [s for s in range(B) if qsl[s + 1] - qsl[s] == 1]
    pre = [s for s in range(B) if qsl[s + 1] - qsl[s] >= 2]
    assert b[5] == len(dec) and b[6] == len(pre)
    # decode: R balanced ranges over the concatenated pages of the decode sequences
    T = sum(-(-ls[s] // P) for s in dec)
    W = b[7]
    if sh.head_dim_qk == 576:   # a latent work-group takes 128 heads when they divide Hq, else 64
        assert W == sh.num_q_heads // (128 if sh.num_q_heads % 128 == 0 else 64)
    else:                       # one work-group per 8 KV heads
        assert W == -(-sh.num_kv_heads // 8)
    if dec:
        min_pps = -(-(o.min_split_tokens or 256) // P)
        wgpc = o.wg_per_cu or (2 if sh.head_dim_qk == 576 else 1)
        assert R == max(1, min(b[12] * wgpc // W, T // min_pps), -(-T // 8192))
        assert ranges[0] == 0 and ranges[-1] == nd
        assert all(x < y for x, y in zip(ranges, ranges[1:]))          # no empty range
        for rr in range(R):
            pages = sum(-(-(it[4] - it[3]) // P) for it in dec_items[ranges[rr]:ranges[rr + 1]])
            assert pages in (T // R, -(-T // R))
    else:
        assert R == 0 and ranges == [0] and nd == 0
    # pieces are listed in slot order; a sequence's pieces are consecutive and tile [0, L)
    assert [it[7] for it in dec_items] == list(range(nd))
    seqs = [it[0] for it in dec_items]
    assert seqs == sorted(seqs) and sorted(set(seqs)) == dec
    for s in dec:
        items = [it for it in dec_items if it[0] == s]
        slot0 = items[0][7]
        pos = 0
        for j, it in enumerate(items):
            seq, jj, n_s, k0, k1, s0, q0, slot = it
            assert (jj, n_s, s0, q0, slot) == (j, len(items), slot0, qsl[s], slot0 + j)
            assert k0 == pos and k1 > k0 and k0 % P == 0
            pos = k1
        assert pos == ls[s]
    # prefill tiles tile [0, n) and carry the causal key end
    bm = b[14]
    rows = {}
    for it in pre_items:
        s, t, r0, r1, kend = it[:5]
        n, L = qsl[s + 1] - qsl[s], ls[s]
        assert r0 == t * bm and r1 == min(n, (t + 1) * bm) and kend == L - n + r1
        rows.setdefault(s, []).append((r0, r1))
    assert sorted(rows) == pre
    for s, rr in rows.items():
        rr.sort()
        assert rr[0][0] == 0 and rr[-1][1] == qsl[s + 1] - qsl[s]
        assert all(a[1] == b_[0] for a, b_ in zip(rr, rr[1:]))
    kends = [it[4] for it in pre_items]
    assert kends == sorted(kends, reverse=True)
    return r


def test_fuzz_invariants():
    rng = random.Random(0)
    for trial in range(300):
        mla = trial % 3 == 0
        sh = shape(mla=mla) if mla else shape(P=rng.choice([16, 64]), d=rng.choice([64, 128]),
                                             Hq=rng.choice([4, 28, 32]), Hkv=rng.choice([1, 4]))
        if sh.num_q_heads % sh.num_kv_heads or sh.num_q_heads // sh.num_kv_heads > 16:
            continue
        qsl, ls, maxp = random_batch(rng, sh.page_size, rng.randint(0, 40), rng.randint(0, 4))
        opts = OP.Opts(cus_decode=rng.choice([0, 64, 128, -1]), max_splits=rng.choice([0, 2, 8]),
                       wg_per_cu=rng.choice([0, 1, 8]))
        check_invariants(sh, opts, qsl, ls, maxp)


def test_workload_configs_plans():
    from paper_2606_04415_amd.workloads import WORKLOADS, draw_lengths
    import torch
    for name, w in WORKLOADS.items():
        ns, ls = draw_lengths(w, torch.Generator().manual_seed(0))
        qsl = [0]
        for n in ns:
            qsl.append(qsl[-1] + n)
        sh = OP.Shape(w.num_q_heads, w.num_kv_heads, w.head_dim_qk, w.head_dim_v, w.page_size,
                      w.sm_scale, int(w.v_aliases_k))
        check_invariants(sh, None, qsl, ls, w.max_pages_per_seq)


@pytest.mark.parametrize("case,status", [
    (dict(qsl=[1, 2], ls=[4]), OP.ERR_INVALID_ARG),          # qsl[0] != 0
    (dict(qsl=[0, 3, 2], ls=[4, 4]), OP.ERR_INVALID_ARG),    # decreasing
    (dict(qsl=[0, 5], ls=[4]), OP.ERR_INVALID_ARG),          # n > L
    (dict(qsl=[0, 1], ls=[10**6]), OP.ERR_INVALID_ARG),      # L > max_pages * P
    (dict(qsl=[0, 0], ls=[0]), OP.OK),                       # empty sequence
    (dict(qsl=[0], ls=[]), OP.OK),                           # empty batch
])
def test_validation(case, status):
    r = OP.build_plan(shape(), None, case["qsl"], case["ls"], 16)
    assert r.status == status


def test_unsupported_shapes():
    assert OP.build_plan(OP.Shape(28, 4, 96, 96, 16, 0.1, 0), None, [0, 1], [5], 4).status == OP.ERR_UNSUPPORTED
    assert OP.build_plan(OP.Shape(28, 4, 128, 128, 32, 0.1, 0), None, [0, 1], [5], 4).status == OP.ERR_UNSUPPORTED
    assert OP.build_plan(OP.Shape(28, 3, 128, 128, 16, 0.1, 0), None, [0, 1], [5], 4).status == OP.ERR_INVALID_ARG
    assert OP.build_plan(OP.Shape(28, 4, 128, 128, 16, -1.0, 0), None, [0, 1], [5], 4).status == OP.ERR_INVALID_ARG
    assert OP.build_plan(OP.Shape(128, 1, 576, 512, 64, 0.1, 0), None, [0, 1], [5], 4).status == OP.ERR_UNSUPPORTED
