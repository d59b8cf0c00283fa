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


def prefill_model(sh, bm, qsl, ls, pre, cus, fl):
    """The plan's prefill time for grouped-query tiles: the work at the
    per-CU rate, or the largest work-group (its rows against every key of
    its sequence) at 0.6 of a CU (flat 4-wave work-groups) or a whole CU
    (32-token groups of up to 8 heads), whichever is longer, plus 10 us."""
    G = sh.num_q_heads // sh.num_kv_heads
    work = 0.0
    big = 0.0
    for s in pre:
        n, L = qsl[s + 1] - qsl[s], ls[s]
        work += sh.num_q_heads * 2 * (sh.head_dim_qk + sh.head_dim_v) * (n * (L - n) + n * (n + 1) / 2)
        rows = min(128, n * G) if bm == 128 else min(bm, n) * min(G, 8)
        big = max(big, rows * L * 2 * (sh.head_dim_qk + sh.head_dim_v) / ((0.6 if bm == 128 else 1.0) * fl))
    return max(work / (cus * fl), big) + 10e-6


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
        # two groups of balanced ranges: [0, TA) for the decode share, the tail [TA, T)
        RB = b[23]
        RA = R - RB
        start = {}
        acc = 0
        for s in dec:
            start[s] = acc
            acc += -(-ls[s] // P)
        TA = start[dec_items[ranges[RA]][0]] + dec_items[ranges[RA]][3] // P if RB else T
        TB = T - TA

        def n_ranges(npages, cus):
            return max(1, min(cus * wgpc // W, npages // min_pps), -(-npages // 8192)) if npages else 0
        assert RA == n_ranges(TA, b[12]) and RB == n_ranges(TB, b[13])
        assert ranges[0] == 0 and ranges[-1] == nd
        assert all(x < y for x, y in zip(ranges, ranges[1:]))          # no empty range
        for rr in range(R):
            pages = sum(-(-(it[4] - it[3]) // P) for it in dec_items[ranges[rr]:ranges[rr + 1]])
            n_g, t_g = (RA, TA) if rr < RA else (RB, TB)
            assert pages in (t_g // n_g, -(-t_g // n_g))
        # a tail only on grouped-query co-run shares; its first page balances the two
        # groups' end times under the cost model (the decode share streams during the
        # prefill, then shares the device with the tail in proportion to CUs)
        N = o.cus_total or 256
        tail_ok = bool(pre) and b[13] < N and sh.head_dim_qk in (64, 128) and o.decode_tail == 0
        if RB:
            assert tail_ok and 1 <= TA < T
        if tail_ok and T > 1:
            n_d, n_p = b[12], b[13]
            hbm = (o.hbm_gbps or OP.DEFAULT_HBM_GBPS) * 1e9
            bw = (o.decode_gbps_per_cu or OP.DEFAULT_DECODE_GBPS_PER_CU) * 1e9
            fl = (o.prefill_tflops_per_cu or OP.DEFAULT_PREFILL_TFLOPS_PER_CU) * 1e12
            D = r.info["decode_bytes"]
            t_p = prefill_model(sh, b[14], qsl, ls, pre, n_p, fl)
            r_s = min(hbm, n_d * bw)
            if r_s * t_p >= D:
                assert RB == 0
            else:
                # t_p + (x - r_s t_p) / (r_a n_d / N) == t_p + (D - x) / (r_a n_p / N)
                x = (n_d * D + n_p * r_s * t_p) / (n_d + n_p)
                assert abs(TA - min(T - 1, max(1, int(x / D * T)))) <= 1
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
    # prefill tiles tile [0, n) (flat tiles: [0, n * G), rows being (token, query
    # head) pairs) and carry the causal key end of their last row's token
    bm = b[14]
    G = sh.num_q_heads // sh.num_kv_heads
    flat = sh.head_dim_qk in (64, 128) and bm == 128
    if sh.head_dim_qk in (64, 128) and not (o.bm or 0):   # default tile height
        flat_wgs = sum(-(-(qsl[s + 1] - qsl[s]) * G // 128) * sh.num_kv_heads for s in pre)
        share = b[13] < (o.cus_total or 256)
        assert bm == (128 if (flat_wgs >= 4 * b[13] or (share and flat_wgs <= 3 * b[13])) else 32)
    assert b[8] == (sh.num_kv_heads if flat else b[8])
    rows = {}
    for it in pre_items:
        s, t, r0, r1, kend = it[:5]
        n, L = qsl[s + 1] - qsl[s], ls[s]
        nrows = n * G if flat else n
        last_token = (r1 - 1) // G if flat else r1 - 1
        assert r0 == t * bm and r1 == min(nrows, (t + 1) * bm) and kend == L - n + last_token + 1
        rows.setdefault(s, []).append((r0, r1))
    assert sorted(rows) == pre
    for s, rr in rows.items():
        rr.sort()
        n = qsl[s + 1] - qsl[s]
        assert rr[0][0] == 0 and rr[-1][1] == (n * G if flat else n)
        assert all(a[1] == b_[0] for a, b_ in zip(rr, rr[1:]))
    kends = [it[4] for it in pre_items]
    assert kends == sorted(kends, reverse=True)
    check_fused(sh, r, b)
    return r


def check_fused(sh, r, b):
    """The one-launch order: every work-group once, on its XCD, each phase in order."""
    nd, npf, R, bm, gy = b[3], b[4], b[16], b[14], b[8]
    off_f, nf = b[20], b[21]
    assert off_f == b[10] + 8 * npf and off_f + nf == b[22] and r.info["n_fused_wgs"] == nf
    B = b[2]
    assert len(b) == b[22] + 2 * B + 1                      # then seq_lens and query_start_loc as given
    fused = b[off_f:off_f + nf]
    G = sh.num_q_heads // sh.num_kv_heads
    fusable = sh.head_dim_qk != 576 and G > 4 and 3 <= sh.num_kv_heads <= 8 and bm == 32 and nd + npf > 0
    assert (nf > 0) == fusable and nf % 8 == 0
    if not nf:
        return
    rpw = 2 if sh.num_kv_heads <= 4 else 1
    n_pre_wg, J = npf * gy, -(-R // rpw)
    assert sorted(e for e in fused if e >= 0) == list(range(n_pre_wg + J)) and min(fused) >= -1
    for x in range(8):
        col = fused[x::8]
        k = len(col)
        while k and col[k - 1] == -1:
            k -= 1
        col = col[:k]
        assert -1 not in col                               # padding only at the end
        for e in col:                                      # work-group b runs on XCD b % 8
            if e < n_pre_wg and 8 % gy == 0:
                assert e % gy == x % gy and (e // gy) % (8 // gy) == x // gy
            elif e >= n_pre_wg:
                assert (e - n_pre_wg) % 8 == x
        # each phase keeps its own order (a pool starts its work-groups in order)
        pre = [e for e in col if e < n_pre_wg]
        dec = [e for e in col if e >= n_pre_wg]
        assert pre == sorted(pre) and dec == sorted(dec)


def test_fuzz_invariants():
    rng = random.Random(0)
    for trial in range(300):
        mla = trial % 3 == 0
        sh = shape(mla=mla) if mla else shape(P=rng.choice([16, 64]), d=rng.choice([64, 128]),
                                             Hq=rng.choice([4, 28, 32, 40, 48]), Hkv=rng.choice([1, 3, 4, 5, 8]))
        if sh.num_q_heads % sh.num_kv_heads or sh.num_q_heads // sh.num_kv_heads > 16:
            continue
        qsl, ls, maxp = random_batch(rng, sh.page_size, rng.randint(0, 40), rng.randint(0, 4))
        cus_total = rng.choice([0, 0, 16])
        opts = OP.Opts(cus_decode=rng.choice([0, 8, -1] if cus_total else [0, 64, 128, -1]),
                       wg_per_cu=rng.choice([0, 1, 8]),
                       bm=0 if mla else rng.choice([0, 0, 16, 32, 128]), cus_total=cus_total,
                       split_granule=8 if cus_total else 0)
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


def test_fused_order_worked_example():
    """A case small enough to schedule by hand.

    16 CUs -> 2 per XCD; no co-run split -> one prefill CU and one decode CU
    per XCD. Four 32-token prompts (one tile each, 528 causal pairs, kend 32,
    tiles in batch order) and 48 one-page decode sequences cut into R =
    16 * 3 = 48 one-page ranges, two per decode work-group (4 KV heads): 24
    decode work-groups. Durations: prefill 528 pairs * 7 heads * 512 flop at
    1 TFLOP/s = 1892.352 ns -> 1893; decode 2 pages * 16 slots * 4 heads *
    256 * 2 B = 65536 B at 80 GB/s = 819.2 ns -> 820. XCD 0 serves tiles 0
    and 2 (column 0 -> entries 0 and 8) and decode work-groups 0, 8, 16
    (entries 16, 24, 32): prefill starts 0, 1893; decode starts 0, 820, 1640;
    by start time: 0 (prefill first), 16, 24, 32, 8.
    """
    sh = OP.Shape(28, 4, 128, 128, 16, 0.088, 0)
    ns = [1] * 48 + [32] * 4
    ls = [16] * 48 + [32] * 4
    qsl = [0]
    for n in ns:
        qsl.append(qsl[-1] + n)
    o = OP.Opts(cus_total=16, wg_per_cu=3, min_split_tokens=16, prefill_tflops_per_cu=1.0, decode_gbps_per_cu=80.0)
    r = OP.build_plan(sh, o, qsl, ls, 2)
    assert r.status == OP.OK and r.blob[16] == 48
    b = r.blob
    fused = b[b[20]:b[20] + b[21]]
    assert fused[0::8][:5] == [0, 16, 24, 32, 8]
    # XCD 4 serves tile 1 and 3 column 0 (entries 4, 12) and decode 4, 12, 20 (entries 20, 28, 36)
    assert fused[4::8][:5] == [4, 20, 28, 36, 12]


def test_decode_tail_on_corun_shares():
    """A mixed-step-shaped batch (128 decodes over 1k-8k keys, one 2048-token
    chunk on 4096 cached keys) planned for each co-run split: a decode tail
    whose first page balances the two groups where the cost model has the
    prefill end first (64 and 96 decode CUs), none where the decode share
    finishes first (check_invariants pins both), with decode_tail = -1, on the
    whole device, or for the latent layout."""
    rng = random.Random(5)
    ls = [rng.randint(1024, 8192) for _ in range(128)] + [6144]
    qsl = list(range(129)) + [128 + 2048]
    sh = shape(P=16, d=128, Hq=28, Hkv=4)
    maxp = max(-(-L // 16) for L in ls)
    for cd in (64, 96, 128, 160, 192):
        o = OP.Opts(cus_decode=cd)
        check_invariants(sh, o, qsl, ls, maxp)
        b = OP.build_plan(sh, o, qsl, ls, maxp).blob
        assert b[12] == cd and (b[23] > 0) == (cd <= 96)
    for o in (OP.Opts(cus_decode=128, decode_tail=-1), OP.Opts(cus_decode=0)):
        check_invariants(sh, o, qsl, ls, maxp)
        assert OP.build_plan(sh, o, qsl, ls, maxp).blob[23] == 0
    lat = shape(mla=True)
    assert OP.build_plan(lat, OP.Opts(cus_decode=128), qsl, ls, max(-(-L // lat.page_size) for L in ls)).blob[23] == 0
    assert OP.build_plan(sh, OP.Opts(decode_tail=1), qsl, ls, maxp).status == OP.ERR_INVALID_ARG


def test_auto_split_with_decode_tail():
    """cus_decode = -1 on the mixed-step-shaped batch: the plan's split is the
    one a time-stepped simulation of the step finds fastest (the decode share
    streams at its rate until the prefill ends, then the whole device at the
    streaming rate), and with the default rates it is 96 decode CUs, the
    split measured fastest for this step (co-run 289 us against 300 us at
    128/128)."""
    rng = random.Random(5)
    ls = [rng.randint(1024, 8192) for _ in range(128)] + [6144]
    qsl = list(range(129)) + [128 + 2048]
    sh = shape(P=16, d=128, Hq=28, Hkv=4)
    maxp = max(-(-L // 16) for L in ls)
    r = OP.build_plan(sh, OP.Opts(cus_decode=-1), qsl, ls, maxp)
    D = r.info["decode_bytes"]
    bw, fl, hbm = 43e9, 4e12, 6500e9

    def simulate(nd, dt=1e-7):
        bm = OP.build_plan(sh, OP.Opts(cus_decode=nd), qsl, ls, maxp).blob[14]   # the tiles of that share
        t, left, t_pre = 0.0, D, prefill_model(sh, bm, qsl, ls, [128], 256 - nd, fl)
        while left > 0:
            left -= (min(hbm, nd * bw) if t < t_pre else hbm) * dt
            t += dt
        return max(t, t_pre)
    times = {nd: simulate(nd) for nd in range(32, 256, 32)}
    assert r.blob[12] == min(times, key=times.get) == 96
