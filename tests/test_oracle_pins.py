"""Pins for the fp64 oracle (oracle/attention.py), CPU only.

Every pin compares the oracle with something other than itself: a closed form,
an invariant of softmax attention, a brute-force scalar loop, torch's fp64
scaled_dot_product_attention with an explicit mask, or the absorbed/
non-absorbed algebra of latent attention. ``test_planted_mistakes`` then plants
plausible mistakes in the oracle's helpers (wrong KV head, wrong slot, top-left
causal alignment, off-by-one mask, no max subtraction, lse without the max) and
checks that each one fails at least one pin.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle.attention as A

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- helpers ---

def pack_pages(seqs_k, seqs_v, P, num_pages=None, rng=None, identity=False):
    """Place per-sequence contiguous K/V [L, Hkv, d] into pages of size P.

    Returns k_cache, v_cache [num_pages, P, Hkv, d], block_table [B, maxp].
    Unused pages and tail slots are NaN, so any stray read poisons the result.
    """
    B = len(seqs_k)
    pages = [-(-k.shape[0] // P) for k in seqs_k]
    used = sum(pages)
    num_pages = num_pages or used + 3
    perm = np.arange(num_pages) if identity else (rng or np.random.default_rng(1)).permutation(num_pages)
    Hkv, dk = seqs_k[0].shape[1:]
    dv = seqs_v[0].shape[2]
    kc = np.full((num_pages, P, Hkv, dk), np.nan)
    vc = np.full((num_pages, P, Hkv, dv), np.nan)
    bt = np.zeros((B, max(pages)), dtype=np.int64)
    logical = 0
    for s in range(B):
        L = seqs_k[s].shape[0]
        for p in range(pages[s]):
            phys = perm[logical]
            logical += 1
            bt[s, p] = phys
            n = min(P, L - p * P)
            kc[phys, :n] = seqs_k[s][p * P:p * P + n]
            vc[phys, :n] = seqs_v[s][p * P:p * P + n]
    return kc, vc, bt


def run(q, kc, vc, bt, Ls, ns, sigma, Hkv, P, **kw):
    qsl = np.concatenate([[0], np.cumsum(ns)]).astype(np.int64)
    return A.paged_attention(q, kc, vc, bt, np.asarray(Ls), qsl, sigma,
                             num_kv_heads=Hkv, page_size=P, **kw)


def rand_problem(rng, Ls, ns, Hq=4, Hkv=2, d=8, dv=None, P=4):
    dv = dv or d
    ks = [rng.standard_normal((L, Hkv, d)) for L in Ls]
    vs = [rng.standard_normal((L, Hkv, dv)) for L in Ls]
    q = rng.standard_normal((sum(ns), Hq, d))
    kc, vc, bt = pack_pages(ks, vs, P, rng=rng)
    return q, ks, vs, kc, vc, bt


def sdpa_reference(q_s, K, V, n, L, sigma, Hq, Hkv):
    """torch fp64 SDPA on gathered K/V with an explicit bottom-right mask."""
    qt = torch.from_numpy(q_s).permute(1, 0, 2)                 # [Hq, n, d]
    rep = Hq // Hkv
    kt = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(rep, 0)   # [Hq, L, d]
    vt = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(rep, 0)
    i = torch.arange(n)[:, None]
    t = torch.arange(L)[None, :]
    mask = t <= (L - n + i)                                      # bottom-right
    out = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=sigma)
    scores = sigma * (qt @ kt.transpose(1, 2))
    lse = torch.logsumexp(scores.masked_fill(~mask, -math.inf), dim=-1)
    return out.permute(1, 0, 2).numpy(), lse.permute(1, 0).numpy()


# ------------------------------------------------------------------- pins ---

def pin_v1_single_key():
    rng = np.random.default_rng(10)
    q, ks, vs, kc, vc, bt = rand_problem(rng, [1], [1], Hq=4, Hkv=2, d=8, P=4)
    out, lse = run(q, kc, vc, bt, [1], [1], 0.3, 2, 4)
    for h in range(4):
        g = h // 2
        if not np.array_equal(out[0, h], vs[0][0, g]):
            return False
        if abs(lse[0, h] - 0.3 * float(q[0, h] @ ks[0][0, g])) > 1e-14:
            return False
    return True


def pin_v2_equal_scores():
    rng = np.random.default_rng(11)
    Ls, ns = [9, 13], [9, 1]
    q, ks, vs, kc, vc, bt = rand_problem(rng, Ls, ns)
    q[:] = 0.0
    out, lse = run(q, kc, vc, bt, Ls, ns, 0.5, 2, 4)
    row = 0
    for s, (L, n) in enumerate(zip(Ls, ns)):
        for i in range(n):
            vis = L - n + i + 1
            for h in range(4):
                mean = vs[s][:vis, h // 2].mean(axis=0)
                if np.max(np.abs(out[row, h] - mean)) > 1e-13 or abs(lse[row, h] - math.log(vis)) > 1e-13:
                    return False
            row += 1
    return True


def pin_v3_constant_values():
    rng = np.random.default_rng(12)
    Ls, ns = [7, 20], [3, 1]
    q, ks, vs, kc, vc, bt = rand_problem(rng, Ls, ns)
    c = rng.standard_normal(8)
    vs = [np.broadcast_to(c, v.shape).copy() for v in vs]
    kc, vc, bt = pack_pages(ks, vs, 4, rng=np.random.default_rng(2))
    out, _ = run(q, kc, vc, bt, Ls, ns, 0.7, 2, 4)
    return np.max(np.abs(out - c)) < 1e-12


def pin_v4_argmax_limit():
    # distinct scores by construction: q = e0, k_t[0] = a permutation of 0..L-1
    rng = np.random.default_rng(13)
    L, Hq, Hkv, d = 12, 2, 1, 4
    k = rng.standard_normal((L, Hkv, d))
    k[:, 0, 0] = rng.permutation(L).astype(float)
    v = rng.standard_normal((L, Hkv, d))
    q = np.zeros((1, Hq, d))
    q[0, :, 0] = 1.0
    kc, vc, bt = pack_pages([k], [v], 4, rng=rng)
    sigma = 1.0e3  # gaps of >= 1000 in the exponent: every other weight underflows
    out, lse = run(q, kc, vc, bt, [L], [1], sigma, Hkv, 4)
    best = int(np.argmax(k[:, 0, 0]))
    return np.array_equal(out[0, 0], v[best, 0]) and abs(lse[0, 0] - sigma * (L - 1)) < 1e-9


def pin_v5_paged_equals_contiguous():
    rng = np.random.default_rng(14)
    Ls, ns = [37, 16, 5], [5, 1, 5]
    q, ks, vs, _, _, _ = rand_problem(rng, Ls, ns, P=4)
    res = []
    for identity, P, seed in ((True, 4, 0), (False, 4, 3), (False, 4, 4), (True, 64, 0)):
        kc, vc, bt = pack_pages(ks, vs, P, rng=np.random.default_rng(seed), identity=identity)
        res.append(run(q, kc, vc, bt, Ls, ns, 0.4, 2, P))
    return all(np.array_equal(res[0][0], r[0]) and np.array_equal(res[0][1], r[1]) for r in res[1:])


def pin_v6_chunked_equals_oneshot():
    rng = np.random.default_rng(15)
    k = rng.standard_normal((64, 2, 8))
    v = rng.standard_normal((64, 2, 8))
    q = rng.standard_normal((64, 4, 8))
    kc, vc, bt = pack_pages([k[:32], k, k], [v[:32], v, v], 16, rng=rng)
    qq = np.concatenate([q[:32], q[32:], q])
    out, lse = run(qq, kc, vc, bt, [32, 64, 64], [32, 32, 64], 0.35, 2, 16)
    one = out[64:]
    return (np.max(np.abs(out[:32] - one[:32])) < 1e-13 and np.max(np.abs(out[32:64] - one[32:])) < 1e-13
            and np.max(np.abs(lse[:64] - lse[64:])) < 1e-13)


def pin_v7_decode_equals_prefill_row():
    rng = np.random.default_rng(16)
    L = 29
    k = rng.standard_normal((L, 2, 8))
    v = rng.standard_normal((L, 2, 8))
    q = rng.standard_normal((L, 4, 8))
    ts = [0, 7, 15, 28]
    kc, vc, bt = pack_pages([k] + [k[:t + 1] for t in ts], [v] + [v[:t + 1] for t in ts], 4, rng=rng)
    qq = np.concatenate([q] + [q[t:t + 1] for t in ts])
    out, _ = run(qq, kc, vc, bt, [L] + [t + 1 for t in ts], [L] + [1] * len(ts), 0.5, 2, 4)
    return all(np.max(np.abs(out[L + j] - out[t])) < 1e-13 for j, t in enumerate(ts))


def pin_v8_causality():
    rng = np.random.default_rng(17)
    L, n = 40, 24
    q, ks, vs, kc, vc, bt = rand_problem(rng, [L], [n])
    out1, _ = run(q, kc, vc, bt, [L], [n], 0.3, 2, 4)
    p = L - n + 10           # absolute position of query 10
    ks2 = [ks[0].copy()]
    vs2 = [vs[0].copy()]
    ks2[0][p + 1:] += 5.0
    vs2[0][p + 1:] *= -3.0
    kc2, vc2, bt2 = pack_pages(ks2, vs2, 4, rng=np.random.default_rng(1))
    out2, _ = run(q, kc2, vc2, bt2, [L], [n], 0.3, 2, 4)
    return np.array_equal(out1[:11], out2[:11]) and not np.allclose(out1[11:], out2[11:])


def pin_v9_gqa_equals_mha():
    rng = np.random.default_rng(18)
    Ls, ns = [21, 9], [6, 1]
    q, ks, vs, kc, vc, bt = rand_problem(rng, Ls, ns, Hq=6, Hkv=2)
    out_g, lse_g = run(q, kc, vc, bt, Ls, ns, 0.4, 2, 4)
    ks_r = [np.repeat(k, 3, axis=1) for k in ks]
    vs_r = [np.repeat(v, 3, axis=1) for v in vs]
    kc2, vc2, bt2 = pack_pages(ks_r, vs_r, 4, rng=rng)
    out_m, lse_m = run(q, kc2, vc2, bt2, Ls, ns, 0.4, 6, 4)
    return np.max(np.abs(out_g - out_m)) < 1e-14 and np.max(np.abs(lse_g - lse_m)) < 1e-14


def pin_v10_linear_in_v():
    rng = np.random.default_rng(19)
    Ls, ns = [17, 30], [17, 1]
    q, ks, vs, _, _, _ = rand_problem(rng, Ls, ns)
    vs2 = [rng.standard_normal(v.shape) for v in vs]
    a, b = 0.75, -1.5
    outs = []
    for vv in (vs, vs2, [a * x + b * y for x, y in zip(vs, vs2)]):
        kc, vc, bt = pack_pages(ks, vv, 4, rng=np.random.default_rng(5))
        outs.append(run(q, kc, vc, bt, Ls, ns, 0.6, 2, 4)[0])
    return np.max(np.abs(outs[2] - (a * outs[0] + b * outs[1]))) < 1e-12


def pin_v11_merge_of_partials():
    rng = np.random.default_rng(20)
    L, P = 53, 4
    q, ks, vs, kc, vc, bt = rand_problem(rng, [L], [1], P=P)
    out, lse = run(q, kc, vc, bt, [L], [1], 0.45, 2, P)
    for trial in range(5):
        cuts = sorted(set([0, L] + [P * int(c) for c in rng.integers(1, -(-L // P), size=trial + 1)]))
        cuts = [c for c in cuts if c <= L]
        if cuts[-1] != L:
            cuts.append(L)
        for h in range(4):
            g = h // 2
            parts = [A.partial_attention(q[0, h], ks[0][:, g], vs[0][:, g], a, b, 0.45)
                     for a, b in zip(cuts[:-1], cuts[1:]) if b > a]
            o, l = A.merge_partials(parts)
            if np.max(np.abs(o - out[0, h])) > 1e-12 or abs(l - lse[0, h]) > 1e-12:
                return False
    return True


def pin_v12_brute_force():
    rng = np.random.default_rng(21)
    Ls, ns = [9, 12, 6], [4, 1, 6]
    q, ks, vs, kc, vc, bt = rand_problem(rng, Ls, ns, Hq=4, Hkv=2, d=5, P=4)
    qsl = np.concatenate([[0], np.cumsum(ns)])
    kw = dict(num_kv_heads=2, page_size=4)
    o1, l1 = A.paged_attention(q, kc, vc, bt, Ls, qsl, 0.55, **kw)
    o2, l2 = A.attention_brute(q, kc, vc, bt, Ls, qsl, 0.55, **kw)
    return np.max(np.abs(o1 - o2)) < 1e-12 and np.max(np.abs(l1 - l2)) < 1e-12


def pin_v13_torch_sdpa():
    rng = np.random.default_rng(22)
    Ls, ns = [50, 33, 18, 64], [20, 1, 18, 2]
    Hq, Hkv = 6, 2
    q, ks, vs, kc, vc, bt = rand_problem(rng, Ls, ns, Hq=Hq, Hkv=Hkv, d=16, P=16)
    out, lse = run(q, kc, vc, bt, Ls, ns, 0.25, Hkv, 16)
    row = 0
    for s, (L, n) in enumerate(zip(Ls, ns)):
        ro, rl = sdpa_reference(q[row:row + n], ks[s], vs[s], n, L, 0.25, Hq, Hkv)
        if np.max(np.abs(out[row:row + n] - ro)) > 1e-12 or np.max(np.abs(lse[row:row + n] - rl)) > 1e-12:
            return False
        row += n
    return True


def pin_v14_latent_absorbed():
    """Absorbed latent attention (V = first d_c columns of the key row) equals the
    non-absorbed form with per-head up-projections, after projecting the
    latent output with W_UV."""
    rng = np.random.default_rng(23)
    H, dc, dr, dn, L, n = 4, 24, 8, 12, 30, 5
    sigma = 1.0 / math.sqrt(dn + dr)
    c = rng.standard_normal((L, dc))
    kr = rng.standard_normal((L, dr))
    qn = rng.standard_normal((n, H, dn))
    qr = rng.standard_normal((n, H, dr))
    Wuk = rng.standard_normal((H, dc, dn)) / math.sqrt(dc)
    Wuv = rng.standard_normal((H, dc, dn)) / math.sqrt(dc)
    # non-absorbed, written directly
    from scipy.special import softmax
    ref = np.empty((n, H, dn))
    for h in range(H):
        kn = c @ Wuk[h]                      # [L, dn]
        vv = c @ Wuv[h]
        for i in range(n):
            z = sigma * (kn @ qn[i, h] + kr @ qr[i, h])
            z[L - n + i + 1:] = -np.inf
            ref[i, h] = softmax(z) @ vv
    # absorbed through the oracle
    q_abs = np.concatenate([np.einsum("hcd,nhd->nhc", Wuk, qn), qr], axis=-1)   # [n, H, dc+dr]
    krow = np.concatenate([c, kr], axis=-1)[:, None, :]                          # [L, 1, dc+dr]
    kc, _, bt = pack_pages([krow], [krow[..., :dc]], 8, rng=rng)
    out, _ = run(q_abs, kc, None, bt, [L], [n], sigma, 1, 8, v_aliases_k=True, head_dim_v=dc)
    proj = np.einsum("nhc,hcd->nhd", out, Wuv)
    return np.max(np.abs(proj - ref)) < 1e-10


def pin_hand_two_keys():
    """Closed form worked by hand (tests/golden/hand_two_keys.txt)."""
    vals = {}
    with open(os.path.join(GOLDEN, "hand_two_keys.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                k, v = line.split("=")
                vals[k.strip()] = [float(x) for x in v.split()]
    sigma = vals["sigma"][0]
    k = np.array([vals["k0"], vals["k1"]])[:, None, :]
    v = np.array([vals["v0"], vals["v1"]])[:, None, :]
    q = np.array(vals["q"])[None, None, :]
    kc, vc, bt = pack_pages([k], [v], 16, rng=np.random.default_rng(0))
    out, lse = run(q, kc, vc, bt, [2], [1], sigma, 1, 16)
    return (np.max(np.abs(out[0, 0] - np.array(vals["out"]))) < 1e-15
            and abs(lse[0, 0] - vals["lse"][0]) < 1e-15)


PINS = {name: fn for name, fn in globals().items() if name.startswith("pin_")}


@pytest.mark.parametrize("name", sorted(PINS))
def test_pin(name):
    assert PINS[name](), name


# ---------------------------------------------------- planted mistakes ---

def _bad_kv_head(h, Hq, Hkv):
    return h % Hkv


def _bad_slot(t, row, P):
    return int(row[t // P]), (t + 1) % P


def _top_left(i, n, L):
    return i + 1


def _no_diagonal(i, n, L):
    return L - n + i


def _no_max_softmax(z):
    w = np.exp(z)
    l = np.sum(w, axis=-1, keepdims=True)
    return w / l, np.log(l)[..., 0]


def _lse_without_max(z):
    M = np.max(z, axis=-1, keepdims=True)
    w = np.exp(z - M)
    l = np.sum(w, axis=-1, keepdims=True)
    return w / l, np.log(l)[..., 0]


MUTANTS = {
    "kv_head_of": _bad_kv_head,
    "key_location": _bad_slot,
    "causal_limit": _top_left,
    "causal_limit_offby1": _no_diagonal,
    "softmax_rows": _no_max_softmax,
    "softmax_rows_lse": _lse_without_max,
}


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_planted_mistakes(mutant, monkeypatch):
    attr = mutant.split("_offby1")[0].split("_lse")[0]
    monkeypatch.setattr(A, attr, MUTANTS[mutant])
    failed = []
    with np.errstate(all="ignore"):
        for name, fn in PINS.items():
            try:
                ok = fn()
            except Exception:
                ok = False
            if not ok:
                failed.append(name)
    assert failed, f"planted mistake {mutant} passed every pin"


def test_attention_rows_matches_batch_oracle():
    """The per-row oracle used for sampled checks at full size (it widens only
    the pages a sequence uses and renumbers them) returns exactly the rows of
    the pinned batch oracle."""
    rng = np.random.default_rng(30)
    Ls, ns = [45, 17, 70, 5], [1, 17, 30, 1]
    q, ks, vs, kc, vc, bt = rand_problem(rng, Ls, ns, Hq=6, Hkv=2, d=8, P=4)
    qsl = np.concatenate([[0], np.cumsum(ns)])
    kw = dict(num_kv_heads=2, page_size=4)
    full_o, full_l = A.paged_attention(q, kc, vc, bt, Ls, qsl, 0.3, **kw)
    picks = [(0, 0), (1, 16), (1, 0), (2, 29), (2, 3), (3, 0)]
    o, l = A.attention_rows(q, kc, vc, bt, Ls, qsl, 0.3, picks, **kw)
    idx = [int(qsl[s]) + i for s, i in picks]
    assert np.array_equal(o, full_o[idx]) and np.array_equal(l, full_l[idx])
    # latent layout: V aliases the first columns of K
    kc2 = kc[..., :8]
    o1, l1 = A.paged_attention(q, kc2, None, bt, Ls, qsl, 0.3, v_aliases_k=True, head_dim_v=5, **kw)
    o2, l2 = A.attention_rows(q, kc2, None, bt, Ls, qsl, 0.3, picks, v_aliases_k=True, head_dim_v=5, **kw)
    assert np.array_equal(o2, o1[idx]) and np.array_equal(l2, l1[idx])
