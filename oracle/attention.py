"""fp64 CPU oracle for paged attention over one mixed prefill/decode batch.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. The library never
does, and this module imports nothing from the library.

What it computes. The paper (FlexNPU) schedules the attention of prefill
chunks and decode steps that share one KV pool (Sec. 3.4, "Memory Locality")
but never writes attention down; it only characterises the phases (prefill is
compute-intensive, decode is bound by memory bandwidth and KV-cache accesses:
Abstract, Sec. 1, Sec. 2.3, Sec. 3). So this oracle is the textbook definition
of scaled dot-product softmax attention, applied per sequence of a batch whose
keys and values sit in fixed-size pages of a shared cache:

  for sequence s with n new query tokens and L keys (n <= L), query i
  (0 <= i < n) sits at absolute position p = L - n + i and sees keys 0..p
  (bottom-right causal alignment; decode is n = 1 and sees all L keys);
  key t of s lives in physical page block_table[s][t // P], slot t % P;
  query head h reads KV head h // (Hq / Hkv);
  z_t = sigma * <q, k_t>,  M = max_t z_t,  w_t = exp(z_t - M),  l = sum_t w_t,
  out = sum_t w_t v_t / l,  lse = M + ln l   (natural log).

With ``v_aliases_k`` (absorbed MLA) the value row of a key is the first d_v
columns of its key row.

Readings taken where the paper is silent that shape this code: page layout [page][slot][kv_head][dim]; bottom-right
causal alignment; consecutive query heads share a KV head; the scale is an
explicit input; n = 0 produces no rows; bf16 inputs are widened exactly to
fp64 and everything after that is fp64 with a two-pass softmax (no online
rescaling, no split-K, no tiling).

Pins: tests/test_oracle_pins.py checks this module against closed forms,
invariants, brute force, and torch's fp64 scaled_dot_product_attention.
"""
from __future__ import annotations

from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np


def _f64(x) -> np.ndarray:
    """Widen an input array (numpy, or a torch CPU tensor of any float dtype) to fp64."""
    if hasattr(x, "detach"):  # torch tensor: bf16 has no numpy dtype, go through fp32 (exact)
        import torch
        x = x.detach().to(torch.float64).cpu().numpy()
    return np.asarray(x, dtype=np.float64)


def _i64(x) -> np.ndarray:
    if hasattr(x, "detach"):
        x = x.detach().cpu().numpy()
    return np.asarray(x, dtype=np.int64)


# ---- the three facts of the paging / causal contract, as small helpers ----

def kv_head_of(h: int, num_q_heads: int, num_kv_heads: int) -> int:
    """KV head read by query head h: consecutive query heads share one KV head."""
    return h // (num_q_heads // num_kv_heads)


def key_location(t: int, block_table_row: np.ndarray, page_size: int) -> Tuple[int, int]:
    """(physical page, slot) of key t of a sequence."""
    return int(block_table_row[t // page_size]), t % page_size


def causal_limit(i: int, n: int, L: int) -> int:
    """Number of keys visible to query i of n new tokens over L keys (bottom-right)."""
    return L - n + i + 1


def gather_sequence(cache: np.ndarray, block_table_row: np.ndarray, L: int,
                    page_size: int) -> np.ndarray:
    """Explicit page gather: rows 0..L-1 of one sequence, [L, Hkv, d] fp64."""
    out = np.empty((L,) + cache.shape[2:], dtype=np.float64)
    for t in range(L):
        page, slot = key_location(t, block_table_row, page_size)
        out[t] = cache[page, slot]
    return out


def softmax_rows(z: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Two-pass softmax over the last axis. Returns (weights / l, lse)."""
    M = np.max(z, axis=-1, keepdims=True)
    w = np.exp(z - M)
    l = np.sum(w, axis=-1, keepdims=True)
    return w / l, (M + np.log(l))[..., 0]


def sequence_attention(q_s: np.ndarray, K: np.ndarray, V: np.ndarray, L: int,
                       num_kv_heads: int, sm_scale: float,
                       rows: Optional[Sequence[int]] = None,
                       block: int = 2048) -> Tuple[np.ndarray, np.ndarray]:
    """Attention of one sequence's n queries over its L gathered keys.

    q_s [n, Hq, d_qk] fp64, K [L, Hkv, d_qk], V [L, Hkv, d_v]. ``rows`` selects
    a subset of the n queries (sampled checks at large sizes). Every (row,
    query head) pair is independent; the pairs whose head reads KV head g are
    stacked into one product with that head's keys, a block of about
    ``block`` pairs at a time to bound memory.
    """
    n, Hq, _ = q_s.shape
    dv = V.shape[-1]
    idx = np.arange(n) if rows is None else np.asarray(list(rows), dtype=np.int64)
    out = np.empty((len(idx), Hq, dv), dtype=np.float64)
    lse = np.empty((len(idx), Hq), dtype=np.float64)
    for g in range(num_kv_heads):
        heads = np.array([h for h in range(Hq) if kv_head_of(h, Hq, num_kv_heads) == g])
        Kg = K[:, g, :]          # [L, d_qk]
        Vg = V[:, g, :]          # [L, d_v]
        rows_per_block = max(1, block // len(heads))
        for b0 in range(0, len(idx), rows_per_block):
            rb = idx[b0:b0 + rows_per_block]
            Qb = q_s[rb][:, heads, :].reshape(len(rb) * len(heads), -1)   # (row, head) pairs
            z = sm_scale * (Qb @ Kg.T)                                    # [pairs, L]
            limits = np.repeat([causal_limit(int(i), n, L) for i in rb], len(heads))
            visible = np.arange(L)[None, :] < limits[:, None]
            z = np.where(visible, z, -np.inf)
            w, ls = softmax_rows(z)
            o = w @ Vg
            out[b0:b0 + len(rb), heads, :] = o.reshape(len(rb), len(heads), dv)
            lse[b0:b0 + len(rb), heads] = ls.reshape(len(rb), len(heads))
    return out, lse


def paged_attention(q, k_cache, v_cache, block_table, seq_lens, query_start_loc,
                    sm_scale: float, *, num_kv_heads: int, page_size: int,
                    head_dim_v: Optional[int] = None, v_aliases_k: bool = False,
                    seqs: Optional[Iterable[int]] = None):
    """Full oracle over a batch.

    q [T, Hq, d_qk]; k_cache [num_pages, P, Hkv, d_qk]; v_cache
    [num_pages, P, Hkv, d_v] (ignored when ``v_aliases_k``: V = K[..., :d_v]);
    block_table [B, max_pages] int; seq_lens [B]; query_start_loc [B+1].
    Returns fp64 (out [T, Hq, d_v], lse [T, Hq]); rows of sequences not in
    ``seqs`` (when given) are left NaN.
    """
    qf = _f64(q)
    kc = _f64(k_cache)
    if v_aliases_k:
        dv = head_dim_v if head_dim_v is not None else kc.shape[-1]
        vc = kc[..., :dv]
    else:
        vc = _f64(v_cache)
        dv = vc.shape[-1]
    bt = _i64(block_table)
    L_all = _i64(seq_lens)
    qsl = _i64(query_start_loc)
    T, Hq, _ = qf.shape
    out = np.full((T, Hq, dv), np.nan)
    lse = np.full((T, Hq), np.nan)
    B = len(L_all)
    for s in (range(B) if seqs is None else seqs):
        q0, q1 = int(qsl[s]), int(qsl[s + 1])
        n, L = q1 - q0, int(L_all[s])
        if n == 0:
            continue
        if not (0 < n <= L):
            raise ValueError(f"sequence {s}: query length {n} not in [0, {L}]")
        K = gather_sequence(kc, bt[s], L, page_size)
        V = gather_sequence(vc, bt[s], L, page_size)
        o, l = sequence_attention(qf[q0:q1], K, V, L, num_kv_heads, sm_scale)
        out[q0:q1] = o
        lse[q0:q1] = l
    return out, lse


def attention_rows(q, k_cache, v_cache, block_table, seq_lens, query_start_loc,
                   sm_scale: float, picks: Sequence[Tuple[int, int]], *, num_kv_heads: int,
                   page_size: int, head_dim_v: Optional[int] = None,
                   v_aliases_k: bool = False):
    """Oracle values of individual output rows, for sampled checks at full size.

    ``picks`` is a list of (sequence, query index within the sequence). Returns
    fp64 (out [len(picks), Hq, d_v], lse [len(picks), Hq]).
    """
    kc = k_cache
    qsl = _i64(query_start_loc)
    L_all = _i64(seq_lens)
    bt = _i64(block_table)
    by_seq = {}
    for j, (s, i) in enumerate(picks):
        by_seq.setdefault(int(s), []).append((j, int(i)))
    Hq = q.shape[1]
    dv = head_dim_v if v_aliases_k else v_cache.shape[-1]
    out = np.empty((len(picks), Hq, dv))
    lse = np.empty((len(picks), Hq))
    for s, items in by_seq.items():
        q0, q1 = int(qsl[s]), int(qsl[s + 1])
        n, L = q1 - q0, int(L_all[s])
        pages = sorted(set(int(bt[s, t // page_size]) for t in range(0, L, page_size)))
        # widen only the pages this sequence uses
        remap = {p: j for j, p in enumerate(pages)}
        kp = _f64(kc[pages])
        vp = kp[..., :dv] if v_aliases_k else _f64(v_cache[pages])
        row = np.array([remap[int(bt[s, t])] for t in range((L + page_size - 1) // page_size)])
        K = gather_sequence(kp, row, L, page_size)
        V = gather_sequence(vp, row, L, page_size)
        qs = _f64(q[q0:q1])
        o, l = sequence_attention(qs, K, V, L, num_kv_heads, sm_scale, rows=[i for _, i in items])
        for r, (j, _) in enumerate(items):
            out[j] = o[r]
            lse[j] = l[r]
    return out, lse


# ---- split-K partials and their merge (flash-decoding combine) ----

def partial_attention(q_row: np.ndarray, K: np.ndarray, V: np.ndarray, k0: int, k1: int,
                      sm_scale: float) -> Tuple[np.ndarray, float, float]:
    """Unnormalised partial over keys [k0, k1) for one query vector and one KV head.

    q_row [d_qk]; K [L, d_qk]; V [L, d_v]. Returns (O_j = sum_t e^{z_t - m_j} v_t,
    m_j = max_t z_t, l_j = sum_t e^{z_t - m_j}).
    """
    z = sm_scale * (K[k0:k1] @ q_row)
    m = float(np.max(z))
    w = np.exp(z - m)
    return w @ V[k0:k1], m, float(np.sum(w))


def merge_partials(parts: List[Tuple[np.ndarray, float, float]]) -> Tuple[np.ndarray, float]:
    """Combine partials over disjoint key ranges: returns (out, lse).

    M = max_j m_j; out = sum_j e^{m_j - M} O_j / sum_j e^{m_j - M} l_j;
    lse = M + ln sum_j e^{m_j - M} l_j.
    """
    M = max(m for _, m, _ in parts)
    num = sum(np.exp(m - M) * O for O, m, _ in parts)
    den = sum(np.exp(m - M) * l for _, m, l in parts)
    return num / den, M + np.log(den)


def attention_brute(q, k_cache, v_cache, block_table, seq_lens, query_start_loc,
                    sm_scale: float, *, num_kv_heads: int, page_size: int,
                    head_dim_v: Optional[int] = None, v_aliases_k: bool = False):
    """Scalar-loop version of ``paged_attention`` for tiny inputs (pure Python)."""
    import math
    qf = _f64(q)
    kc = _f64(k_cache)
    vc = kc[..., :head_dim_v] if v_aliases_k else _f64(v_cache)
    bt = _i64(block_table)
    L_all = _i64(seq_lens)
    qsl = _i64(query_start_loc)
    T, Hq, dqk = qf.shape
    dv = vc.shape[-1]
    group = Hq // num_kv_heads
    out = np.full((T, Hq, dv), np.nan)
    lse = np.full((T, Hq), np.nan)
    for s in range(len(L_all)):
        q0, q1 = int(qsl[s]), int(qsl[s + 1])
        n, L = q1 - q0, int(L_all[s])
        for i in range(n):
            last = L - n + i
            for h in range(Hq):
                g = h // group
                z = []
                for t in range(last + 1):
                    page = int(bt[s][t // page_size])
                    acc = 0.0
                    for d in range(dqk):
                        acc += float(qf[q0 + i, h, d]) * float(kc[page, t % page_size, g, d])
                    z.append(sm_scale * acc)
                M = max(z)
                w = [math.exp(x - M) for x in z]
                l = sum(w)
                for d in range(dv):
                    acc = 0.0
                    for t in range(last + 1):
                        page = int(bt[s][t // page_size])
                        acc += w[t] * float(vc[page, t % page_size, g, d])
                    out[q0 + i, h, d] = acc / l
                lse[q0 + i, h] = M + math.log(l)
    return out, lse
