"""Integer re-derivation of the host plan: validation, phase classification,
split-K partition of decode sequences and the prefill tile list.

TEST INFRASTRUCTURE (same rules as oracle/attention.py): imported only by
tests/. Written from the plan contract below, not from the library's C++; the
two are compared bit-exactly through ``flex_attn_plan_export``.

Role in the method. The paper's daemon validates every request before dispatch
(Sec. 3.2) and keeps separate prefill and decode queues (Sec. 3.4,
"Phase-Aware Dispatch"); the plan is that step for one mixed batch: it
classifies each sequence by its number of new tokens and lays out the work of
each phase. The partition itself is not in the paper (it defines no kernel);
the contract is:

* classification: n = 1 -> decode, n >= 2 -> prefill, n = 0 -> nothing; in
  the (192, 128) layout (latent attention with heads split out, prefill only)
  every n >= 1 is prefill.
* decode partition (balanced split-K): P_s = ceil(L_s / P); the pages of
  all decode sequences, concatenated in batch order, form a list of
  T = sum_s P_s pages; W = work-groups per key range (grouped-query
  attention: one per group of up to 8 KV heads, W = ceil(Hkv / 8), so a
  work-group reads whole slot rows; the 576/512 latent layout: Hq / 128 when
  128 divides Hq, else Hq / 64). The list is cut into
  R = max(1, min(floor(cus_decode * wg_per_cu / W), floor(T / min_pps)),
  ceil(T / 8192)) ranges, range r = pages [floor(r T / R), floor((r + 1) T / R)),
  min_pps = ceil(min_split_tokens / P). A piece is the non-empty overlap of a
  range with one sequence, keys [k0, k1) = [first page * P,
  min(L_s, end page * P)); pieces are listed by range, i.e. in batch order
  with keys ascending, and the list index is the piece's workspace slot.
  Item words: [s, j, n_s, k0, k1, slot of piece 0 of s, qsl[s], slot], j the
  piece's rank within its sequence and n_s the sequence's piece count. A range
  table of R + 1 words gives the first piece of each range (the last word is
  the piece count), a launch order of the pieces for one-work-group-per-
  piece launches lists them by key count descending, ties by slot, and a
  merge list gives the first piece of every sequence cut into several pieces
  (batch order).
* prefill tiles of BM rows (128 for the latent layout, which also takes 64):
  rows [t*BM, min(n, (t+1)*BM)), key_end = L - n + row_end; ordered by
  key_end descending, then sequence, then tile. Each tile is served by
  Hkv * ceil(G / 8) work-groups (grouped-query) or Hq (latent layouts).
  Grouped-query BM is 16, 32 or 128; BM = 128 makes flat tiles: a row is a
  (token, query head) pair of one KV head, r = token * G + head, so a
  sequence has n * G rows; tile rows [t*BM, min(n*G, (t+1)*BM)), key_end =
  L - n + (row_end - 1) // G + 1 (the causal limit of the last row's token);
  one work-group per (tile, KV head), Hkv of them. With BM unset the
  grouped-query default is 128 when F = sum over prefill sequences of
  ceil(n * G / 128) * Hkv satisfies F >= 4 * cus_prefill, or
  F <= 3 * cus_prefill with cus_prefill < cus_total (a co-run share), else 32.
* co-run CU split: explicit, or (cus_decode = -1) the argmin over multiples of
  the granule of the step time, smallest n_d on ties: with t_p =
  prefill_flops / ((cus_total - n_d) * flops_cu) and r_s = min(hbm, n_d *
  bw_cu), max(decode_bytes / r_s, t_p), or, where a decode tail can form
  (grouped-query heads, decode_tail 0), t_p + max(0, decode_bytes - r_s t_p)
  / min(hbm, cus_total * bw_cu).

* fused order (one launch for both phases), only for grouped-query heads
  with G > 4, W = 1, 3 <= Hkv <= 8 and BM = 32 (else empty): prefill
  work-group e = tile * grid_y + column, decode work-group j holding ranges
  [rpw j, rpw j + rpw) (rpw = 2 when Hkv <= 4, else 1) as entry
  n_tiles * grid_y + j. Launch work-group b runs on XCD b % 8; prefill
  column c belongs to XCD c + grid_y * (tile % (8 / grid_y)) when grid_y
  divides 8 (else to XCD entry % 8), decode work-group j to XCD j % 8. Each
  XCD's entries are listed by their start time in a simulation of its
  cus_total / 8 CUs split into a decode pool of cus_decode / cus_total of
  them (half without a split; at least one CU each; all of them when the
  other phase has no work there) and a prefill pool of the rest, each pool
  giving its phase's work-groups, in order, to its earliest-free CU (lowest
  index on ties). Durations in whole ns plus one: prefill
  2 (d_qk + d_v) x heads of the column x causal pairs of the tile /
  (prefill_tflops_per_cu 1e12); decode pages of the ranges x page bytes /
  (decode_gbps_per_cu 1e9). Ties in start time: prefill first, then phase
  order. Entry 8 k + x is the k-th of XCD x's list, -1 past its end.

Blob layout (int32, version 7): 24-word header (word 19: offset of the
merge list, 20: offset of the fused order, 21: its length, 22: offset of the
lengths, 23: ranges of the decode tail, the last ones of the range table),
8 words per decode item, the range table, the piece launch order,
the merge list, 8 words per prefill item, the fused order, then seq_lens [B]
and query_start_loc [B+1] as given; see ``build_plan``.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED = 0, -1, -2
MAGIC = 0x46504C58
VERSION = 7
HEADER = 24
ITEM = 8
# cost-model rates of one CU when the options leave them 0 (the library's
# defaults: measured with half of an MI355X running one phase alone)
DEFAULT_DECODE_GBPS_PER_CU = 43.0
DEFAULT_PREFILL_TFLOPS_PER_CU = 4.0
DEFAULT_HBM_GBPS = 6500.0
FLAT_WG_CU_SHARE = 0.6        # rate of one flat 4-wave prefill work-group alone, in CUs
PREFILL_LAUNCH_S = 10e-6      # prefill launch latency in the cost model


def cdiv(a: int, b: int) -> int:
    return (a + b - 1) // b


@dataclass
class Shape:
    num_q_heads: int
    num_kv_heads: int
    head_dim_qk: int
    head_dim_v: int
    page_size: int
    sm_scale: float
    v_aliases_k: int


@dataclass
class Opts:
    cus_total: int = 0           # 0 -> 256
    cus_decode: int = 0          # 0 -> all; -1 -> cost model
    bm: int = 0                  # 0 -> 32 or 128 by batch size (128 for the latent layouts)
    min_split_tokens: int = 0    # 0 -> 256
    wg_per_cu: int = 0           # 0 -> 1 (grouped-query), 2 (576/512 latent layout)
    split_granule: int = 0       # 0 -> 32
    hbm_gbps: float = 0.0        # 0 -> 6500
    decode_gbps_per_cu: float = 0.0   # 0 -> 43
    prefill_tflops_per_cu: float = 0.0  # 0 -> 4
    decode_tail: int = 0         # 0 -> a tail group of ranges on grouped-query co-run plans; -1 -> none


@dataclass
class PlanResult:
    status: int
    blob: Optional[List[int]] = None
    info: Optional[dict] = None


MLA_ROWS_PER_WG = 64        # latent heads must be a multiple of this
MLA_ROWS_PER_WG_WIDE = 128  # latent decode work-group rows when they divide Hq
MAX_RANGE_PAGES = 8192


def _supported(sh: Shape) -> bool:
    pair = (sh.head_dim_qk, sh.head_dim_v)
    if pair not in ((64, 64), (128, 128), (576, 512), (192, 128)):
        return False
    if sh.page_size not in (16, 64):
        return False
    if pair == (576, 512):
        return bool(sh.v_aliases_k) and sh.num_q_heads % MLA_ROWS_PER_WG == 0
    if pair == (192, 128):
        return not sh.v_aliases_k and sh.page_size == 64 and (sh.num_q_heads // sh.num_kv_heads) <= 16
    return (sh.num_q_heads // sh.num_kv_heads) <= 16


def build_plan(sh: Shape, opts: Optional[Opts], qsl: Sequence[int], seq_lens: Sequence[int],
               max_pages_per_seq: int) -> PlanResult:
    o = opts or Opts()
    B = len(seq_lens)
    if len(qsl) != B + 1:
        return PlanResult(ERR_INVALID_ARG)
    # --- shape checks
    if sh.num_q_heads <= 0 or sh.num_kv_heads <= 0 or sh.num_q_heads % sh.num_kv_heads:
        return PlanResult(ERR_INVALID_ARG)
    if not (math.isfinite(sh.sm_scale) and sh.sm_scale > 0):
        return PlanResult(ERR_INVALID_ARG)
    if sh.v_aliases_k and (sh.num_kv_heads != 1 or sh.head_dim_v > sh.head_dim_qk):
        return PlanResult(ERR_INVALID_ARG)
    if not _supported(sh):
        return PlanResult(ERR_UNSUPPORTED)
    # --- option checks / defaults
    cus_total = o.cus_total or 256
    wg_per_cu = o.wg_per_cu or (2 if sh.head_dim_qk == 576 else 1)
    min_tokens = o.min_split_tokens or 256
    granule = o.split_granule or 32
    mla = sh.head_dim_qk == 576
    split = sh.head_dim_qk == 192     # heads split out: prefill only, one tile per query head
    bm = o.bm or (128 if mla or split else 0)      # grouped-query default chosen after the CU split
    if cus_total < 1 or wg_per_cu < 1 or min_tokens < 1 or granule < 1:
        return PlanResult(ERR_INVALID_ARG)
    if o.decode_tail not in (0, -1):
        return PlanResult(ERR_INVALID_ARG)
    if o.cus_decode < -1 or o.cus_decode > cus_total:
        return PlanResult(ERR_INVALID_ARG)
    if (mla and bm not in (64, 128)) or (split and bm != 128) or (
            not mla and not split and bm not in (0, 16, 32, 128)):
        return PlanResult(ERR_UNSUPPORTED)
    # --- integer metadata checks
    if max_pages_per_seq < 0:
        return PlanResult(ERR_INVALID_ARG)
    if B > 0 and qsl[0] != 0:
        return PlanResult(ERR_INVALID_ARG)
    P = sh.page_size
    for s in range(B):
        n = qsl[s + 1] - qsl[s]
        L = seq_lens[s]
        if n < 0 or L < 0 or n > L or L > max_pages_per_seq * P:
            return PlanResult(ERR_INVALID_ARG)
    if B > 0 and qsl[B] > 2**31 - 1:
        return PlanResult(ERR_INVALID_ARG)

    heads_per_wg = min(sh.num_kv_heads, 8)
    mla_rows = MLA_ROWS_PER_WG_WIDE if sh.num_q_heads % MLA_ROWS_PER_WG_WIDE == 0 else MLA_ROWS_PER_WG
    W = (sh.num_q_heads // mla_rows) if mla else cdiv(sh.num_kv_heads, heads_per_wg)
    rows_per_wg = mla_rows if mla else heads_per_wg * (sh.num_q_heads // sh.num_kv_heads)
    dec = [s for s in range(B) if qsl[s + 1] - qsl[s] == 1 and not split]
    pre = [s for s in range(B) if qsl[s + 1] - qsl[s] >= (1 if split else 2)]

    # --- co-run CU split
    dec_bytes = 0
    kv_row = sh.num_kv_heads * (sh.head_dim_qk if sh.v_aliases_k else sh.head_dim_qk + sh.head_dim_v) * 2
    for s in dec:
        dec_bytes += seq_lens[s] * kv_row
    pre_flops = 0
    for s in pre:
        n, L = qsl[s + 1] - qsl[s], seq_lens[s]
        pre_flops += sh.num_q_heads * 2 * (sh.head_dim_qk + sh.head_dim_v) * (n * (L - n) + n * (n + 1) // 2)
    # --- grouped-query tile height (used by the cost model below too): 128 flat rows
    # when every prefill CU gets at least four such work-groups or, on a co-run
    # share, when all of them fit in one round (three per CU), else 32 tokens
    G = sh.num_q_heads // sh.num_kv_heads
    flat_wgs = sum(cdiv((qsl[s + 1] - qsl[s]) * G, 128) * sh.num_kv_heads for s in pre)

    def default_bm(cus):
        share = cus < cus_total
        return 128 if (flat_wgs >= 4 * cus or (share and flat_wgs <= 3 * cus)) else 32

    # --- cost-model prefill time on `cus` CUs: grouped-query shapes take the longer of
    # the work at the per-CU rate and the largest work-group (every key of its
    # sequence) at one work-group's rate, plus a launch latency
    bm_opt = bm

    def prefill_time(cus, fl_cu):
        t_work = float(pre_flops) / (float(cus) * fl_cu)
        if mla or split:
            return t_work
        b = bm_opt if bm_opt else default_bm(cus)
        tile = 0.0
        for s in pre:
            n = qsl[s + 1] - qsl[s]
            rows = min(128, n * G) if b == 128 else min(b, n) * min(G, 8)
            tile = max(tile, float(rows) * float(seq_lens[s]) * float(2 * (sh.head_dim_qk + sh.head_dim_v)))
        share = FLAT_WG_CU_SHARE if b == 128 else 1.0
        return max(t_work, tile / (share * fl_cu)) + PREFILL_LAUNCH_S

    if o.cus_decode == 0 or not dec or not pre:
        cus_decode = cus_total
    elif o.cus_decode > 0:
        cus_decode = o.cus_decode
    else:
        hbm = (o.hbm_gbps or DEFAULT_HBM_GBPS) * 1e9
        bw_cu = (o.decode_gbps_per_cu or DEFAULT_DECODE_GBPS_PER_CU) * 1e9
        fl_cu = (o.prefill_tflops_per_cu or DEFAULT_PREFILL_TFLOPS_PER_CU) * 1e12
        tail_model = not mla and not split and o.decode_tail == 0
        r_all = min(hbm, float(cus_total) * bw_cu)
        best, best_t = None, None
        nd = granule
        while nd < cus_total:
            r_share = min(hbm, float(nd) * bw_cu)
            t_pre = prefill_time(cus_total - nd, fl_cu)
            t = max(float(dec_bytes) / r_share, t_pre)
            if tail_model:   # the prefill, then decode's rest on all CUs
                rest = float(dec_bytes) - r_share * t_pre
                t = t_pre + rest / r_all if rest > 0.0 else t_pre
            if best_t is None or t < best_t:
                best, best_t = nd, t
            nd += granule
        cus_decode = best if best is not None else cus_total
    cus_prefill = cus_total - cus_decode if (dec and pre and cus_decode < cus_total) else cus_total

    if bm == 0:
        bm = default_bm(cus_prefill)
    flat = not mla and not split and bm == 128   # rows are (token, query head) pairs of one KV head

    # --- decode partition: balanced page ranges over the concatenated decode sequences;
    # on a grouped-query co-run share, pages [0, TA) for the decode share and a tail
    # group [TA, T) sized for the prefill share (run after the prefill), TA from the
    # cost model: what the decode share covers during the prefill plus its share
    # of the rest at the device's streaming rate
    min_pps = cdiv(min_tokens, P)
    pages = [cdiv(seq_lens[s], P) for s in dec]
    T = sum(pages)
    TA = T
    if not mla and not split and o.decode_tail == 0 and cus_prefill < cus_total and T > 1:
        hbm = (o.hbm_gbps or DEFAULT_HBM_GBPS) * 1e9
        bw_cu = (o.decode_gbps_per_cu or DEFAULT_DECODE_GBPS_PER_CU) * 1e9
        fl_cu = (o.prefill_tflops_per_cu or DEFAULT_PREFILL_TFLOPS_PER_CU) * 1e12
        r_share = min(hbm, float(cus_decode) * bw_cu)
        r_all = min(hbm, float(cus_total) * bw_cu)
        t_pre = prefill_time(cus_prefill, fl_cu)
        during = r_share * t_pre
        if during < float(dec_bytes):
            t_rest = (float(dec_bytes) - during) / r_all
            share_rest = r_all * (float(cus_decode) / float(cus_total)) * t_rest
            frac = (during + share_rest) / float(dec_bytes)
            TA = min(T - 1, max(1, math.floor(frac * float(T))))
    TB = T - TA

    def n_ranges(npages, cus):
        if npages == 0:
            return 0
        return max(1, min((cus * wg_per_cu) // W, npages // min_pps), cdiv(npages, MAX_RANGE_PAGES))
    RA = n_ranges(TA, cus_decode) if dec else 0
    RB = n_ranges(TB, cus_prefill) if dec else 0
    R = RA + RB
    bounds = ([(r * TA) // RA for r in range(RA + 1)] + [TA + (r * TB) // RB for r in range(1, RB + 1)]
              if dec else [0])
    start = [0]
    for n_p in pages:
        start.append(start[-1] + n_p)       # first global page of each decode sequence
    pieces, ranges = [], []
    for r in range(R):
        ranges.append(len(pieces))
        for d, s in enumerate(dec):
            lo, hi = max(bounds[r], start[d]), min(bounds[r + 1], start[d + 1])
            if lo < hi:
                k0 = (lo - start[d]) * P
                k1 = min(seq_lens[s], (hi - start[d]) * P)
                pieces.append([s, d, k0, k1])
    ranges.append(len(pieces))
    dec_items = []
    n_split = 0
    for d, s in enumerate(dec):
        mine = [i for i, pc in enumerate(pieces) if pc[1] == d]
        n_split += len(mine) > 1
        for j, i in enumerate(mine):
            dec_items.append((i, [s, j, len(mine), pieces[i][2], pieces[i][3], mine[0], qsl[s], i]))
    dec_items = [it for _, it in sorted(dec_items, key=lambda x: x[0])]
    ppr = max(cdiv(TA, RA) if RA else 0, cdiv(TB, RB) if RB else 0)

    # --- prefill tiles, longest key range first
    tiles = []
    for s in pre:
        n, L = qsl[s + 1] - qsl[s], seq_lens[s]
        rows = n * G if flat else n          # flat: row r is (token r // G, query head r % G)
        if rows > 2**31 - 1:
            return PlanResult(ERR_INVALID_ARG)
        for t in range(cdiv(rows, bm)):
            r0, r1 = t * bm, min(rows, (t + 1) * bm)
            last_token = (r1 - 1) // G if flat else r1 - 1
            tiles.append([s, t, r0, r1, L - n + last_token + 1, 0, 0, 0])
    tiles.sort(key=lambda it: (-it[4], it[0], it[1]))

    nd_, np_ = len(dec_items), len(tiles)
    order = sorted(range(nd_), key=lambda i: (-(dec_items[i][4] - dec_items[i][3]), i))
    off_ranges = HEADER + ITEM * nd_
    off_order = off_ranges + len(ranges)
    # merge list: the first piece of every decode sequence cut into several pieces
    merge = [it[5] for it in dec_items if it[1] == 0 and it[2] > 1]
    off_merge = off_order + nd_
    off_pre = off_merge + len(merge)
    total = off_pre + ITEM * np_
    pre_height = sh.num_q_heads if mla or split else sh.num_kv_heads * (1 if flat else cdiv(G, 8))
    fused = fused_order(tiles, pre_height, R, T, heads_per_wg,
                        not mla and not split and G > 4 and W == 1 and heads_per_wg >= 3 and bm == 32,
                        G=G, sh=sh, o=o, cus_total=cus_total, cus_decode=cus_decode)
    off_fused = total
    total += len(fused)
    off_lens = total
    total += 2 * B + 1
    hdr = [MAGIC, VERSION, B, nd_, np_, len(dec), len(pre), W, pre_height,
           HEADER, off_pre, ppr, cus_decode, cus_prefill, bm, total, R, off_ranges, off_order, off_merge,
           off_fused, len(fused), off_lens, RB]
    blob = (hdr + [x for it in dec_items for x in it] + ranges + order + merge + [x for it in tiles for x in it]
            + fused + list(seq_lens) + list(qsl))
    # workspace: (max, sum) per decode item, column and row, then the partial outputs;
    # only needed when some decode sequence is split
    if n_split == 0:
        ws = 0
    else:
        stats = nd_ * W * rows_per_wg * 2 * 4
        ws = cdiv(stats, 256) * 256 + nd_ * W * rows_per_wg * sh.head_dim_v * 4
    info = dict(num_seqs=B, n_decode_seqs=len(dec), n_prefill_seqs=len(pre),
                n_decode_items=nd_, n_prefill_items=np_, n_split_seqs=n_split, decode_wg_width=W,
                n_decode_ranges=R, prefill_grid_y=pre_height, pages_per_split=ppr,
                cus_decode=cus_decode, cus_prefill=cus_prefill, bm=bm,
                plan_words=total, device_plan_bytes=cdiv(total * 4, 256) * 256,
                workspace_bytes=ws, decode_bytes=dec_bytes, prefill_flops=pre_flops, n_fused_wgs=len(fused))
    return PlanResult(OK, blob, info)


def fused_order(tiles, grid_y: int, R: int, T: int, kv_heads_per_wg: int, fusable: bool, *, G: int,
                sh: "Shape", o: "Opts", cus_total: int, cus_decode: int) -> List[int]:
    """Work of each work-group of the one-launch form (see the module contract)."""
    if not fusable or (not tiles and R == 0):
        return []
    per_wg = 2 if kv_heads_per_wg <= 4 else 1        # decode ranges per work-group
    n_pre_wg = len(tiles) * grid_y
    fl_cu = (o.prefill_tflops_per_cu or DEFAULT_PREFILL_TFLOPS_PER_CU) * 1e12
    bw_cu = (o.decode_gbps_per_cu or DEFAULT_DECODE_GBPS_PER_CU) * 1e9
    pre_q = [[] for _ in range(8)]                  # per XCD: (entry, duration in ns)
    dec_q = [[] for _ in range(8)]
    columns_per_kv = cdiv(G, 8)
    for i, t in enumerate(tiles):
        r0, r1, kend = t[2], t[3], t[4]
        # query row r of the tile sees keys 0 .. kend - r1 + r (inclusive)
        pairs = sum(kend - r1 + r + 1 for r in range(r0, r1))
        for c in range(grid_y):
            e = i * grid_y + c
            x = c + grid_y * (i % (8 // grid_y)) if 8 % grid_y == 0 else e % 8
            heads = min(8, G - 8 * (c % columns_per_kv))
            flops = float(pairs) * float(heads) * float(2 * (sh.head_dim_qk + sh.head_dim_v))
            pre_q[x].append((e, int(flops / fl_cu * 1e9) + 1))
    page_bytes = sh.page_size * sh.num_kv_heads * (sh.head_dim_qk + sh.head_dim_v) * 2
    for j in range(cdiv(R, per_wg)):
        lo, hi = per_wg * j, min(R, per_wg * j + per_wg)
        nbytes = float((hi * T) // R - (lo * T) // R) * float(page_bytes)
        dec_q[j % 8].append((n_pre_wg + j, int(nbytes / bw_cu * 1e9) + 1))
    cap = max(2, cus_total // 8)                     # CUs of one XCD
    n_dec_cus = cus_decode * cap // cus_total if cus_decode < cus_total else cap // 2
    n_dec_cus = min(cap - 1, max(1, n_dec_cus))

    def starts(queue, machines):
        # each work-group, in order, to the CU that frees up first (lowest index on ties)
        free_at = [0] * machines
        out = []
        for _, dur in queue:
            q = free_at.index(min(free_at))
            out.append(free_at[q])
            free_at[q] += dur
        return out

    lists = []
    for x in range(8):
        sp = starts(pre_q[x], cap if not dec_q[x] else cap - n_dec_cus)
        sd = starts(dec_q[x], cap if not pre_q[x] else n_dec_cus)
        ev = [(t0, 0, k) for k, t0 in enumerate(sp)] + [(t0, 1, k) for k, t0 in enumerate(sd)]
        ev.sort()
        lists.append([pre_q[x][k][0] if kind == 0 else dec_q[x][k][0] for _, kind, k in ev])
    longest = max(len(l) for l in lists)
    order = [-1] * (8 * longest)
    for x in range(8):
        for k, e in enumerate(lists[x]):
            order[8 * k + x] = e
    return order
