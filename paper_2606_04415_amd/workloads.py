"""Seeded synthetic workloads for mixed prefill/decode paged attention.

This module only draws inputs: shapes, lengths, page permutations and random
tensors. It holds none of the attention arithmetic, so both the fp64 oracle
(test infrastructure) and the HIP path can consume its batches without sharing
any computation.

The paper characterises the two phases that share one device (prefill is
compute-heavy, decode is bound by KV-cache traffic; Abstract, Sec. 1, Sec. 3.4)
and evaluates on Qwen2.5-7B and DeepSeek-R1 (Sec. 4.1, Sec. 4.3, Sec. 4.4). It
gives no attention shapes, so the five workloads below take the standard
attention geometry of those two models:

* Qwen2.5-7B: 28 query heads, 4 KV heads (GQA 7:1), head_dim 128.
* DeepSeek-R1 MLA in absorbed form: 128 query heads, one latent KV head of
  width 576 (512 latent + 64 rope), value width 512 (the first 512 columns of
  the latent row), softmax scale 1/sqrt(192); and for prefill with its heads
  split out: 128 heads with keys of 192 (128 + 64 rope) and values of 128.

Draw order for a workload (one torch CPU generator, seeded):
  1. ``seq_lens`` per segment, in batch order, via ``randint(lo, hi + 1)``;
  2. the physical page permutation, ``randperm(num_pages)``;
  3. q, 4. k_cache, 5. v_cache (skipped when V aliases K): ``randn`` in fp32,
     rounded to bf16 (round-to-nearest-even, by torch).
Logical page k of the batch (sequences in batch order, pages in order within a
sequence) lives in physical page ``perm[k]``.

Poisoning (optional, used by correctness runs): physical pages that no
sequence references are filled with NaN, and cache slots past a sequence's
last key inside its last page are filled with +/-1e4, so that a wrong page
index or an unmasked tail read shows up in the output. Block-table entries
past a sequence's last page point at a NaN page.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import torch


@dataclass(frozen=True)
class Segment:
    """A run of sequences with the same query-length rule.

    ``n`` is the number of new query tokens per sequence (``None`` means the
    whole context is new, i.e. n == L). ``seq_len`` is either a fixed length or
    an inclusive (lo, hi) range drawn uniformly per sequence.
    """
    count: int
    n: Optional[int]
    seq_len: Tuple[int, int]


@dataclass(frozen=True)
class Workload:
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim_qk: int
    head_dim_v: int
    page_size: int
    sm_scale: float
    v_aliases_k: bool
    segments: Tuple[Segment, ...]
    num_pages: Optional[int] = None      # None: exactly the pages referenced
    description: str = ""

    @property
    def batch(self) -> int:
        return sum(s.count for s in self.segments)

    @property
    def max_pages_per_seq(self) -> int:
        return max(-(-s.seq_len[1] // self.page_size) for s in self.segments)


WORKLOADS = {
    "tiny": Workload(
        name="tiny", num_q_heads=4, num_kv_heads=1, head_dim_qk=64, head_dim_v=64,
        page_size=16, sm_scale=1.0 / 8.0, v_aliases_k=False,
        segments=(Segment(2, None, (64, 64)), Segment(4, 1, (128, 128))),
        num_pages=64,
        description="tiny mixed batch: 2 prompts of 64 tokens + 4 decodes over 128-token "
                    "contexts; GQA 4/1, head_dim 64, page 16, 64 physical pages"),
    "decode": Workload(
        name="decode", num_q_heads=28, num_kv_heads=4, head_dim_qk=128, head_dim_v=128,
        page_size=16, sm_scale=1.0 / math.sqrt(128.0), v_aliases_k=False,
        segments=(Segment(64, 1, (512, 4096)),),
        description="Qwen2.5-7B-shaped decode: 64 sequences, context U[512,4096], page 16"),
    "prefill": Workload(
        name="prefill", num_q_heads=28, num_kv_heads=4, head_dim_qk=128, head_dim_v=128,
        page_size=16, sm_scale=1.0 / math.sqrt(128.0), v_aliases_k=False,
        segments=(Segment(8, None, (2048, 2048)),),
        description="Qwen2.5-7B-shaped prefill: 8 causal prompts of 2048 tokens, page 16"),
    "mixed": Workload(
        name="mixed", num_q_heads=28, num_kv_heads=4, head_dim_qk=128, head_dim_v=128,
        page_size=16, sm_scale=1.0 / math.sqrt(128.0), v_aliases_k=False,
        segments=(Segment(1, 2048, (6144, 6144)), Segment(128, 1, (1024, 8192))),
        description="Qwen2.5-7B-shaped mixed step: one 2048-token chunk on 4096 cached tokens "
                    "+ 128 decodes with context U[1024,8192], page 16"),
    "mla": Workload(
        name="mla", num_q_heads=128, num_kv_heads=1, head_dim_qk=576, head_dim_v=512,
        page_size=64, sm_scale=1.0 / math.sqrt(192.0), v_aliases_k=True,
        segments=(Segment(256, 1, (1024, 16384)), Segment(1, None, (4096, 4096))),
        description="DeepSeek-R1-style absorbed MLA, one GPU's share: 128 heads, latent 576 "
                    "(V = first 512), page 64; 256 decodes U[1024,16384] + one 4096-token prompt"),
    "mla_split": Workload(
        name="mla_split", num_q_heads=128, num_kv_heads=128, head_dim_qk=192, head_dim_v=128,
        page_size=64, sm_scale=1.0 / math.sqrt(192.0), v_aliases_k=False,
        segments=(Segment(1, None, (4096, 4096)),),
        description="DeepSeek-R1-style MLA prefill with heads split out (keys 128 + 64 rope, values 128, "
                    "128 heads), page 64; one 4096-token prompt"),
}


@dataclass
class Batch:
    """One synthetic batch on the host (torch CPU tensors)."""
    workload: Workload
    seq_lens: torch.Tensor          # int32 [B]
    query_start_loc: torch.Tensor   # int32 [B+1]
    block_table: torch.Tensor       # int32 [B, max_pages_per_seq]
    q: torch.Tensor                 # bf16 [T, Hq, d_qk]
    k_cache: torch.Tensor           # bf16 [num_pages, P, Hkv, d_qk]
    v_cache: Optional[torch.Tensor]  # bf16 [num_pages, P, Hkv, d_v] (None when V aliases K)
    num_pages: int
    used_pages: int
    extra: dict = field(default_factory=dict)

    @property
    def total_q(self) -> int:
        return int(self.query_start_loc[-1])


def draw_lengths(w: Workload, gen: torch.Generator) -> Tuple[List[int], List[int]]:
    """Step 1 of the draw order: per-sequence (n, L) in batch order."""
    ns: List[int] = []
    ls: List[int] = []
    for seg in w.segments:
        lo, hi = seg.seq_len
        if lo == hi:
            lens = [lo] * seg.count
        else:
            lens = torch.randint(lo, hi + 1, (seg.count,), generator=gen).tolist()
        for L in lens:
            ls.append(int(L))
            ns.append(int(L) if seg.n is None else seg.n)
    return ns, ls


def make_batch(w: Workload, seed: int = 0, poison: bool = True,
               ns: Optional[List[int]] = None, ls: Optional[List[int]] = None,
               num_pages: Optional[int] = None, device=None) -> Batch:
    """Draw one batch of ``w``. ``ns``/``ls`` override the drawn lengths (tests).

    With ``device`` (e.g. "cuda"), steps 3-5 of the draw order run on that
    device with a generator of its own seeded with ``seed``: the same shapes
    and distributions, other values than the CPU draw, and the tensors stay
    on the device (the benchmark draws its large workloads this way)."""
    gen = torch.Generator().manual_seed(seed)
    if ns is None or ls is None:
        ns, ls = draw_lengths(w, gen)
    P = w.page_size
    B = len(ls)
    pages_per_seq = [-(-L // P) for L in ls]
    used = sum(pages_per_seq)
    npages = num_pages if num_pages is not None else (w.num_pages or used)
    if npages < used:
        raise ValueError(f"{npages} physical pages cannot hold {used} logical pages")
    trap_page = None
    if npages == used:
        # one extra NaN page that unused block-table entries point at
        npages_alloc = npages + 1
        trap_page = npages
    else:
        npages_alloc = npages
    perm = torch.randperm(npages, generator=gen)
    T = sum(ns)
    tgen, tdev = gen, None
    if device is not None:
        tdev = torch.device(device)
        tgen = torch.Generator(device=tdev).manual_seed(seed)
    q = torch.randn((T, w.num_q_heads, w.head_dim_qk), generator=tgen, device=tdev).to(torch.bfloat16)
    k = torch.randn((npages_alloc, P, w.num_kv_heads, w.head_dim_qk), generator=tgen, device=tdev).to(torch.bfloat16)
    v = None
    if not w.v_aliases_k:
        v = torch.randn((npages_alloc, P, w.num_kv_heads, w.head_dim_v), generator=tgen,
                        device=tdev).to(torch.bfloat16)

    max_pages = max([w.max_pages_per_seq] + pages_per_seq)
    bt = torch.empty((B, max_pages), dtype=torch.int32)
    logical = 0
    for s, np_ in enumerate(pages_per_seq):
        bt[s, :np_] = perm[logical:logical + np_].to(torch.int32)
        logical += np_
    used_phys = set(perm[:used].tolist())
    unused = [p for p in range(npages_alloc) if p not in used_phys]
    if trap_page is None:
        trap_page = unused[0]
    for s, np_ in enumerate(pages_per_seq):
        bt[s, np_:] = trap_page

    if poison:
        nan = float("nan")
        for p in unused:
            k[p] = nan
            if v is not None:
                v[p] = nan
        for s, L in enumerate(ls):
            tail = L % P
            if tail:
                last = int(bt[s, pages_per_seq[s] - 1])
                k[last, tail:] = 1.0e4
                if v is not None:
                    v[last, tail:] = -1.0e4
    else:
        for p in unused:
            k[p] = 0
            if v is not None:
                v[p] = 0

    qsl = torch.zeros(B + 1, dtype=torch.int32)
    qsl[1:] = torch.cumsum(torch.tensor(ns, dtype=torch.int64), 0).to(torch.int32)
    return Batch(workload=w, seq_lens=torch.tensor(ls, dtype=torch.int32), query_start_loc=qsl,
                 block_table=bt, q=q, k_cache=k, v_cache=v, num_pages=npages_alloc,
                 used_pages=used, extra={"ns": ns, "ls": ls})


def algorithmic_work(w: Workload, ns: List[int], ls: List[int]) -> dict:
    """Bytes the method must move and flops it must do (causal pairs only).

    Bytes: each referenced key/value row once (V counted with K when it aliases
    K), the query rows, the output rows and the block-table entries in use.
    Flops: 2*(d_qk + d_v) per (query head, causal query-key pair).
    Split by phase: sequences with one new token are decode, longer ones prefill.
    """
    Hq, Hkv, dqk, dv, P = w.num_q_heads, w.num_kv_heads, w.head_dim_qk, w.head_dim_v, w.page_size
    out = {"decode": {"bytes": 0, "flops": 0}, "prefill": {"bytes": 0, "flops": 0}}
    kv_row = Hkv * (dqk if w.v_aliases_k else dqk + dv) * 2
    for n, L in zip(ns, ls):
        if n == 0:
            continue
        ph = "decode" if n == 1 else "prefill"
        pairs = n * (L - n) + n * (n + 1) // 2
        out[ph]["flops"] += Hq * 2 * (dqk + dv) * pairs
        out[ph]["bytes"] += L * kv_row + n * Hq * (dqk + dv) * 2 + 4 * (-(-L // P))
    return out


@dataclass
class AppendBatch:
    """New tokens' rows and their cache slots (torch CPU tensors)."""
    k_new: torch.Tensor             # bf16 [n, Hkv, d_qk]
    v_new: Optional[torch.Tensor]   # bf16 [n, Hkv, d_v] (None when V aliases K)
    slot_mapping: torch.Tensor      # int32 [n]
    n_pad: int                      # entries set to -1
    n_out_of_range: int             # entries at or past num_pages * P


def make_append(b: Batch, seed: int = 0, n_pad: int = 0, n_out_of_range: int = 0) -> AppendBatch:
    """The new tokens of batch ``b`` as a serving step would append them before
    its attention: query i of sequence s is key position L - n + i, whose slot
    is ``block_table[s][pos // P] * P + pos % P`` (the position-to-slot map an
    engine keeps). ``n_pad`` padding entries (-1) and ``n_out_of_range`` entries
    past the pool are then inserted at seeded random positions.

    Draw order (one torch CPU generator, seeded): k_new, v_new (skipped when V
    aliases K) as ``randn`` rounded to bf16; then ``randperm`` of the final
    token count to place the padding and out-of-range entries.
    """
    w = b.workload
    gen = torch.Generator().manual_seed(seed)
    ns, ls = b.extra["ns"], b.extra["ls"]
    P = w.page_size
    slots = []
    for s, (n, L) in enumerate(zip(ns, ls)):
        for i in range(n):
            pos = L - n + i
            slots.append(int(b.block_table[s, pos // P]) * P + pos % P)
    extra = [-1] * n_pad + [b.num_pages * P + 7 * j for j in range(n_out_of_range)]
    n_tot = len(slots) + len(extra)
    k_new = torch.randn((n_tot, w.num_kv_heads, w.head_dim_qk), generator=gen).to(torch.bfloat16)
    v_new = None
    if not w.v_aliases_k:
        v_new = torch.randn((n_tot, w.num_kv_heads, w.head_dim_v), generator=gen).to(torch.bfloat16)
    order = torch.randperm(n_tot, generator=gen).tolist()
    merged = [0] * n_tot
    vals = slots + extra
    for dst, src in zip(order, range(n_tot)):
        merged[dst] = vals[src]
    return AppendBatch(k_new=k_new, v_new=v_new, slot_mapping=torch.tensor(merged, dtype=torch.int32),
                       n_pad=n_pad, n_out_of_range=n_out_of_range)
