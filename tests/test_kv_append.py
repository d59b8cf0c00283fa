"""Pins of the KV-append oracle (CPU only).

The append has a plain definition (a paged row write), so the oracle is that
definition; these tests pin it to something other than itself: reading the
appended rows back through the attention oracle's independent block-table
gather, rows that must not change, and the skip rules.
"""
import numpy as np
import torch

import oracle.attention as OA
import oracle.kv_append as KA
from paper_2606_04415_amd.workloads import WORKLOADS, make_append, make_batch


def u16(t):
    return None if t is None else t.view(torch.int16).numpy().astype(np.int64)


def test_round_trip_through_block_table_gather():
    # Append every key of fresh sequences (all tokens new); gathering each
    # sequence back through its block table must return the new rows exactly.
    w = WORKLOADS["tiny"]
    b = make_batch(w, seed=5, ns=[40, 1, 17], ls=[40, 33, 17])
    a = make_append(b, seed=6)
    k, v, bad = KA.kv_append(u16(b.k_cache), u16(b.v_cache), u16(a.k_new), u16(a.v_new), a.slot_mapping.numpy())
    assert bad == 0
    qsl = b.query_start_loc.tolist()
    # token order of make_append before shuffling: sequences in order, queries in order
    sm = a.slot_mapping.tolist()
    for s, (n, L) in enumerate(zip(b.extra["ns"], b.extra["ls"])):
        Kg = OA.gather_sequence(k, b.block_table[s].numpy(), L, w.page_size)
        Vg = OA.gather_sequence(v, b.block_table[s].numpy(), L, w.page_size)
        for i in range(n):
            pos = L - n + i
            slot = int(b.block_table[s, pos // w.page_size]) * w.page_size + pos % w.page_size
            t = sm.index(slot)
            assert np.array_equal(Kg[pos], u16(a.k_new)[t])
            assert np.array_equal(Vg[pos], u16(a.v_new)[t])
        # keys before the new ones keep the batch's rows
        old = OA.gather_sequence(u16(b.k_cache), b.block_table[s].numpy(), L - n, w.page_size)
        assert np.array_equal(Kg[:L - n], old)
    assert qsl[-1] == len(sm)


def test_untouched_rows_and_skip_rules():
    w = WORKLOADS["tiny"]
    b = make_batch(w, seed=1, poison=False)
    a = make_append(b, seed=2, n_pad=5, n_out_of_range=3)
    k0, v0 = u16(b.k_cache), u16(b.v_cache)
    k, v, bad = KA.kv_append(k0, v0, u16(a.k_new), u16(a.v_new), a.slot_mapping.numpy())
    assert bad == 3
    P = w.page_size
    written = {s for s in a.slot_mapping.tolist() if 0 <= s < k0.shape[0] * P}
    assert len(written) == len(a.slot_mapping) - 8
    changed = {p * P + r for p in range(k0.shape[0]) for r in range(P)
               if not np.array_equal(k[p, r], k0[p, r])}
    assert changed <= written                 # nothing outside the slots moved
    for p in range(k0.shape[0]):
        for r in range(P):
            if p * P + r not in written:
                assert np.array_equal(v[p, r], v0[p, r])
    # inputs are not modified
    assert np.array_equal(k0, u16(b.k_cache))


def test_aliased_values_and_empty_append():
    w = WORKLOADS["mla"]
    b = make_batch(w, seed=0, ns=[1, 3], ls=[70, 3], poison=False)
    a = make_append(b, seed=3)
    assert a.v_new is None
    k, v, bad = KA.kv_append(u16(b.k_cache), None, u16(a.k_new), None, a.slot_mapping.numpy())
    assert v is None and bad == 0
    for t, slot in enumerate(a.slot_mapping.tolist()):
        assert np.array_equal(k[slot // 64, slot % 64], u16(a.k_new)[t])
    k2, _, bad2 = KA.kv_append(k, None, u16(a.k_new)[:0], None, np.zeros(0, dtype=np.int32))
    assert bad2 == 0 and np.array_equal(k2, k)


def test_planted_mistake_is_caught():
    # A write to the transposed (row, page) location must fail the round trip.
    w = WORKLOADS["tiny"]
    b = make_batch(w, seed=5, ns=[20], ls=[40])
    a = make_append(b, seed=6)
    k0 = u16(b.k_cache)
    k = k0.copy()
    P = w.page_size
    for t, slot in enumerate(a.slot_mapping.tolist()):
        page, row = divmod(slot, P)
        k[row % k.shape[0], page % P] = u16(a.k_new)[t]     # wrong index order
    ref, _, _ = KA.kv_append(k0, None, u16(a.k_new), None, a.slot_mapping.numpy())
    assert not np.array_equal(k, ref)
