"""CPU oracle for appending new tokens' key/value rows to the paged KV pool.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module. The library never
does, and this module imports nothing from the library.

What it computes. Co-located prefill and decode extend and read one shared KV
pool in place (Sec. 3.4, "Memory Locality"); the paper gives no write rule, so
this is the plain definition of a paged write: token t's key row (and value row
unless values alias keys) goes to page ``slot_mapping[t] // P``, row
``slot_mapping[t] % P`` of the caches laid out [page][slot][kv_head][dim]. A
negative slot skips its token; a slot at or past ``num_pages * P`` skips it
too and counts it as out of range. Rows are copied bit for bit (uint16 views
of bf16), so the comparison with the device is exact.

Pins: tests/test_kv_append.py (round trip through a block-table gather,
untouched rows, skip rules).
"""
from __future__ import annotations

from typing import Optional, Tuple

import numpy as np


def kv_append(k_cache: np.ndarray, v_cache: Optional[np.ndarray], k_new: np.ndarray,
              v_new: Optional[np.ndarray], slot_mapping: np.ndarray) -> Tuple[np.ndarray, Optional[np.ndarray], int]:
    """Return (k_cache', v_cache', out_of_range) after the append; inputs are not modified.

    k_cache [pages, P, Hkv, d_qk], v_cache [pages, P, Hkv, d_v] or None (aliased),
    k_new [n, Hkv, d_qk], v_new [n, Hkv, d_v] or None, slot_mapping [n] ints.
    Tokens are written in order, so a later token given the same slot wins
    (the device leaves one of them; tests use distinct slots).
    """
    k = k_cache.copy()
    v = None if v_cache is None else v_cache.copy()
    pages, P = k.shape[0], k.shape[1]
    bad = 0
    for t, slot in enumerate(np.asarray(slot_mapping).tolist()):
        if slot < 0:
            continue
        if slot >= pages * P:
            bad += 1
            continue
        page, row = divmod(slot, P)
        k[page, row] = k_new[t]
        if v is not None:
            v[page, row] = v_new[t]
    return k, v, bad
