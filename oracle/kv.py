"""Commit / rollback of the KV index (test infrastructure, imported only by the
tests, the smoke check and the benchmark's CPU-baseline leg).

A cycle that accepted n of its k drafts commits n + 1 tokens (Sec. 2.2): the
block entries written by verification at positions m .. m+n stay, those at
m+n+1 .. m+k are rolled back.  Closed form: m' = m + n + 1.  Physical slot of
position t of sequence b in a paged cache: block_table[b][t // P] * P + t % P.
"""
from __future__ import annotations

import numpy as np


def kv_commit(lens, n_accept, k: int, block_table, page_size: int):
    """Returns (new_lens [B], committed_slots [B, k+1]: slot of block position i
    if i <= n_b else -1)."""
    lens = np.asarray(lens, dtype=np.int64)
    n = np.asarray(n_accept, dtype=np.int64)
    bt = np.asarray(block_table, dtype=np.int64)
    B = lens.shape[0]
    slots = np.full((B, k + 1), -1, dtype=np.int64)
    for b in range(B):
        for i in range(int(n[b]) + 1):
            t = lens[b] + i
            slots[b, i] = bt[b, t // page_size] * page_size + t % page_size
    return lens + n + 1, slots
