"""Top-1 mixing draft construction (an input recipe of the benchmark
workloads, not part of the method).  Test infrastructure: imported only by the
tests, the smoke check and the benchmark's CPU-baseline leg.

Draft i of a sequence is the target's top-1 token at block position i given
[t_m, d_1 .. d_{i-1}] with a fixed probability, otherwise a uniform token.
Because the block is causal, top-1 at position i depends only on the drafts
before it, so the drafts are built left to right, one target forward per
position.  The top-1 is taken on the float32 logits in the given rounding
mode, lowest id on ties.
"""
from __future__ import annotations

import numpy as np

from .model import verify_forward


def mixing_drafts(shape, W, caches, lens, pending, take_top1, alt, rnd):
    """pending [B] tokens t_m; take_top1 [B, k] bool; alt [B, k] uniform tokens."""
    B, k = take_top1.shape
    block = np.asarray(pending, dtype=np.int64).reshape(B, 1)
    drafts = np.zeros((B, k), dtype=np.int64)
    for i in range(k):
        logits, _, _ = verify_forward(shape, W, caches, block, lens, rnd, lm_rows=[i])
        top1 = np.argmax(logits[:, 0].astype(np.float32), axis=-1)
        drafts[:, i] = np.where(take_top1[:, i], top1, alt[:, i])
        block = np.concatenate([block, drafts[:, i:i + 1]], axis=1)
    return drafts
