"""Cycle record of one verification (test infrastructure; see the package docstring).

App. "Implementing Draft-Path Reconstruction in verl" (recording in rollout):
the record of a cycle keeps, at every draft position, the target's
verification distribution truncated to its 64 largest entries, as
log-probabilities stored in bf16 that keep the full-vocabulary normalisation
(they are not renormalised over the kept set).  The distribution at draft
position i is p_i = softmax(z_i / T) of the block row that verifies d_i
(Sec. 2.2), i.e. block rows 0 .. k-1 of the verification.

Reading where the paper is silent: entries come in decreasing probability,
equal probabilities in increasing id.  The order is taken on the logits
themselves, which for T > 0 is the order of z / T and of p.
"""
import numpy as np

from .numerics import round_bf16


def record_topk(target_logits: np.ndarray, k: int, temperature: float = 1.0, topk: int = 64):
    """Top-`topk` entries of p_i = softmax(z_i / T) for block rows i = 0 .. k-1.

    target_logits: [B, k+1, V] (float32 values).  Returns (ids [B, k, topk] int64,
    logp [B, k, topk] float64 holding bf16 values: log p_i(id) with the
    full-vocabulary normaliser, rounded to bf16)."""
    z = np.asarray(target_logits, dtype=np.float64)
    B, k1, V = z.shape
    if k1 != k + 1 or not (1 <= topk <= V) or not temperature > 0:
        raise ValueError("record_topk: bad shapes or arguments")
    ids = np.zeros((B, k, topk), dtype=np.int64)
    logp = np.zeros((B, k, topk), dtype=np.float64)
    for b in range(B):
        for i in range(k):
            row = z[b, i]
            # decreasing logit, then increasing id (lexsort sorts by the last key first)
            order = np.lexsort((np.arange(V), -row))[:topk]
            s = row / temperature
            m = s.max()
            lse = m + np.log(np.sum(np.exp(s - m)))      # log of the full-vocabulary normaliser
            ids[b, i] = order
            logp[b, i] = round_bf16(s[order] - lse)
    return ids, logp
