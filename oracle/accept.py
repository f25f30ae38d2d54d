"""Accept / reject of a draft block (float64).

Test infrastructure: imported only by the tests, the smoke check and the
benchmark's CPU-baseline leg.

Sec. 2.2: the target verifies the K drafts in one forward and accepts draft
d_i with probability min(1, p_i(d_i) / q_i(d_i)) (Eq. accept-rule), scanning
i = 1..K and stopping at the first rejection, so the accepted positions form a
prefix and one integer n per sequence records the decision (App. "Implementing
Draft-Path Reconstruction in verl": the accepted length; first rejection
j = n + 1, with j = K + 1 when all are accepted).  At the first rejection a
replacement is drawn from the corrected distribution; if all K are accepted a
bonus token is drawn from p_{K+1}.  The cycle commits n + 1 tokens, so the
acceptance length tau lies in [1, K + 1].

Readings where the paper is silent:
* the corrected distribution is norm(max(0, p - q)), the residual of the
  speculative-sampling papers the section cites;
* a draft is accepted iff u < p(d) / q(d) with the supplied u in [0, 1), so
  p(d) >= q(d) always accepts; the ratio is taken in the kernel's precision
  (float32) before the comparison;
* every draw is an inverse-CDF draw in ascending id order with a supplied
  uniform (u_final serves either the residual or the bonus draw); if the
  residual mass is zero the draw falls back to p;
* both p and q are softmax(z / T) with the same temperature T;
* greedy mode (not used by the paper, whose rollouts sample at T = 1) accepts
  d_i iff d_i is the argmax of the float32 target logits (lowest id on ties)
  and commits the argmax of row n + 1;
* top-p (the evaluation setting: T = 1, top-p 0.7, rejection sampling, App.
  "Evaluation Configuration"): every p_i and q_i is replaced by its nucleus
  (``numerics.nucleus``) before the rule, so the drafts are samples of the
  truncated head distribution and the committed tokens are distributed as the
  truncated target; greedy mode ignores top_p (the argmax is always kept).

Flags mark decisions that a correct float32 evaluation could take the other
way: an examined accept test with |u - min(1, p/q)| < accept_eps, a greedy
row whose top-2 logit margin is < margin_eps, a final draw whose target
u * Z lies within final_eps * Z + final_abs of an edge of the chosen id's CDF
interval (final_abs in probability units, a scalar or one value per
sequence), and a nucleus whose boundary lies within nucleus_eps of top_p.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

from .numerics import softmax, inverse_cdf_rows, nucleus


@dataclasses.dataclass
class AcceptResult:
    n_accept: np.ndarray        # [B] accepted drafts n_b in [0, k]
    out_tokens: np.ndarray      # [B, k+1] accepted drafts then the final token, -1 after
    flagged: np.ndarray         # [B] some decision of this sequence lies within a flag window
    flag_accept: np.ndarray     # [B] an examined accept test / greedy row is near its threshold
    flag_final: np.ndarray      # [B] the final draw / greedy final row is near its threshold
    alpha: Optional[np.ndarray] = None   # [B, k] sum_x min(p_i, q_i) (sample mode)


def _top2_margin(z: np.ndarray) -> float:
    if z.size < 2:
        return np.inf
    s = np.partition(z, z.size - 2)
    return float(s[-1] - s[-2])


def spec_accept(target_logits, draft_logits, drafts, u_accept, u_final, mode: str = "sample",
                temperature: float = 1.0, accept_eps: float = 1e-3, margin_eps: float = 1e-2,
                final_eps: float = 0.0, top_p: float = 1.0, nucleus_eps: float = 0.0,
                final_abs=0.0) -> AcceptResult:
    """target_logits [B, k+1, V]; draft_logits [B, k, V] (None in greedy mode);
    drafts [B, k]; u_accept [B, k]; u_final [B]."""
    zt = np.asarray(target_logits, dtype=np.float64)
    B, k1, V = zt.shape
    k = k1 - 1
    drafts = np.asarray(drafts).reshape(B, k)
    n = np.zeros(B, dtype=np.int64)
    out = np.full((B, k + 1), -1, dtype=np.int64)
    f_acc = np.zeros(B, dtype=bool)
    f_fin = np.zeros(B, dtype=bool)
    alpha = None

    if mode == "greedy":
        for b in range(B):
            i = 0
            while i < k:
                row = zt[b, i].astype(np.float32)
                if _top2_margin(row) < margin_eps:
                    f_acc[b] = True
                if drafts[b, i] != int(np.argmax(row)):
                    break
                i += 1
            n[b] = i
            row = zt[b, i].astype(np.float32)
            if _top2_margin(row) < margin_eps:
                f_fin[b] = True
            out[b, :i] = drafts[b, :i]
            out[b, i] = int(np.argmax(row))
    elif mode == "sample":
        zq = np.asarray(draft_logits, dtype=np.float64)
        p = softmax(zt / temperature, axis=-1)                      # [B, k+1, V]
        q = softmax(zq / temperature, axis=-1)                      # [B, k, V]
        if top_p < 1.0:
            p, dist_p = nucleus(zt, p, top_p)
            q, dist_q = nucleus(zq, q, top_p)
            f_acc |= (dist_p < nucleus_eps).any(axis=-1)
            if k:
                f_acc |= (dist_q < nucleus_eps).any(axis=-1)
        alpha = np.minimum(p[:, :k], q).sum(axis=-1)                # Eq. alpha
        rows = np.arange(B)
        alive = np.ones(B, dtype=bool)       # no rejection yet: position i is examined
        for i in range(k):
            d = drafts[:, i]
            pd, qd = p[rows, i, d], q[rows, i, d]
            with np.errstate(divide="ignore", invalid="ignore"):
                ratio = np.where(qd > 0, pd / np.where(qd > 0, qd, 1.0), np.inf).astype(np.float32)
            u = np.asarray(u_accept[:, i], dtype=np.float32)
            f_acc |= alive & (np.abs(u.astype(np.float64) - np.minimum(1.0, ratio)) < accept_eps)
            alive &= u < ratio                                       # Eq. accept-rule
            n += alive
        # first rejection at row n < k: residual max(0, p - q); all accepted: bonus from p_{k+1}
        q_rows = np.concatenate([q, np.zeros((B, 1, V))], axis=1)[rows, n]
        p_rows = p[rows, n]
        w = np.maximum(p_rows - q_rows, 0.0)
        empty = ~(w.sum(axis=-1) > 0.0)
        w[empty] = p_rows[empty]
        x, dist, z = inverse_cdf_rows(w, u_final)
        f_fin = dist < final_eps * z + np.broadcast_to(np.asarray(final_abs, dtype=np.float64), (B,))
        for b in range(B):
            out[b, :n[b]] = drafts[b, :n[b]]
            out[b, n[b]] = x[b]
    else:
        raise ValueError(mode)
    return AcceptResult(n, out, f_acc | f_fin, f_acc, f_fin, alpha)
