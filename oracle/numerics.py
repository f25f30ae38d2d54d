"""Elementary numerics of the oracle, float64.

Test infrastructure: imported only by the tests, the smoke check and the
benchmark's CPU-baseline leg.
"""
from __future__ import annotations

import numpy as np


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values as the GPU does: to float32 first, then to bfloat16
    by round-to-nearest-even on the upper 16 bits.  Returns float64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    b = f.view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    b = (b + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


class Rounding:
    """Where the bf16 GPU path rounds, the oracle may round too.

    ``exact``    -- no rounding (float64 end to end).
    ``contract`` -- round to bf16 the operands of the matrix products: the
                    normed activations entering the QKV, gate/up, LM-head and
                    MTP projections, Q/K/V after RoPE (K and V as stored in the
                    cache), the attention output entering O and the SwiGLU
                    output entering the down projection.
    """

    def __init__(self, mode: str = "exact"):
        if mode not in ("exact", "contract"):
            raise ValueError(mode)
        self.mode = mode

    def __call__(self, x: np.ndarray) -> np.ndarray:
        return round_bf16(x) if self.mode == "contract" else np.asarray(x, dtype=np.float64)


def softmax(z: np.ndarray, axis: int = -1) -> np.ndarray:
    """exp(z - max z) / sum exp(z - max z), float64; -inf entries get 0."""
    z = np.asarray(z, dtype=np.float64)
    m = np.max(z, axis=axis, keepdims=True)
    e = np.exp(z - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def rmsnorm(x: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    """x * rsqrt(mean(x^2) + eps) * w over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(w, dtype=np.float64)


def silu(x: np.ndarray) -> np.ndarray:
    """x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotary position embedding, rotate-half form.

    x [..., R, heads, d] with positions pos [..., R].  Pairs (i, i + d/2) are
    rotated by the angle pos * base^(-2i/d)."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv          # [..., R, half]
    c = np.cos(ang)[..., None, :]
    s = np.sin(ang)[..., None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def inverse_cdf(w: np.ndarray, u: float):
    """Inverse-CDF draw from unnormalised non-negative weights over ids 0..V-1.

    Returns (x, dist, Z): the smallest id x with C(x) > u * Z, where C is the
    running sum in ascending id order and Z = C(V-1); ``dist`` is the distance
    from u * Z to the nearer edge of x's interval [C(x-1), C(x)), used to flag
    draws that another correct summation order could move."""
    c = np.cumsum(np.asarray(w, dtype=np.float64))
    z = c[-1]
    t = float(u) * z
    x = int(np.argmax(c > t))
    lo = c[x - 1] if x > 0 else 0.0
    return x, min(t - lo, c[x] - t), z


def inverse_cdf_rows(w: np.ndarray, u: np.ndarray):
    """Row-wise ``inverse_cdf``: w [B, V] non-negative, u [B].
    Returns (x [B], dist [B], Z [B])."""
    c = np.cumsum(np.asarray(w, dtype=np.float64), axis=-1)
    z = c[:, -1]
    t = np.asarray(u, dtype=np.float64) * z
    x = np.argmax(c > t[:, None], axis=-1)
    rows = np.arange(c.shape[0])
    lo = np.where(x > 0, c[rows, np.maximum(x - 1, 0)], 0.0)
    return x, np.minimum(t - lo, c[rows, x] - t), z


def nucleus(z: np.ndarray, p: np.ndarray, top_p: float):
    """Nucleus (top-p) truncation of distributions p [..., V] whose logits are
    z [..., V] (the order of p is the order of z).

    The kept set of a row is the shortest prefix of its ids ranked by logit
    (float32, larger first, the lower id first among equal logits) whose total
    probability reaches top_p: the top-p sampling of the paper's evaluation
    setting (App. "Evaluation Configuration").  p is restricted to it and
    renormalised; top_p >= 1 keeps every id.  Returns (p', dist): dist [...] is
    the distance from top_p to the nearer of the two running sums around the
    last kept id (before it and with it), used to flag sets that a correct
    evaluation of the sums in another order could change."""
    p = np.asarray(p, dtype=np.float64)
    if top_p >= 1.0:
        return p / p.sum(axis=-1, keepdims=True), np.full(p.shape[:-1], np.inf)
    z32 = np.asarray(z, dtype=np.float32).astype(np.float64)
    order = np.argsort(-z32, axis=-1, kind="stable")         # stable: lower ids first on ties
    c = np.cumsum(np.take_along_axis(p, order, axis=-1), axis=-1)
    reach = c >= top_p
    n = np.where(reach.any(axis=-1), np.argmax(reach, axis=-1), p.shape[-1] - 1)   # last kept rank
    rank = np.empty_like(order)
    np.put_along_axis(rank, order, np.arange(p.shape[-1]) + np.zeros_like(order), axis=-1)
    out = np.where(rank <= n[..., None], p, 0.0)
    at = np.take_along_axis(c, n[..., None], axis=-1)[..., 0]
    before = np.where(n > 0, np.take_along_axis(c, np.maximum(n - 1, 0)[..., None], axis=-1)[..., 0], 0.0)
    return out / out.sum(axis=-1, keepdims=True), np.minimum(np.abs(at - top_p), np.abs(before - top_p))
