"""Target-model forward of the oracle (float64).

Test infrastructure: imported only by the tests, the smoke check and the
benchmark's CPU-baseline leg.

Verification (Sec. 3.1, Eq. verification-context) feeds the target the
committed context followed by the draft block and reads the target
distribution at every block position; it is one forward over the draft path
(App. "Draft-Path Reconstruction").  The plain definition of that forward is
a causal forward over the whole sequence with no cache, read at the block
positions: ``full_forward``.  ``verify_forward`` computes the same rows from a
KV cache of the committed prefix, as a rollout engine does.

The decoder is the pre-norm layer of the paper's backbones (Qwen3 / Qwen2
family, App. "Models and Draft Heads"):
    x <- x + W_o . Attn(RoPE(W_q n), RoPE(W_k n), W_v n),   n = RMSNorm(x)
    x <- x + W_down (silu(W_gate n) * W_up n),             n = RMSNorm(x)
followed by a final RMSNorm and the LM head.  Attention is causal, grouped
(query head h reads KV head h // (n_heads / n_kv_heads)) and scaled by
1/sqrt(head_dim).  The hidden state handed to the draft head is the last
layer's output before the final RMSNorm.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np

from .numerics import Rounding, rmsnorm, rope, silu, softmax, inverse_cdf


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_visible: np.ndarray) -> np.ndarray:
    """Grouped causal attention of one sequence.

    q [R, n_heads, d]; k, v [L, n_kv_heads, d]; row r attends to keys
    0 .. n_visible[r]-1.  Returns [R, n_heads, d]."""
    R, nq, d = q.shape
    L, nkv, _ = k.shape
    group = nq // nkv
    visible = np.arange(L)[None, :] < np.asarray(n_visible)[:, None]
    out = np.empty((R, nq, d))
    for h in range(nq):
        j = h // group
        s = (q[:, h, :] @ k[:, j, :].T) / np.sqrt(d)
        s = np.where(visible, s, -np.inf)
        out[:, h, :] = softmax(s, axis=-1) @ v[:, j, :]
    return out


def layer_forward(shape, Wl, x: np.ndarray, pos: np.ndarray,
                  cache_k: Sequence[np.ndarray], cache_v: Sequence[np.ndarray],
                  rnd: Rounding):
    """One decoder layer over R consecutive positions of each of B sequences.

    x [B, R, H]; pos [B, R] absolute positions; cache_k[b] / cache_v[b]
    [m_b, n_kv, d] hold the entries of positions 0 .. m_b-1, and pos[b] starts
    at m_b.  Row r of sequence b sees the cache and rows 0..r.
    Returns (x_out [B, R, H], k_new [B, R, n_kv, d], v_new [B, R, n_kv, d])."""
    B, R, H = x.shape
    nq, nkv, d = shape.n_heads, shape.n_kv_heads, shape.head_dim
    n = rnd(rmsnorm(x, Wl["attn_norm"], shape.rms_eps))
    q = (n @ _f64(Wl["wq"]).T).reshape(B, R, nq, d)
    k = (n @ _f64(Wl["wk"]).T).reshape(B, R, nkv, d)
    v = (n @ _f64(Wl["wv"]).T).reshape(B, R, nkv, d)
    if shape.qk_norm:
        q = rmsnorm(q, Wl["q_norm"], shape.rms_eps)
        k = rmsnorm(k, Wl["k_norm"], shape.rms_eps)
    q = rnd(rope(q, pos, shape.rope_base))
    k = rnd(rope(k, pos, shape.rope_base))
    v = rnd(v)
    o = np.empty((B, R, nq, d))
    for b in range(B):
        m = cache_k[b].shape[0]
        K = np.concatenate([_f64(cache_k[b]), k[b]], axis=0)
        V = np.concatenate([_f64(cache_v[b]), v[b]], axis=0)
        o[b] = attention(q[b], K, V, m + np.arange(R) + 1)
    o = rnd(o).reshape(B, R, nq * d)
    x = x + o @ _f64(Wl["wo"]).T
    n2 = rnd(rmsnorm(x, Wl["ffn_norm"], shape.rms_eps))
    h = rnd(silu(n2 @ _f64(Wl["w_gate"]).T) * (n2 @ _f64(Wl["w_up"]).T))
    x = x + h @ _f64(Wl["w_down"]).T
    return x, k, v


def lm_head(shape, W, hidden: np.ndarray, rnd: Rounding) -> np.ndarray:
    """Final RMSNorm then the LM head: logits over the vocabulary."""
    return rnd(rmsnorm(hidden, W["final_norm"], shape.rms_eps)) @ _f64(W["lm_head"]).T


def verify_forward(shape, W, caches, tokens: np.ndarray, lens: np.ndarray, rnd: Rounding,
                   lm_rows: Optional[Sequence[int]] = None):
    """Target forward over the block [t_m, d_1 .. d_k] of every sequence.

    caches: per layer a pair (K list, V list) of the committed entries
    [m_b, n_kv, d]; tokens [B, R]; lens [B] = m_b.  The block occupies
    positions m_b .. m_b+R-1.  Returns (logits [B, R', V], hidden [B, R, H],
    new_kv: per layer (k [B,R,n_kv,d], v [B,R,n_kv,d])); R' = R unless
    lm_rows selects the block rows whose logits are wanted."""
    tokens = np.asarray(tokens)
    B, R = tokens.shape
    x = _f64(np.asarray(W["embed"])[tokens])
    pos = np.asarray(lens, dtype=np.int64)[:, None] + np.arange(R)[None, :]
    new_kv = []
    for li, Wl in enumerate(W["layers"]):
        x, k, v = layer_forward(shape, Wl, x, pos, caches[li][0], caches[li][1], rnd)
        new_kv.append((k, v))
    rows = x if lm_rows is None else x[:, list(lm_rows)]
    return lm_head(shape, W, rows, rnd), x, new_kv


def full_forward(shape, W, tokens: np.ndarray, rnd: Rounding):
    """Causal forward of whole sequences [B, T] from position 0 with no cache:
    the plain definition the cached forward must reproduce."""
    tokens = np.asarray(tokens)
    B = tokens.shape[0]
    empty = np.zeros((0, shape.n_kv_heads, shape.head_dim))
    caches = [([empty] * B, [empty] * B) for _ in range(shape.n_layers)]
    return verify_forward(shape, W, caches, tokens, np.zeros(B, np.int64), rnd)


def prefill(shape, W, tokens: np.ndarray, rnd: Rounding):
    """KV entries of a prompt [B, T] (no cache): per layer (K list, V list)."""
    _, _, kv = full_forward(shape, W, tokens, rnd)
    return [([k[b] for b in range(k.shape[0])], [v[b] for b in range(v.shape[0])]) for k, v in kv]


def ar_decode(shape, W, prompt: np.ndarray, u: np.ndarray, temperature: float, rnd: Rounding):
    """Plain autoregressive decoding by full recomputation: at every step the
    next token is the inverse-CDF draw from softmax(z / T) of the last row of
    a no-cache forward over the sequence so far, with the supplied uniform.
    prompt [B, T0]; u [B, steps].  Returns the generated tokens [B, steps]."""
    seq = np.asarray(prompt).copy()
    B, steps = u.shape
    out = np.zeros((B, steps), dtype=np.int64)
    for t in range(steps):
        logits, _, _ = full_forward(shape, W, seq, rnd)
        z = logits[:, -1, :].astype(np.float32).astype(np.float64)
        for b in range(B):
            out[b, t] = inverse_cdf(softmax(z[b] / temperature), u[b, t])[0]
        seq = np.concatenate([seq, out[:, t:t + 1]], axis=1)
    return out
