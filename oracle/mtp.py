"""Recurrent MTP draft head of the oracle (float64).

Test infrastructure: imported only by the tests, the smoke check and the
benchmark's CPU-baseline leg.

The head (App. "Models and Draft Heads") is recurrent: each step consumes one
(conditioning hidden, token) pair.  Each half gets its own RMSNorm, the two
results are joined with the hidden half first, a bias-free linear map takes
the 2H values to H, and a single decoder layer with a private KV cache (one
entry per position) follows.  The token embedding and the output head are
shared with the backbone.  Reading where the paper is silent: one final
RMSNorm precedes the shared LM head, and the hidden carried along the chain
is the decoder layer's output before that norm.

Cycle restart (App. "Train--Inference Inconsistency under Teacher Forcing",
Eqs. tf-restart and tf-restart-kv): behind the boundary every cache entry is
computed from a target feature; the chain's own features enter the cache only
through the current cycle's writes, which the next cycle discards, also when
every draft was accepted.

Indexing used here.  Let h_t be the target's last-layer hidden at position t
(it predicts token x_{t+1}).  Cache slot s of the head holds the entry of the
pair (h_s, x_{s+1}), rotated at position s + 1.  With m committed target
positions before a step, the head's committed length is also m.  After the
step accepted n drafts and drew the final token f, the extend rows are
(h_m, d_1) .. (h_{m+n-1}, d_n), (h_{m+n}, f) at slots m .. m+n; the last row's
output g_1 gives q_1 and the first new draft; chain step i feeds
(g_{i-1}, d'_{i-1}) at slot m+n+i-1.  The committed length becomes m+n+1.

Draft-path reconstruction (App. "Draft-Path Reconstruction"; "Parallelizing
GrowMTP Training"): the training side re-runs the chain of every recorded cycle
with the recorded drafts as inputs and nothing sampled.  A cycle that starts
with s committed head entries (slot s holds its first row, the pair of the
boundary hidden and the last committed token) is rebuilt from those s entries
alone: depth 1 feeds the recorded start pair at slot s, depth j feeds
(g_{j-1}, d_{j-1}) at slot s + j - 1, each rotated at its slot + 1, and every
depth sees only the prefix and its own chain's earlier entries.

Pins (tests/test_oracle_mtp.py): pass-through special cases fix the concat
order, the shared embedding and head, the final norm and the chain's feed; two
special cases in which the decoder layer has a closed form that reads its
cache (uniform attention with W_q = W_k = 0; scores a b cos(P - P') with Q/K in
the first rotary pair only) fix which (hidden, token) pair fills every extend
slot, what each row sees, and every entry's rotary position.  The decoder
layer itself is the target's, pinned against a float64 Hugging Face decoder.
The reconstruction is further pinned by reproducing the drafting's own
distributions.
"""
from __future__ import annotations

import numpy as np

from .numerics import Rounding, rmsnorm, softmax, inverse_cdf, nucleus
from .model import layer_forward, lm_head


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def mtp_apply(shape, Wm, W, h: np.ndarray, toks: np.ndarray, pos: np.ndarray,
              cache_k: np.ndarray, cache_v: np.ndarray, rnd: Rounding):
    """The head over R consecutive rows of one sequence.

    h [R, H] conditioning hiddens, toks [R] tokens, pos [R] rotary positions,
    cache [s, n_kv, d] entries the rows attend before their own.
    Returns (g [R, H] layer outputs, logits [R, V], k [R,n_kv,d], v [R,n_kv,d])."""
    a = rmsnorm(h, Wm["norm_h"], shape.rms_eps)
    e = rmsnorm(_f64(np.asarray(W["embed"])[np.asarray(toks)]), Wm["norm_e"], shape.rms_eps)
    x = rnd(np.concatenate([a, e], axis=-1)) @ _f64(Wm["w_proj"]).T
    g, k, v = layer_forward(shape, Wm["layer"], x[None], np.asarray(pos)[None],
                            [cache_k], [cache_v], rnd)
    head = {"final_norm": Wm["final_norm"], "lm_head": W["lm_head"]}
    return g[0], lm_head(shape, head, g[0], rnd), k[0], v[0]


def _draw(z: np.ndarray, u: float, mode: str, temperature: float, top_p: float = 1.0) -> int:
    z32 = z.astype(np.float32)
    if mode == "greedy":
        return int(np.argmax(z32))
    q = softmax(z32.astype(np.float64) / temperature)
    if top_p < 1.0:                       # a sample of the head's nucleus (evaluation setting)
        q = nucleus(z32, q, top_p)[0]
    return inverse_cdf(q, u)[0]


def mtp_draft(shape, Wm, W, cache_k, cache_v, mtp_lens, hidden, n_accept, out_tokens,
              u_draft, k: int, mode: str, temperature: float, rnd: Rounding, top_p: float = 1.0):
    """Draft the next block of every sequence.

    cache_k[b] / cache_v[b] [>= mtp_lens[b], n_kv, d]: the head's cache;
    hidden [B, k+1, H] target hiddens of the last verification; n_accept [B];
    out_tokens [B, k+1] (accepted drafts then the final token); u_draft [B, k].
    Returns dict(drafts [B, k], draft_logits [B, k, V], new_lens [B],
    ext_k / ext_v: per sequence the committed extend entries [n_b+1, n_kv, d],
    chain_k / chain_v: per sequence the transient chain entries [k-1, n_kv, d])."""
    B = len(mtp_lens)
    V = np.asarray(W["lm_head"]).shape[0]
    drafts = np.zeros((B, k), dtype=np.int64)
    dlog = np.zeros((B, k, V))
    new_lens = np.zeros(B, dtype=np.int64)
    ext_k, ext_v, ch_k, ch_v = [], [], [], []
    for b in range(B):
        m = int(mtp_lens[b])
        R = int(n_accept[b]) + 1
        kc, vc = _f64(cache_k[b][:m]), _f64(cache_v[b][:m])
        g, logits, kn, vn = mtp_apply(shape, Wm, W, _f64(hidden[b, :R]), out_tokens[b, :R],
                                      m + 1 + np.arange(R), kc, vc, rnd)
        ext_k.append(kn)
        ext_v.append(vn)
        kc, vc = np.concatenate([kc, kn]), np.concatenate([vc, vn])
        g_prev, z = g[-1], logits[-1]
        ck, cv = [], []
        for i in range(k):
            dlog[b, i] = z
            drafts[b, i] = _draw(z, u_draft[b, i], mode, temperature, top_p)
            if i + 1 < k:
                slot = m + R + i
                g1, l1, k1, v1 = mtp_apply(shape, Wm, W, g_prev[None], [drafts[b, i]],
                                           [slot + 1], kc, vc, rnd)
                kc, vc = np.concatenate([kc, k1]), np.concatenate([vc, v1])
                ck.append(k1[0])
                cv.append(v1[0])
                g_prev, z = g1[0], l1[0]
        ch_k.append(np.array(ck))
        ch_v.append(np.array(cv))
        new_lens[b] = m + R
    return dict(drafts=drafts, draft_logits=dlog, new_lens=new_lens,
                ext_k=ext_k, ext_v=ext_v, chain_k=ch_k, chain_v=ch_v)


def mtp_reconstruct(shape, Wm, W, cache_k, cache_v, starts, start_hidden, start_tokens, drafts, K: int,
                    rnd: Rounding):
    """Reconstruct the head's distributions along recorded draft paths.

    For cycle r: cache_k[r] / cache_v[r] [>= starts[r], n_kv, d] hold the head's
    committed entries (the first starts[r] are visible); start_hidden [R, H] and
    start_tokens [R] are the recorded start pair; drafts [R, >= K-1] the recorded
    drafts, fed back in order (d_1 .. d_{K-1}).  Returns dict(logits [R, K, V] --
    the head logits whose softmax is q_{r,k} -- and chain_k / chain_v [R][K, n_kv, d],
    the entries the chain writes at slots starts[r] .. starts[r] + K - 1)."""
    R = len(starts)
    V = np.asarray(W["lm_head"]).shape[0]
    logits = np.zeros((R, K, V))
    ck, cv = [], []
    for r in range(R):
        s = int(starts[r])
        kc, vc = _f64(cache_k[r][:s]), _f64(cache_v[r][:s])
        h, t = _f64(start_hidden[r]), int(start_tokens[r])
        ks, vs = [], []
        for j in range(K):
            g, lg, k1, v1 = mtp_apply(shape, Wm, W, h[None], [t], [s + j + 1], kc, vc, rnd)
            logits[r, j] = lg[0]
            kc, vc = np.concatenate([kc, k1]), np.concatenate([vc, v1])
            ks.append(k1[0])
            vs.append(v1[0])
            if j + 1 < K:
                h, t = g[0], int(drafts[r][j])
        ck.append(np.array(ks))
        cv.append(np.array(vs))
    return dict(logits=logits, chain_k=ck, chain_v=cv)
