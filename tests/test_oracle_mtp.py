"""Pins of the oracle's MTP draft head (CPU only).

The paper describes the head in prose (App. "Models and Draft Heads"; Eqs.
tf-restart / tf-restart-kv); these special cases pin it:
* a zero decoder layer with W_proj = [0 | I] reduces the head to
  W_lm . RMSNorm_f(RMSNorm_e(E[t])): pins the concat order, the shared
  embedding / LM head, the final norm and that chain step i consumes the
  previous draft;
* W_proj = [I | 0] reduces it to W_lm . RMSNorm_f(RMSNorm_h(h)): pins that the
  first draft of a cycle starts from the target feature at the boundary
  (verify row n) and that the chain carries the layer output forward;
* the restart: the committed length becomes the boundary m + n + 1 and only
  the n + 1 extend rows are committed entries;
* the cache composition (closed forms of a layer that reads its cache, see
  below): the (hidden, token) pair of every extend slot, what each row sees,
  the chain's feed and every entry's rotary position."""
import dataclasses

import numpy as np

import oracle
import synth

EXACT = oracle.Rounding("exact")
SHAPE = synth.ModelShape(n_layers=1, hidden=32, n_heads=4, n_kv_heads=2, head_dim=8, ffn=48,
                         vocab=40, dtype="f32")


def _rms(x, w, eps=1e-6):
    return x / np.sqrt((x * x).mean(-1, keepdims=True) + eps) * w


def _setup(seed, proj):
    W = synth.model_weights(SHAPE, seed)
    Wm = synth.mtp_weights(SHAPE, seed)
    for key in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down"):
        Wm["layer"][key] = np.zeros_like(Wm["layer"][key])
    g = np.random.default_rng(seed)
    Wm["norm_h"] = (1 + 0.3 * g.standard_normal(SHAPE.hidden))
    Wm["norm_e"] = (1 + 0.3 * g.standard_normal(SHAPE.hidden))
    Wm["final_norm"] = (1 + 0.3 * g.standard_normal(SHAPE.hidden))
    H = SHAPE.hidden
    eye, zero = np.eye(H), np.zeros((H, H))
    Wm["w_proj"] = np.concatenate([zero, eye], 1) if proj == "embed" else np.concatenate([eye, zero], 1)
    return W, Wm


def _inputs(seed, B=3, k=3):
    g = np.random.default_rng(seed)
    lens = g.integers(2, 9, B)
    ck = [g.standard_normal((m + 6, SHAPE.n_kv_heads, SHAPE.head_dim)) for m in lens]
    cv = [g.standard_normal((m + 6, SHAPE.n_kv_heads, SHAPE.head_dim)) for m in lens]
    hidden = g.standard_normal((B, k + 1, SHAPE.hidden))
    n = g.integers(0, k + 1, B)
    out = g.integers(0, SHAPE.vocab, (B, k + 1))
    u = g.random((B, k)).astype(np.float32)
    return lens, ck, cv, hidden, n, out, u


def test_embedding_path_special_case():
    W, Wm = _setup(1, "embed")
    k = 3
    lens, ck, cv, hidden, n, out, u = _inputs(1, k=k)
    r = oracle.mtp_draft(SHAPE, Wm, W, ck, cv, lens, hidden, n, out, u, k, "greedy", 1.0, EXACT)
    E, L = W["embed"].astype(np.float64), W["lm_head"].astype(np.float64)
    head = lambda t: _rms(_rms(E[t], Wm["norm_e"]), Wm["final_norm"]) @ L.T
    for b in range(len(lens)):
        prev = out[b, n[b]]                         # the cycle's final token opens the next cycle
        for i in range(k):
            z = head(prev)
            np.testing.assert_allclose(r["draft_logits"][b, i], z, rtol=1e-12, atol=1e-12)
            assert r["drafts"][b, i] == int(np.argmax(z.astype(np.float32)))
            prev = r["drafts"][b, i]


def test_hidden_path_special_case():
    W, Wm = _setup(2, "hidden")
    k = 3
    lens, ck, cv, hidden, n, out, u = _inputs(2, k=k)
    r = oracle.mtp_draft(SHAPE, Wm, W, ck, cv, lens, hidden, n, out, u, k, "sample", 1.0, EXACT)
    L = W["lm_head"].astype(np.float64)
    for b in range(len(lens)):
        g = _rms(hidden[b, n[b]], Wm["norm_h"])      # target feature at the boundary
        for i in range(k):
            np.testing.assert_allclose(r["draft_logits"][b, i], _rms(g, Wm["final_norm"]) @ L.T,
                                       rtol=1e-12, atol=1e-12)
            g = _rms(g, Wm["norm_h"])                # the chain feeds the layer output back


def test_restart_lengths_and_entries():
    shape = SHAPE
    W = synth.model_weights(shape, 3)
    Wm = synth.mtp_weights(shape, 3)
    k = 4
    lens, ck, cv, hidden, n, out, u = _inputs(3, B=4, k=k)
    r = oracle.mtp_draft(shape, Wm, W, ck, cv, lens, hidden, n, out, u, k, "sample", 1.0, EXACT)
    np.testing.assert_array_equal(r["new_lens"], lens + n + 1)
    for b in range(4):
        assert r["ext_k"][b].shape[0] == n[b] + 1
        assert r["chain_k"][b].shape[0] == k - 1
    # the extend rows computed together equal the rows computed one at a time
    b = int(np.argmax(n))
    m = int(lens[b])
    kc, vc = ck[b][:m], cv[b][:m]
    for i in range(n[b] + 1):
        _, _, k1, v1 = oracle.mtp_apply(shape, Wm, W, hidden[b, i:i + 1], out[b, i:i + 1],
                                        [m + 1 + i], kc, vc, EXACT)
        np.testing.assert_allclose(k1[0], r["ext_k"][b][i], atol=1e-12)
        kc, vc = np.concatenate([kc, k1]), np.concatenate([vc, v1])


def test_stale_cache_beyond_length_is_ignored():
    # entries past the committed length (an earlier chain's writes) never enter a draft
    W = synth.model_weights(SHAPE, 4)
    Wm = synth.mtp_weights(SHAPE, 4)
    lens, ck, cv, hidden, n, out, u = _inputs(4)
    a = oracle.mtp_draft(SHAPE, Wm, W, ck, cv, lens, hidden, n, out, u, 3, "sample", 1.0, EXACT)
    ck2 = [c.copy() for c in ck]
    for b, m in enumerate(lens):
        ck2[b][m:] = 1e3
    b_ = oracle.mtp_draft(SHAPE, Wm, W, ck2, cv, lens, hidden, n, out, u, 3, "sample", 1.0, EXACT)
    np.testing.assert_array_equal(a["draft_logits"], b_["draft_logits"])


# ------------------------------------------------------------------ draft-path reconstruction
def _reconstruct_inputs(r, lens, ck, cv, hidden, n, out):
    """The record of the cycles mtp_draft just drafted: each starts with the committed
    entries before the boundary row (the head's old entries and extend rows 0..n-1),
    from the boundary hidden and the cycle's final token."""
    B = len(lens)
    starts = np.array([int(lens[b]) + int(n[b]) for b in range(B)])
    pk = [np.concatenate([ck[b][:lens[b]], r["ext_k"][b][:n[b]]]) for b in range(B)]
    pv = [np.concatenate([cv[b][:lens[b]], r["ext_v"][b][:n[b]]]) for b in range(B)]
    return starts, pk, pv, hidden[np.arange(B), n], out[np.arange(B), n]


def test_reconstruction_reproduces_the_drafting():
    # Fed the recorded drafts from the recorded start, every depth sees the context the
    # drafting saw (App. "Draft-Path Reconstruction": the drafts turn from outputs into
    # inputs; the start state is the one drafting consumed), so the reconstructed head
    # logits are the draft logits and the chain rewrites the same cache entries
    shape = SHAPE
    W = synth.model_weights(shape, 5)
    Wm = synth.mtp_weights(shape, 5)
    k = 4
    for mode in ("sample", "greedy"):
        lens, ck, cv, hidden, n, out, u = _inputs(5, B=5, k=k)
        r = oracle.mtp_draft(shape, Wm, W, ck, cv, lens, hidden, n, out, u, k, mode, 1.0, EXACT)
        starts, pk, pv, h0, t0 = _reconstruct_inputs(r, lens, ck, cv, hidden, n, out)
        rec = oracle.mtp_reconstruct(shape, Wm, W, pk, pv, starts, h0, t0, r["drafts"], k, EXACT)
        np.testing.assert_allclose(rec["logits"], r["draft_logits"], rtol=1e-12, atol=1e-12)
        for b in range(len(lens)):
            np.testing.assert_allclose(rec["chain_k"][b][0], r["ext_k"][b][n[b]], atol=1e-12)   # the boundary row
            np.testing.assert_allclose(rec["chain_k"][b][1:], r["chain_k"][b], atol=1e-12)


def test_reconstruction_feeds_the_recorded_drafts_in_order():
    # embedding path (W_proj = [0 | I], zero layer): depth 1 reads the start token, depth
    # j the recorded draft d_{j-1}, whatever the head itself would have drawn
    W, Wm = _setup(6, "embed")
    K, R = 4, 3
    g = np.random.default_rng(6)
    starts = g.integers(1, 7, R)
    ck = [g.standard_normal((s + K, SHAPE.n_kv_heads, SHAPE.head_dim)) for s in starts]
    drafts = g.integers(0, SHAPE.vocab, (R, K))
    t0 = g.integers(0, SHAPE.vocab, R)
    rec = oracle.mtp_reconstruct(SHAPE, Wm, W, ck, ck, starts, g.standard_normal((R, SHAPE.hidden)), t0, drafts, K,
                                 EXACT)
    E, L = W["embed"].astype(np.float64), W["lm_head"].astype(np.float64)
    head = lambda t: _rms(_rms(E[t], Wm["norm_e"]), Wm["final_norm"]) @ L.T
    for r_ in range(R):
        fed = [t0[r_]] + list(drafts[r_, :K - 1])
        for j in range(K):
            np.testing.assert_allclose(rec["logits"][r_, j], head(fed[j]), rtol=1e-12, atol=1e-12)


def test_reconstructed_cycles_are_independent():
    # chains share only recorded inputs: a cycle's result does not depend on the others
    # in the batch (App. "Parallelizing GrowMTP Training"), nor on entries past its start
    shape = SHAPE
    W = synth.model_weights(shape, 7)
    Wm = synth.mtp_weights(shape, 7)
    K, R = 3, 4
    g = np.random.default_rng(7)
    starts = g.integers(2, 9, R)
    ck = [g.standard_normal((s + 5, shape.n_kv_heads, shape.head_dim)) for s in starts]
    cv = [g.standard_normal((s + 5, shape.n_kv_heads, shape.head_dim)) for s in starts]
    h0 = g.standard_normal((R, shape.hidden))
    t0 = g.integers(0, shape.vocab, R)
    drafts = g.integers(0, shape.vocab, (R, K))
    full = oracle.mtp_reconstruct(shape, Wm, W, ck, cv, starts, h0, t0, drafts, K, EXACT)
    ck2 = [c.copy() for c in ck]
    for r_, s in enumerate(starts):
        ck2[r_][s:] = 1e3
    for r_ in (2, 0):
        one = oracle.mtp_reconstruct(shape, Wm, W, ck2[r_:r_ + 1], cv[r_:r_ + 1], starts[r_:r_ + 1], h0[r_:r_ + 1],
                                     t0[r_:r_ + 1], drafts[r_:r_ + 1], K, EXACT)
        np.testing.assert_array_equal(one["logits"][0], full["logits"][r_])


# ------------------------------------------------------------------ cache composition
# Two special cases in which the head's decoder layer has a closed form that does
# depend on its cache, written out below without the oracle's layer code:
#  * W_q = W_k = 0: every score is 0, so each row attends uniformly to everything it
#    sees, and the output is x + W_o (mean of the visible V entries);
#  * W_q and W_k non-zero only in the first channel of each head (the rotary pair
#    (0, d/2), whose angle is the position itself): a query at position P and a key
#    at position P' then score a * b * cos(P - P') / sqrt(d) (RoPE's relative-position
#    property), with a and b the raw first channels.
# The FFN is zero in both.  With the pairing of App. "Models and Draft Heads" and Eq.
# tf-restart (slot s holds the pair (h_s, x_{s+1}) at position s + 1) the closed form
# fixes which (hidden, token) pair fills each extend slot, that row i sees the prefix
# and rows 0..i, which rows the chain feeds, and every entry's rotary position, both
# through the scores and through the stored (rotated) keys.
def _composition_setup(seed, rotary):
    shape = SHAPE
    H, d, nq, nkv = shape.hidden, shape.head_dim, shape.n_heads, shape.n_kv_heads
    W = synth.model_weights(shape, seed)
    Wm = synth.mtp_weights(shape, seed)
    g = np.random.default_rng(100 + seed)
    Wm["w_proj"] = 0.3 * g.standard_normal((H, 2 * H))          # both halves act
    Wl = Wm["layer"]
    Wl["wq"] = np.zeros((nq * d, H))
    Wl["wk"] = np.zeros((nkv * d, H))
    if rotary:
        for h in range(nq):
            Wl["wq"][h * d] = 0.5 * g.standard_normal(H)
        for j in range(nkv):
            Wl["wk"][j * d] = 0.5 * g.standard_normal(H)
    Wl["wv"] = g.standard_normal((nkv * d, H))
    Wl["wo"] = 0.3 * g.standard_normal((H, nq * d))
    for key in ("w_gate", "w_up", "w_down"):
        Wl[key] = np.zeros_like(Wl[key])
    Wl["attn_norm"] = 1 + 0.3 * g.standard_normal(H)
    Wm["norm_h"] = 1 + 0.3 * g.standard_normal(H)
    Wm["norm_e"] = 1 + 0.3 * g.standard_normal(H)
    Wm["final_norm"] = 1 + 0.3 * g.standard_normal(H)
    return W, Wm


def _prefix_entries(g, m, rotary):
    """m committed entries: key b e^{i P} in the first rotary pair at P = slot + 1 (as the
    head writes them), random values.  Returns the cache arrays and the entry list."""
    nkv, d = SHAPE.n_kv_heads, SHAPE.head_dim
    kb = 3.0 * g.standard_normal((m, nkv)) if rotary else np.zeros((m, nkv))
    vv = g.standard_normal((m, nkv, d))
    P = np.arange(m) + 1.0
    K = np.zeros((m, nkv, d))
    K[:, :, 0] = kb * np.cos(P)[:, None]
    K[:, :, d // 2] = kb * np.sin(P)[:, None]
    return K, vv, [(kb[j], P[j], vv[j]) for j in range(m)]


def _closed_form_row(Wm, x, P, entries):
    """One row of the special-case layer: input x at position P after the visible entries.
    Returns (layer output, its own entry (b, P, v))."""
    Wl = Wm["layer"]
    nq, nkv, d = SHAPE.n_heads, SHAPE.n_kv_heads, SHAPE.head_dim
    n = _rms(x, Wl["attn_norm"])
    a = (Wl["wq"] @ n).reshape(nq, d)[:, 0]
    own = ((Wl["wk"] @ n).reshape(nkv, d)[:, 0], P, (Wl["wv"] @ n).reshape(nkv, d))
    seen = entries + [own]
    o = np.zeros((nq, d))
    for h in range(nq):
        j = h // (nq // nkv)
        s = np.array([a[h] * kb[j] * np.cos(P - Pe) for kb, Pe, _ in seen]) / np.sqrt(d)
        w = np.exp(s - s.max())
        w /= w.sum()
        o[h] = sum(wi * ve[j] for wi, (_, _, ve) in zip(w, seen))
    return x + Wl["wo"] @ o.reshape(-1), own


def _closed_form_draft(W, Wm, h_rows, tok_rows, m, prefix, k):
    """The greedy draft of one sequence by the closed form: extend rows (h_rows[i],
    tok_rows[i]) at slots m + i, then the chain."""
    E, L = W["embed"].astype(np.float64), W["lm_head"].astype(np.float64)
    feed = lambda h, t: Wm["w_proj"] @ np.concatenate([_rms(h, Wm["norm_h"]), _rms(E[t], Wm["norm_e"])])
    entries = list(prefix)
    for i in range(len(h_rows)):
        g, own = _closed_form_row(Wm, feed(h_rows[i], tok_rows[i]), m + i + 1.0, entries)
        entries.append(own)
    logits, drafts = [], []
    for j in range(k):
        z = L @ _rms(g, Wm["final_norm"])
        logits.append(z)
        drafts.append(int(np.argmax(z.astype(np.float32))))
        if j + 1 < k:
            g, own = _closed_form_row(Wm, feed(g, drafts[-1]), m + len(h_rows) + j + 1.0, entries)
            entries.append(own)
    return np.array(logits), drafts, entries[len(prefix):]


def _check_composition(seed, rotary):
    W, Wm = _composition_setup(seed, rotary)
    k, B = 4, 4
    g = np.random.default_rng(seed)
    lens = g.integers(3, 9, B)
    pre = [_prefix_entries(g, int(m), rotary) for m in lens]
    hidden = g.standard_normal((B, k + 1, SHAPE.hidden))
    n = np.array([0, 1, 3, 4])
    out = g.integers(0, SHAPE.vocab, (B, k + 1))
    u = np.zeros((B, k), np.float32)
    r = oracle.mtp_draft(SHAPE, Wm, W, [p[0] for p in pre], [p[1] for p in pre], lens, hidden, n, out, u, k,
                         "greedy", 1.0, EXACT)
    d = SHAPE.head_dim
    for b in range(B):
        R = int(n[b]) + 1
        z, dr, new = _closed_form_draft(W, Wm, hidden[b, :R], out[b, :R], int(lens[b]), pre[b][2], k)
        np.testing.assert_allclose(r["draft_logits"][b], z, rtol=1e-10, atol=1e-10)
        assert list(r["drafts"][b]) == dr
        # the stored keys: entry (b, P) rotated to b e^{i P} in the first pair
        keys = np.concatenate([r["ext_k"][b], r["chain_k"][b].reshape(-1, SHAPE.n_kv_heads, d)])
        assert keys.shape[0] == len(new) == R + k - 1
        for e, (kb, P, vv) in enumerate(new):
            np.testing.assert_allclose(keys[e][:, 0], kb * np.cos(P), atol=1e-10)
            np.testing.assert_allclose(keys[e][:, d // 2], kb * np.sin(P), atol=1e-10)
        vals = np.concatenate([r["ext_v"][b], r["chain_v"][b].reshape(-1, SHAPE.n_kv_heads, d)])
        np.testing.assert_allclose(vals, np.array([vv for _, _, vv in new]), atol=1e-10)


def test_cache_pairing_uniform_attention():
    # W_q = W_k = 0: the first draft is a closed form in the extend pairs and the prefix
    # values; shifting the pairing (h_i with x_{i+2}, or h_{i+1} with x_{i+1}) or the
    # visible set changes it
    for seed in (11, 12):
        _check_composition(seed, rotary=False)


def test_cache_rotary_positions():
    # first-pair Q/K: scores depend on the position differences, so an extend or chain
    # entry rotated one position off (slot instead of slot + 1) against the prefix fails
    for seed in (13, 14):
        _check_composition(seed, rotary=True)
