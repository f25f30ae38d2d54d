"""Pins of the oracle's MTP draft head (CPU only).

The paper describes the head in prose (App. "Models and Draft Heads"; Eqs.
tf-restart / tf-restart-kv), so parity past these special cases is unpinned:
* a zero decoder layer with W_proj = [0 | I] reduces the head to
  W_lm . RMSNorm_f(RMSNorm_e(E[t])): pins the concat order, the shared
  embedding / LM head, the final norm and that chain step i consumes the
  previous draft;
* W_proj = [I | 0] reduces it to W_lm . RMSNorm_f(RMSNorm_h(h)): pins that the
  first draft of a cycle starts from the target feature at the boundary
  (verify row n) and that the chain carries the layer output forward;
* the restart: the committed length becomes the boundary m + n + 1 and only
  the n + 1 extend rows are committed entries."""
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
