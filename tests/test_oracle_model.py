"""Pins of the oracle's target forward (CPU only).

The forward is pinned by (1) an independent implementation of the same
pre-norm decoder (Hugging Face Llama / Qwen3 modules, random-init from a
config, run in float64), (2) its plain definition (the cached block forward
equals a no-cache forward of the whole sequence), and (3) closed-form special
cases of attention."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import synth

EXACT = oracle.Rounding("exact")
SMALL = synth.ModelShape(n_layers=2, hidden=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn=96,
                         vocab=100, dtype="f32")


# ---------------------------------------------------------------- attention
def test_attention_single_key_returns_value():
    g = np.random.default_rng(0)
    q, k, v = g.standard_normal((3, 4, 8)), g.standard_normal((1, 2, 8)), g.standard_normal((1, 2, 8))
    out = oracle.attention(q, k, v, np.array([1, 1, 1]))
    for h in range(4):
        np.testing.assert_allclose(out[:, h], np.broadcast_to(v[0, h // 2], (3, 8)), rtol=1e-14)


def test_attention_equal_keys_average_visible_values():
    g = np.random.default_rng(1)
    L = 9
    k = np.broadcast_to(g.standard_normal((1, 1, 8)), (L, 1, 8)).copy()
    v = g.standard_normal((L, 1, 8))
    q = g.standard_normal((4, 2, 8))
    vis = np.array([1, 4, 7, 9])
    out = oracle.attention(q, k, v, vis)
    for r in range(4):
        np.testing.assert_allclose(out[r, 0], v[:vis[r], 0].mean(0), rtol=1e-12)
        np.testing.assert_allclose(out[r, 1], v[:vis[r], 0].mean(0), rtol=1e-12)


def test_attention_one_hot_focus():
    # key j is a large multiple of the query, all others orthogonal to it
    L, d = 6, 8
    k = np.zeros((L, 1, d))
    for j in range(L):
        k[j, 0, j] = 1.0
    v = np.arange(L * d, dtype=np.float64).reshape(L, 1, d)
    for j in range(L):
        q = np.zeros((1, 1, d))
        q[0, 0, j] = 400.0
        out = oracle.attention(q, k, v, np.array([L]))
        np.testing.assert_allclose(out[0, 0], v[j, 0], atol=1e-9)


def test_attention_gqa_head_mapping():
    # zero queries give uniform weights: query head h reads KV head h // (n_q / n_kv)
    g = np.random.default_rng(2)
    v = g.standard_normal((5, 2, 4))
    out = oracle.attention(np.zeros((1, 6, 4)), g.standard_normal((5, 2, 4)), v, np.array([5]))
    for h in range(6):
        np.testing.assert_allclose(out[0, h], v[:, h // 3].mean(0), rtol=1e-12)


def test_attention_matches_torch_sdpa():
    g = np.random.default_rng(3)
    R, L, nq, nkv, d = 5, 40, 8, 2, 16
    q, k, v = g.standard_normal((R, nq, d)), g.standard_normal((L, nkv, d)), g.standard_normal((L, nkv, d))
    vis = np.array([36, 37, 38, 39, 40])
    out = oracle.attention(q, k, v, vis)
    mask = torch.tensor(np.arange(L)[None, :] < vis[:, None])
    rep = nq // nkv
    kt = torch.tensor(k).permute(1, 0, 2).repeat_interleave(rep, 0)
    vt = torch.tensor(v).permute(1, 0, 2).repeat_interleave(rep, 0)
    ref = torch.nn.functional.scaled_dot_product_attention(torch.tensor(q).permute(1, 0, 2), kt, vt,
                                                           attn_mask=mask)
    np.testing.assert_allclose(out, ref.permute(1, 0, 2).numpy(), rtol=1e-11, atol=1e-12)


# ---------------------------------------------------------------- full model
def _hf_model(shape, W):
    from transformers import LlamaConfig, LlamaForCausalLM, Qwen3Config, Qwen3ForCausalLM
    kw = dict(hidden_size=shape.hidden, intermediate_size=shape.ffn, num_hidden_layers=shape.n_layers,
              num_attention_heads=shape.n_heads, num_key_value_heads=shape.n_kv_heads,
              head_dim=shape.head_dim, vocab_size=shape.vocab, rms_norm_eps=shape.rms_eps,
              max_position_embeddings=8192, tie_word_embeddings=shape.tie_embed,
              rope_parameters={"rope_type": "default", "rope_theta": shape.rope_base})
    if shape.qk_norm:
        model = Qwen3ForCausalLM(Qwen3Config(attention_bias=False, **kw))
    else:
        model = LlamaForCausalLM(LlamaConfig(attention_bias=False, mlp_bias=False, **kw))
    model = model.to(torch.float64).eval()
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    sd = {"model.embed_tokens.weight": t(W["embed"]), "model.norm.weight": t(W["final_norm"]),
          "lm_head.weight": t(W["lm_head"])}
    for i, L in enumerate(W["layers"]):
        p = "model.layers.%d." % i
        sd.update({p + "self_attn.q_proj.weight": t(L["wq"]), p + "self_attn.k_proj.weight": t(L["wk"]),
                   p + "self_attn.v_proj.weight": t(L["wv"]), p + "self_attn.o_proj.weight": t(L["wo"]),
                   p + "mlp.gate_proj.weight": t(L["w_gate"]), p + "mlp.up_proj.weight": t(L["w_up"]),
                   p + "mlp.down_proj.weight": t(L["w_down"]), p + "input_layernorm.weight": t(L["attn_norm"]),
                   p + "post_attention_layernorm.weight": t(L["ffn_norm"])})
        if shape.qk_norm:
            sd[p + "self_attn.q_norm.weight"] = t(L["q_norm"])
            sd[p + "self_attn.k_norm.weight"] = t(L["k_norm"])
    model.load_state_dict(sd, strict=True)
    return model


def _perturbed_norms(shape, seed):
    # non-unit norm weights so that a dropped or misplaced norm weight shows
    W = synth.model_weights(shape, seed)
    g = np.random.default_rng(seed + 100)
    for L in W["layers"]:
        for key in ("attn_norm", "ffn_norm", "q_norm", "k_norm"):
            if key in L:
                L[key] = (1.0 + 0.3 * g.standard_normal(L[key].shape)).astype(np.float32)
    W["final_norm"] = (1.0 + 0.3 * g.standard_normal(shape.hidden)).astype(np.float32)
    for L in W["layers"]:                      # larger weights: a non-trivial attention pattern
        for key in ("wq", "wk"):
            L[key] = L[key] * 20
    return W


@pytest.mark.parametrize("qk_norm", [False, True])
def test_full_forward_matches_hf_decoder(qk_norm):
    shape = dataclasses.replace(SMALL, qk_norm=qk_norm)
    W = _perturbed_norms(shape, 7)
    tokens = synth.token_ids(2 * 37, shape.vocab, 1, "hf").reshape(2, 37)
    logits, hidden, _ = oracle.full_forward(shape, W, tokens, EXACT)
    with torch.no_grad():
        out = _hf_model(shape, W)(torch.tensor(tokens, dtype=torch.long), output_hidden_states=True)
    ref = out.logits.numpy()
    # the library evaluates its norms and rotary tables in float32
    scale = np.abs(ref).max()
    assert np.abs(logits - ref).max() / scale < 2e-6
    assert np.abs(logits).max() > 0.1


def test_cached_block_equals_no_cache_forward():
    W = _perturbed_norms(SMALL, 8)
    B, T0, k = 3, 21, 4
    seq = synth.token_ids(B * (T0 + k + 1), SMALL.vocab, 1, "cache").reshape(B, T0 + k + 1)
    full, hid_full, kv_full = oracle.full_forward(SMALL, W, seq, EXACT)
    caches = oracle.prefill(SMALL, W, seq[:, :T0], EXACT)
    logits, hidden, new_kv = oracle.verify_forward(SMALL, W, caches, seq[:, T0:], np.full(B, T0), EXACT)
    np.testing.assert_allclose(logits, full[:, T0:], rtol=0, atol=1e-12 * np.abs(full).max())
    np.testing.assert_allclose(hidden, hid_full[:, T0:], rtol=0, atol=1e-12 * np.abs(hid_full).max())
    for (k1, v1), (k2, v2) in zip(new_kv, kv_full):
        np.testing.assert_allclose(k1, k2[:, T0:], atol=1e-12)
        np.testing.assert_allclose(v1, v2[:, T0:], atol=1e-12)


def test_ragged_cache_lengths():
    # sequences of different committed lengths in one batch equal their single-sequence forwards
    W = _perturbed_norms(SMALL, 9)
    lens = np.array([3, 17, 9])
    seqs = [synth.token_ids(int(m) + 4, SMALL.vocab, 1, "rag", b) for b, m in enumerate(lens)]
    caches = [([], []) for _ in range(SMALL.n_layers)]
    for s, m in zip(seqs, lens):
        c = oracle.prefill(SMALL, W, s[None, :m], EXACT)
        for l in range(SMALL.n_layers):
            caches[l][0].append(c[l][0][0])
            caches[l][1].append(c[l][1][0])
    block = np.stack([s[m:] for s, m in zip(seqs, lens)])
    logits, _, _ = oracle.verify_forward(SMALL, W, caches, block, lens, EXACT)
    for b, (s, m) in enumerate(zip(seqs, lens)):
        ref, _, _ = oracle.full_forward(SMALL, W, s[None], EXACT)
        np.testing.assert_allclose(logits[b], ref[0, m:], atol=1e-12 * np.abs(ref).max())


def test_block_is_causal():
    # changing the last draft leaves every earlier block row unchanged
    W = _perturbed_norms(SMALL, 10)
    seq = synth.token_ids(30, SMALL.vocab, 1, "causal").reshape(1, 30)
    caches = oracle.prefill(SMALL, W, seq[:, :26], EXACT)
    a, _, _ = oracle.verify_forward(SMALL, W, caches, seq[:, 26:], np.array([26]), EXACT)
    blk = seq[:, 26:].copy()
    blk[0, -1] = (blk[0, -1] + 1) % SMALL.vocab
    b, _, _ = oracle.verify_forward(SMALL, W, caches, blk, np.array([26]), EXACT)
    np.testing.assert_array_equal(a[:, :-1], b[:, :-1])
    assert np.abs(a[:, -1] - b[:, -1]).max() > 0


def _zero_layers(W):
    for L in W["layers"]:
        for key in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down"):
            L[key] = np.zeros_like(L[key])
    return W


def test_zero_layers_reduce_to_one_matmul():
    # layers with zero weights pass the residual through: logits = W_lm . RMSNorm(E[t])
    W = _zero_layers(synth.model_weights(SMALL, 11))
    W["final_norm"] = np.linspace(0.5, 1.5, SMALL.hidden).astype(np.float32)
    tok = synth.token_ids(10, SMALL.vocab, 1, "zero").reshape(2, 5)
    logits, hidden, _ = oracle.full_forward(SMALL, W, tok, EXACT)
    e = W["embed"][tok].astype(np.float64)
    np.testing.assert_array_equal(hidden, e)
    n = e / np.sqrt((e * e).mean(-1, keepdims=True) + SMALL.rms_eps) * W["final_norm"]
    np.testing.assert_allclose(logits, n @ W["lm_head"].astype(np.float64).T, rtol=1e-12, atol=1e-14)


def test_embedding_and_head_orientation():
    # tied orthogonal embedding rows, zero layers: the top logit of a row is its own token
    shape = dataclasses.replace(SMALL, vocab=48, tie_embed=True)
    W = _zero_layers(synth.model_weights(shape, 12))
    qmat, _ = np.linalg.qr(np.random.default_rng(0).standard_normal((shape.hidden, shape.vocab)))
    W["embed"] = W["lm_head"] = qmat.T.astype(np.float64)
    tok = np.arange(shape.vocab).reshape(4, 12)
    logits, _, _ = oracle.full_forward(shape, W, tok, EXACT)
    np.testing.assert_array_equal(np.argmax(logits, -1), tok)


def test_contract_rounding_stays_close_to_exact():
    shape = dataclasses.replace(SMALL, dtype="bf16")
    W = synth.model_weights(shape, 13)
    tok = synth.token_ids(24, shape.vocab, 1, "contract").reshape(2, 12)
    a, _, _ = oracle.full_forward(shape, W, tok, EXACT)
    b, _, _ = oracle.full_forward(shape, W, tok, oracle.Rounding("contract"))
    rel = np.abs(a - b).max() / np.abs(a).max()
    assert 0 < rel < 2e-2
