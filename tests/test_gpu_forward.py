"""GPU parity of gm_verify_forward against the oracle: logits and hiddens
within 1e-4 (float32 model) or 2e-2 (bf16 model) relative error, the block's
K/V entries written at positions m_b .. m_b + k, and greedy accept counts on
the GPU's logits bit-exact with the oracle's outside the flag window."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import need_gpu, rel_err, device_cache, synth_caches, t32, i32, flag_report, CONTRACT, EXACT
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu


def _gpu_forward(model, cache, tokens):
    B, k1 = tokens.shape
    s = model.shape
    logits = torch.empty((B, k1, s.vocab), dtype=torch.float32, device="cuda")
    hidden = torch.empty((B, k1, s.hidden), dtype=torch.float32, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    gm.verify_forward(model, cache, i32(tokens), logits, hidden, gm.Workspace(), err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return logits.cpu().numpy(), hidden.cpu().numpy()


def _gpu_greedy(logits, drafts):
    B, k1, V = logits.shape
    n = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, k1), dtype=torch.int32, device="cuda")
    gm.spec_accept(t32(logits), None, i32(drafts), None, None, n, out, gm.GM_GREEDY, gm.Workspace())
    torch.cuda.synchronize()
    return n.cpu().numpy(), out.cpu().numpy()


@pytest.mark.parametrize("qk_norm", [False, True])
def test_tiny_f32_forward(qk_norm):
    need_gpu()
    wl = synth.WORKLOADS["tiny"]
    shape = dataclasses.replace(wl.shape, qk_norm=qk_norm)
    W = synth.model_weights(shape)
    B, k, T0 = wl.batch, wl.k, wl.ctx_lo
    prompt = synth.token_ids(B * T0, shape.vocab, 1, "tiny-prompt").reshape(B, T0)
    caches = oracle.prefill(shape, W, prompt, EXACT)
    # the cache holds what the GPU stores: float32 entries
    caches = [([a.astype(np.float32) for a in ks], [a.astype(np.float32) for a in vs]) for ks, vs in caches]
    lens = np.full(B, T0)
    tokens = synth.token_ids(B * (k + 1), shape.vocab, 1, "tiny-block").reshape(B, k + 1)
    model = gm.DeviceModel(shape, W)
    cache = device_cache(shape, caches, lens, k + 1)
    logits, hidden = _gpu_forward(model, cache, tokens)
    ref, ref_h, new_kv = oracle.verify_forward(shape, W, caches, tokens, lens, EXACT)
    e = rel_err(logits, ref)
    print("[forward tiny f32 qk_norm=%d] logits rel err %.3e" % (qk_norm, e), flush=True)
    assert e < 1e-4
    assert rel_err(hidden, ref_h) < 1e-4
    for l in range(shape.n_layers):
        for b in range(B):
            kk, vv = cache.read(l, b, lens[b] + np.arange(k + 1))
            assert rel_err(kk, new_kv[l][0][b]) < 1e-5
            assert rel_err(vv, new_kv[l][1][b]) < 1e-5
    # no-cache definition: the block rows of a full causal forward
    full, _, _ = oracle.full_forward(shape, W, np.concatenate([prompt, tokens], 1), EXACT)
    assert rel_err(logits, full[:, T0:]) < 1e-4


@pytest.fixture(scope="module")
def qwen_layer():
    wl = synth.WORKLOADS["qwen3_4b_layer"]
    shape = wl.shape
    W = synth.model_weights(shape)
    lens = synth.context_lengths(wl)
    caches = synth_caches(shape, lens, shape.n_layers)
    pending = synth.token_ids(wl.batch, shape.vocab, 1, "pending")
    take, alt = synth.mixing_draws(wl.batch, wl.k, shape.vocab, wl.mix_prob)
    drafts = oracle.mixing_drafts(shape, W, caches, lens, pending, take, alt, CONTRACT)
    return wl, shape, W, lens, caches, np.concatenate([pending[:, None], drafts], 1)


def test_qwen_layer_bf16_forward(qwen_layer):
    need_gpu()
    wl, shape, W, lens, caches, tokens = qwen_layer
    k = wl.k
    model = gm.DeviceModel(shape, W)
    cache = device_cache(shape, caches, lens, k + 1)
    logits, hidden = _gpu_forward(model, cache, tokens)
    ref_c, ref_hc, kv_c = oracle.verify_forward(shape, W, caches, tokens, lens, CONTRACT)
    ref_e, _, _ = oracle.verify_forward(shape, W, caches, tokens, lens, EXACT)
    e_exact, e_contract = rel_err(logits, ref_e), rel_err(logits, ref_c)
    print("[forward qwen3 layer bf16] logits rel err vs exact %.3e, vs contract %.3e; hidden %.3e"
          % (e_exact, e_contract, rel_err(hidden, ref_hc)), flush=True)
    assert e_exact < 2e-2
    # float32 accumulation still flips ~0.1% of the bf16 roundings the contract mirrors; a float32
    # CPU emulation of the same arithmetic lands 4-5e-3 from the float64 contract oracle
    assert e_contract < 1e-2
    assert rel_err(hidden, ref_hc) < 1e-2
    for b in range(0, wl.batch, 9):
        kk, vv = cache.read(0, b, lens[b] + np.arange(k + 1))
        assert np.abs(kk - kv_c[0][0][b]).max() <= 2.0 ** -7 * np.abs(kv_c[0][0][b]).max()
        assert np.abs(vv - kv_c[0][1][b]).max() <= 2.0 ** -7 * np.abs(kv_c[0][1][b]).max()
    # greedy acceptance on the GPU's logits equals the oracle's outside the flags
    drafts = tokens[:, 1:]
    ref = oracle.spec_accept(ref_c, None, drafts, None, None, mode="greedy")
    n, out = _gpu_greedy(logits, drafts)
    flag_report("forward+greedy qwen3 layer", ref.flagged, len(n))
    ok = ~ref.flagged
    np.testing.assert_array_equal(n[ok], ref.n_accept[ok])
    np.testing.assert_array_equal(out[ok], ref.out_tokens[ok])
    tau = 1 + n.mean()
    print("[forward+greedy qwen3 layer] tau %.3f (0.7 mixing predicts %.3f)" % (tau, (1 - 0.7 ** 4) / 0.3), flush=True)


def test_qwen_layer_bf16_forward_mid_batch(qwen_layer):
    # 24 sequences: M = 96 block rows takes the 128-row GEMM tile on the LM head and
    # 64-row tiles with K splits on the narrow projections
    need_gpu()
    wl, shape, W, lens, caches, tokens = qwen_layer
    B, k = 24, wl.k
    lens, tokens = lens[:B], tokens[:B]
    caches = [(ks[:B], vs[:B]) for ks, vs in caches]
    model = gm.DeviceModel(shape, W)
    cache = device_cache(shape, caches, lens, k + 1, page_size=32)
    logits, hidden = _gpu_forward(model, cache, tokens)
    ref_c, ref_hc, _ = oracle.verify_forward(shape, W, caches, tokens, lens, CONTRACT)
    print("[forward qwen3 layer bf16 B=24] logits rel err vs contract %.3e, hidden %.3e"
          % (rel_err(logits, ref_c), rel_err(hidden, ref_hc)), flush=True)
    assert rel_err(logits, ref_c) < 1e-2 and rel_err(hidden, ref_hc) < 1e-2


def test_qwen_layer_bf16_forward_k7_block(qwen_layer):
    # a k = 7 block of the 64 sequences: M = 512 verify rows, which take 256 x 224 tiles on the
    # SwiGLU projection (385..768 rows) and two 256-row M tiles of 224 columns on the LM head
    need_gpu()
    wl, shape, W, lens, caches, _ = qwen_layer
    B, k = wl.batch, 7
    tokens = synth.token_ids(B * (k + 1), shape.vocab, 1, "k7-block").reshape(B, k + 1)
    model = gm.DeviceModel(shape, W)
    cache = device_cache(shape, caches, lens, k + 1)
    logits, hidden = _gpu_forward(model, cache, tokens)
    ref_c, ref_hc, _ = oracle.verify_forward(shape, W, caches, tokens, lens, CONTRACT)
    print("[forward qwen3 layer bf16 k=7] logits rel err vs contract %.3e, hidden %.3e"
          % (rel_err(logits, ref_c), rel_err(hidden, ref_hc)), flush=True)
    assert rel_err(logits, ref_c) < 1e-2 and rel_err(hidden, ref_hc) < 1e-2


def test_qwen_layer_bf16_block_is_causal(qwen_layer):
    # Changing the last draft d_k leaves every earlier block row's logits and hidden
    # bit-identical (a block position sees only the positions before it, Sec. 3.1's
    # one-forward verification; outputs are deterministic), and does change row k
    need_gpu()
    wl, shape, W, lens, caches, tokens = qwen_layer
    k = wl.k
    model = gm.DeviceModel(shape, W)
    alt = tokens.copy()
    alt[:, k] = (alt[:, k] + 1 + np.arange(len(alt)) * 7919) % shape.vocab
    l0, h0 = _gpu_forward(model, device_cache(shape, caches, lens, k + 1), tokens)
    l1, h1 = _gpu_forward(model, device_cache(shape, caches, lens, k + 1), alt)
    np.testing.assert_array_equal(l0[:, :k], l1[:, :k])
    np.testing.assert_array_equal(h0[:, :k], h1[:, :k])
    assert (np.abs(l0[:, k] - l1[:, k]).max(-1) > 0).all()


# ------------------------------------------------------------------ target statistics handoff
def _stats_definition(z, temperature):
    """gm_row_stats of rows of float32 logits by definition: max of z * (1/T) in float32,
    the lowest id attaining it, sum of exp(z/T - max) in float64."""
    inv_t = np.float32(1.0) / np.float32(temperature)
    v = z.astype(np.float32) * inv_t
    m = v.max(-1)
    return m, v.argmax(-1), np.exp(v.astype(np.float64) - m[..., None].astype(np.float64)).sum(-1)


def _forward_with_stats(model, cache, tokens, temperature):
    B, k1 = tokens.shape
    s = model.shape
    logits = torch.empty((B, k1, s.vocab), dtype=torch.float32, device="cuda")
    hidden = torch.empty((B, k1, s.hidden), dtype=torch.float32, device="cuda")
    stats = gm.new_row_stats(B, k1)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    gm.verify_forward(model, cache, i32(tokens), logits, hidden, gm.Workspace(), err, target_stats=stats,
                      temperature=temperature)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return logits, stats


def _check_stats(name, stats, logits, temperature):
    # the handed-over statistics describe the logits they come with
    mx, am, sm = gm.decode_row_stats(stats)
    rm, ram, rs = _stats_definition(logits.cpu().numpy(), temperature)
    np.testing.assert_array_equal(mx, rm)
    np.testing.assert_array_equal(am, ram)
    e = float(np.abs(sm / rs - 1).max())
    print("[%s] T=%.2f statistics: max and arg-max exact, normaliser rel err %.2e" % (name, temperature, e), flush=True)
    assert e < 2e-6


def _accept_with_stats(logits, stats, zq, drafts, ua, uf, mode, temperature):
    B, k1, V = logits.shape
    n = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, k1), dtype=torch.int32, device="cuda")
    gm.spec_accept(logits, t32(zq) if zq is not None else None, i32(drafts), t32(ua) if ua is not None else None,
                   t32(uf) if uf is not None else None, n, out, mode, gm.Workspace(), temperature=temperature,
                   target_stats=stats)
    torch.cuda.synchronize()
    return n.cpu().numpy(), out.cpu().numpy()


def _handoff_parity(name, logits, stats, ref_logits, drafts, temperature, seed, final_floor):
    """Greedy and sampled acceptance with the forward's statistics against the oracle's
    accept on its own logits.  The flag windows widen with the measured deviation d of the
    two sets of logits: a ratio p/q moves by at most ~2d/T, a top-2 margin by 2d, a CDF edge
    by 2d/T of the mass."""
    B, k1, V = ref_logits.shape
    k = k1 - 1
    d = float(np.abs(logits.cpu().numpy().astype(np.float64) - ref_logits).max())
    # greedy
    ref = oracle.spec_accept(ref_logits, None, drafts, None, None, mode="greedy", margin_eps=max(1e-2, 2.5 * d))
    n, out = _accept_with_stats(logits, stats, None, drafts, None, None, gm.GM_GREEDY, temperature)
    ok = ~ref.flagged
    flag_report("%s greedy with target stats" % name, ref.flagged, B)
    assert ok.any()
    np.testing.assert_array_equal(n[ok], ref.n_accept[ok])
    np.testing.assert_array_equal(out[ok], ref.out_tokens[ok])
    # sample: q close to p (so deep prefixes and the bonus draw are reached), drafts ~ q
    zq = ref_logits[:, :k] + 0.3 * synth.normal_logits((B, k, V), seed, name, "zq").astype(np.float64)
    ua, uf, ud = synth.uniforms(B, k, seed, name)
    qd = oracle.softmax(zq / temperature)
    dr = np.stack([oracle.inverse_cdf_rows(qd[:, i], ud[:, i])[0] for i in range(k)], 1)
    zq32 = zq.astype(np.float32)
    ref = oracle.spec_accept(ref_logits, zq32, dr, ua, uf, temperature=temperature,
                             accept_eps=max(1e-3, 3 * d / temperature), final_eps=max(final_floor, 3 * d / temperature))
    n, out = _accept_with_stats(logits, stats, zq32, dr, ua, uf, gm.GM_SAMPLE, temperature)
    oka, ok = ~ref.flag_accept, ~ref.flagged
    print("[%s sample with target stats] logit deviation %.2e; accept decisions compared %d of %d, whole outputs %d; "
          "mean accepted %.2f" % (name, d, oka.sum(), B, ok.sum(), n.mean()), flush=True)
    assert oka.any()
    np.testing.assert_array_equal(n[oka], ref.n_accept[oka])
    np.testing.assert_array_equal(out[ok], ref.out_tokens[ok])
    return n


def test_target_stats_handoff_tiny_f32():
    # float32 model: the forward's statistics (a pass over the stored rows on this path) and
    # the accept that takes them, against the oracle's exact forward and accept
    need_gpu()
    wl = synth.WORKLOADS["tiny"]
    shape = wl.shape
    W = synth.model_weights(shape)
    B, k, T0 = wl.batch, wl.k, wl.ctx_lo
    prompt = synth.token_ids(B * T0, shape.vocab, 1, "tiny-prompt").reshape(B, T0)
    caches = oracle.prefill(shape, W, prompt, EXACT)
    caches = [([a.astype(np.float32) for a in ks], [a.astype(np.float32) for a in vs]) for ks, vs in caches]
    lens = np.full(B, T0)
    tokens = synth.token_ids(B * (k + 1), shape.vocab, 1, "tiny-block").reshape(B, k + 1)
    ref, _, _ = oracle.verify_forward(shape, W, caches, tokens, lens, EXACT)
    model = gm.DeviceModel(shape, W)
    for T in (1.0, 0.7):
        logits, stats = _forward_with_stats(model, device_cache(shape, caches, lens, k + 1), tokens, T)
        _check_stats("tiny f32", stats, logits, T)
        _handoff_parity("tiny f32 T=%.1f" % T, logits, stats, ref, tokens[:, 1:], T, 11, 1e-5)


@pytest.mark.parametrize("B", [64, 16])
def test_target_stats_handoff_qwen_layer(qwen_layer, B):
    # bf16 Qwen3-4B-shaped layer: M = 256 block rows take the tiled LM head's statistics
    # epilogue, M = 64 the strip-range kernel's; greedy and sampled decisions with the
    # handed-over statistics against the oracle (rounding-contract logits)
    need_gpu()
    wl, shape, W, lens, caches, tokens = qwen_layer
    k = wl.k
    lens, tokens = lens[:B], tokens[:B]
    caches = [(ks[:B], vs[:B]) for ks, vs in caches]
    ref, _, _ = oracle.verify_forward(shape, W, caches, tokens, lens, CONTRACT)
    model = gm.DeviceModel(shape, W)
    for T in ((1.0, 0.7) if B == 64 else (1.0,)):
        logits, stats = _forward_with_stats(model, device_cache(shape, caches, lens, k + 1), tokens, T)
        _check_stats("qwen3 layer B=%d" % B, stats, logits, T)
        n = _handoff_parity("qwen3 layer B=%d T=%.1f" % (B, T), logits, stats, ref, tokens[:, 1:], T, 12, 1e-8)
        # the statistics pass and the handoff decide alike on the same logits
        zq = ref[:, :k] + 0.3 * synth.normal_logits((B, k, shape.vocab), 12, "qwen3 layer B=%d T=%.1f" % (B, T), "zq")
        ua, uf, ud = synth.uniforms(B, k, 12, "qwen3 layer B=%d T=%.1f" % (B, T))
        qd = oracle.softmax(zq / T)
        dr = np.stack([oracle.inverse_cdf_rows(qd[:, i], ud[:, i])[0] for i in range(k)], 1)
        n_pass = torch.zeros(B, dtype=torch.int32, device="cuda")
        o_pass = torch.zeros((B, k + 1), dtype=torch.int32, device="cuda")
        gm.spec_accept(logits, t32(zq.astype(np.float32)), i32(dr), t32(ua), t32(uf), n_pass, o_pass, gm.GM_SAMPLE,
                       gm.Workspace(), temperature=T)
        torch.cuda.synchronize()
        assert (n_pass.cpu().numpy() == n).mean() >= 0.98


def test_qwen_layer_bf16_forward_200_rows(qwen_layer):
    # 50 of the sequences with k = 3: M = 200 verify rows, so the SwiGLU projection takes two
    # 128-row M tiles (the second holds 72 rows) of 160 columns with five compute waves, the
    # last column tile ragged (9728 features in 122 tiles of 80), and the LM head one 256-row
    # tile of 224 columns
    need_gpu()
    wl, shape, W, lens, caches, tokens = qwen_layer
    B = 50
    lens_b = lens[:B]
    caches_b = [(ks[:B], vs[:B]) for ks, vs in caches]
    tok_b = tokens[:B]
    model = gm.DeviceModel(shape, W)
    logits, hidden = _gpu_forward(model, device_cache(shape, caches_b, lens_b, wl.k + 1), tok_b)
    ref_c, ref_hc, _ = oracle.verify_forward(shape, W, caches_b, tok_b, lens_b, CONTRACT)
    print("[forward qwen3 layer bf16, 200 rows] logits rel err vs contract %.3e, hidden %.3e"
          % (rel_err(logits, ref_c), rel_err(hidden, ref_hc)), flush=True)
    assert rel_err(logits, ref_c) < 1e-2 and rel_err(hidden, ref_hc) < 1e-2


def test_strip_ranges_with_idle_waves():
    # A bf16 model whose vocabulary is 10248 strips of 16 ids (163968 ids): more strips than
    # 1024 waves hold at ten each, so the LM head at M = 64 rows runs 1025 strip ranges (1023 of
    # ten strips, two of nine) in 257 workgroups, the last of which holds three waves with no
    # range (they stage their share of the activations and meet the barriers, then leave).
    # Both K loops (ten and nine strips) and the idle waves run; logits against the oracle,
    # statistics against their definition.
    need_gpu()
    shape = synth.ModelShape(1, 256, 2, 2, 128, 512, 10248 * 16, dtype="bf16")
    W = synth.model_weights(shape)
    B, k = 16, 3
    lens = 96 + 16 * np.arange(B)
    caches = synth_caches(shape, lens, shape.n_layers)
    tokens = synth.token_ids(B * (k + 1), shape.vocab, 1, "idle-waves").reshape(B, k + 1)
    ref, _, _ = oracle.verify_forward(shape, W, caches, tokens, lens, CONTRACT)
    model = gm.DeviceModel(shape, W)
    logits, stats = _forward_with_stats(model, device_cache(shape, caches, lens, k + 1), tokens, 1.0)
    err = rel_err(logits.cpu().numpy(), ref)
    print("[strip ranges, 10248 strips] logits rel err vs contract %.3e" % err, flush=True)
    assert err < 1e-2
    _check_stats("strip ranges, 10248 strips", stats, logits, 1.0)
