"""Pins of the oracle's accept rule and KV commit (CPU only).

The four checks of the method: draft length 0 reproduces autoregressive
decoding; a draft equal to the target's greedy choice is fully accepted;
greedy acceptance is the longest argmax-matching prefix; and on a 4-token
vocabulary the committed tokens are distributed as the target (chi-square over
10^6 seeded trials).  Further pins: the acceptance rate equals
alpha = sum min(p, q) (Eq. alpha), the residual mass equals 1 - alpha, the
structure of the output, and the commit closed form."""
import json
import os

import numpy as np
import pytest
import scipy.stats

import oracle
import synth

EXACT = oracle.Rounding("exact")
HERE = os.path.dirname(os.path.abspath(__file__))


def _logits_of(p):
    return np.log(np.asarray(p, dtype=np.float64))


# ------------------------------------------------------------ check 1: k = 0 is AR decoding
def test_k0_reproduces_autoregressive_decoding():
    shape = synth.TINY
    W = synth.model_weights(shape, 0)
    B, T0, steps = 2, 24, 16
    prompt = synth.token_ids(B * (T0 + 1), shape.vocab, 1, "ar").reshape(B, T0 + 1)
    u = synth.stream(4, "ar-u").random((B, steps), dtype=np.float32)
    ref = oracle.ar_decode(shape, W, prompt, u, 1.0, EXACT)

    # speculative loop with k = 0: verify [t_m], accept (bonus draw), commit one token
    caches = oracle.prefill(shape, W, prompt[:, :T0], EXACT)
    lens = np.full(B, T0)
    pending = prompt[:, T0].copy()
    got = np.zeros((B, steps), dtype=np.int64)
    bt = np.arange(B * 8).reshape(B, 8)           # page table of 8 pages of 16 slots each
    for t in range(steps):
        logits, _, kv = oracle.verify_forward(shape, W, caches, pending[:, None], lens, EXACT)
        res = oracle.spec_accept(logits.astype(np.float32), np.zeros((B, 0, shape.vocab)),
                                 np.zeros((B, 0), np.int64), np.zeros((B, 0), np.float32), u[:, t])
        assert (res.n_accept == 0).all()
        new_lens, slots = oracle.kv_commit(lens, res.n_accept, 0, bt, 16)
        for l, (k, v) in enumerate(kv):
            for b in range(B):
                caches[l][0][b] = np.concatenate([caches[l][0][b], k[b, :1]])
                caches[l][1][b] = np.concatenate([caches[l][1][b], v[b, :1]])
        got[:, t] = res.out_tokens[:, 0]
        pending = res.out_tokens[:, 0]
        lens = new_lens
    np.testing.assert_array_equal(got, ref)
    assert (lens == T0 + steps).all()


# ------------------------------------------------------------ check 2: greedy drafts accepted
def test_draft_equal_to_greedy_choice_is_fully_accepted():
    shape = synth.TINY
    W = synth.model_weights(shape, 0)
    B, T0, k = 4, 32, 5
    prompt = synth.token_ids(B * T0, shape.vocab, 1, "g").reshape(B, T0)
    caches = oracle.prefill(shape, W, prompt[:, :-1], EXACT)
    lens = np.full(B, T0 - 1)
    drafts = oracle.mixing_drafts(shape, W, caches, lens, prompt[:, -1], np.ones((B, k), bool),
                                  np.zeros((B, k), np.int64), EXACT)
    # the plain definition: drafts are the argmax continuation of a no-cache forward
    seq = prompt.copy()
    for i in range(k):
        full, _, _ = oracle.full_forward(shape, W, seq, EXACT)
        nxt = np.argmax(full[:, -1].astype(np.float32), -1)
        np.testing.assert_array_equal(nxt, drafts[:, i])
        seq = np.concatenate([seq, nxt[:, None]], 1)
    block = np.concatenate([prompt[:, -1:], drafts], 1)
    logits, _, _ = oracle.verify_forward(shape, W, caches, block, lens, EXACT)
    res = oracle.spec_accept(logits, None, drafts, None, None, mode="greedy")
    np.testing.assert_array_equal(res.n_accept, k)
    np.testing.assert_array_equal(res.out_tokens[:, :k], drafts)
    np.testing.assert_array_equal(res.out_tokens[:, k], np.argmax(logits[:, k].astype(np.float32), -1))


def test_q_equal_p_accepts_every_draft():
    g = np.random.default_rng(1)
    B, k, V = 2000, 4, 9
    zt = g.standard_normal((B, k + 1, V))
    drafts = g.integers(0, V, (B, k))
    u = g.random((B, k)).astype(np.float32)
    res = oracle.spec_accept(zt, zt[:, :k], drafts, u, g.random(B))
    np.testing.assert_array_equal(res.n_accept, k)


# ------------------------------------------------------------ check 3: longest argmax prefix
def test_greedy_is_longest_argmax_matching_prefix():
    g = np.random.default_rng(2)
    B, k, V = 500, 6, 13
    z = g.standard_normal((B, k + 1, V)).astype(np.float32)
    z[:, :, 3] = z[:, :, 7]                          # plant exact ties: lowest id must win
    top = np.array([[min(np.flatnonzero(row == row.max())) for row in zb] for zb in z])
    plant = g.random((B, k)) < 0.8
    drafts = np.where(plant, top[:, :k], g.integers(0, V, (B, k)))
    res = oracle.spec_accept(z, None, drafts, None, None, mode="greedy")
    for b in range(B):
        n = 0
        while n < k and drafts[b, n] == top[b, n]:
            n += 1
        assert res.n_accept[b] == n
        assert list(res.out_tokens[b, :n]) == list(drafts[b, :n])
        assert res.out_tokens[b, n] == top[b, n]
        assert (res.out_tokens[b, n + 1:] == -1).all()


# ------------------------------------------------------------ check 4: distribution preserved
def _draw_from(q, u):
    x, _, _ = oracle.inverse_cdf_rows(q, u)
    return x


@pytest.mark.slow
def test_chi_square_single_position():
    trials, V = 1_000_000, 4
    p = np.array([0.1, 0.2, 0.3, 0.4])
    q = np.array([0.4, 0.3, 0.2, 0.1])
    g = synth.stream(4, "chi1")
    d = _draw_from(np.tile(q, (trials, 1)), g.random(trials))
    res = oracle.spec_accept(np.tile(_logits_of([p, p]), (trials, 1, 1)),
                             np.tile(_logits_of([q]), (trials, 1, 1)), d[:, None],
                             g.random((trials, 1), dtype=np.float32), g.random(trials))
    first = res.out_tokens[:, 0]
    counts = np.bincount(first, minlength=V)
    assert scipy.stats.chisquare(counts, trials * p).pvalue > 0.01
    # empirical acceptance = alpha = sum min(p, q) (Eq. alpha), within 5 sigma
    alpha = np.minimum(p, q).sum()
    acc = res.n_accept.mean()
    assert abs(acc - alpha) < 5 * np.sqrt(alpha * (1 - alpha) / trials)
    np.testing.assert_allclose(res.alpha[:, 0], alpha, rtol=1e-12)


@pytest.mark.slow
def test_chi_square_markov_chain_k3():
    # context-dependent target P(x | prev) and head Q(x | prev); drafts d_i ~ Q(. | d_{i-1});
    # cycles repeat until two tokens are committed; the joint of the first two must be P x P
    trials, V, k = 1_000_000, 4, 3
    g = synth.stream(4, "chi3")
    P = g.dirichlet(np.ones(V), size=V)
    Q = g.dirichlet(np.ones(V), size=V)
    start = 2
    ctx = np.full(trials, start)
    committed = [[] for _ in range(2)]
    firsts = np.full(trials, -1)
    seconds = np.full(trials, -1)
    live = np.arange(trials)
    while live.size:
        n = live.size
        drafts = np.zeros((n, k), np.int64)
        prev = ctx[live]
        qz = np.zeros((n, k, V))
        pz = np.zeros((n, k + 1, V))
        for i in range(k):
            pz[:, i] = np.log(P[prev])
            qz[:, i] = np.log(Q[prev])
            drafts[:, i] = _draw_from(Q[prev], g.random(n))
            prev = drafts[:, i]
        pz[:, k] = np.log(P[prev])
        res = oracle.spec_accept(pz, qz, drafts, g.random((n, k), dtype=np.float32), g.random(n))
        for j in range(k + 1):
            tok = res.out_tokens[:, j]
            ok = tok >= 0
            idx = live[ok]
            need1 = firsts[idx] < 0
            firsts[idx[need1]] = tok[ok][need1]
            need2 = (~need1) & (seconds[idx] < 0)
            seconds[idx[need2]] = tok[ok][need2]
        last = res.out_tokens[np.arange(n), res.n_accept]
        ctx[live] = last
        live = live[seconds[live] < 0]
    joint = np.bincount(firsts * V + seconds, minlength=V * V)
    expect = (P[start][:, None] * P).reshape(-1) * trials
    assert scipy.stats.chisquare(joint, expect).pvalue > 0.01


def test_residual_mass_is_one_minus_alpha():
    g = np.random.default_rng(3)
    for _ in range(100):
        p = g.dirichlet(np.ones(50) * 0.3)
        q = g.dirichlet(np.ones(50) * 0.3)
        assert abs(np.maximum(p - q, 0).sum() - (1 - np.minimum(p, q).sum())) < 1e-12


def test_output_structure_and_bounds():
    g = np.random.default_rng(4)
    B, k, V = 3000, 5, 6
    zt, zq = g.standard_normal((B, k + 1, V)), g.standard_normal((B, k, V))
    drafts = g.integers(0, V, (B, k))
    res = oracle.spec_accept(zt, zq, drafts, g.random((B, k)).astype(np.float32), g.random(B))
    assert res.n_accept.min() >= 0 and res.n_accept.max() <= k
    for b in range(0, B, 7):
        n = res.n_accept[b]
        assert list(res.out_tokens[b, :n]) == list(drafts[b, :n])
        assert 0 <= res.out_tokens[b, n] < V
        assert (res.out_tokens[b, n + 1:] == -1).all()
    tau = 1 + res.n_accept.mean()
    assert 1 <= tau <= k + 1
    # a rejected draft is never re-drawn as the replacement: the residual is zero there
    rej = res.n_accept < k
    b = np.flatnonzero(rej)
    assert (res.out_tokens[b, res.n_accept[b]] != drafts[b, res.n_accept[b]]).all()


def test_accept_is_strict_and_ratio_above_one_always_accepts():
    p = np.array([[0.5, 0.5], [0.5, 0.5]])
    q = np.array([[0.25, 0.75]])
    # p(0)/q(0) = 2 > any u in [0, 1): accepted; p(1)/q(1) = 2/3: accepted iff u < 2/3
    lt, lq = _logits_of(p)[None], _logits_of(q)[None]
    assert oracle.spec_accept(lt, lq, [[0]], np.array([[0.9999]], np.float32), [0.5]).n_accept[0] == 1
    r = np.float32(2.0 / 3.0)
    assert oracle.spec_accept(lt, lq, [[1]], np.array([[np.nextafter(r, 0)]], np.float32), [0.5]).n_accept[0] == 1
    assert oracle.spec_accept(lt, lq, [[1]], np.array([[r]], np.float32), [0.5]).n_accept[0] == 0


def test_flags_mark_near_threshold_decisions():
    lt = _logits_of([[0.5, 0.5], [0.5, 0.5]])[None]
    lq = _logits_of([[0.25, 0.75]])[None]
    near = oracle.spec_accept(lt, lq, [[1]], np.array([[0.6665]], np.float32), [0.3])
    far = oracle.spec_accept(lt, lq, [[1]], np.array([[0.2]], np.float32), [0.3])
    assert near.flag_accept[0] and not far.flag_accept[0]
    z = np.array([[[1.0, 1.004, 0.0]]], np.float32)
    assert oracle.spec_accept(z, None, np.zeros((1, 0), int), None, None, mode="greedy").flagged[0]


# ------------------------------------------------------------ commit closed form
def test_final_draw_window_in_probability_units():
    # k = 0: the final draw is the bonus draw from p.  With p = (0.1, 0.2, 0.3, 0.4) and u placed
    # 1e-6 above the edge C(1) = 0.3, the draw is id 2 and is flagged exactly when the absolute window
    # exceeds 1e-6 (a scalar, or one value per sequence); the relative window scales with Z = 1
    p = np.array([0.1, 0.2, 0.3, 0.4])
    z = np.log(p)[None, None, :].repeat(2, 0)
    u = np.array([0.3 + 1e-6, 0.3 + 1e-6])
    none = np.zeros((2, 0), dtype=np.int64)
    r = oracle.spec_accept(z, np.zeros((2, 0, 4)), none, np.zeros((2, 0)), u)
    assert (r.out_tokens[:, 0] == 2).all() and not r.flagged.any()
    assert oracle.spec_accept(z, np.zeros((2, 0, 4)), none, np.zeros((2, 0)), u, final_abs=2e-6).flagged.all()
    assert not oracle.spec_accept(z, np.zeros((2, 0, 4)), none, np.zeros((2, 0)), u, final_abs=5e-7).flagged.any()
    r = oracle.spec_accept(z, np.zeros((2, 0, 4)), none, np.zeros((2, 0)), u, final_abs=np.array([2e-6, 5e-7]))
    assert r.flagged.tolist() == [True, False]
    assert oracle.spec_accept(z, np.zeros((2, 0, 4)), none, np.zeros((2, 0)), u, final_eps=2e-6).flagged.all()


def test_kv_commit_golden_example():
    with open(os.path.join(HERE, "golden", "kv_commit_example.json")) as f:
        ex = json.load(f)
    new_lens, slots = oracle.kv_commit(ex["lens"], ex["n_accept"], ex["k"], ex["block_table"], ex["page_size"])
    assert new_lens.tolist() == ex["new_lens"]
    assert slots.tolist() == ex["committed_slots"]


def test_kv_commit_closed_form():
    g = np.random.default_rng(5)
    B, k, P = 50, 7, 16
    lens = g.integers(1, 1000, B)
    n = g.integers(0, k + 1, B)
    bt = g.permutation(B * 70).reshape(B, 70)
    new_lens, slots = oracle.kv_commit(lens, n, k, bt, P)
    np.testing.assert_array_equal(new_lens, lens + n + 1)
    assert ((slots >= 0).sum(1) == n + 1).all()
    allslots = slots[slots >= 0]
    assert len(set(allslots.tolist())) == allslots.size        # distinct physical slots
