"""Pins of the oracle's top-p variant (CPU only).

The paper's evaluation decodes at T = 1 and top-p 0.7 with rejection sampling
(App. "Evaluation Configuration").  The oracle replaces every p_i and q_i by
its nucleus before the accept rule.  Pinned by hand-worked nuclei, by the
distribution check of rejection sampling (the committed tokens, first and
bonus, are distributed as the nucleus of the target when the drafts are
samples of the head's nucleus), and by the limit top_p -> 0, where every
nucleus is the argmax and sampled acceptance becomes greedy decoding."""
import numpy as np
import pytest
import scipy.stats

import oracle
import synth


def _lg(p):
    return np.log(np.asarray(p, dtype=np.float64))


def test_nucleus_hand_examples():
    z = _lg([0.1, 0.4, 0.3, 0.2])
    p = oracle.softmax(z)
    # ranked 1 (0.4), 2 (0.3), 3 (0.2), 0 (0.1): 0.4 < 0.65 <= 0.7 keeps {1, 2}
    got, dist = oracle.nucleus(z, p, 0.65)
    np.testing.assert_allclose(got, [0, 4 / 7, 3 / 7, 0], rtol=1e-12)
    assert abs(dist - 0.05) < 1e-12
    got, _ = oracle.nucleus(z, p, 0.35)                 # the top id alone reaches 0.35
    np.testing.assert_allclose(got, [0, 1, 0, 0])
    got, _ = oracle.nucleus(z, p, 0.95)                 # 0.9 < 0.95: all four
    np.testing.assert_allclose(got, p, rtol=1e-12)
    got, dist = oracle.nucleus(z, p, 1.0)               # top_p = 1: no truncation
    np.testing.assert_allclose(got, p, rtol=1e-12)
    assert np.isinf(dist)
    # equal logits: the lower ids come first
    got, _ = oracle.nucleus(np.zeros(4), np.full(4, 0.25), 0.6)
    np.testing.assert_allclose(got, [1 / 3, 1 / 3, 1 / 3, 0], rtol=1e-12)
    # a tie at the boundary behind a larger entry: 0.4 + 0.2 + 0.2 reaches 0.75 with ids 1, 0, 2
    zt = _lg([0.2, 0.4, 0.2, 0.2])
    got, _ = oracle.nucleus(zt, oracle.softmax(zt), 0.75)
    np.testing.assert_allclose(got, [0.25, 0.5, 0.25, 0], rtol=1e-12)
    # rows are independent
    zz = np.stack([z, zt])
    got, _ = oracle.nucleus(zz, oracle.softmax(zz), 0.65)
    np.testing.assert_allclose(got[0], [0, 4 / 7, 3 / 7, 0], rtol=1e-12)
    np.testing.assert_allclose(got[1], [0.25, 0.5, 0.25, 0], rtol=1e-12)   # 0.6 < 0.65: id 2 too


def test_nucleus_matches_brute_force_sort():
    # against a plain per-row loop over a full sort, on random rows with repeated values
    g = np.random.default_rng(11)
    for trial in range(200):
        V = int(g.integers(1, 40))
        z = np.round(g.standard_normal(V) * 2, 1).astype(np.float32)   # ties are common
        p = oracle.softmax(z.astype(np.float64))
        top_p = float(g.uniform(0.05, 0.999))
        got, _ = oracle.nucleus(z, p, top_p)
        ranked = sorted(range(V), key=lambda x: (-float(z[x]), x))
        kept, run = [], 0.0
        for x in ranked:
            kept.append(x)
            run += p[x]
            if run >= top_p:
                break
        ref = np.zeros(V)
        ref[kept] = p[kept]
        np.testing.assert_allclose(got, ref / ref.sum(), rtol=1e-12, atol=1e-300)


def _draw(q, u):
    return oracle.inverse_cdf_rows(q, u)[0]


@pytest.mark.slow
def test_committed_tokens_follow_the_target_nucleus():
    # k = 2.  Drafts are samples of the head's nucleus; the first committed token
    # must follow nucleus(p_1), and the bonus token (both accepted) nucleus(p_3)
    trials, V, top_p = 600_000, 6, 0.6
    p1 = np.array([0.05, 0.10, 0.15, 0.20, 0.22, 0.28])     # nucleus {5, 4, 3}
    q1 = np.array([0.05, 0.10, 0.30, 0.25, 0.20, 0.10])     # nucleus {2, 3, 4}
    p2 = np.array([0.30, 0.25, 0.20, 0.10, 0.10, 0.05])
    q2 = np.array([0.25, 0.30, 0.15, 0.10, 0.10, 0.10])
    p3 = np.array([0.12, 0.18, 0.10, 0.35, 0.15, 0.10])
    g = synth.stream(4, "top-p-chi")
    pz = np.tile(_lg([p1, p2, p3]), (trials, 1, 1))
    qz = np.tile(_lg([q1, q2]), (trials, 1, 1))
    nq1 = oracle.nucleus(_lg(q1), q1, top_p)[0]
    nq2 = oracle.nucleus(_lg(q2), q2, top_p)[0]
    d = np.stack([_draw(np.tile(nq1, (trials, 1)), g.random(trials)),
                  _draw(np.tile(nq2, (trials, 1)), g.random(trials))], axis=1)
    res = oracle.spec_accept(pz, qz, d, g.random((trials, 2), dtype=np.float32), g.random(trials),
                             top_p=top_p)
    np1 = oracle.nucleus(_lg(p1), p1, top_p)[0]
    np3 = oracle.nucleus(_lg(p3), p3, top_p)[0]
    first = res.out_tokens[:, 0]
    assert ((first == 3) | (first == 4) | (first == 5)).all()         # never outside the nucleus
    c1 = np.bincount(first, minlength=V)[3:]
    assert scipy.stats.chisquare(c1, trials * np1[3:]).pvalue > 0.01
    both = res.n_accept == 2
    bonus = res.out_tokens[both, 2]
    keep3 = np.nonzero(np3)[0]
    cb = np.bincount(bonus, minlength=V)
    assert cb[np3 == 0].sum() == 0
    assert scipy.stats.chisquare(cb[keep3], both.sum() * np3[keep3]).pvalue > 0.01
    # acceptance of the first draft = sum min(p', q') (Eq. alpha on the nuclei)
    alpha = np.minimum(np1, nq1).sum()
    acc = (res.n_accept >= 1).mean()
    assert abs(acc - alpha) < 5 * np.sqrt(alpha * (1 - alpha) / trials)
    np.testing.assert_allclose(res.alpha[:, 0], alpha, rtol=1e-12)


def test_top_p_to_zero_is_greedy_decoding():
    # as top_p -> 0 every nucleus is the argmax: a draft sampled from the head's nucleus
    # is its argmax, accepted iff it is the target's argmax, and the final token is the
    # argmax of row n + 1 -- the greedy rule
    g = np.random.default_rng(5)
    B, k, V = 64, 3, 50
    zt = g.standard_normal((B, k + 1, V)).astype(np.float32)
    zq = g.standard_normal((B, k, V)).astype(np.float32)
    agree = g.random((B, k)) < 0.6                   # head row equal to the target row: accepted
    zq[agree] = zt[:, :k][agree]
    drafts = zq.argmax(-1)
    u = g.random((B, k), dtype=np.float32)
    uf = g.random(B)
    res = oracle.spec_accept(zt, zq, drafts, u, uf, top_p=1e-12)
    ref = oracle.spec_accept(zt, None, drafts, u, uf, mode="greedy")
    np.testing.assert_array_equal(res.n_accept, ref.n_accept)
    np.testing.assert_array_equal(res.out_tokens, ref.out_tokens)
    assert 0 < ref.n_accept.mean() < k


def test_top_p_one_is_the_plain_rule_and_flags():
    g = np.random.default_rng(8)
    B, k, V = 16, 3, 30
    zt = g.standard_normal((B, k + 1, V))
    zq = g.standard_normal((B, k, V))
    d = g.integers(0, V, (B, k))
    u = g.random((B, k), dtype=np.float32)
    uf = g.random(B)
    a = oracle.spec_accept(zt, zq, d, u, uf)
    b = oracle.spec_accept(zt, zq, d, u, uf, top_p=1.0)
    np.testing.assert_array_equal(a.out_tokens, b.out_tokens)
    # a nucleus boundary within nucleus_eps of top_p flags its sequence
    p = oracle.softmax(zt[0, 0])
    c = np.cumsum(np.sort(p)[::-1])
    near = float(c[5]) + 1e-12
    r = oracle.spec_accept(zt[:1], zq[:1], d[:1], u[:1], uf[:1], top_p=near, nucleus_eps=1e-9)
    assert r.flag_accept[0]
    r = oracle.spec_accept(zt[:1], zq[:1], d[:1], u[:1], uf[:1], top_p=float(c[5]) + 0.5 * (c[6] - c[5]),
                           nucleus_eps=1e-9, accept_eps=0.0)
    assert not r.flag_accept[0]
