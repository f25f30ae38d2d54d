"""Pins of the oracle's elementary numerics against library routines, closed
forms and invariants (CPU only)."""
import numpy as np
import pytest
import scipy.special
import torch

import oracle
from oracle import numerics as nx


def test_round_bf16_matches_torch_conversion():
    # torch's float32 -> bfloat16 conversion (round to nearest even) is the library routine
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(20000) * 10.0 ** g.integers(-6, 6, 20000),
                        1.0 + np.arange(16) * 2.0 ** -8])              # halfway cases
    ref = torch.tensor(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(nx.round_bf16(x), ref)


def test_round_bf16_ties_to_even():
    # 1 + 2^-8 lies halfway between 1 and 1 + 2^-7 (bf16 has 7 stored mantissa bits)
    assert nx.round_bf16(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    assert nx.round_bf16(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6


def test_softmax_matches_scipy_and_invariants():
    g = np.random.default_rng(1)
    z = g.standard_normal((7, 33)) * 5
    p = nx.softmax(z)
    np.testing.assert_allclose(p, scipy.special.softmax(z, axis=-1), rtol=1e-13, atol=0)
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=1e-14)
    np.testing.assert_allclose(nx.softmax(z + 123.0), p, rtol=1e-12)


def test_rmsnorm_matches_torch():
    g = np.random.default_rng(2)
    x = g.standard_normal((5, 64))
    w = g.standard_normal(64)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (64,), torch.tensor(w), eps=1e-6).numpy()
    np.testing.assert_allclose(nx.rmsnorm(x, w, 1e-6), ref, rtol=1e-12, atol=1e-14)
    # unit weight gives unit root-mean-square
    y = nx.rmsnorm(x, np.ones(64), 0.0)
    np.testing.assert_allclose(np.sqrt((y * y).mean(-1)), 1.0, rtol=1e-12)


def test_silu_matches_torch():
    x = np.linspace(-30, 30, 1001)
    ref = torch.nn.functional.silu(torch.tensor(x)).numpy()
    np.testing.assert_allclose(nx.silu(x), ref, rtol=1e-13, atol=1e-300)


def test_rope_is_complex_rotation():
    # textbook form: the pair (x_i, x_{i+d/2}) is the complex number x_i + j x_{i+d/2}
    # multiplied by exp(j * pos * base^(-2i/d))
    g = np.random.default_rng(3)
    d, base = 16, 10000.0
    x = g.standard_normal((6, 3, d))
    pos = np.array([0, 1, 7, 100, 4095, 32767])
    y = nx.rope(x, pos, base)
    half = d // 2
    cz = x[..., :half] + 1j * x[..., half:]
    theta = pos[:, None] * base ** (-2.0 * np.arange(half) / d)
    rot = cz * np.exp(1j * theta)[:, None, :]
    np.testing.assert_allclose(y[..., :half], rot.real, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y[..., half:], rot.imag, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(y[0], x[0])                              # position 0: identity
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)


def test_rope_relative_positions():
    # <R(m) q, R(n) k> depends on m - n only
    g = np.random.default_rng(4)
    q, k = g.standard_normal((1, 1, 32)), g.standard_normal((1, 1, 32))
    a = np.sum(nx.rope(q, np.array([50]), 1e4) * nx.rope(k, np.array([20]), 1e4))
    b = np.sum(nx.rope(q, np.array([1030]), 1e4) * nx.rope(k, np.array([1000]), 1e4))
    assert abs(a - b) < 1e-10


def test_inverse_cdf_matches_searchsorted():
    g = np.random.default_rng(5)
    for _ in range(200):
        w = g.random(50) * (g.random(50) < 0.7)
        if w.sum() == 0:
            continue
        u = g.random()
        x, dist, z = nx.inverse_cdf(w, u)
        c = np.cumsum(w)
        assert x == int(np.searchsorted(c, u * c[-1], side="right"))
        assert w[x] > 0 and dist >= 0
    # batched form agrees with the single-row form
    W = g.random((30, 20))
    U = g.random(30)
    xs, _, _ = nx.inverse_cdf_rows(W, U)
    assert [nx.inverse_cdf(W[i], U[i])[0] for i in range(30)] == list(xs)


def test_inverse_cdf_frequencies():
    # over an even grid of u the draw hits each id in proportion to its weight
    w = np.array([0.1, 0.0, 0.45, 0.25, 0.2])
    grid = (np.arange(100000) + 0.5) / 100000
    xs, _, _ = nx.inverse_cdf_rows(np.tile(w, (grid.size, 1)), grid)
    freq = np.bincount(xs, minlength=5) / grid.size
    np.testing.assert_allclose(freq, w, atol=2e-5)


def test_rounding_modes():
    x = np.array([1.0 + 2.0 ** -10, -3.14159])
    np.testing.assert_array_equal(oracle.Rounding("exact")(x), x)
    np.testing.assert_array_equal(oracle.Rounding("contract")(x), nx.round_bf16(x))
    with pytest.raises(ValueError):
        oracle.Rounding("bf16")


def test_inverse_cdf_edges():
    # a zero-weight id is never drawn, and a target exactly on an edge belongs to the next id
    assert nx.inverse_cdf(np.array([0.0, 1.0, 1.0]), 0.0)[0] == 1
    assert nx.inverse_cdf(np.array([1.0, 1.0, 1.0, 1.0]), 0.5)[0] == 2
    xs, _, _ = nx.inverse_cdf_rows(np.array([[0.0, 1.0, 1.0], [1.0, 1.0, 1.0, 1.0][:3]]), np.array([0.0, 1 / 3]))
    assert list(xs) == [1, 1]
