"""Pins of the oracle's DCA + VGM loss and its gradient (Sec. "The Depth-Coupled
Acceptance Loss", "Learning up to the First Rejection"; App. "DCA"; the sparse
top-64 overlap with a residual bin of App. "Implementing Draft-Path
Reconstruction in verl")."""
import numpy as np
import pytest
import torch

import oracle


def _case(N, K, V, W, seed, exact_logp=True):
    g = np.random.default_rng(seed)
    zt = g.standard_normal((N, K, V)) * 1.5                      # target logits
    zq = zt + g.standard_normal((N, K, V)) * 0.8                  # a head near the target
    lp_full = zt - np.log(np.exp(zt).sum(-1, keepdims=True))
    ids = np.argsort(-zt, -1, kind="stable")[..., :W]
    logp = np.take_along_axis(lp_full, ids, -1)
    if not exact_logp:
        logp = oracle.round_bf16(logp)
    n = g.integers(0, K + 1, N)
    return zq, ids, logp, n, lp_full


def _torch_loss(zq, ids, logp, n, vgm, tv=False):
    """The same objective written with torch ops; float64 autograd gives the gradient."""
    z = torch.tensor(zq, dtype=torch.float64, requires_grad=True)
    q = torch.softmax(z, -1)
    qS = torch.gather(q, -1, torch.tensor(ids))
    pS = torch.exp(torch.tensor(logp, dtype=torch.float64))
    pR = torch.clamp(1 - pS.sum(-1), min=0)
    qR = 1 - qS.sum(-1)
    alpha = torch.minimum(pS, qS).sum(-1) + torch.minimum(pR, qR)
    K = zq.shape[1]
    losses = []
    for b in range(zq.shape[0]):
        L = min(int(n[b]) + 1, K) if vgm else K
        chain = torch.cumprod(alpha[b, :L], 0).sum()
        losses.append(-chain if tv else -torch.log(chain))
    total = torch.stack(losses)
    total.sum().backward()
    return total.detach().numpy(), alpha.detach().numpy(), z.grad.numpy()


@pytest.mark.parametrize("vgm", [True, False])
@pytest.mark.parametrize("N,K,V,W", [(6, 3, 300, 64), (4, 7, 200, 16), (3, 1, 100, 64)])
def test_dca_matches_autograd(N, K, V, W, vgm):
    zq, ids, logp, n, _ = _case(N, K, V, W, N + K + V, exact_logp=False)
    loss, alpha, grad = oracle.dca_loss(zq, ids, logp, n, vgm)
    tl, ta, tg = _torch_loss(zq, ids, logp, n, vgm)
    np.testing.assert_allclose(loss, tl, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(alpha, ta, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(grad, tg, rtol=1e-9, atol=1e-15)


def test_alpha_is_one_minus_total_variation_when_the_record_covers_the_vocabulary():
    # Eq. alpha: sum_d min(p, q) = 1 - TV(p, q)
    zq, ids, logp, n, lp_full = _case(5, 3, 48, 48, 7)
    _, alpha, _ = oracle.dca_loss(zq, ids, logp, n)
    p = np.exp(lp_full)
    q = np.exp(zq - np.log(np.exp(zq).sum(-1, keepdims=True)))
    np.testing.assert_allclose(alpha, 1 - 0.5 * np.abs(p - q).sum(-1), rtol=1e-12, atol=1e-12)


def test_sparse_overlap_bounds_the_full_overlap():
    # the top-64 overlap with a residual bin exceeds the full one by at most the target mass outside
    zq, ids, logp, n, lp_full = _case(6, 3, 400, 64, 8)
    _, alpha, _ = oracle.dca_loss(zq, ids, logp, n)
    p = np.exp(lp_full)
    q = np.exp(zq - np.log(np.exp(zq).sum(-1, keepdims=True)))
    full = np.minimum(p, q).sum(-1)
    outside = 1 - np.exp(logp).sum(-1)
    assert (alpha >= full - 1e-12).all() and (alpha <= full + outside + 1e-12).all()


def test_dca_gradient_is_the_tv_gradient_over_the_chain_value():
    # Eq. dca-identity: grad L_DCA = grad L_TV / M with M = -L_TV
    zq, ids, logp, n, _ = _case(5, 4, 250, 64, 9, exact_logp=False)
    loss, _, grad = oracle.dca_loss(zq, ids, logp, n, True)
    tv, _, tv_grad = _torch_loss(zq, ids, logp, n, True, tv=True)
    M = -tv
    np.testing.assert_allclose(np.exp(-loss), M, rtol=1e-12)
    np.testing.assert_allclose(grad, tv_grad / M[:, None, None], rtol=1e-9, atol=1e-15)


def test_vgm_truncates_at_the_first_rejection():
    zq, ids, logp, _, _ = _case(4, 3, 200, 64, 10)
    n0 = np.zeros(4, dtype=np.int64)                       # rejected at the first draft
    loss, alpha, grad = oracle.dca_loss(zq, ids, logp, n0, True)
    np.testing.assert_allclose(loss, -np.log(alpha[:, 0]), rtol=1e-13)
    assert (grad[:, 1:] == 0).all() and (np.abs(grad[:, 0]).max(-1) > 0).all()
    nK = np.full(4, 3)                                      # every draft accepted: the full chain
    np.testing.assert_allclose(oracle.dca_loss(zq, ids, logp, nK, True)[0],
                               oracle.dca_loss(zq, ids, logp, nK, False)[0], rtol=0)


def test_perfect_head_gives_minus_log_chain_length():
    # q = p and the record covers the vocabulary: alpha = 1, M = L, loss = -log L (min is not
    # differentiable where q = p, so no gradient value is pinned here)
    g = np.random.default_rng(11)
    V, K = 32, 3
    z = g.standard_normal((3, K, V))
    lp = z - np.log(np.exp(z).sum(-1, keepdims=True))
    ids = np.tile(np.arange(V), (3, K, 1))
    n = np.array([0, 1, 3])
    loss, alpha, grad = oracle.dca_loss(z, ids, lp, n, True)
    np.testing.assert_allclose(alpha, 1, atol=1e-13)
    np.testing.assert_allclose(loss, -np.log([1, 2, 3]), atol=1e-13)
