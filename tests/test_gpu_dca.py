"""GPU parity of gm_dca_loss (the DCA loss with verify-gated masking over the
cycle record's top-k support plus a residual bin, and its gradient in the head
logits) against the oracle on the same seeded inputs: loss and alpha within
1e-6 relative (both are float64 sums of the same float32 logits), the gradient
within 1e-5 of its largest entry (float32 on the GPU)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import need_gpu, t32, i32
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu


def _inputs(N, K, V, topk, seed):
    g = np.random.default_rng(seed)
    zt = synth.normal_logits((N, K + 1, V), 3, "dca", N, K, V) * np.float32(2.0)
    zq = (zt[:, :K] + g.standard_normal((N, K, V)).astype(np.float32)).astype(np.float32)
    ids, logp = oracle.record_topk(zt, K, 1.0, topk)
    n = g.integers(0, K + 1, N)
    return zq, ids, logp, n


def _gpu(zq, ids, logp, n, vgm, with_grad=True):
    N, K, V = zq.shape
    topk = ids.shape[-1]
    loss = torch.zeros(N, dtype=torch.float32, device="cuda")
    alpha = torch.zeros((N, K), dtype=torch.float32, device="cuda")
    grad = torch.full((N, K, V), 7.0, dtype=torch.float32, device="cuda") if with_grad else None
    lp = torch.from_numpy(logp.astype(np.float32)).to("cuda").to(torch.bfloat16)   # bf16 values: exact
    gm.dca_loss(t32(zq), lp, i32(ids), i32(n), loss, alpha, grad, gm.Workspace(), vgm=vgm)
    torch.cuda.synchronize()
    return loss.cpu().numpy(), alpha.cpu().numpy(), grad.cpu().numpy() if with_grad else None


@pytest.mark.parametrize("N,K,V,topk,vgm", [(16, 3, 151936, 64, True), (16, 3, 151936, 64, False),
                                            (8, 7, 20000, 64, True), (33, 1, 1000, 16, True), (5, 2, 64, 64, True)])
def test_dca_matches_oracle(N, K, V, topk, vgm):
    need_gpu()
    zq, ids, logp, n = _inputs(N, K, V, topk, N + K + V)
    loss, alpha, grad = _gpu(zq, ids, logp, n, vgm)
    rl, ra, rg = oracle.dca_loss(zq, ids, logp, n, vgm)
    np.testing.assert_allclose(alpha, ra, rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(loss, rl, rtol=1e-6, atol=1e-7)
    err = np.abs(grad - rg).max() / np.abs(rg).max()
    print("[dca N=%d K=%d V=%d top%d vgm=%d] loss %.4f, grad rel err %.2e" % (N, K, V, topk, vgm, rl.mean(), err),
          flush=True)
    assert err < 1e-5
    if vgm:   # positions past the first rejection get no gradient
        for b in range(N):
            assert (grad[b, min(int(n[b]) + 1, K):] == 0).all()


def test_dca_without_gradient_and_on_the_accepts_own_record():
    # the record taken by gm_spec_accept feeds the loss directly
    need_gpu()
    N, K, V = 24, 3, 151936
    zt = synth.normal_logits((N, K + 1, V), 3, "dca2", N, K, V) * np.float32(2.0)
    zq = (zt[:, :K] + np.random.default_rng(2).standard_normal((N, K, V)).astype(np.float32)).astype(np.float32)
    rec_lp = torch.zeros((N, K, 64), dtype=torch.bfloat16, device="cuda")
    rec_id = torch.zeros((N, K, 64), dtype=torch.int32, device="cuda")
    n = torch.zeros(N, dtype=torch.int32, device="cuda")
    out = torch.zeros((N, K + 1), dtype=torch.int32, device="cuda")
    drafts = np.argmax(zq, -1)
    gm.spec_accept(t32(zt), None, i32(drafts), None, None, n, out, gm.GM_GREEDY, gm.Workspace(), record=(rec_lp, rec_id))
    torch.cuda.synchronize()
    ids, logp, na = rec_id.cpu().numpy(), rec_lp.float().cpu().numpy().astype(np.float64), n.cpu().numpy()
    loss, alpha, _ = _gpu(zq, ids, logp, na, True, with_grad=False)
    rl, ra, _ = oracle.dca_loss(zq, ids, logp, na, True)
    np.testing.assert_allclose(alpha, ra, rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(loss, rl, rtol=1e-6, atol=1e-7)
