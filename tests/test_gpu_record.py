"""GPU parity of the cycle record taken in gm_spec_accept's vocabulary pass
(App. "Implementing Draft-Path Reconstruction in verl": the target's top-64
log-probabilities per draft position, full-vocabulary normalised, in bf16)
against the oracle: ids bit-exact (the order is that of the logits, ties to the
lower id), log-probabilities within one bf16 step of the oracle's (both round a
value that agrees to ~1e-7 relative)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import need_gpu, t32, i32
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu


def _gpu_record(zt, drafts, topk, T, mode=None, zq=None, ua=None, uf=None):
    B, k1, V = zt.shape
    k = k1 - 1
    mode = gm.GM_GREEDY if mode is None else mode
    n = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, k1), dtype=torch.int32, device="cuda")
    logp = torch.zeros((B, k, topk), dtype=torch.bfloat16, device="cuda")
    ids = torch.full((B, k, topk), -7, dtype=torch.int32, device="cuda")
    gm.spec_accept(t32(zt), t32(zq) if zq is not None else None, i32(drafts), t32(ua) if ua is not None else None,
                   t32(uf) if uf is not None else None, n, out, mode, gm.Workspace(), temperature=T,
                   record=(logp, ids))
    torch.cuda.synchronize()
    return ids.cpu().numpy(), logp.float().cpu().numpy().astype(np.float64), n.cpu().numpy(), out.cpu().numpy()


def _check(zt, k, T, topk, ids, logp):
    ref_ids, ref_lp = oracle.record_topk(zt, k, T, topk)
    np.testing.assert_array_equal(ids, ref_ids)
    step = np.abs(ref_lp) * 2.0 ** -8 + 1e-30          # one bf16 step at that magnitude
    assert (np.abs(logp - ref_lp) <= step).all(), np.abs(logp - ref_lp).max()
    return float((logp == ref_lp).mean())


@pytest.mark.parametrize("B,k,V,topk,T", [(64, 3, 151936, 64, 1.0), (16, 7, 151936, 64, 0.7), (8, 3, 151680, 10, 1.0),
                                          (4, 2, 1000, 64, 1.0), (3, 1, 20000, 64, 1.0), (5, 2, 5000, 64, 1.0)])
def test_record_matches_oracle(B, k, V, topk, T):
    # V = 5000: fewer runs of 256 ids than the record is wide, so every id qualifies and the
    # selection takes the exact bisection; V = 1000 and 20000: the sorted-candidate path
    need_gpu()
    zt = synth.normal_logits((B, k + 1, V), 3, "rec", B, k, V) * np.float32(3.0)
    drafts = np.zeros((B, k), dtype=np.int64)
    ids, logp, _, _ = _gpu_record(zt, drafts, topk, T)
    same = _check(zt, k, T, topk, ids, logp)
    print("[record B=%d k=%d V=%d top%d T=%.1f] ids exact, log-probs bit-equal %.4f" % (B, k, V, topk, T, same),
          flush=True)


def test_record_ties_and_flat_rows():
    # row 0: 300 ids share the maximum, the record takes the 64 lowest of them; row 1: a flat
    # row (every id ties, the bisection path), ids 0..63 at log(1/V)
    need_gpu()
    B, k, V = 2, 2, 151936
    g = np.random.default_rng(3)
    zt = g.standard_normal((B, k + 1, V)).astype(np.float32)
    tied = np.sort(g.choice(V, 300, replace=False))
    zt[0, 0, tied] = 9.0
    zt[1, 1, :] = 0.5
    ids, logp, _, _ = _gpu_record(zt, np.zeros((B, k), np.int64), 64, 1.0)
    _check(zt, k, 1.0, 64, ids, logp)
    assert ids[0, 0].tolist() == tied[:64].tolist()
    assert ids[1, 1].tolist() == list(range(64))


def test_record_leaves_the_accept_unchanged():
    need_gpu()
    B, k, V = 32, 3, 151936
    zt = synth.normal_logits((B, k + 1, V), 3, "rec2", B, k, V)
    zq = synth.normal_logits((B, k, V), 3, "rec2q", B, k, V)
    ua, uf, _ = synth.uniforms(B, k, 4, "rec2")
    drafts = np.argmax(zq, -1)
    ids, logp, n1, o1 = _gpu_record(zt, drafts, 64, 1.0, gm.GM_SAMPLE, zq, ua, uf)
    n0 = torch.zeros(B, dtype=torch.int32, device="cuda")
    o0 = torch.zeros((B, k + 1), dtype=torch.int32, device="cuda")
    gm.spec_accept(t32(zt), t32(zq), i32(drafts), t32(ua), t32(uf), n0, o0, gm.GM_SAMPLE, gm.Workspace())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(n0.cpu().numpy(), n1)
    np.testing.assert_array_equal(o0.cpu().numpy(), o1)
    _check(zt, k, 1.0, 64, ids, logp)
