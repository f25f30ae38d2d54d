"""The no-allocation accept (gm_spec_accept_noalloc, the library's fixed device scratch)
against gm_spec_accept with a caller workspace: identical decisions and tokens, bit for
bit, on two calls in a row -- the second smaller, so it runs on scratch the first left
behind -- in sample mode (with top-p on the second) and greedy mode."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import need_gpu, t32, i32
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu


def _inputs(B, k, V, tag):
    zt = synth.normal_logits((B, k + 1, V), 3, "noalloc-t", tag)
    zq = synth.normal_logits((B, k, V), 3, "noalloc-q", tag)
    ua, uf, ud = synth.uniforms(B, k, 4, "noalloc", tag)
    q = oracle.softmax(zq.astype(np.float64))
    drafts = np.stack([oracle.inverse_cdf_rows(q[:, i], ud[:, i])[0] for i in range(k)], 1) if k else np.zeros((B, 0))
    return t32(zt), t32(zq), i32(drafts), t32(ua), t32(uf)


def _both(zt, zq, drafts, ua, uf, mode, top_p):
    B, k1, _ = zt.shape
    outs = []
    for noalloc in (False, True):
        n = torch.full((B,), -7, dtype=torch.int32, device="cuda")
        out = torch.full((B, k1), -7, dtype=torch.int32, device="cuda")
        if noalloc:
            gm.spec_accept_noalloc(zt, zq if mode == gm.GM_SAMPLE else None, drafts, ua, uf, n, out, mode, top_p=top_p)
        else:
            gm.spec_accept(zt, zq if mode == gm.GM_SAMPLE else None, drafts, ua, uf, n, out, mode, gm.Workspace(),
                           top_p=top_p)
        torch.cuda.synchronize()
        outs.append((n.cpu().numpy(), out.cpu().numpy()))
    return outs


def test_noalloc_accept_matches_workspace_accept():
    need_gpu()
    cases = [(64, 3, 151936, gm.GM_SAMPLE, 1.0), (16, 2, 32000, gm.GM_SAMPLE, 0.7), (8, 1, 1000, gm.GM_GREEDY, 1.0)]
    for B, k, V, mode, top_p in cases:
        (n0, o0), (n1, o1) = _both(*_inputs(B, k, V, "%d-%d-%d" % (B, k, V)), mode, top_p)
        print("[noalloc] B=%d k=%d V=%d mode=%d top_p=%.1f: mean accepted %.2f" % (B, k, V, mode, top_p, n0.mean()),
              flush=True)
        assert (n0 >= 0).all() and (n0 <= k).all()
        np.testing.assert_array_equal(n1, n0)
        np.testing.assert_array_equal(o1, o0)
