"""End-to-end GPU parity of the step: the four entry points chained over
several cycles, against the oracle chained the same way.

* draft length 0 on the GPU reproduces plain autoregressive decoding of the
  oracle (no-cache recomputation, same uniforms);
* a greedy loop verify -> accept -> commit -> MTP draft commits the same
  tokens as the oracle's loop, cycle after cycle."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import need_gpu, device_cache, t32, i32, EXACT
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu


def test_k0_gpu_reproduces_autoregressive_decoding():
    need_gpu()
    shape = synth.TINY
    W = synth.model_weights(shape)
    B, T0, steps = 3, 40, 16
    prompt = synth.token_ids(B * (T0 + 1), shape.vocab, 1, "gpu-ar").reshape(B, T0 + 1)
    u = synth.stream(4, "gpu-ar-u").random((B, steps), dtype=np.float32)
    ref = oracle.ar_decode(shape, W, prompt, u, 1.0, EXACT)

    caches = oracle.prefill(shape, W, prompt[:, :T0], EXACT)
    caches = [([a.astype(np.float32) for a in ks], [a.astype(np.float32) for a in vs]) for ks, vs in caches]
    model = gm.DeviceModel(shape, W)
    cache = device_cache(shape, caches, np.full(B, T0), steps + 1)
    cache.max_ctx = T0 + steps
    ws = gm.Workspace()
    logits = torch.empty((B, 1, shape.vocab), dtype=torch.float32, device="cuda")
    hidden = torch.empty((B, 1, shape.hidden), dtype=torch.float32, device="cuda")
    n = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, 1), dtype=torch.int32, device="cuda")
    empty_i = torch.zeros((B, 0), dtype=torch.int32, device="cuda")
    pending = i32(prompt[:, T0:T0 + 1])
    got = []
    for t in range(steps):
        gm.verify_forward(model, cache, pending, logits, hidden, ws)
        gm.spec_accept(logits, None, empty_i, None, t32(u[:, t]), n, out, gm.GM_SAMPLE, ws)
        gm.kv_commit(cache, 0, n)
        pending = out.clone()
        got.append(out[:, 0].clone())
    torch.cuda.synchronize()
    got = torch.stack(got, 1).cpu().numpy()
    np.testing.assert_array_equal(got, ref)
    np.testing.assert_array_equal(cache.seq_lens.cpu().numpy(), T0 + steps)


@pytest.mark.parametrize("k", [3, 7])
def test_greedy_loop_with_mtp_matches_oracle(k):
    # k = 7: the deeper chains of the paper's depth study
    need_gpu()
    shape = synth.TINY
    W = synth.model_weights(shape)
    Wm = synth.mtp_weights(shape)
    B, T0, cycles = 4, 48, 5
    prompt = synth.token_ids(B * (T0 + 1), shape.vocab, 1, "loop").reshape(B, T0 + 1)
    caches = oracle.prefill(shape, W, prompt[:, :T0], EXACT)
    caches = [([a.astype(np.float32) for a in ks], [a.astype(np.float32) for a in vs]) for ks, vs in caches]
    lens = np.full(B, T0)
    mk, mv = synth.kv_prefix(shape, lens, layer=77)
    mcaches = [(list(mk), list(mv))]
    drafts = synth.token_ids(B * k, shape.vocab, 1, "loop-d0").reshape(B, k)
    pending = prompt[:, T0]

    # ---- GPU loop
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cap = (k + 1) * cycles + 2 * k + 2
    cache = device_cache(shape, caches, lens, cap)
    mcache = device_cache(shape, mcaches, lens, cap)
    cache.max_ctx = mcache.max_ctx = T0 + (k + 1) * cycles
    ws, ws2 = gm.Workspace(), gm.Workspace()
    logits = torch.empty((B, k + 1, shape.vocab), dtype=torch.float32, device="cuda")
    hidden = torch.empty((B, k + 1, shape.hidden), dtype=torch.float32, device="cuda")
    n = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, k + 1), dtype=torch.int32, device="cuda")
    d_dev = i32(drafts)
    dlog = torch.zeros((B, k, shape.vocab), dtype=torch.float32, device="cuda")
    p_dev = i32(pending)
    gpu_out = []
    for c in range(cycles):
        tokens = torch.cat([p_dev[:, None], d_dev], 1).contiguous()
        gm.verify_forward(model, cache, tokens, logits, hidden, ws)
        gm.spec_accept(logits, None, d_dev, None, None, n, out, gm.GM_GREEDY, ws)
        gm.kv_commit(cache, k, n)
        nxt = torch.zeros((B, k), dtype=torch.int32, device="cuda")
        gm.mtp_draft(model, mtp, mcache, k, gm.GM_GREEDY, hidden, n, out, None, nxt, dlog, ws2)
        p_dev = out.gather(1, n.long()[:, None])[:, 0].contiguous()
        d_dev = nxt
        gpu_out.append(out.cpu().numpy())
    torch.cuda.synchronize()

    # ---- oracle loop
    lens_o = lens.copy()
    mlens = lens.copy()
    pend = pending.copy()
    dr = drafts.copy()
    compared = 0
    for c in range(cycles):
        block = np.concatenate([pend[:, None], dr], 1)
        lg, hid, kv = oracle.verify_forward(shape, W, caches, block, lens_o, EXACT)
        # float32 logits agree to ~1e-6: a 1e-4 top-2 margin is the flag window here
        res = oracle.spec_accept(lg.astype(np.float32), None, dr, None, None, mode="greedy", margin_eps=1e-4)
        if res.flagged.any():
            break
        np.testing.assert_array_equal(gpu_out[c], res.out_tokens)
        compared += 1
        for l, (kk, vv) in enumerate(kv):
            for b in range(B):
                m = res.n_accept[b] + 1
                caches[l][0][b] = np.concatenate([caches[l][0][b], kk[b, :m].astype(np.float32)])
                caches[l][1][b] = np.concatenate([caches[l][1][b], vv[b, :m].astype(np.float32)])
        lens_o = lens_o + res.n_accept + 1
        r = oracle.mtp_draft(shape, Wm, W, mcaches[0][0], mcaches[0][1], mlens, hid, res.n_accept,
                             res.out_tokens, np.zeros((B, k), np.float32), k, "greedy", 1.0, EXACT)
        for b in range(B):
            mcaches[0][0][b] = np.concatenate([mcaches[0][0][b][:mlens[b]], r["ext_k"][b]])
            mcaches[0][1][b] = np.concatenate([mcaches[0][1][b][:mlens[b]], r["ext_v"][b]])
        mlens = r["new_lens"]
        pend = res.out_tokens[np.arange(B), res.n_accept]
        dr = r["drafts"]
        z = np.sort(r["draft_logits"].astype(np.float32), -1)
        if (z[..., -1] - z[..., -2] < 1e-4).any():
            break
    print("[greedy loop] %d of %d cycles compared" % (compared, cycles), flush=True)
    assert compared >= 3
    if compared == cycles:
        np.testing.assert_array_equal(cache.seq_lens.cpu().numpy(), lens_o)
        np.testing.assert_array_equal(mcache.seq_lens.cpu().numpy(), mlens)
