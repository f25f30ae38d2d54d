"""The whole speculative step captured in a HIP graph and replayed.

The four entry points enqueue kernels only (no allocation, memset, copy or host
synchronisation inside a call), so a caller can capture verify -> accept ->
commit -> draft once and replay it.  The graph is replayed several times, with
the caches' lengths restored and the outputs cleared by eager work between the
replays and an eager step run in between; every replay and every eager step
must reproduce the first eager step bit for bit (the kernels are
deterministic: fixed reduction orders, integer atomics only).  The
no-allocation accept, meant for such callers, is captured and replayed the
same way."""
import numpy as np
import pytest
import torch

import synth
from helpers import need_gpu, device_cache, synth_caches, t32, i32
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("top_p", [1.0, 0.7])
def test_step_graph_replays_match_eager(top_p):
    need_gpu()
    shape = synth.ModelShape(1, 256, 2, 2, 128, 512, 16384, dtype="bf16")
    W = synth.model_weights(shape)
    Wm = synth.mtp_weights(shape)
    B, k = 16, 3
    lens = 96 + 16 * np.arange(B)
    caches = synth_caches(shape, lens, shape.n_layers)
    mk, mv = synth.kv_prefix(shape, lens, layer=77)
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cache = device_cache(shape, caches, lens, 2 * k + 2)
    mcache = device_cache(shape, [(list(mk), list(mv))], lens, 2 * k + 2)
    tokens = i32(synth.token_ids(B * (k + 1), shape.vocab, 1, "graph").reshape(B, k + 1))
    drafts = tokens[:, 1:].contiguous()
    zq = t32(synth.normal_logits((B, k, shape.vocab), 3, "graph", "zq"))
    ua, uf, ud = (t32(a) for a in synth.uniforms(B, k, 5, "graph"))
    lens0, mlens0 = cache.seq_lens.clone(), mcache.seq_lens.clone()

    logits = torch.empty((B, k + 1, shape.vocab), dtype=torch.float32, device="cuda")
    hidden = torch.empty((B, k + 1, shape.hidden), dtype=torch.float32, device="cuda")
    n = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, k + 1), dtype=torch.int32, device="cuda")
    nxt = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    dlog = torch.zeros((B, k, shape.vocab), dtype=torch.float32, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws, ws2 = gm.Workspace(), gm.Workspace()
    outputs = (logits, hidden, n, out, nxt, dlog, cache.seq_lens, mcache.seq_lens)

    def reset():   # eager work outside the graph: lengths restored, outputs cleared
        cache.seq_lens.copy_(lens0)
        mcache.seq_lens.copy_(mlens0)
        for t in (logits, hidden, dlog):
            t.fill_(float("nan"))
        for t in (n, out, nxt):
            t.fill_(-7)

    def step():    # library calls only
        gm.verify_forward(model, cache, tokens, logits, hidden, ws, err)
        gm.spec_accept(logits, zq, drafts, ua, uf, n, out, gm.GM_SAMPLE, ws, top_p=top_p)
        gm.kv_commit(cache, k, n)
        gm.mtp_draft(model, mtp, mcache, k, gm.GM_SAMPLE, hidden, n, out, ud, nxt, dlog, ws2, dev_err=err,
                     top_p=top_p)

    reset()
    step()
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = [t.clone() for t in outputs]
    assert bool(torch.isfinite(ref[0]).all()) and bool(torch.isfinite(ref[5]).all())

    def check(what):
        torch.cuda.synchronize()
        for name, got, want in zip(("logits", "hidden", "n_accept", "out_tokens", "drafts", "draft_logits",
                                    "seq_lens", "head seq_lens"), outputs, ref):
            assert torch.equal(got, want), "%s: %s differs from the first eager step" % (what, name)

    # warm-up on a side stream (torch's capture recipe), then the capture itself
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        reset()
        step()
    torch.cuda.current_stream().wait_stream(side)
    check("side-stream warm-up")
    reset()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(3):
        reset()
        g.replay()
        check("replay %d" % r)
        reset()
        step()
        check("eager step after replay %d" % r)
    assert int(err.item()) == 0
    print("[graph top_p=%.1f] 3 replays and 3 eager steps identical to the first eager step (n_accept %s)"
          % (top_p, ref[2].cpu().numpy().tolist()), flush=True)


@pytest.mark.parametrize("top_p", [1.0, 0.7])
def test_noalloc_accept_graph_replays_match_eager(top_p):
    # the no-allocation accept is meant for callers under graph capture: captured once, its
    # replays (with the workspace accept run eagerly between them, on its own scratch) give
    # the eager call's decisions and tokens bit for bit
    need_gpu()
    import oracle
    B, k, V = 32, 3, 32768
    zt = t32(synth.normal_logits((B, k + 1, V), 3, "graph-noalloc-t"))
    zq_np = synth.normal_logits((B, k, V), 3, "graph-noalloc-q")
    ua, uf, ud = synth.uniforms(B, k, 4, "graph-noalloc")
    q = oracle.softmax(zq_np.astype(np.float64))
    drafts = i32(np.stack([oracle.inverse_cdf_rows(q[:, i], ud[:, i])[0] for i in range(k)], 1))
    zq, ua, uf = t32(zq_np), t32(ua), t32(uf)
    n = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, k + 1), dtype=torch.int32, device="cuda")
    n2, out2 = torch.zeros_like(n), torch.zeros_like(out)
    ws = gm.Workspace()

    def reset():
        for t in (n, out, n2, out2):
            t.fill_(-7)

    def call():
        gm.spec_accept_noalloc(zt, zq, drafts, ua, uf, n, out, gm.GM_SAMPLE, top_p=top_p)

    reset()
    call()
    torch.cuda.synchronize()
    ref_n, ref_out = n.clone(), out.clone()
    assert int((ref_n >= 0).sum()) == B

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    for r in range(3):
        reset()
        g.replay()
        gm.spec_accept(zt, zq, drafts, ua, uf, n2, out2, gm.GM_SAMPLE, ws, top_p=top_p)   # eager, between replays
        torch.cuda.synchronize()
        assert torch.equal(n, ref_n) and torch.equal(out, ref_out), "replay %d differs from the eager call" % r
        assert torch.equal(n2, ref_n) and torch.equal(out2, ref_out), "workspace accept after replay %d differs" % r
    print("[graph no-alloc accept top_p=%.1f] 3 replays identical to the eager call (mean accepted %.2f)"
          % (top_p, float(ref_n.float().mean())), flush=True)
