"""GPU parity of the top-p variant of gm_spec_accept (the evaluation setting of
App. "Evaluation Configuration": rejection sampling at T = 1, top-p 0.7) against
the oracle on the same seeded logits.  The drafts are samples of the head's
nucleus.  Accept counts and committed tokens must match bit for bit outside the
flag windows (those of the plain rule, plus a nucleus whose boundary lies within
5e-9 of top_p); the flagged count is printed."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import need_gpu, t32, i32, flag_report
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu
FINAL_EPS = 1e-8
NUC_EPS = 5e-9         # >= V 2^-45, the largest distance of the kernel's fixed-point sums from float64


def _nucleus_drafts(zq, ud, top_p, temperature):
    """d_i ~ nucleus(q_i) by the inverse CDF."""
    B, k, V = zq.shape
    q = oracle.softmax(zq.astype(np.float64) / temperature)
    qn = oracle.nucleus(zq, q, top_p)[0]
    d = np.zeros((B, k), np.int64)
    for i in range(k):
        d[:, i] = oracle.inverse_cdf_rows(qn[:, i], ud[:, i])[0]
    return d


def _run(zt, zq, drafts, ua, uf, mode, temperature, top_p):
    B, k1, V = zt.shape
    n = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, k1), dtype=torch.int32, device="cuda")
    gm.spec_accept(t32(zt), t32(zq) if zq is not None else None, i32(drafts), t32(ua) if ua is not None else None,
                   t32(uf) if uf is not None else None, n, out, mode, gm.Workspace(), temperature=temperature,
                   top_p=top_p)
    torch.cuda.synchronize()
    return n.cpu().numpy(), out.cpu().numpy()


def _logits(shape, kind, *tags):
    z = synth.normal_logits(shape, 3, *tags)
    if kind == "ties":          # values on a 0.5 grid: long runs of equal logits at every boundary
        z = np.round(z * 2.0) / 2.0
    elif kind == "flat":        # nearly every logit equal: the boundary inside a run of ~10^5 ties
        z = np.where(synth.stream(3, "flat", *tags).random(shape) < 1e-3, z * 3.0, 0.0)
    return z.astype(np.float32)


@pytest.mark.parametrize("B,k,V,T,top_p,kind", [
    (64, 3, 151936, 1.0, 0.7, "normal"),       # the evaluation setting at the layer workload's shape
    (32, 7, 151936, 0.7, 0.9, "normal"),
    (257, 2, 1000, 1.0, 0.5, "normal"),        # ragged vocabulary, more sequences than CUs
    (40, 3, 5000, 1.0, 0.7, "ties"),           # the boundary inside a run of equal logits
    (8, 1, 4096, 1.3, 0.2, "ties"),
    (8, 2, 151936, 1.0, 0.5, "flat"),          # too many ties for LDS: the passes over the row
    (3, 0, 5000, 1.0, 0.7, "normal"),          # no drafts: the bonus draw from the target's nucleus
    (16, 2, 1001, 1.0, 0.6, "normal"),         # rows not a multiple of 4 ids: unaligned row reads
    (1, 1, 151936, 1.0, 0.7, "normal"),        # one sequence: the first pass split over 8 workgroups
])
def test_top_p_accept_matches_oracle(B, k, V, T, top_p, kind):
    need_gpu()
    zt = _logits((B, k + 1, V), kind, "tp-t", B, k, V)
    zq = _logits((B, k, V), kind, "tp-q", B, k, V)
    ua, uf, ud = synth.uniforms(B, k, 4, "tp", B, k, V)
    drafts = _nucleus_drafts(zq, ud, top_p, T)
    ref = oracle.spec_accept(zt, zq, drafts, ua, uf, temperature=T, final_eps=FINAL_EPS, top_p=top_p,
                             nucleus_eps=NUC_EPS)
    n, out = _run(zt, zq, drafts, ua, uf, gm.GM_SAMPLE, T, top_p)
    name = "top-p %.2f T=%.1f B=%d k=%d V=%d %s" % (top_p, T, B, k, V, kind)
    flag_report(name, ref.flagged, B)
    ok = ~ref.flagged
    np.testing.assert_array_equal(n[ok], ref.n_accept[ok])
    np.testing.assert_array_equal(out[ok], ref.out_tokens[ok])
    assert ref.flagged.mean() < 0.1
    # every committed final token lies in the nucleus of its target row (all sequences)
    p = oracle.softmax(zt.astype(np.float64) / T)
    for b in range(B):
        row = oracle.nucleus(zt[b, n[b]], p[b, n[b]], top_p)
        if row[1] >= NUC_EPS:
            assert row[0][out[b, n[b]]] > 0, (b, n[b], out[b, n[b]])
    print("[%s] mean accepted %.2f" % (name, n.mean()), flush=True)


def test_top_p_one_is_the_plain_rule():
    need_gpu()
    B, k, V = 32, 3, 151936
    zt = _logits((B, k + 1, V), "normal", "tp1-t")
    zq = _logits((B, k, V), "normal", "tp1-q")
    ua, uf, ud = synth.uniforms(B, k, 4, "tp1")
    drafts = _nucleus_drafts(zq, ud, 1.0, 1.0)
    a = _run(zt, zq, drafts, ua, uf, gm.GM_SAMPLE, 1.0, 1.0)
    b = _run(zt, zq, drafts, ua, uf, gm.GM_SAMPLE, 1.0, 0.999999)   # a nucleus of nearly all ids
    np.testing.assert_array_equal(a[0], b[0])


def test_tiny_top_p_is_greedy():
    # every nucleus is the row's argmax: with drafts = the head's argmax, sampled
    # acceptance at top_p -> 0 takes the greedy rule's decisions and tokens
    need_gpu()
    B, k, V = 48, 3, 151936
    zt = _logits((B, k + 1, V), "normal", "tp0-t")
    zq = _logits((B, k, V), "normal", "tp0-q")
    agree = np.random.default_rng(4).random((B, k)) < 0.6
    zq[agree] = zt[:, :k][agree]
    drafts = zq.argmax(-1)
    ua, uf, _ = synth.uniforms(B, k, 4, "tp0")
    n, out = _run(zt, zq, drafts, ua, uf, gm.GM_SAMPLE, 1.0, 1e-6)
    ng, outg = _run(zt, None, drafts, None, None, gm.GM_GREEDY, 1.0, 1.0)
    np.testing.assert_array_equal(n, ng)
    np.testing.assert_array_equal(out, outg)
    assert 0 < n.mean() < k


def test_top_p_nucleus_handoff():
    # gm_mtp_draft's nuclei handed to gm_spec_accept stand in for the accept's own passes
    # over the draft rows: the same decisions and tokens, bit for bit
    need_gpu()
    from helpers import device_cache
    shape = synth.QWEN3_4B_LAYER
    W, Wm = synth.model_weights(shape), synth.mtp_weights(shape)
    B, k, top_p = 32, 3, 0.7
    g = np.random.default_rng(21)
    lens = g.integers(1, 600, B)
    ks, vs = synth.kv_prefix(shape, lens, layer=500)
    hidden = g.standard_normal((B, k + 1, shape.hidden)).astype(np.float32)
    n0 = g.integers(0, k + 1, B).astype(np.int32)
    out0 = g.integers(0, shape.vocab, (B, k + 1)).astype(np.int32)
    ua, uf, ud = synth.uniforms(B, k, 4, "handoff")
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cache = device_cache(shape, [(ks, vs)], lens, 2 * k + 2)
    drafts = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    dlog = torch.zeros((B, k, shape.vocab), dtype=torch.float32, device="cuda")
    nuc = gm.new_nuclei(B, k)
    gm.mtp_draft(model, mtp, cache, k, gm.GM_SAMPLE, t32(hidden), i32(n0), i32(out0), t32(ud), drafts, dlog,
                 gm.Workspace(), top_p=top_p, draft_nucleus=nuc)
    zt = t32(_logits((B, k + 1, shape.vocab), "normal", "handoff-t"))
    res = []
    for handoff in (None, nuc):
        n = torch.zeros(B, dtype=torch.int32, device="cuda")
        out = torch.zeros((B, k + 1), dtype=torch.int32, device="cuda")
        gm.spec_accept(zt, dlog, drafts, t32(ua), t32(uf), n, out, gm.GM_SAMPLE, gm.Workspace(), top_p=top_p,
                       draft_nucleus=handoff)
        torch.cuda.synchronize()
        res.append((n.cpu().numpy(), out.cpu().numpy()))
    np.testing.assert_array_equal(res[0][0], res[1][0])
    np.testing.assert_array_equal(res[0][1], res[1][1])
    # the handed-over nuclei hold the head's own masses: every draft lies in its nucleus
    h = nuc.cpu().numpy().reshape(B, k, 24)
    key = h[..., 16:20].copy().view(np.uint32)[..., 0]
    last = h[..., 20:24].copy().view(np.int32)[..., 0]
    z = dlog.cpu().numpy()
    d = drafts.cpu().numpy()
    zd = np.take_along_axis(z, d[..., None], -1)[..., 0].astype(np.float32)
    u = zd.view(np.uint32)
    okey = np.where(u & 0x80000000, ~u, u | 0x80000000).astype(np.uint32)
    assert ((okey > key) | ((okey == key) & (d <= last))).all()
    print("[top-p handoff] mean accepted %.2f" % res[0][0].mean(), flush=True)
