"""GPU parity of the top-p variant of gm_spec_accept (the evaluation setting of
App. "Evaluation Configuration": rejection sampling at T = 1, top-p 0.7) against
the oracle on the same seeded logits.  The drafts are samples of the head's
nucleus (and, in the handoff test, the oracle's own draft head's draws).  Accept
counts and committed tokens must match bit for bit outside the flag windows (|u - min(1, p/q)| < 1e-3, a final draw within the derived float32
bound ``draw_window`` of a CDF edge, and a nucleus whose boundary lies within
5e-9 of top_p); the flagged count is printed."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import need_gpu, t32, i32, flag_report, draw_window
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu
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
    # a head close to the target (zq = zt + 0.1 N(0, 1)): most drafts accepted, so the deep
    # prefixes and the bonus draw from the last target row's nucleus are compared
    (64, 3, 151936, 1.0, 0.7, "overlap"),
    (32, 7, 151936, 1.0, 0.7, "overlap"),
])
def test_top_p_accept_matches_oracle(B, k, V, T, top_p, kind):
    need_gpu()
    zt = _logits((B, k + 1, V), kind, "tp-t", B, k, V)
    if kind == "overlap":
        zq = (zt[:, :k] + np.float32(0.1) * synth.normal_logits((B, k, V), 3, "tp-q", B, k, V)).astype(np.float32)
    else:
        zq = _logits((B, k, V), kind, "tp-q", B, k, V)
    ua, uf, ud = synth.uniforms(B, k, 4, "tp", B, k, V)
    drafts = _nucleus_drafts(zq, ud, top_p, T)
    ref = oracle.spec_accept(zt, zq, drafts, ua, uf, temperature=T, top_p=top_p, nucleus_eps=NUC_EPS,
                             final_abs=draw_window(zt, zq, T, top_p))
    n, out = _run(zt, zq, drafts, ua, uf, gm.GM_SAMPLE, T, top_p)
    name = "top-p %.2f T=%.1f B=%d k=%d V=%d %s" % (top_p, T, B, k, V, kind)
    flag_report(name, ref.flagged, B)
    ok, oka = ~ref.flagged, ~ref.flag_accept     # a flagged final draw leaves the accept count comparable
    np.testing.assert_array_equal(n[oka], ref.n_accept[oka])
    np.testing.assert_array_equal(out[ok], ref.out_tokens[ok])
    assert ref.flagged.sum() <= max(1, 0.1 * B)
    if kind == "overlap":       # deep prefixes and bonus draws are among the compared sequences
        assert n[ok].mean() > k / 2 and (n[ok] == k).sum() >= 4, (n.mean(), (n == k).sum())
    # every committed final token lies in the nucleus of its target row (all sequences)
    p = oracle.softmax(zt.astype(np.float64) / T)
    for b in range(B):
        row = oracle.nucleus(zt[b, n[b]], p[b, n[b]], top_p)
        if row[1] >= NUC_EPS:
            assert row[0][out[b, n[b]]] > 0, (b, n[b], out[b, n[b]])
    print("[%s] mean accepted %.2f, all k accepted in %d" % (name, n.mean(), (n == k).sum()), flush=True)


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



def _chain_flags(zt, zq, d_ref, n_ref, dev, ua, uf, ud, top_p, window):
    """Per sequence, how far the oracle's draft-and-accept chain (at T = 1) stays comparable when
    the GPU's draft logits sit within dev[b, j] (max over the row) of the oracle's.  Walks the examined
    events in order -- draw j, accept test j, then the final draw -- and stops at the first one
    that such a deviation D could move:
      * the draw of d_j from the nucleus of q_j: the nucleus changes if the logit just below its
        boundary lies within 2 D of the boundary's, or its running masses lie within e^{2D} - 1
        (+ 5e-9) of top_p; the inverse-CDF draw moves if u lies within e^{4D} - 1 (+ 1e-6) of an
        edge (each nucleus mass moves by a factor within e^{+-4D});
      * accept test j: |u - min(1, p'/q')| < max(1e-3, 5 D), or p's nucleus within 5e-9 of top_p;
      * the final draw: within window[b] + 8 D / top_p of an edge (residual) or window[b] (bonus).
    Returns per sequence: drawn (leading drafts that must be the oracle's), upto (leading accept
    decisions that must agree), known (the accept count must agree) and whole (every committed
    token must agree)."""
    B, k1, V = zt.shape
    k = k1 - 1
    drawn = np.zeros(B, np.int64)
    upto = np.zeros(B, np.int64)
    known = np.zeros(B, bool)
    whole = np.zeros(B, bool)
    for b in range(B):
        n = int(n_ref[b])
        stopped = False
        for j in range(min(n + 1, k)):
            D = float(dev[b, j])
            qn, dist_n = oracle.nucleus(zq[b, j], oracle.softmax(zq[b, j].astype(np.float64)), top_p)
            zs = np.sort(zq[b, j].astype(np.float32))[::-1]
            m = int((qn > 0).sum())
            gap = zs[m - 1] - zs[m] if m < V else np.inf
            dist_d = oracle.inverse_cdf(qn, ud[b, j])[1]
            if gap < 2 * D or dist_n < np.expm1(2 * D) + 5e-9 or dist_d < np.expm1(4 * D) + 1e-6:
                stopped = True
                break
            drawn[b] = j + 1
            pn, dist_p = oracle.nucleus(zt[b, j], oracle.softmax(zt[b, j].astype(np.float64)), top_p)
            r = min(1.0, pn[d_ref[b, j]] / qn[d_ref[b, j]])
            if dist_p < 5e-9 or abs(float(ua[b, j]) - r) < max(1e-3, 5 * D):
                stopped = True
                break
            upto[b] = min(j + 1, n)
        if stopped:
            continue
        known[b] = True
        pn, dist_p = oracle.nucleus(zt[b, n], oracle.softmax(zt[b, n].astype(np.float64)), top_p)
        if dist_p < 5e-9:
            continue
        if n < k:
            qn = oracle.nucleus(zq[b, n], oracle.softmax(zq[b, n].astype(np.float64)), top_p)[0]
            w = np.maximum(pn - qn, 0.0)
            if not w.sum() > 0:
                w = pn
            lim = window[b] + 8 * float(dev[b, n]) / top_p
        else:
            w, lim = pn, window[b]
        whole[b] = oracle.inverse_cdf(w, uf[b])[1] >= lim
    return drawn, upto, known, whole


def test_top_p_nucleus_handoff_matches_oracle():
    # The whole top-p step with the handoff -- gm_mtp_draft's nuclei, draws and logits taken by
    # gm_spec_accept in place of its own passes over the draft rows -- against the oracle's draft
    # head and accept on the same seeded inputs.  A float32 head over a 151936-id vocabulary
    # whose final norm is scaled by 16 (logits ~ N(0, 5^2): nuclei of tens of ids, so a 1e-5
    # deviation moves few draws) and a target within 0.1 N(0, 1) of the oracle's draft logits
    # (most drafts accepted).  Decisions are compared up to each sequence's first event that the
    # measured logit deviation could move (``_chain_flags``).
    need_gpu()
    import dataclasses
    from helpers import device_cache, EXACT
    shape = dataclasses.replace(synth.TINY, vocab=151936)
    W = synth.model_weights(shape)
    Wm = dict(synth.mtp_weights(shape))
    Wm["final_norm"] = (Wm["final_norm"] * np.float32(16.0)).astype(np.float32)
    B, k, top_p = 32, 3, 0.7
    g = np.random.default_rng(31)
    lens = g.integers(1, 200, B)
    caches = [synth.kv_prefix(shape, lens, layer=131)]
    hidden = g.standard_normal((B, k + 1, shape.hidden)).astype(np.float32)
    n0 = g.integers(0, k + 1, B).astype(np.int32)
    out0 = g.integers(0, shape.vocab, (B, k + 1)).astype(np.int32)
    for b in range(B):
        out0[b, n0[b] + 1:] = -1
    ua, uf, ud = synth.uniforms(B, k, 4, "handoff-f32")
    ref_d = oracle.mtp_draft(shape, Wm, W, caches[0][0], caches[0][1], lens, hidden, n0, out0, ud, k, "sample", 1.0,
                             EXACT, top_p=top_p)
    zq = ref_d["draft_logits"].astype(np.float32)
    noise = synth.normal_logits((B, k + 1, shape.vocab), 31, "handoff-f32-t")
    zt = np.concatenate([zq, np.zeros((B, 1, shape.vocab), np.float32)], 1) + np.float32(0.1) * noise
    zt[:, k] = np.float32(5.0) * noise[:, k]
    zt = zt.astype(np.float32)
    ref = oracle.spec_accept(zt, zq, ref_d["drafts"], ua, uf, top_p=top_p, nucleus_eps=NUC_EPS)

    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cache = device_cache(shape, caches, lens, 2 * k + 2)
    drafts = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    dlog = torch.zeros((B, k, shape.vocab), dtype=torch.float32, device="cuda")
    nuc = gm.new_nuclei(B, k)
    gm.mtp_draft(model, mtp, cache, k, gm.GM_SAMPLE, t32(hidden), i32(n0), i32(out0), t32(ud), drafts, dlog,
                 gm.Workspace(), top_p=top_p, draft_nucleus=nuc)
    n = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, k + 1), dtype=torch.int32, device="cuda")
    gm.spec_accept(t32(zt), dlog, drafts, t32(ua), t32(uf), n, out, gm.GM_SAMPLE, gm.Workspace(), top_p=top_p,
                   draft_nucleus=nuc)
    torch.cuda.synchronize()
    n, out = n.cpu().numpy(), out.cpu().numpy()
    got_d, got_l = drafts.cpu().numpy(), dlog.cpu().numpy()

    dev = np.abs(got_l.astype(np.float64) - zq).max(-1)          # [B, k]
    drawn, upto, known, whole = _chain_flags(zt, zq, ref_d["drafts"], ref.n_accept, dev, ua, uf, ud, top_p,
                                             draw_window(zt, zq, 1.0, top_p))
    for b in range(B):
        np.testing.assert_array_equal(got_d[b, :drawn[b]], ref_d["drafts"][b, :drawn[b]])
        assert n[b] >= upto[b], (b, n[b], upto[b])
        np.testing.assert_array_equal(out[b, :upto[b]], ref.out_tokens[b, :upto[b]])
        if known[b]:
            assert n[b] == ref.n_accept[b], (b, n[b], ref.n_accept[b])
        if whole[b]:
            np.testing.assert_array_equal(out[b, :n[b] + 1], ref.out_tokens[b, :n[b] + 1])
    examined = np.minimum(ref.n_accept + 1, k)
    print("[top-p handoff vs oracle] logit deviation max %.2e; drafts compared %d, accept decisions compared "
          "%d of %d examined (counts known %d), whole sequences %d of %d; mean accepted %.2f (oracle %.2f)"
          % (dev.max(), drawn.sum(), upto.sum() + (known & (ref.n_accept < k)).sum(), examined.sum(), known.sum(),
             whole.sum(), B, n.mean(), ref.n_accept.mean()), flush=True)
    assert known.sum() >= B // 2 and whole.sum() >= B // 4 and upto.sum() >= B
