"""GPU parity of gm_mtp_draft against the oracle's draft head: draft logits
within 1e-4 (float32) / 1e-2 of the rounding-contract oracle (bf16), drafts
identical up to the first flagged position, the extend entries written at
the committed slots and the head's length moved to the new boundary."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import need_gpu, rel_err, device_cache, t32, i32, flag_report, row_window, CONTRACT, EXACT
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu


def _inputs(shape, B, k, lo, hi, seed):
    g = np.random.default_rng(seed)
    lens = g.integers(lo, hi, B)
    caches = [synth.kv_prefix(shape, lens, layer=100 + seed)]
    hidden = g.standard_normal((B, k + 1, shape.hidden)).astype(np.float32)
    n = g.integers(0, k + 1, B).astype(np.int32)
    out = g.integers(0, shape.vocab, (B, k + 1)).astype(np.int32)
    for b in range(B):
        out[b, n[b] + 1:] = -1
    u = synth.uniforms(B, k, 4, "mtp", seed)[2]
    return lens, caches, hidden, n, out, u


def _flags(logits, drafts, u, mode, margin=1e-2, final_eps=1e-8):
    """First position of every sequence whose draft a correct float32 evaluation could change."""
    B, k, V = logits.shape
    first = np.full(B, k)
    for b in range(B):
        for j in range(k):
            z = logits[b, j].astype(np.float32)
            if mode == gm.GM_GREEDY:
                s = np.partition(z, V - 2)
                bad = s[-1] - s[-2] < margin
            else:
                _, dist, zz = oracle.inverse_cdf(oracle.softmax(z.astype(np.float64)), u[b, j])
                bad = dist < final_eps * zz
            if bad:
                first[b] = j
                break
    return first


def _run(shape, W, Wm, lens, caches, hidden, n, out, u, k, mode, rnd, tol):
    B = len(lens)
    model = gm.DeviceModel(shape, W)
    mtp = gm.DeviceMtp(shape, Wm)
    cache = device_cache(shape, caches, lens, 2 * k + 2)
    drafts = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    dlog = torch.zeros((B, k, shape.vocab), dtype=torch.float32, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    gm.mtp_draft(model, mtp, cache, k, mode, t32(hidden), i32(n), i32(out), t32(u), drafts, dlog, gm.Workspace(),
                 dev_err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = oracle.mtp_draft(shape, Wm, W, caches[0][0], caches[0][1], lens, hidden, n, out, u, k,
                           "greedy" if mode == gm.GM_GREEDY else "sample", 1.0, rnd)
    got_d, got_l = drafts.cpu().numpy(), dlog.cpu().numpy()
    np.testing.assert_array_equal(cache.seq_lens.cpu().numpy(), ref["new_lens"])
    first = _flags(ref["draft_logits"], ref["drafts"], u, mode)
    flag_report("mtp mode=%d" % mode, first < k, B)
    worst = 0.0
    for b in range(B):
        f = first[b]
        np.testing.assert_array_equal(got_d[b, :f], ref["drafts"][b, :f])
        upto = min(f + 1, k)         # logits up to the first flagged draw are still comparable
        worst = max(worst, rel_err(got_l[b, :upto], ref["draft_logits"][b, :upto]))
        ek, ev = cache.read(0, b, lens[b] + np.arange(n[b] + 1))
        assert rel_err(ek, ref["ext_k"][b]) < tol and rel_err(ev, ref["ext_v"][b]) < tol
    print("[mtp mode=%d] draft logits rel err %.3e" % (mode, worst), flush=True)
    assert worst < tol
    return got_d


@pytest.mark.parametrize("mode", [gm.GM_GREEDY, gm.GM_SAMPLE])
def test_tiny_f32_mtp(mode):
    need_gpu()
    shape = synth.TINY
    W = synth.model_weights(shape)
    Wm = synth.mtp_weights(shape)
    k = 3
    lens, caches, hidden, n, out, u = _inputs(shape, 6, k, 1, 150, 1)
    _run(shape, W, Wm, lens, caches, hidden, n, out, u, k, mode, EXACT, 1e-4)


@pytest.fixture(scope="module")
def qwen_mtp():
    shape = synth.QWEN3_4B_LAYER
    return shape, synth.model_weights(shape), synth.mtp_weights(shape)


@pytest.mark.parametrize("k", [3, 7])
def test_qwen_layer_bf16_mtp_greedy(qwen_mtp, k):
    # bf16 logits sit ~1e-3 from the oracle's: drafts are compared in greedy mode (top-2 margin flags);
    # k = 7 runs the extend with 32-row GQA tiles (the deeper chains of the paper's depth study)
    need_gpu()
    shape, W, Wm = qwen_mtp
    lens, caches, hidden, n, out, u = _inputs(shape, 8, k, 1, 3000, 2)
    _run(shape, W, Wm, lens, caches, hidden, n, out, u, k, gm.GM_GREEDY, CONTRACT, 1e-2)


def test_qwen_layer_bf16_mtp_sample_logits(qwen_mtp):
    # sample mode: the first draft's logits do not depend on any draw; report the draw match rate
    need_gpu()
    shape, W, Wm = qwen_mtp
    k = 3
    lens, caches, hidden, n, out, u = _inputs(shape, 8, k, 1, 3000, 3)
    B = len(lens)
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cache = device_cache(shape, caches, lens, 2 * k + 2)
    drafts = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    dlog = torch.zeros((B, k, shape.vocab), dtype=torch.float32, device="cuda")
    gm.mtp_draft(model, mtp, cache, k, gm.GM_SAMPLE, t32(hidden), i32(n), i32(out), t32(u), drafts, dlog,
                 gm.Workspace())
    torch.cuda.synchronize()
    ref = oracle.mtp_draft(shape, Wm, W, caches[0][0], caches[0][1], lens, hidden, n, out, u, k, "sample", 1.0,
                           CONTRACT)
    got_l = dlog.cpu().numpy()
    e = rel_err(got_l[:, 0], ref["draft_logits"][:, 0])
    got = drafts.cpu().numpy()
    assert ((got >= 0) & (got < shape.vocab)).all()
    # the first draw, against the oracle's from its own logits: with every logit within D of the
    # oracle's, each mass of softmax(z) moves by a factor within e^{+-2D}, so every running sum
    # by at most e^{2D} - 1 of the total; a draw whose u lies farther than that (+ 1e-6 for the
    # float32 terms) from both edges of the oracle's interval must pick the same id.  At bf16's
    # D ~ 1e-2 over ~1.5e5 ids of ~1e-5 mass each the window holds every draw, so the draws are
    # compared with the oracle on the head's own logits in the test below
    compared = 0
    for b in range(B):
        D = float(np.abs(got_l[b, 0].astype(np.float64) - ref["draft_logits"][b, 0]).max())
        _, dist, Z = oracle.inverse_cdf(oracle.softmax(ref["draft_logits"][b, 0]), u[b, 0])
        if dist >= (np.expm1(2 * D) + 1e-6) * Z:
            assert got[b, 0] == ref["drafts"][b, 0], (b, got[b, 0], ref["drafts"][b, 0], D, dist / Z)
            compared += 1
    match = float((got[:, 0] == ref["drafts"][:, 0]).mean())
    print("[mtp bf16 sample] first-draft logits rel err %.3e, first-draft match rate %.2f, %d of %d draws outside "
          "the deviation window (all identical)" % (e, match, compared, B), flush=True)
    assert e < 1e-2


@pytest.mark.parametrize("B,temperature,max_ctx", [(64, 1.0, 3000), (64, 0.7, 3000), (96, 1.0, 600), (300, 0.7, 600)])
def test_qwen_layer_bf16_mtp_sample_draw_from_own_logits(qwen_mtp, B, temperature, max_ctx):
    # Each sampled draft is the inverse-CDF draw from softmax(z / T) of the logits the
    # head itself wrote (Sec. 2.2: drafts are samples of q).  For every row, u * Z must
    # fall in the drawn id's CDF interval [C(x - 1), C(x)) of those logits, widened by the
    # derived float32 window of the kernel's terms (``row_window``, twice: the running sums
    # and u * Z), and a draw outside that window must be the oracle's id.  At 64 rows the LM
    # head's statistics tiles are strip ranges of up to 160 ids; at 96 and 300 rows they are
    # the 128-id tiles of the 128- and 256-row GEMM tiles (300: two M tiles, the second
    # ragged).  A draw that reached only part of a tile lands intervals away and fails within
    # a few rows; the row statistics are checked exactly.
    need_gpu()
    shape, W, Wm = qwen_mtp
    k = 3
    lens, caches, hidden, n, out, u = _inputs(shape, B, k, 1, max_ctx, 6)
    B = len(lens)
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cache = device_cache(shape, caches, lens, 2 * k + 2)
    drafts = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    dlog = torch.zeros((B, k, shape.vocab), dtype=torch.float32, device="cuda")
    stats = gm.new_row_stats(B, k)
    gm.mtp_draft(model, mtp, cache, k, gm.GM_SAMPLE, t32(hidden), i32(n), i32(out), t32(u), drafts, dlog,
                 gm.Workspace(), temperature=temperature, draft_stats=stats)
    torch.cuda.synchronize()
    z = dlog.cpu().numpy()
    got = drafts.cpu().numpy()
    inv_t = float(np.float32(1.0 / temperature))
    # the row statistics handed to the accept: max of z / T, lowest arg-max, and the normaliser
    smax, sarg, ssum = gm.decode_row_stats(stats)
    v = z * np.float32(inv_t)
    np.testing.assert_array_equal(smax, v.max(-1))
    np.testing.assert_array_equal(sarg, v.argmax(-1))
    ref_sum = np.exp(v.astype(np.float64) - v.max(-1, keepdims=True).astype(np.float64)).sum(-1)
    assert np.abs(ssum / ref_sum - 1).max() < 1e-6
    exact, in_tail, outside = 0, 0, 0
    strips = shape.vocab // 16
    first = (np.arange(1025) * strips) // 1024   # first strip of each range when the chip holds 1024 waves
    for b in range(B):
        for j in range(k):
            c = np.cumsum(oracle.softmax(z[b, j].astype(np.float64) * inv_t))
            t, x = float(u[b, j]) * c[-1], int(got[b, j])
            assert 0 <= x < shape.vocab
            lo = c[x - 1] if x > 0 else 0.0
            win = 2.0 * float(row_window(z[b, j], temperature)) * c[-1]
            assert lo - win <= t < c[x] + win, (b, j, x, (t - lo) / c[-1], (c[x] - t) / c[-1])
            ref, dist, zz = oracle.inverse_cdf(oracle.softmax(z[b, j].astype(np.float64) * inv_t), u[b, j])
            exact += int(ref == x)
            if dist >= win:                  # outside the window: the same id as the oracle's draw
                assert x == ref, (b, j, x, ref, dist / zz)
                outside += 1
            r = int(np.searchsorted(first, ref // 16, side="right")) - 1
            in_tail += int(ref - 16 * first[r] >= 128)
    print("[mtp bf16 draw B=%d T=%.1f] %d draws, %d identical to the oracle's (%d outside the window, all "
          "identical), %d past the 128th id of their range" % (B, temperature, B * k, exact, outside, in_tail),
          flush=True)
    assert outside >= B * k * 9 // 10


def test_f32_mtp_large_vocab_sample():
    # sampled drafts over a 151936-id vocabulary: float32 logits agree with the oracle to ~1e-6
    # relative, so a draw is compared outside a 1e-6 window around the CDF edges
    need_gpu()
    import dataclasses
    shape = dataclasses.replace(synth.TINY, vocab=151936)
    W = synth.model_weights(shape)
    Wm = synth.mtp_weights(shape)
    k = 3
    lens, caches, hidden, n, out, u = _inputs(shape, 8, k, 1, 200, 5)
    B = len(lens)
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cache = device_cache(shape, caches, lens, 2 * k + 2)
    drafts = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    dlog = torch.zeros((B, k, shape.vocab), dtype=torch.float32, device="cuda")
    gm.mtp_draft(model, mtp, cache, k, gm.GM_SAMPLE, t32(hidden), i32(n), i32(out), t32(u), drafts, dlog,
                 gm.Workspace())
    torch.cuda.synchronize()
    ref = oracle.mtp_draft(shape, Wm, W, caches[0][0], caches[0][1], lens, hidden, n, out, u, k, "sample", 1.0, EXACT)
    first = _flags(ref["draft_logits"], ref["drafts"], u, gm.GM_SAMPLE, final_eps=1e-6)
    flag_report("mtp f32 V=151936 sample", first < k, B)
    got = drafts.cpu().numpy()
    for b in range(B):
        np.testing.assert_array_equal(got[b, :first[b]], ref["drafts"][b, :first[b]])
    assert rel_err(dlog.cpu().numpy()[:, 0], ref["draft_logits"][:, 0]) < 1e-4


@pytest.mark.parametrize("B,temperature,top_p", [(64, 1.0, 0.7), (96, 0.7, 0.9)])
def test_qwen_layer_bf16_mtp_top_p_draw_from_own_logits(qwen_mtp, B, temperature, top_p):
    # top-p drafting (the evaluation setting): each draft is the inverse-CDF draw from the
    # nucleus of softmax(z / T) of the logits the head wrote.  u * Z' (Z' the nucleus
    # mass) must fall in the drawn id's interval of the nucleus's CDF, widened by 1e-6 Z'
    # for the float32 terms, and the draw equals the oracle's from the same logits unless
    # the nucleus boundary lies within 5e-9 of top_p
    need_gpu()
    shape, W, Wm = qwen_mtp
    k = 3
    lens, caches, hidden, n, out, u = _inputs(shape, B, k, 1, 600, 9)
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cache = device_cache(shape, caches, lens, 2 * k + 2)
    drafts = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    dlog = torch.zeros((B, k, shape.vocab), dtype=torch.float32, device="cuda")
    gm.mtp_draft(model, mtp, cache, k, gm.GM_SAMPLE, t32(hidden), i32(n), i32(out), t32(u), drafts, dlog,
                 gm.Workspace(), temperature=temperature, top_p=top_p)
    torch.cuda.synchronize()
    z = dlog.cpu().numpy()
    got = drafts.cpu().numpy()
    exact, flagged = 0, 0
    for b in range(B):
        for j in range(k):
            pn, dist = oracle.nucleus(z[b, j], oracle.softmax(z[b, j].astype(np.float64) / temperature), top_p)
            if dist < 5e-9:
                flagged += 1
                continue
            x = int(got[b, j])
            assert pn[x] > 0, (b, j, x)
            c = np.cumsum(pn)
            t = float(u[b, j])
            lo = c[x - 1] if x > 0 else 0.0
            assert lo - 1e-6 <= t < c[x] + 1e-6, (b, j, x, t - lo, c[x] - t)
            exact += int(oracle.inverse_cdf(pn, u[b, j])[0] == x)
    print("[mtp bf16 top-p %.1f B=%d T=%.1f] %d draws, %d identical to the oracle's, %d flagged"
          % (top_p, B, temperature, B * k, exact, flagged), flush=True)
    assert exact >= B * k - flagged - 2
