"""GPU parity of gm_mtp_reconstruct (the draft-path reconstruction of App.
"Draft-Path Reconstruction" and "Parallelizing GrowMTP Training") against the
oracle: head logits within 1e-4 (float32) / 1e-2 of the rounding-contract
oracle (bf16), and the chain's cache entries; and, on the GPU alone, that
reconstructing the cycles gm_mtp_draft just drafted, from the recorded start
with the recorded drafts, reproduces the drafting's logits and drafts."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import need_gpu, rel_err, device_cache, t32, i32, CONTRACT, EXACT
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu


def _cycles(shape, R, K, lo, hi, seed):
    g = np.random.default_rng(seed)
    starts = g.integers(lo, hi, R)
    ks, vs = synth.kv_prefix(shape, starts, layer=300 + seed)
    h0 = g.standard_normal((R, shape.hidden)).astype(np.float32)
    t0 = g.integers(0, shape.vocab, R).astype(np.int32)
    drafts = g.integers(0, shape.vocab, (R, K)).astype(np.int32)
    return starts, ks, vs, h0, t0, drafts


def _run(shape, W, Wm, starts, ks, vs, h0, t0, drafts, K):
    R = len(starts)
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cache = device_cache(shape, [(ks, vs)], starts, K + 1)
    out = torch.zeros((R, K, shape.vocab), dtype=torch.float32, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    gm.mtp_reconstruct(model, mtp, cache, K, t32(h0), i32(t0), i32(drafts) if K > 1 else None, out, gm.Workspace(),
                       dev_err=err)   # depth 1 alone reads no draft
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    np.testing.assert_array_equal(cache.seq_lens.cpu().numpy(), starts)      # lengths untouched
    return cache, out.cpu().numpy()


@pytest.mark.parametrize("shape_name,R,K,hi,tol", [("tiny", 7, 4, 150, 1e-4), ("qwen", 12, 3, 2000, 1e-2),
                                                    ("qwen", 5, 7, 700, 1e-2), ("tiny", 1, 1, 40, 1e-4)])
def test_reconstruct_matches_oracle(shape_name, R, K, hi, tol):
    need_gpu()
    shape = synth.TINY if shape_name == "tiny" else synth.QWEN3_4B_LAYER
    rnd = EXACT if shape.dtype == "f32" else CONTRACT
    W, Wm = synth.model_weights(shape), synth.mtp_weights(shape)
    starts, ks, vs, h0, t0, drafts = _cycles(shape, R, K, 1, hi, 11)
    cache, got = _run(shape, W, Wm, starts, ks, vs, h0, t0, drafts, K)
    ref = oracle.mtp_reconstruct(shape, Wm, W, ks, vs, starts, h0, t0, drafts, K, rnd)
    e = rel_err(got, ref["logits"])
    print("[reconstruct %s R=%d K=%d] head logits rel err %.3e" % (shape_name, R, K, e), flush=True)
    assert e < tol
    for r in range(R):
        ck, cv = cache.read(0, r, starts[r] + np.arange(K))
        assert rel_err(ck, ref["chain_k"][r]) < tol and rel_err(cv, ref["chain_v"][r]) < tol


def test_reconstruct_reproduces_gpu_drafting():
    # draft a block with gm_mtp_draft (greedy), then rebuild the same cycles from their
    # record: start slot m_b + n_b (the entries before the boundary row), the boundary
    # hidden and the cycle's final token, the drafts fed back.  The two launches tile their
    # GEMMs differently (the extend runs B (k + 1) rows, the reconstruction B), so float32
    # accumulation orders differ and flip some bf16 roundings of the activations: the
    # logits agree within the bf16 parity bound (1e-2), the drafts exactly where the
    # top-2 margin is clear
    need_gpu()
    shape = synth.QWEN3_4B_LAYER
    W, Wm = synth.model_weights(shape), synth.mtp_weights(shape)
    B, k = 16, 3
    g = np.random.default_rng(12)
    lens = g.integers(1, 2500, B)
    ks, vs = synth.kv_prefix(shape, lens, layer=400)
    hidden = g.standard_normal((B, k + 1, shape.hidden)).astype(np.float32)
    n = g.integers(0, k + 1, B).astype(np.int32)
    out = g.integers(0, shape.vocab, (B, k + 1)).astype(np.int32)
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cache = device_cache(shape, [(ks, vs)], lens, 2 * k + 2)
    drafts = torch.zeros((B, k), dtype=torch.int32, device="cuda")
    dlog = torch.zeros((B, k, shape.vocab), dtype=torch.float32, device="cuda")
    gm.mtp_draft(model, mtp, cache, k, gm.GM_GREEDY, t32(hidden), i32(n), i32(out), None, drafts, dlog,
                 gm.Workspace())
    torch.cuda.synchronize()
    cache.seq_lens.copy_(i32(lens + n))                  # the cycle's start: entries before the boundary row
    rec = torch.zeros_like(dlog)
    gm.mtp_reconstruct(model, mtp, cache, k, t32(hidden[np.arange(B), n]), i32(out[np.arange(B), n]), drafts, rec,
                       gm.Workspace())
    torch.cuda.synchronize()
    a, b = rec.cpu().numpy(), dlog.cpu().numpy()
    e = rel_err(a, b)
    top = np.sort(b, -1)
    clear = (top[..., -1] - top[..., -2]) > 1e-2
    same = (a.argmax(-1) == drafts.cpu().numpy())[clear].mean()
    print("[reconstruct vs drafting] rel err %.3e, argmax = draft on %.3f of %d clear rows"
          % (e, same, int(clear.sum())), flush=True)
    assert e < 1e-2
    assert same == 1.0


def test_reconstruct_full_size_sampled():
    # the bench's launch configuration: 1024 cycles (the paper's chunk) at the Qwen3-4B
    # shape, K = 3, starts from the layer workload's contexts U[1024, 4096]; the head
    # cache is filled on the device, and four sampled cycles (first, last, two inside)
    # are checked against the oracle from the entries read back
    need_gpu()
    shape = synth.QWEN3_4B_LAYER
    W, Wm = synth.model_weights(shape), synth.mtp_weights(shape)
    R, K = 1024, 3
    g = np.random.default_rng(13)
    starts = g.integers(1024, 4097, R)
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    cache = gm.PagedCache(shape, 1, starts, starts + K + 1, fill="empty")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(13)
    for t in cache.k + cache.v:
        t.normal_(generator=gen)
    h0 = g.standard_normal((R, shape.hidden)).astype(np.float32)
    t0 = g.integers(0, shape.vocab, R).astype(np.int32)
    drafts = g.integers(0, shape.vocab, (R, K)).astype(np.int32)
    out = torch.zeros((R, K, shape.vocab), dtype=torch.float32, device="cuda")
    gm.mtp_reconstruct(model, mtp, cache, K, t32(h0), i32(t0), i32(drafts), out, gm.Workspace())
    torch.cuda.synchronize()
    worst = 0.0
    for r in (0, 377, 800, R - 1):
        ks, vs = cache.read(0, r, np.arange(starts[r]))
        ref = oracle.mtp_reconstruct(shape, Wm, W, [ks], [vs], starts[r:r + 1], h0[r:r + 1], t0[r:r + 1],
                                     drafts[r:r + 1], K, CONTRACT)
        worst = max(worst, rel_err(out[r].cpu().numpy(), ref["logits"][0]))
    print("[reconstruct R=1024 K=3] sampled cycles' head logits rel err %.3e" % worst, flush=True)
    assert worst < 1e-2


@pytest.mark.parametrize("shape_name,K,P,tol", [("tiny", 4, 300, 1e-4), ("qwen", 3, 1500, 1e-2)])
def test_reconstruct_over_shared_prefix_pages(shape_name, K, P, tol):
    # All cycles of one response attend over one shared cache (App. "Parallelizing GrowMTP
    # Training"): the pages that hold only committed prefix entries are the same physical
    # pages in every cycle's table; the page holding cycle r's start s_r and those after it
    # are the cycle's own (the start page begins with a copy of the prefix entries before
    # s_r).  Starts include page boundaries and a repeated start.  The head logits and the
    # chain entries match the oracle over the prefix truncated at each start, and the
    # shared pages still hold the prefix afterwards.
    need_gpu()
    shape = synth.TINY if shape_name == "tiny" else synth.QWEN3_4B_LAYER
    rnd = EXACT if shape.dtype == "f32" else CONTRACT
    W, Wm = synth.model_weights(shape), synth.mtp_weights(shape)
    ps = 16
    g = np.random.default_rng(17)
    starts = np.sort(np.concatenate([g.integers(1, P, 6), [ps, 4 * ps, P, P // 2, P // 2]])).astype(np.int64)
    R = len(starts)
    pk, pv = synth.kv_prefix(shape, [P], layer=333)
    ks, vs = [pk[0][:s] for s in starts], [pv[0][:s] for s in starts]
    h0 = g.standard_normal((R, shape.hidden)).astype(np.float32)
    t0 = g.integers(0, shape.vocab, R).astype(np.int32)
    drafts = g.integers(0, shape.vocab, (R, K)).astype(np.int32)
    # page table: shared pages 0 .. ceil(P / ps) - 1 hold the prefix; cycle r takes the first
    # s_r // ps of them and private pages from s_r's page on
    n_shared = -(-P // ps)
    max_pages = -(-(P + K) // ps)
    table = np.full((R, max_pages), -1, dtype=np.int32)
    nxt = n_shared
    for r, s in enumerate(starts):
        full = s // ps
        table[r, :full] = np.arange(full)
        own = -(-(s + K) // ps) - full
        table[r, full:full + own] = np.arange(nxt, nxt + own)
        nxt += own
    cache = gm.PagedCache(shape, 1, starts, starts + K, page_size=ps, table=table)
    for r, s in enumerate(starts):     # shared pages are written once per cycle, with the same entries
        cache.write(0, r, np.arange(s), ks[r], vs[r])
    model, mtp = gm.DeviceModel(shape, W), gm.DeviceMtp(shape, Wm)
    out = torch.zeros((R, K, shape.vocab), dtype=torch.float32, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    gm.mtp_reconstruct(model, mtp, cache, K, t32(h0), i32(t0), i32(drafts), out, gm.Workspace(), dev_err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = oracle.mtp_reconstruct(shape, Wm, W, ks, vs, starts, h0, t0, drafts, K, rnd)
    e = rel_err(out.cpu().numpy(), ref["logits"])
    print("[reconstruct shared prefix %s R=%d K=%d P=%d] head logits rel err %.3e" % (shape_name, R, K, P, e),
          flush=True)
    assert e < tol
    for r in range(R):
        ck, cv = cache.read(0, r, starts[r] + np.arange(K))
        assert rel_err(ck, ref["chain_k"][r]) < tol and rel_err(cv, ref["chain_v"][r]) < tol
    # the longest cycle's table reads the whole shared prefix back unchanged
    r = int(np.argmax(starts))
    k_back, v_back = cache.read(0, r, np.arange(starts[r]))
    q = (lambda a: a) if shape.dtype == "f32" else (lambda a: oracle.round_bf16(a))
    np.testing.assert_array_equal(k_back, q(np.asarray(pk[0][:starts[r]], np.float32)))
    np.testing.assert_array_equal(v_back, q(np.asarray(pv[0][:starts[r]], np.float32)))
