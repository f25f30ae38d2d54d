#!/usr/bin/env python3
"""Benchmark of the batched speculative-decoding step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--mode sample|greedy]

One step is the whole hot path over one batch: gm_verify_forward (target
forward over the k+1 block positions), gm_spec_accept, gm_kv_commit and
gm_mtp_draft (the draft of the next block).  Inputs are seeded synthetic
tensors with the shapes of the workload (weights N(0, 0.02), KV N(0, 1));
they are resident in HBM before the timed region.  Each step restarts from
the same committed lengths, so every timed step does identical work.

Prints one JSON line: throughput (committed tokens/s), the roofline of the
dominant kernel measured with HIP events inside the timed region, the
per-kernel breakdown, and the CPU oracle timed on a bounded sample of the
same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402

HBM_GBS = 8000.0            # MI355X HBM3E peak, GB/s
BF16_TFLOPS = 2500.0        # MI355X dense bf16 matrix peak, TFLOP/s
METRIC = "accepted tokens/s per verify step; verify-attn HBM GB/s & GEMM MFMA % of peak"

DESCRIPTIONS = {
    "tiny": "random-init float32 decoder: 2 layers, hidden 256, 4 heads x 64, FFN 1024, vocab 1024; B=4, 128-token "
            "contexts, k=3 uniform drafts; T=1",
    "qwen3_4b_layer": "one Qwen3-4B-shaped layer (H 2560, 32/8 heads x 128, FFN 9728) + LM head (V 151936) "
                      "+ 1-layer MTP head of the same shape; B=64, contexts U[1024,4096], k=3, drafts = target "
                      "top-1 w.p. 0.7 else uniform; T=1",
    "qwen3_4b_full": "36-layer Qwen3-4B shape + 1-layer MTP head; B=256, contexts 512+U[0,8192], k=3; T=1",
    "qwen3_4b_layer_k7": "the qwen3_4b_layer workload at k=7 (the deepest chain of the depth study): B=64, "
                         "contexts U[1024,4096], drafts = target top-1 w.p. 0.7 else uniform; T=1",
    "mimo_7b": "36-layer MiMo-7B shape (H 4096, 32/8 heads x 128, FFN 11008, V 151680) + 1-layer MTP head; B=128, "
               "contexts U[2048,16384], k=1, drafts = target top-1 w.p. 0.5 else uniform; T=1",
    "long_ctx": "Qwen3-4B-shaped verify attention + accept only; B=32, contexts U[16384,32768], k=7, "
                "drafts sampled from q = softmax(N(0,1)); T=1",
}


# workloads whose two input sets fit in HBM side by side (the rest run one set: a step of theirs
# touches far more than the 256 MB Infinity Cache anyway)
ROTATED = ("tiny", "qwen3_4b_layer", "qwen3_4b_layer_k7", "long_ctx")
# the other configurations, measured after the headline workload in the same run
EXTRA = ("tiny", "long_ctx", "qwen3_4b_full", "mimo_7b")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# ----------------------------------------------------------------------------- accounting
def accounting(wl, lens, top_p=1.0, record=0, target_stats=False):
    """Algorithmic flops and HBM bytes per step, per kernel name."""
    s, B, k = wl.shape, wl.batch, wl.k
    R, M = k + 1, wl.batch * (k + 1)
    H, F, V, d = s.hidden, s.ffn, s.vocab, s.head_dim
    nq, nkv, L = s.n_heads, s.n_kv_heads, s.n_layers
    qw, qd = (nq + 2 * nkv) * d, nq * d
    ctx = lens.astype(np.float64) + R
    kv_bytes = float((ctx * nkv * d * 2 * 2).sum())            # K and V, bf16
    attn_flops = float((4.0 * R * nq * ctx * d).sum())

    def gemm(m, n, kk, out_bytes, add=False):
        return 2.0 * m * n * kk, 2.0 * n * kk + 2.0 * m * kk + m * n * out_bytes * (2 if add else 1)

    acc = {}

    def put(name, fb, launches):
        f, b = fb
        acc[name] = dict(flops=f * launches, bytes=b * launches, launches=launches)

    if wl.name != "long_ctx":
        put("gemm_qkv", gemm(M, qw, H, 4), L)
        put("gemm_o", gemm(M, H, qd, 4, add=True), L)
        put("gemm_gate_up", (2.0 * M * 2 * F * H, 2.0 * 2 * F * H + 2.0 * M * H + 2.0 * M * F), L)
        put("gemm_down", gemm(M, H, F, 4, add=True), L)
        put("gemm_lm_head", gemm(M, V, H, 4), 1)
    put("attn_verify", (attn_flops, kv_bytes + 2.0 * 2 * M * qd), L)
    # rows the accept's statistics pass reads: the target rows' statistics come from the verify
    # forward's LM-head epilogue (unless a cycle record needs the pass's run maxima); the draft
    # rows' from the draft head when it runs in the step (not under top-p, whose draws produce none)
    handoff = wl.with_mtp and top_p >= 1.0
    rows = (0 if (target_stats and wl.name != "long_ctx" and not record) else k + 1) + (0 if handoff else k)
    if rows:
        put("accept_row_stats", (0.0, 4.0 * B * rows * V), 1)
    if top_p < 1.0:   # three passes over every target and draft row (the selection's bins)
        put("accept_nucleus", (0.0, 3 * 4.0 * B * (2 * k + 1) * V), 1)
    if wl.with_mtp:
        mkv = float((lens.astype(np.float64) * nkv * d * 2 * 2).sum())
        put("mtp_gemm_lm_head", gemm(B, V, H, 4), k)
        put("mtp_gemm_proj", ((2.0 * (M + (k - 1) * B) * H * 2 * H) / k, 2.0 * H * 2 * H), k)
        put("mtp_gemm_qkv", ((2.0 * (M + (k - 1) * B) * qw * H) / k, 2.0 * qw * H), k)
        put("mtp_gemm_o", gemm(B, H, qd, 4, add=True), k)
        put("mtp_gemm_gate_up", (2.0 * B * 2 * F * H, 2.0 * 2 * F * H + 2.0 * B * H + 2.0 * B * F), k)
        put("mtp_gemm_down", gemm(B, H, F, 4, add=True), k)
        put("attn_mtp", (4.0 * nq * float(lens.sum()) * d * k, mkv), k)
        put("draft_row_stats", (0.0, 4.0 * B * V), k)
        if top_p < 1.0:
            put("draft_nucleus", (0.0, 3 * 4.0 * B * V), k)
    return acc


# ----------------------------------------------------------------------------- workloads
class StepEvents:
    """HIP timing events on torch's current stream that record without the system-scope fence
    of a default event (hipEventDisableSystemFence).  Only their timestamps are read; the
    fence's cache write-back would leave the stream idle for several microseconds at every
    record, inside the timed region."""
    _FLAG = 0x20000000

    def __init__(self, n):
        import ctypes
        import torch
        self._c, self._torch = ctypes, torch
        hip = ctypes.CDLL("libamdhip64.so.7")   # resolves to the HIP runtime torch has loaded
        hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self._hip = hip
        self._ev = []
        for _ in range(n):
            e = ctypes.c_void_p()
            self._check(hip.hipEventCreateWithFlags(ctypes.byref(e), self._FLAG), "CreateWithFlags")
            self._ev.append(e)

    @staticmethod
    def _check(rc, what):
        if rc != 0:
            raise RuntimeError("hipEvent%s failed with HIP error %d" % (what, rc))

    def record(self, i):
        self._check(self._hip.hipEventRecord(self._ev[i], self._torch.cuda.current_stream().cuda_stream), "Record")

    def elapsed(self, i, j):
        """Milliseconds from event i to event j (waits for j)."""
        ms = self._c.c_float()
        self._check(self._hip.hipEventSynchronize(self._ev[j]), "Synchronize")
        self._check(self._hip.hipEventElapsedTime(self._c.byref(ms), self._ev[i], self._ev[j]), "ElapsedTime")
        return ms.value

    def per_step(self):
        return [self.elapsed(i, i + 1) for i in range(len(self._ev) - 1)]

    def close(self):
        for e in self._ev:
            self._hip.hipEventDestroy(e)
        self._ev = []


class Step:
    """Device state of one workload and the enqueue of one step."""

    def __init__(self, wl, mode, device="cuda", record=0, top_p=1.0, target_stats=False, host=None, chain=False,
                 headroom=0):
        """host: host_state() of another Step of the same workload (a second input set with the
        same values in separate buffers); chain: each step verifies the drafts the head proposed
        in the step before (the committed lengths advance; headroom: positions to reserve)."""
        import torch
        from paper_2609_16648_amd import gm
        self.torch, self.gm, self.wl = torch, gm, wl
        # top-p below 1 (sample mode): the accept and the draft work on the nuclei; the
        # draft then hands no row statistics to the accept
        self.top_p = top_p
        s, B, k = wl.shape, wl.batch, wl.k
        self.mode = gm.GM_SAMPLE if mode == "sample" else gm.GM_GREEDY
        # the cycle record's top-k log-probabilities per draft position, taken in the accept's pass
        self.record = None
        if record:
            self.record = (torch.zeros((wl.batch, wl.k, record), dtype=torch.bfloat16, device=device),
                           torch.zeros((wl.batch, wl.k, record), dtype=torch.int32, device=device))
        t0 = time.time()
        self.lens = synth.context_lengths(wl)
        cap = self.lens + 2 * k + 2 + headroom
        self.chain = chain and wl.with_mtp
        gen = torch.Generator(device=device)
        gen.manual_seed(synth.SEED_KV)

        def random_pools(cache):
            for t in cache.k + cache.v:
                t.normal_(generator=gen)

        self.cache = gm.PagedCache(s, 1 if wl.name == "long_ctx" else s.n_layers, self.lens, cap,
                                   page_size=wl.page_size, fill="empty")
        random_pools(self.cache)
        self.lens0 = self.cache.seq_lens.clone()
        self.lens_both = None
        V = s.vocab
        u_acc, u_fin, u_dr = synth.uniforms(B, k)
        dev = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dt)
        self.ua, self.uf, self.ud = dev(u_acc), dev(u_fin), dev(u_dr)
        self.zq = dev(synth.normal_logits((B, k, V), synth.SEED_DRAFT, wl.name, "zq"))
        self.n = torch.zeros(B, dtype=torch.int32, device=device)
        self.out = torch.zeros((B, k + 1), dtype=torch.int32, device=device)
        self.slots = torch.zeros((B, k + 1), dtype=torch.int32, device=device)
        self.ws_v, self.ws_a, self.ws_m = gm.Workspace(device), gm.Workspace(device), gm.Workspace(device)
        self.cfg = gm.model_config(s)
        if wl.name == "long_ctx":
            R = k + 1
            self.q = torch.empty((B, R, s.n_heads, s.head_dim), dtype=torch.bfloat16, device=device)
            self.q.normal_(generator=gen)
            self.attn_out = torch.empty_like(self.q)
            self.zt = dev(synth.normal_logits((B, R, V), synth.SEED_DRAFT, wl.name, "zt"))
            # drafts d_i ~ q_i by the inverse CDF with u_draft (set-up, not timed)
            p = torch.softmax(self.zq.double(), -1).cumsum(-1)
            tgt = self.ud.double()[..., None] * p[..., -1:]
            self.drafts = torch.searchsorted(p, tgt, right=True).clamp_(max=V - 1)[..., 0].to(torch.int32)
        else:
            self.W = host["W"] if host else synth.model_weights(s, threads=16)
            self.model = gm.DeviceModel(s, self.W, device)
            self.logits = torch.empty((B, k + 1, V), dtype=torch.float32, device=device)
            # optionally the target rows' softmax statistics from the LM head's epilogue, for the
            # accept (in place of its pass over the target rows)
            self.tstats = gm.new_row_stats(B, k + 1, device) if target_stats else None
            self.hidden = torch.empty((B, k + 1, s.hidden), dtype=torch.float32, device=device)
            if wl.with_mtp:
                # zq stands in for the draft logits the previous step's head wrote; the head
                # also hands the accept their softmax statistics, so those come with them
                zq = self.zq.cpu().numpy()
                st = np.zeros((B, k), dtype=[("max", "<f4"), ("argmax", "<i4"), ("sum", "<f8")])
                st["max"] = zq.max(-1)
                st["argmax"] = zq.argmax(-1)
                st["sum"] = np.exp(zq.astype(np.float64) - st["max"][..., None].astype(np.float64)).sum(-1)
                self.zq_stats = torch.from_numpy(st.view(np.uint8).reshape(B, k, gm.ROW_STATS_BYTES).copy()).to(device)
                self.next_stats = gm.new_row_stats(B, k, device)
                self.Wm = host["Wm"] if host else synth.mtp_weights(s)
                self.mtp = gm.DeviceMtp(s, self.Wm, device)
                self.mcache = gm.PagedCache(s, 1, self.lens, cap, page_size=wl.page_size, fill="empty")
                random_pools(self.mcache)
                # both caches' lengths in one tensor: one copy per step puts them back
                both = torch.stack([self.cache.seq_lens, self.mcache.seq_lens])
                self.cache.seq_lens, self.mcache.seq_lens = both[0], both[1]
                self.lens_both, self.lens_both0 = both, both.clone()
                self.next_drafts = torch.zeros((B, k), dtype=torch.int32, device=device)
                self.dlog = torch.zeros((B, k, V), dtype=torch.float32, device=device)
                if self.chain:   # the head writes one pair while the accept reads the other
                    self.next_drafts2 = torch.zeros_like(self.next_drafts)
                    self.dlog2 = torch.zeros_like(self.dlog)
                    self.next_stats2 = gm.new_row_stats(B, k, device)
                    self.accept_in = (self.zq, self.zq_stats)
            self.pending = dev(synth.token_ids(B, V, synth.SEED_TOKENS, wl.name, "pending"), torch.int32)
            self.drafts = host["drafts"].to(device) if host else self._mixing_drafts(device)
            self.tokens = torch.cat([self.pending[:, None], self.drafts], 1).contiguous()
        torch.cuda.synchronize()
        log("[bench] set-up of %s took %.1f s" % (wl.name, time.time() - t0))

    def _mixing_drafts(self, device):
        """Draft i = the target's top-1 at block position i given the drafts before it with
        probability mix_prob, else a uniform token (set-up: one verify forward per position)."""
        torch, gm, wl = self.torch, self.gm, self.wl
        B, k, V = wl.batch, wl.k, wl.shape.vocab
        prob = wl.mix_prob if wl.mix_prob is not None else 0.0
        take, alt = synth.mixing_draws(B, k, V, prob, synth.SEED_DRAFT, wl.name)
        take, alt = torch.from_numpy(take).to(device), torch.from_numpy(alt).to(device)
        drafts = alt.clone()
        for i in range(k):
            toks = torch.cat([self.pending[:, None], drafts], 1).contiguous()
            self.cache.seq_lens.copy_(self.lens0)
            gm.verify_forward(self.model, self.cache, toks, self.logits, self.hidden, self.ws_v)
            top1 = torch.argmax(self.logits[:, i], -1).to(torch.int32)
            drafts[:, i] = torch.where(take[:, i], top1, alt[:, i])
        return drafts.contiguous()

    def host_state(self):
        return {"W": getattr(self, "W", None), "Wm": getattr(self, "Wm", None), "drafts": self.drafts.cpu()}

    def __call__(self, draft=True):
        """One step; draft=False leaves out the draft head (verify, accept and commit only)."""
        gm, wl = self.gm, self.wl
        k = wl.k
        if self.chain:
            return self._chain_step()
        if self.lens_both is not None:
            self.lens_both.copy_(self.lens_both0)
        else:
            self.cache.seq_lens.copy_(self.lens0)
        if wl.name == "long_ctx":
            gm.verify_attention(self.cfg, self.cache, 0, self.q, self.attn_out, self.ws_v)
            gm.spec_accept(self.zt, self.zq, self.drafts, self.ua, self.uf, self.n, self.out, self.mode, self.ws_a,
                           record=self.record, top_p=self.top_p)
            gm.kv_commit(self.cache, k, self.n, self.slots)
            return
        gm.verify_forward(self.model, self.cache, self.tokens, self.logits, self.hidden, self.ws_v,
                          target_stats=self.tstats)
        handoff = wl.with_mtp and self.top_p >= 1.0
        gm.spec_accept(self.logits, self.zq, self.drafts, self.ua, self.uf, self.n, self.out, self.mode, self.ws_a,
                       draft_stats=self.zq_stats if handoff else None, record=self.record, top_p=self.top_p,
                       target_stats=self.tstats)
        gm.kv_commit(self.cache, k, self.n, self.slots)
        if wl.with_mtp and draft:
            gm.mtp_draft(self.model, self.mtp, self.mcache, k, self.mode, self.hidden, self.n, self.out, self.ud,
                         self.next_drafts, self.dlog, self.ws_m, draft_stats=self.next_stats if handoff else None,
                         top_p=self.top_p)


    def _chain_step(self):
        """Verify the block [pending, drafts], accept, commit, then the head drafts the next
        block from this step's hiddens; the next step verifies those drafts after the token
        this step drew."""
        torch, gm, wl = self.torch, self.gm, self.wl
        k = wl.k
        zq, zq_stats = self.accept_in
        gm.verify_forward(self.model, self.cache, self.tokens, self.logits, self.hidden, self.ws_v)
        gm.spec_accept(self.logits, zq, self.drafts, self.ua, self.uf, self.n, self.out, self.mode, self.ws_a,
                       draft_stats=zq_stats if self.top_p >= 1.0 else None, top_p=self.top_p)
        gm.kv_commit(self.cache, k, self.n, self.slots)
        gm.mtp_draft(self.model, self.mtp, self.mcache, k, self.mode, self.hidden, self.n, self.out, self.ud,
                     self.next_drafts, self.dlog, self.ws_m,
                     draft_stats=self.next_stats if self.top_p >= 1.0 else None, top_p=self.top_p)
        final = torch.gather(self.out, 1, self.n.long()[:, None])
        self.tokens = torch.cat([final, self.next_drafts], 1).contiguous()
        self.drafts = self.next_drafts
        self.accept_in = (self.dlog, self.next_stats)
        # the head writes the other pair next time
        self.next_drafts, self.next_drafts2 = self.next_drafts2, self.next_drafts
        self.dlog, self.dlog2 = self.dlog2, self.dlog
        self.next_stats, self.next_stats2 = self.next_stats2, self.next_stats


# ----------------------------------------------------------------------------- DCA loss timing
def time_dca(wl, N, iters=5):
    """The DCA loss with verify-gated masking and its gradient (the head-training side
    of the cycle record) over N synthetic records: head logits N(0,1) [N, k, V], a
    top-64 record of other N(0,1) logits, accepted lengths uniform in 0..k.  The pass
    reads the logits twice (statistics, gradient) and writes the gradient once."""
    import torch
    from paper_2609_16648_amd import gm
    K, V = wl.k, wl.shape.vocab
    gen = torch.Generator(device="cuda")
    gen.manual_seed(synth.SEED_DRAFT)
    z = torch.empty((N, K, V), dtype=torch.float32, device="cuda").normal_(generator=gen)
    zt = torch.empty((N, K, V), dtype=torch.float32, device="cuda").normal_(generator=gen)
    top = torch.topk(zt, 64, dim=-1)
    lse = torch.logsumexp(zt, -1, keepdim=True)
    rec_lp = (top.values - lse).to(torch.bfloat16)
    rec_id = top.indices.to(torch.int32).contiguous()
    del zt, top, lse
    n = torch.randint(0, K + 1, (N,), generator=gen, device="cuda", dtype=torch.int32)
    loss = torch.empty(N, dtype=torch.float32, device="cuda")
    alpha = torch.empty((N, K), dtype=torch.float32, device="cuda")
    grad = torch.empty_like(z)
    ws = gm.Workspace()
    gm.dca_loss(z, rec_lp, rec_id, n, loss, alpha, grad, ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(iters):
        gm.dca_loss(z, rec_lp, rec_id, n, loss, alpha, grad, ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / iters
    nbytes = 3.0 * N * K * V * 4
    out = {"cycles": N, "k": K, "vocab": V, "ms": round(ms, 4), "GB_s": round(nbytes / (ms * 1e-3) / 1e9, 1),
           "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_GBS, 3), "mean_loss": round(float(loss.mean()), 5)}
    del z, grad
    torch.cuda.empty_cache()
    return out


def time_reconstruct(step, wl, R, iters=3):
    """Draft-path reconstruction (gm_mtp_reconstruct) of R recorded cycles over the
    workload's depth K, with the workload's head weights: cycle r starts after the
    committed prefix of the workload's context lengths (repeated to R), N(0,1) head
    cache, start hiddens N(0,1), uniform start tokens and drafts.  One call runs the K
    batched depths; its algorithmic bytes are K x (head weights incl. the LM head
    + every cycle's visible KV + the head logits)."""
    import torch
    from paper_2609_16648_amd import gm
    s, K, V, H = wl.shape, wl.k, wl.shape.vocab, wl.shape.hidden
    starts = np.resize(step.lens, R)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(synth.SEED_KV + 7)
    cache = gm.PagedCache(s, 1, starts, starts + K + 1, page_size=wl.page_size, fill="empty")
    for t in cache.k + cache.v:
        t.normal_(generator=gen)
    h0 = torch.empty((R, H), dtype=torch.float32, device="cuda").normal_(generator=gen)
    t0 = torch.randint(0, V, (R,), generator=gen, device="cuda", dtype=torch.int32)
    drafts = torch.randint(0, V, (R, K), generator=gen, device="cuda", dtype=torch.int32)
    out = torch.empty((R, K, V), dtype=torch.float32, device="cuda")
    ws = gm.Workspace()
    gm.mtp_reconstruct(step.model, step.mtp, cache, K, h0, t0, drafts, out, ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(iters):
        gm.mtp_reconstruct(step.model, step.mtp, cache, K, h0, t0, drafts, out, ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / iters
    d, nkv, nq, F = s.head_dim, s.n_kv_heads, s.n_heads, s.ffn
    params = 2 * H * H + H * (nq + 2 * nkv) * d + nq * d * H + 2 * F * H + F * H + V * H
    kv = float(sum((starts.astype(np.float64) + j + 1).sum() for j in range(K))) * nkv * d * 2 * 2
    flops = K * 2.0 * R * params + 4.0 * nq * d * kv / (nkv * d * 2 * 2)
    nbytes = K * (2.0 * params + R * V * 4.0) + kv
    out_ = {"cycles": R, "k": K, "ms": round(ms, 3), "ms_per_depth": round(ms / K, 3),
            "TFLOP_s": round(flops / (ms * 1e-3) / 1e12, 1), "mfma_frac": round(flops / (ms * 1e-3) / 1e12 / BF16_TFLOPS, 3),
            "GB_s": round(nbytes / (ms * 1e-3) / 1e9, 1)}
    del cache, out
    torch.cuda.empty_cache()
    return out_


# ----------------------------------------------------------------------------- CPU baseline
def cpu_baseline(wl, mode, budget_s, weights=None, top_p=1.0):
    """The oracle, as it stands, on a bounded sample of the same workload: the
    same step (verify forward in the rounding-contract mode, accept, commit,
    MTP draft) for the first few sequences."""
    import oracle
    from threadpoolctl import threadpool_info
    s, k = wl.shape, wl.k
    rnd = oracle.Rounding("contract" if s.dtype == "bf16" else "exact")
    lens_all = synth.context_lengths(wl)
    W = weights[0] if weights else (synth.model_weights(s) if wl.name != "long_ctx" else None)
    Wm = weights[1] if weights and len(weights) > 1 else (synth.mtp_weights(s) if wl.with_mtp else None)
    V = s.vocab
    u_acc, u_fin, u_dr = synth.uniforms(wl.batch, k)
    zq_all = synth.normal_logits((wl.batch, k, V), synth.SEED_DRAFT, wl.name, "zq")

    def run(nseq):
        idx = list(range(nseq))
        lens = lens_all[:nseq]
        if wl.name == "long_ctx":
            ks, vs = synth.kv_prefix(s, lens + k + 1, 0, seqs=idx)
            q = synth.normal_tensor((nseq, k + 1, s.n_heads, s.head_dim), 5, "bf16", "cpu-q")
            zt = synth.normal_logits((nseq, k + 1, V), synth.SEED_DRAFT, wl.name, "cpu-zt")
            dr = np.stack([oracle.inverse_cdf_rows(oracle.softmax(zq_all[:nseq, i].astype(np.float64)),
                                                   u_dr[:nseq, i])[0] for i in range(k)], 1)
            t0 = time.perf_counter()
            for b in range(nseq):
                oracle.attention(q[b].astype(np.float64), ks[b].astype(np.float64), vs[b].astype(np.float64),
                                 lens[b] + np.arange(k + 1) + 1)
            res = oracle.spec_accept(zt, zq_all[:nseq], dr, u_acc[:nseq], u_fin[:nseq], top_p=top_p)
            oracle.kv_commit(lens, res.n_accept, k, np.arange(nseq * 4096).reshape(nseq, 4096), 16)
            return time.perf_counter() - t0, int((res.n_accept + 1).sum())
        caches = [synth.kv_prefix(s, lens, l, seqs=idx) for l in range(s.n_layers)]
        pending = synth.token_ids(wl.batch, V, synth.SEED_TOKENS, wl.name, "pending")[:nseq]
        prob = wl.mix_prob if wl.mix_prob is not None else 0.0
        take, alt = synth.mixing_draws(wl.batch, k, V, prob, synth.SEED_DRAFT, wl.name)
        dr = oracle.mixing_drafts(s, W, caches, lens, pending, take[:nseq], alt[:nseq], rnd)
        block = np.concatenate([pending[:, None], dr], 1)
        mk, mv = (synth.kv_prefix(s, lens, 99, seqs=idx) if wl.with_mtp else (None, None))
        t0 = time.perf_counter()
        logits, hid, _ = oracle.verify_forward(s, W, caches, block, lens, rnd)
        if mode == "sample":
            res = oracle.spec_accept(logits.astype(np.float32), zq_all[:nseq], dr, u_acc[:nseq], u_fin[:nseq],
                                     top_p=top_p)
        else:
            res = oracle.spec_accept(logits.astype(np.float32), None, dr, None, None, mode="greedy")
        oracle.kv_commit(lens, res.n_accept, k, np.arange(nseq * 4096).reshape(nseq, 4096), 16)
        if wl.with_mtp:
            oracle.mtp_draft(s, Wm, W, mk, mv, lens, hid, res.n_accept, res.out_tokens, u_dr[:nseq], k, mode, 1.0, rnd,
                             top_p=top_p)
        return time.perf_counter() - t0, int((res.n_accept + 1).sum())

    # the oracle works in float64: hand it float64 weights once, outside the timed runs
    def f64(w):
        if isinstance(w, dict):
            return {kk: f64(vv) for kk, vv in w.items()}
        if isinstance(w, list):
            return [f64(vv) for vv in w]
        return np.asarray(w, dtype=np.float64)
    if W is not None:
        tied = W["lm_head"] is W["embed"]
        W = f64(W)
        if tied:
            W["lm_head"] = W["embed"]
    if Wm is not None:
        Wm = f64(Wm)
    t1, c1 = run(1)
    per_seq = max(t1, 1e-3)
    nseq = int(max(1, min(wl.batch, budget_s / per_seq)))
    t, c = run(nseq) if nseq > 1 else (t1, c1)
    reps = 1
    while nseq == wl.batch and t < 10.0 and reps < 4:   # a whole batch in under 10 s: repeat it
        t2, c2 = run(nseq)
        t, c, reps = t + t2, c + c2, reps + 1
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": c / t, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": "%d of %d sequences of the %s workload, %d full step%s (%s, accept, commit%s) in %.1f s, "
                      "%d committed tokens"
                      % (nseq, wl.batch, wl.name, reps, "s" if reps > 1 else "",
                         "verify attention" if wl.name == "long_ctx" else
                         ("verify forward in the bf16 rounding-contract mode" if s.dtype == "bf16" else
                          "verify forward in float64"),
                         ", MTP draft" if wl.with_mtp else "", t, c)}


def cpu_layer_extrapolated(wl, layer_wl, weights, mode, budget_s, tau):
    """The oracle's cost of one step of a deep workload, from one of its layers: the layer (in
    the rounding-contract mode) timed on a few sequences at the workload's own context mix and
    scaled to all its layers, plus the LM head, the accept, the commit and the MTP draft timed
    once.  layer_wl: the one-layer workload of the same layer shape, whose weights are given;
    tau: committed tokens per sequence per step, from the GPU run of `wl`."""
    import oracle
    from threadpoolctl import threadpool_info
    s1, k, V = layer_wl.shape, wl.k, wl.shape.vocab
    rnd = oracle.Rounding("contract")
    W = {kk: (vv if kk == "layers" else np.asarray(vv, dtype=np.float64)) for kk, vv in weights[0].items()}
    W["layers"] = [{kk: np.asarray(vv, dtype=np.float64) for kk, vv in Wl.items()} for Wl in weights[0]["layers"]]
    Wm = weights[1]
    Wm = {kk: ({k2: np.asarray(v2, dtype=np.float64) for k2, v2 in vv.items()} if isinstance(vv, dict)
                else np.asarray(vv, dtype=np.float64)) for kk, vv in Wm.items()}
    lens_all = synth.context_lengths(wl)
    u_acc, u_fin, u_dr = synth.uniforms(wl.batch, k)
    zq = synth.normal_logits((wl.batch, k, V), synth.SEED_DRAFT, wl.name, "zq")
    t_layer = t_rest = 0.0
    nseq = 0
    while nseq < wl.batch and (nseq == 0 or t_layer + t_rest < budget_s):
        b = nseq
        lens = lens_all[b:b + 1]
        caches = [synth.kv_prefix(s1, lens_all, 0, seqs=[b])]
        block = synth.token_ids(k + 1, V, synth.SEED_TOKENS, wl.name, "cpu-block", b).reshape(1, k + 1)
        t0 = time.perf_counter()
        logits, hid, _ = oracle.verify_forward(s1, W, caches, block, lens, rnd)
        t1 = time.perf_counter()
        oracle.model.lm_head(s1, W, hid[0], rnd)
        t2 = time.perf_counter()
        dr = block[:, 1:]
        if mode == "sample":
            res = oracle.spec_accept(logits.astype(np.float32), zq[b:b + 1], dr, u_acc[b:b + 1], u_fin[b:b + 1])
        else:
            res = oracle.spec_accept(logits.astype(np.float32), None, dr, None, None, mode="greedy")
        oracle.kv_commit(lens, res.n_accept, k, np.arange(4096).reshape(1, 4096), 16)
        mk, mv = synth.kv_prefix(s1, lens_all, 99, seqs=[b])
        oracle.mtp_draft(s1, Wm, W, mk, mv, lens, hid, res.n_accept, res.out_tokens, u_dr[b:b + 1], k, mode, 1.0,
                         rnd)
        t3 = time.perf_counter()
        head = t2 - t1
        t_layer += (t1 - t0) - head        # the layer alone: the forward less its LM head
        t_rest += head + (t3 - t2)
        nseq += 1
    t_step = wl.shape.n_layers * t_layer + t_rest
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": tau * nseq / t_step, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": "extrapolated: one of the %d layers timed on %d of %d sequences of this workload's context mix "
                      "(%.1f s), scaled to %d layers, plus the LM head, accept, commit and MTP draft timed once per "
                      "sequence (%.1f s); committed tokens per sequence per step from the GPU run (%.2f)"
                      % (wl.shape.n_layers, nseq, wl.batch, t_layer, wl.shape.n_layers, t_rest, tau)}


# ----------------------------------------------------------------------------- other configurations
def measure_workload(name, mode, steps, warmup=2):
    """One configuration besides the headline: set-up, warm-up, one traced step for the kernel
    fractions, then `steps` steps timed with a HIP event after each (median reported).  The
    36-layer Qwen3-4B workload runs as a chain: each step verifies the drafts the head proposed
    in the step before, so its committed tokens are counted step by step on the device."""
    import torch
    from paper_2609_16648_amd import gm
    wl = synth.WORKLOADS[name]
    chain = name == "qwen3_4b_full"
    t0 = time.time()
    st = Step(wl, mode, chain=chain, headroom=(warmup + 1 + steps) * (wl.k + 1) if chain else 0)
    setup_s = time.time() - t0
    for _ in range(warmup):
        st()
    torch.cuda.synchronize()
    gm.trace_start()
    st()
    per_kernel = gm.trace_stop()
    committed = torch.zeros((), dtype=torch.int64, device="cuda")
    evs = StepEvents(steps + 1)
    evs.record(0)
    for i in range(steps):
        st()
        evs.record(i + 1)
        if chain:
            committed += (st.n + 1).sum()
    torch.cuda.synchronize()
    per_step = evs.per_step()
    ms_all = evs.elapsed(0, steps) / steps
    evs.close()
    med = float(np.median(per_step))
    tokens = int(committed.item()) / steps if chain else int((st.n + 1).sum().item())
    acc = accounting(wl, st.lens)
    out = {"description": DESCRIPTIONS[name], "batch": wl.batch, "k": wl.k, "steps": steps,
           "ms_per_step": round(ms_all, 4), "ms_per_step_median": round(med, 4),
           "tokens_per_s_median": round(tokens / (med / 1e3), 1), "committed_tokens_per_step": tokens,
           "tau": round(tokens / wl.batch, 4), "setup_s": round(setup_s, 1),
           "drafts": "the head's own chain, fed back step to step" if chain else
                     ("target top-1 w.p. %.1f else uniform" % wl.mix_prob if wl.mix_prob else
                      ("drawn from q" if name == "long_ctx" else "uniform"))}
    if name == "mimo_7b":
        # this configuration is specified in both modes: greedy acceptance on the same set
        other = gm.GM_GREEDY if st.mode == gm.GM_SAMPLE else gm.GM_SAMPLE
        st.mode = other
        for _ in range(warmup):
            st()
        ev = StepEvents(steps + 1)
        ev.record(0)
        for i in range(steps):
            st()
            ev.record(i + 1)
        torch.cuda.synchronize()
        med2 = float(np.median(ev.per_step()))
        ev.close()
        tok2 = int((st.n + 1).sum().item())
        out["greedy" if other == gm.GM_GREEDY else "sample"] = {
            "ms_per_step_median": round(med2, 4), "tokens_per_s_median": round(tok2 / (med2 / 1e3), 1),
            "committed_tokens_per_step": tok2, "tau": round(tok2 / wl.batch, 4)}
    if "attn_verify" in per_kernel and "attn_verify" in acc:
        ms_a = per_kernel["attn_verify"][1]
        out["verify_attn_hbm_frac"] = round(acc["attn_verify"]["bytes"] / (ms_a * 1e-3) / 1e9 / HBM_GBS, 3)
    gn = [x for x in per_kernel if x.startswith("gemm_") and x in acc]
    if gn:
        gms = sum(per_kernel[x][1] for x in gn)
        out["verify_gemm_mfma_frac"] = round(sum(acc[x]["flops"] for x in gn) / (gms * 1e-3) / 1e12 / BF16_TFLOPS, 3)
    log("[bench] %s: %s" % (name, out))
    del st
    torch.cuda.empty_cache()
    return out


# ----------------------------------------------------------------------------- main
def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter record
    (profiles/hbm_traffic_<kernel>.json), or None when there is none for this
    workload or a source file it was taken from has changed since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "hbm_traffic_%s.json" % kernel)
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel") != kernel or rec.get("workload") != workload:
        return None
    for rel, digest in rec.get("sources_sha256", {}).items():
        f = os.path.join(ROOT, rel)
        if not os.path.exists(f) or hashlib.sha256(open(f, "rb").read()).hexdigest() != digest:
            return None
    return int(rec["traffic_bytes_per_launch"])


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen3_4b_layer", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--mode", default="sample", choices=["sample", "greedy"])
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work for the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--dca", type=int, default=0, metavar="N",
                    help="also time the DCA loss forward and gradient over N cycle records of the workload's shape")
    ap.add_argument("--record", type=int, default=0, metavar="K",
                    help="also take the cycle record's top-K log-probabilities in the accept (0: off)")
    ap.add_argument("--reconstruct", type=int, default=0, metavar="R",
                    help="also time the draft-path reconstruction of R recorded cycles (the paper's chunks: 1024)")
    ap.add_argument("--top-p", type=float, default=1.0,
                    help="top-p of the accept and the draft (the paper's evaluation decodes at 0.7; 1: off)")
    ap.add_argument("--target-stats", action="store_true",
                    help="hand the verify LM head's epilogue statistics to the accept (off: the accept's own pass)")
    ap.add_argument("--one-set", action="store_true", help="one input set (no rotation between steps)")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the other configurations (tiny, long_ctx, qwen3_4b_full, mimo_7b) after the headline")
    ap.add_argument("--extra-steps", type=int, default=5, help="timed steps of each other configuration")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also time a plain device copy of this many MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs the step on one GPU only; N > 1 is not supported "
              "(sequences are independent: data parallelism would need no exchange)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_16648_amd import gm
    gm.lib()
    torch.cuda.set_device(0)
    wl = synth.WORKLOADS[args.workload]
    step = Step(wl, args.mode, record=args.record, top_p=args.top_p, target_stats=args.target_stats)
    # Two input sets (weights, KV, logits and every step buffer; the same values in separate
    # buffers) alternate between steps, so that no step finds the previous step's data in the
    # 256 MB Infinity Cache.  Large workloads, whose step touches far more than that cache,
    # run one set.
    sets = [step]
    if not args.one_set and wl.name in ROTATED:
        sets.append(Step(wl, args.mode, record=args.record, top_p=args.top_p, target_stats=args.target_stats,
                         host=step.host_state()))

    for i in range(args.warmup):
        sets[i % len(sets)]()
    torch.cuda.synchronize()
    # every set holds the same values, so every step of every set accepts alike
    n_ref = sets[0].n.clone() if args.warmup > 0 else None

    # all kernels of a few steps (a separate pass), to find the dominant one and the breakdown
    gm.trace_start()
    probe_steps = 2 * len(sets)
    for i in range(probe_steps):
        sets[i % len(sets)]()
    per_kernel = gm.trace_stop()
    dominant = max(per_kernel, key=lambda n: per_kernel[n][1])

    # timed region: K steps, a HIP event after each; launches of the dominant kernel are also
    # bracketed by HIP events on their stream (its average launch duration for the roofline).
    # Each pair of events leaves the stream idle for a few microseconds, so only every
    # (L + 1)-th of its launches is bracketed, L its launches per step: about one per step,
    # each of its L places in the step in turn.
    dom_per_step = max(1, per_kernel[dominant][0] // probe_steps)
    torch.cuda.synchronize()
    evs = StepEvents(args.steps + 1)
    gm.trace_start(dominant, every=dom_per_step + 1)
    evs.record(0)
    for i in range(args.steps):
        sets[i % len(sets)]()
        evs.record(i + 1)
    torch.cuda.synchronize()
    dom = gm.trace_stop()[dominant]
    per_step = evs.per_step()
    ms = evs.elapsed(0, args.steps) / args.steps
    evs.close()
    ms_median = float(np.median(per_step))
    if n_ref is None:
        n_ref = sets[0].n.clone()
    for st in sets:
        if not torch.equal(st.n, n_ref):
            raise RuntimeError("steps are not identical: accept counts changed between steps")
    n = step.n.cpu().numpy()
    committed = int((n + 1).sum())
    value = committed / (ms / 1e3)

    acc = accounting(wl, step.lens, args.top_p, args.record, args.target_stats)
    kernels = {}
    for name, (launches, tot) in sorted(per_kernel.items(), key=lambda kv: -kv[1][1]):
        ms_step = tot / probe_steps
        row = {"ms_per_step": round(ms_step, 4), "launches_per_step": launches // probe_steps}
        if name in acc and ms_step > 0:
            a = acc[name]
            row["GB_s"] = round(a["bytes"] / (ms_step * 1e-3) / 1e9, 1)
            row["hbm_frac"] = round(row["GB_s"] / HBM_GBS, 3)
            if a["flops"]:
                row["TFLOP_s"] = round(a["flops"] / (ms_step * 1e-3) / 1e12, 1)
                row["mfma_frac"] = round(row["TFLOP_s"] / BF16_TFLOPS, 3)
        kernels[name] = row

    a = acc.get(dominant)
    dom_ms = dom[1] / dom[0]
    if a is not None:
        per_launch_bytes = a["bytes"] / a["launches"]
        per_launch_flops = a["flops"] / a["launches"]
        intensity = per_launch_flops / per_launch_bytes if per_launch_bytes else 0.0
        if intensity * HBM_GBS * 1e9 > BF16_TFLOPS * 1e12:
            roof = {"bound": "mfma", "achieved": round(per_launch_flops / (dom_ms * 1e-3) / 1e12, 1),
                    "peak": BF16_TFLOPS, "unit": "TFLOP/s"}
        else:
            roof = {"bound": "hbm", "achieved": round(per_launch_bytes / (dom_ms * 1e-3) / 1e9, 1),
                    "peak": HBM_GBS, "unit": "GB/s"}
        roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
        roof["traffic"] = measured_traffic(dominant, args.workload)
        if roof["traffic"] is not None:
            roof["traffic_unit"] = "bytes/launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
            roof["traffic_vs_algorithmic"] = round(roof["traffic"] / per_launch_bytes, 3)
        roof["kernel"] = dominant
        roof["avg_launch_ms"] = round(dom_ms, 4)
        roof["launches"] = dom[0]
        roof["launch_sample"] = "every %d-th launch of the timed region" % (dom_per_step + 1)
    else:
        roof = {"bound": None, "achieved": None, "peak": None, "unit": None, "frac": None, "traffic": None,
                "kernel": dominant}

    # configuration 2 as specified (one layer and the LM head, no draft head): verify, accept and
    # commit only, on the same sets (reported beside the full step; not the headline)
    verify_only = None
    if wl.with_mtp:
        for i in range(2 * len(sets)):
            sets[i % len(sets)](draft=False)
        torch.cuda.synchronize()
        ev = StepEvents(args.steps + 1)
        ev.record(0)
        for i in range(args.steps):
            sets[i % len(sets)](draft=False)
            ev.record(i + 1)
        torch.cuda.synchronize()
        vo = ev.per_step()
        ev.close()
        verify_only = {"ms_per_step_median": round(float(np.median(vo)), 4),
                       "tokens_per_s": round(committed / (float(np.median(vo)) / 1e3), 1),
                       "what": "verify forward + accept + commit, no draft head"}

    gemm_names = [x for x in kernels if x.startswith("gemm_")]
    verify_gemm_ms = sum(kernels[x]["ms_per_step"] for x in gemm_names)
    verify_gemm_flops = sum(acc[x]["flops"] for x in gemm_names if x in acc)
    summary = {
        "verify_attn_GB_s": kernels.get("attn_verify", {}).get("GB_s"),
        "verify_attn_hbm_frac": kernels.get("attn_verify", {}).get("hbm_frac"),
        "verify_gemm_TFLOP_s": round(verify_gemm_flops / (verify_gemm_ms * 1e-3) / 1e12, 1) if verify_gemm_ms else None,
        "verify_gemm_mfma_frac": round(verify_gemm_flops / (verify_gemm_ms * 1e-3) / 1e12 / BF16_TFLOPS, 3)
        if verify_gemm_ms else None,
        "tau": round(1.0 + float(n.mean()), 4),
        "committed_tokens_per_step": committed,
    }

    summary["ms_per_step_median"] = round(ms_median, 4)
    summary["tokens_per_s_median"] = round(committed / (ms_median / 1e3), 1)
    summary["input_sets"] = len(sets)
    if verify_only:
        summary["config2_as_specified"] = verify_only
    if args.dca:
        summary["dca"] = time_dca(wl, args.dca)
    if args.reconstruct:
        if not wl.with_mtp:
            raise SystemExit("--reconstruct needs a workload with the MTP head")
        summary["reconstruct"] = time_reconstruct(step, wl, args.reconstruct)

    if args.copy_probe_mib:
        src = torch.empty(args.copy_probe_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        summary["copy_probe_mib"] = args.copy_probe_mib

    # the two stated targets of the step (verify attention >= 0.70 of HBM, verify GEMMs >= 0.50 of MFMA),
    # beside the dominant kernel's roofline
    targets = {}
    if "attn_verify" in kernels and "GB_s" in kernels["attn_verify"]:
        targets["verify_attention"] = {"bound": "hbm", "achieved": kernels["attn_verify"]["GB_s"], "peak": HBM_GBS,
                                       "unit": "GB/s", "frac": kernels["attn_verify"]["hbm_frac"], "target_frac": 0.70}
    if summary.get("verify_gemm_TFLOP_s"):
        targets["verify_gemms"] = {"bound": "mfma", "achieved": summary["verify_gemm_TFLOP_s"], "peak": BF16_TFLOPS,
                                   "unit": "TFLOP/s", "frac": summary["verify_gemm_mfma_frac"], "target_frac": 0.50}

    line = {"metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": args.workload, "description": DESCRIPTIONS[args.workload],
                       "batch": wl.batch, "k": wl.k, "accept_mode": args.mode, "parallelism": "none (1 GPU)",
                       "record_topk": args.record, "top_p": args.top_p,
                       "target_stats": args.target_stats},
            "roofline": roof, "roofline_targets": targets, "summary": summary, "kernels": kernels}
    weights = None
    if not args.no_cpu_baseline:
        if hasattr(step, "W"):
            weights = (step.W, step.Wm) if wl.with_mtp else (step.W,)
        line["cpu_baseline"] = cpu_baseline(wl, args.mode, args.cpu_budget, weights, args.top_p)
    else:
        line["cpu_baseline"] = None
    if not args.no_extra:
        del sets, step
        torch.cuda.empty_cache()
        line["workloads"] = {}
        for name in EXTRA:
            if name != args.workload:
                line["workloads"][name] = measure_workload(name, args.mode, args.extra_steps)
        # the oracle beside them, on bounded samples: the small configurations directly, the
        # 36-layer Qwen3-4B shape from one of its layers (the layer workload's weights)
        if not args.no_cpu_baseline:
            for name, budget in (("tiny", 3.0), ("long_ctx", 8.0)):
                if name in line["workloads"]:
                    line["workloads"][name]["cpu_baseline"] = cpu_baseline(synth.WORKLOADS[name], args.mode, budget)
            if "qwen3_4b_full" in line["workloads"] and weights is not None and wl.name == "qwen3_4b_layer":
                w3 = line["workloads"]["qwen3_4b_full"]
                w3["cpu_baseline"] = cpu_layer_extrapolated(synth.WORKLOADS["qwen3_4b_full"], wl, weights, args.mode,
                                                            10.0, w3["tau"])
    for name, row in kernels.items():
        log("[bench] %-24s %s" % (name, row))
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
