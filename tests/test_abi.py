"""The C ABI without a GPU: the library loads, exports every entry point that
include/gm.h declares, sizes its workspaces, and rejects bad arguments on the
host before launching anything."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2609_16648_amd import gm, layout
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = ctypes.c_void_p(1 << 20)          # never dereferenced: every call below fails validation first


def _declared():
    src = open(os.path.join(ROOT, "include", "gm.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(gm_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    L = gm.lib()
    names = _declared()
    assert "gm_verify_forward" in names and "gm_spec_accept" in names
    for n in names:
        assert hasattr(L, n), n
    assert sorted(gm.EXPORTS) == names


def _cfg(shape=synth.QWEN3_4B_LAYER):
    return gm.model_config(shape)


def test_workspace_sizes():
    cfg = _cfg()
    for op in (gm.GM_OP_VERIFY_FORWARD, gm.GM_OP_VERIFY_ATTENTION, gm.GM_OP_SPEC_ACCEPT, gm.GM_OP_MTP_DRAFT,
               gm.GM_OP_MTP_RECONSTRUCT):
        assert gm.workspace_size(op, cfg, 64, 3, 4096) > 0
    assert gm.workspace_size(99, cfg, 64, 3, 4096) == 0
    assert gm.workspace_size(gm.GM_OP_VERIFY_FORWARD, cfg, 64, 16, 4096) == 0      # k beyond the limit
    bad = _cfg(synth.ModelShape(1, 256, 4, 4, 64, 1024, 1024, dtype="bf16"))       # bf16 needs head_dim 128
    assert gm.workspace_size(gm.GM_OP_VERIFY_FORWARD, bad, 4, 3, 128) == 0
    # the attention partials grow with the context bound
    a = gm.workspace_size(gm.GM_OP_VERIFY_ATTENTION, cfg, 32, 7, 32768)
    b = gm.workspace_size(gm.GM_OP_VERIFY_ATTENTION, cfg, 32, 7, 1024)
    assert a > b


def test_spec_accept_rejects_bad_arguments():
    L = gm.lib()
    ws = ctypes.c_void_p(1 << 20)
    args = lambda **kw: dict(dict(B=4, k=3, V=100, mode=gm.GM_SAMPLE, T=1.0, top_p=1.0, tl=FAKE, dl=FAKE, dt=FAKE,
                                  ua=FAKE, uf=FAKE, n=FAKE, out=FAKE, ws=ws, nbytes=1 << 30), **kw)

    def call(a):
        return L.gm_spec_accept(a["B"], a["k"], a["V"], a["mode"], a["T"], a["top_p"], a["tl"], a["dl"], None, None, None,
                                a["dt"],
                                a["ua"], a["uf"], a["n"], a["out"], a.get("rec"), a["ws"], a["nbytes"], None)

    assert call(args(k=16)) == gm.GM_ERR_INVALID_ARG
    assert call(args(mode=7)) == gm.GM_ERR_INVALID_ARG
    assert call(args(T=0.0)) == gm.GM_ERR_INVALID_ARG
    for bad in (0.0, -0.5, 1.5, float("nan")):
        assert call(args(top_p=bad)) == gm.GM_ERR_INVALID_ARG and "top_p" in gm.last_error()
    assert call(args(dl=None)) == gm.GM_ERR_INVALID_ARG
    assert "draft_logits" in gm.last_error()
    assert call(args(uf=None)) == gm.GM_ERR_INVALID_ARG
    assert call(args(tl=None)) == gm.GM_ERR_INVALID_ARG
    assert call(args(nbytes=16)) == gm.GM_ERR_WORKSPACE
    assert call(args(ws=ctypes.c_void_p((1 << 20) + 8))) == gm.GM_ERR_WORKSPACE      # misaligned
    assert call(args(B=0)) == gm.GM_OK                                               # nothing to do
    rec = gm.Record(65, FAKE, FAKE)                                                  # record width above 64
    assert call(args(rec=ctypes.byref(rec))) == gm.GM_ERR_INVALID_ARG and "topk" in gm.last_error()
    rec = gm.Record(64, FAKE, None)
    assert call(args(rec=ctypes.byref(rec))) == gm.GM_ERR_INVALID_ARG
    rec = gm.Record(64, FAKE, FAKE)
    assert call(args(V=40, rec=ctypes.byref(rec))) == gm.GM_ERR_INVALID_ARG         # wider than the vocabulary


class _FakeCache:
    def __init__(self, n_layers, max_ctx, page_size=16, max_pages=10):
        self.kp = (ctypes.c_void_p * n_layers)(*([1 << 20] * n_layers))
        self.desc = gm.KVCacheDesc(self.kp, self.kp, n_layers, page_size, 100, max_pages, FAKE, FAKE, max_ctx)


def _weights(n_layers):
    lw = gm.LayerWeights(*([FAKE] * 8))
    arr = (gm.LayerWeights * n_layers)(*([lw] * n_layers))
    return arr, gm.ModelWeights(FAKE, FAKE, FAKE, ctypes.cast(arr, ctypes.POINTER(gm.LayerWeights)))


def test_verify_forward_rejects_bad_arguments():
    L = gm.lib()
    shape = synth.ModelShape(2, 256, 4, 4, 64, 1024, 1024, dtype="f32")
    cfg = gm.model_config(shape)
    keep, w = _weights(2)

    def call(cfg_=cfg, cache=None, B=4, k=3, nbytes=1 << 30, T=1.0, stats=None):
        cache = cache or _FakeCache(2, 100)
        return L.gm_verify_forward(ctypes.byref(cfg_), ctypes.byref(w), ctypes.byref(cache.desc), B, k, FAKE, FAKE,
                                   FAKE, T, stats, FAKE, nbytes, None, None)

    assert call(cache=_FakeCache(2, 157)) == gm.GM_ERR_CAPACITY      # 157 + 4 > 10 pages of 16
    assert "exceed" in gm.last_error()
    assert call(cache=_FakeCache(1, 100)) == gm.GM_ERR_INVALID_ARG   # cache layers != model layers
    assert call(cache=_FakeCache(2, 100, page_size=24)) == gm.GM_ERR_UNSUPPORTED
    assert call(k=-1) == gm.GM_ERR_UNSUPPORTED
    assert call(nbytes=100) == gm.GM_ERR_WORKSPACE
    bad = gm.model_config(synth.ModelShape(2, 256, 4, 3, 64, 1024, 1024, dtype="f32"))   # 4 % 3 != 0
    assert call(cfg_=bad) == gm.GM_ERR_INVALID_ARG
    big_group = gm.model_config(synth.ModelShape(2, 256, 32, 2, 64, 1024, 1024, dtype="f32"))  # 16 * 4 rows ok
    assert call(cfg_=big_group, k=4) == gm.GM_ERR_UNSUPPORTED                               # 16 * 5 > 64
    assert call(stats=FAKE, T=0.0) == gm.GM_ERR_INVALID_ARG and "temperature" in gm.last_error()
    assert call(B=0) == gm.GM_OK


def test_mtp_and_attention_reject_bad_arguments():
    L = gm.lib()
    shape = synth.ModelShape(1, 256, 4, 4, 64, 1024, 1024, dtype="f32")
    cfg = gm.model_config(shape)
    keep, w = _weights(1)
    mtp = gm.MtpWeights(FAKE, FAKE, FAKE, FAKE, gm.LayerWeights(*([FAKE] * 8)))
    c = _FakeCache(1, 100)
    st = L.gm_mtp_draft(ctypes.byref(cfg), ctypes.byref(mtp), ctypes.byref(w), ctypes.byref(c.desc), 4, 3,
                        gm.GM_SAMPLE, 1.0, 1.0, FAKE, FAKE, FAKE, None, FAKE, FAKE, None, None, FAKE, 1 << 30, None, None)
    assert st == gm.GM_ERR_INVALID_ARG and "u_draft" in gm.last_error()
    c2 = _FakeCache(1, 150)                                         # 150 + 2k + 1 > 160
    st = L.gm_mtp_draft(ctypes.byref(cfg), ctypes.byref(mtp), ctypes.byref(w), ctypes.byref(c2.desc), 4, 5,
                        gm.GM_GREEDY, 1.0, 1.0, FAKE, FAKE, FAKE, None, FAKE, FAKE, None, None, FAKE, 1 << 30, None, None)
    assert st == gm.GM_ERR_CAPACITY
    for bad in (0.0, 2.0):
        st = L.gm_mtp_draft(ctypes.byref(cfg), ctypes.byref(mtp), ctypes.byref(w), ctypes.byref(c.desc), 4, 3,
                            gm.GM_SAMPLE, 1.0, bad, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, FAKE, 1 << 30, None, None)
        assert st == gm.GM_ERR_INVALID_ARG and "top_p" in gm.last_error()
    # top-p draws do not produce the row statistics of the accept handoff
    st = L.gm_mtp_draft(ctypes.byref(cfg), ctypes.byref(mtp), ctypes.byref(w), ctypes.byref(c.desc), 4, 3,
                        gm.GM_SAMPLE, 1.0, 0.7, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 1 << 30, None, None)
    assert st == gm.GM_ERR_UNSUPPORTED and "draft_stats" in gm.last_error()
    # reconstruction: K >= 1, inputs, and room for the K chain entries past max_ctx
    rc = lambda cache, K, hid=FAKE, toks=FAKE, dr=FAKE: L.gm_mtp_reconstruct(
        ctypes.byref(cfg), ctypes.byref(mtp), ctypes.byref(w), ctypes.byref(cache.desc), 4, K, hid, toks, dr, FAKE,
        FAKE, 1 << 30, None, None)
    assert rc(c, 0) == gm.GM_ERR_INVALID_ARG
    assert rc(c, 3, hid=None) == gm.GM_ERR_INVALID_ARG and "reconstruction" in gm.last_error()
    assert rc(c, 3, dr=None) == gm.GM_ERR_INVALID_ARG
    assert rc(_FakeCache(1, 150), 11) == gm.GM_ERR_CAPACITY           # 150 + 11 > 160
    assert gm.workspace_size(gm.GM_OP_MTP_RECONSTRUCT, cfg, 4, 0, 100) == 0
    st = L.gm_verify_attention(ctypes.byref(cfg), ctypes.byref(c.desc), 1, 4, 3, FAKE, FAKE, FAKE, 1 << 30, None, None)
    assert st == gm.GM_ERR_INVALID_ARG                              # layer out of range
    st = L.gm_kv_commit(ctypes.byref(c.desc), 4, 3, None, None, None)
    assert st == gm.GM_ERR_INVALID_ARG


# ------------------------------------------------------------------ layout
@pytest.mark.parametrize("head_dim", [64, 128])
def test_tile_layout_is_a_bijection(head_dim):
    k, v = layout.tile_offsets(head_dim)
    for t in (k, v):
        assert sorted(t.ravel().tolist()) == list(range(16 * head_dim))


def test_tile_layout_matches_operand_order():
    # one 16-byte load per lane (8 bf16) at instruction i reads elements i*512 + 8*lane .. +7
    k, v = layout.tile_offsets(128)
    inv_k = {int(o): (s, c) for (s, c), o in np.ndenumerate(k)}
    inv_v = {int(o): (s, c) for (s, c), o in np.ndenumerate(v)}
    for i in range(4):
        for lane in range(64):
            got = [inv_k[i * 512 + 8 * lane + e] for e in range(8)]
            # K: token lane % 16, eight consecutive channels of one 32-channel slice
            assert all(s == lane % 16 for s, _ in got)
            assert [c for _, c in got] == [32 * i + 8 * (lane // 16) + e for e in range(8)]
            got = [inv_v[i * 512 + 8 * lane + e] for e in range(8)]
            # V: channels 32i + lane % 16 (first four) and 32i + 16 + lane % 16 (last four),
            #    tokens 4 (lane // 16) .. +3 in each half
            assert [c for _, c in got] == [32 * i + lane % 16] * 4 + [32 * i + 16 + lane % 16] * 4
            assert [s for s, _ in got] == [4 * (lane // 16) + e for e in range(4)] * 2


def test_scatter_gather_round_trip():
    g = np.random.default_rng(0)
    page_size, n_kv, d = 32, 2, 64
    table, num_pages = layout.block_table([3, 5], 5, seed=1)
    pool = np.zeros((num_pages, n_kv, page_size * d), np.float32)
    ent = g.standard_normal((150, n_kv, d)).astype(np.float32)
    pos = np.arange(150)
    layout.scatter(pool, ent, pos, table[1], page_size, "v")
    np.testing.assert_array_equal(layout.gather(pool, pos, table[1], page_size, n_kv, d, "v"), ent)
    assert (table[0, 3:] == -1).all() and sorted(table[table >= 0].tolist()) == list(range(8))


def test_weight_tiling_matches_header_formula():
    g = np.random.default_rng(1)
    n, k = 256, 96
    w = g.standard_normal((n, k)).astype(np.float32)
    flat = layout.tile_weight(w)
    r, c = np.meshgrid(np.arange(n), np.arange(k), indexing="ij")
    off = (((r // 128) * (k // 32) + c // 32) * 8 + (r // 16) % 8) * 512 + ((c % 32) // 8) * 128 + (r % 16) * 8 + c % 8
    np.testing.assert_array_equal(flat[off], w)
    np.testing.assert_array_equal(layout.untile_weight(flat, n, k), w)
    # one 16-byte load per lane at lane * 8 of a tile: row lane % 16, columns 8 (lane // 16) .. +7
    t = flat[:512].reshape(64, 8)
    for lane in range(64):
        np.testing.assert_array_equal(t[lane], w[lane % 16, 8 * (lane // 16): 8 * (lane // 16) + 8])


def test_dca_loss_rejects_bad_arguments():
    L = gm.lib()
    ws = ctypes.c_void_p(1 << 20)

    def call(N=4, K=3, V=1000, topk=64, n=FAKE, vgm=1, nbytes=1 << 30):
        return L.gm_dca_loss(N, K, V, topk, FAKE, FAKE, FAKE, n, vgm, FAKE, FAKE, None, ws, nbytes, None)

    assert call(K=0) == gm.GM_ERR_INVALID_ARG
    assert call(K=16) == gm.GM_ERR_INVALID_ARG
    assert call(topk=65) == gm.GM_ERR_INVALID_ARG and "topk" in gm.last_error()
    assert call(V=40) == gm.GM_ERR_INVALID_ARG                 # record wider than the vocabulary
    assert call(n=None) == gm.GM_ERR_INVALID_ARG               # verify-gated masking needs n_accept
    assert call(nbytes=64) == gm.GM_ERR_WORKSPACE
    assert call(N=0) == gm.GM_OK
    cfg = gm.ModelConfig()
    cfg.vocab = 151936
    assert gm.workspace_size(gm.GM_OP_DCA_LOSS, cfg, 1024, 3, 0) > gm.workspace_size(gm.GM_OP_DCA_LOSS, cfg, 8, 3, 0)


def test_workspace_size_null_config():
    # every op reports 0 for a NULL config instead of reading through it
    L = gm.lib()
    for op in (gm.GM_OP_VERIFY_FORWARD, gm.GM_OP_VERIFY_ATTENTION, gm.GM_OP_SPEC_ACCEPT, gm.GM_OP_MTP_DRAFT,
               gm.GM_OP_DCA_LOSS, gm.GM_OP_MTP_RECONSTRUCT):
        assert L.gm_workspace_size(op, None, 8, 3, 1024) == 0


def test_trace_sampling_argument():
    # the sampling stride is checked on the host (no GPU here)
    L = gm.lib()
    assert L.gm_trace_every(0) == gm.GM_ERR_INVALID_ARG and "gm_trace_every" in gm.last_error()
    assert L.gm_trace_every(-3) == gm.GM_ERR_INVALID_ARG
    assert L.gm_trace_every(4) == gm.GM_OK
    assert L.gm_trace_every(1) == gm.GM_OK


def test_spec_accept_noalloc_rejects_on_the_host():
    # oversized calls and bad shapes fail before the device is touched (no GPU here)
    L = gm.lib()
    call = lambda B, k, V: L.gm_spec_accept_noalloc(B, k, V, gm.GM_SAMPLE, 1.0, 1.0, FAKE, FAKE, None, None, None,
                                                    FAKE, FAKE, FAKE, FAKE, FAKE, None, None)
    assert call(4, 16, 100) == gm.GM_ERR_INVALID_ARG
    assert call(-1, 3, 100) == gm.GM_ERR_INVALID_ARG
    assert call(0, 3, 100) == gm.GM_OK
    assert call(4096, 15, 524288) == gm.GM_ERR_CAPACITY and "fixed scratch" in gm.last_error()
    cfg = gm.ModelConfig()
    cfg.vocab = 151936
    assert gm.workspace_size(gm.GM_OP_SPEC_ACCEPT, cfg, 256, 7, 0) <= 16 << 20     # the stated fit
