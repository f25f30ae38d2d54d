"""Python binding of libgm (include/gm.h): argument marshalling only.

Every function here converts torch tensors to raw device pointers, calls the
C entry point of the same name on the current HIP stream and raises GMError
on a non-OK status.  All arithmetic of the step runs in libgm's HIP kernels;
if libgm.so is missing, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import layout

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgm.so")

GM_OK, GM_ERR_INVALID_ARG, GM_ERR_UNSUPPORTED, GM_ERR_CAPACITY, GM_ERR_WORKSPACE, GM_ERR_DEVICE = 0, -1, -2, -3, -4, -5
GM_F32, GM_BF16 = 0, 1
GM_GREEDY, GM_SAMPLE = 0, 1
GM_OP_VERIFY_FORWARD, GM_OP_VERIFY_ATTENTION, GM_OP_SPEC_ACCEPT, GM_OP_MTP_DRAFT, GM_OP_DCA_LOSS = 0, 1, 2, 3, 4
GM_OP_MTP_RECONSTRUCT = 5
GM_DEVERR_TOKEN, GM_DEVERR_PAGE = 1, 2

c_int, c_float, c_void_p, c_size_t, c_double = ctypes.c_int, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_double


class GMError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("libgm status %d: %s" % (status, msg))
        self.status = status


class ModelConfig(ctypes.Structure):
    _fields_ = [("n_layers", c_int), ("hidden", c_int), ("n_heads", c_int), ("n_kv_heads", c_int),
                ("head_dim", c_int), ("ffn", c_int), ("vocab", c_int), ("rope_base", c_float),
                ("rms_eps", c_float), ("dtype", c_int), ("qk_norm", c_int), ("tie_embed", c_int)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("attn_norm", "w_qkv", "q_norm", "k_norm", "w_o", "ffn_norm",
                                        "w_gate_up", "w_down")]


class ModelWeights(ctypes.Structure):
    _fields_ = [("embed", c_void_p), ("final_norm", c_void_p), ("lm_head", c_void_p),
                ("layers", ctypes.POINTER(LayerWeights))]


class MtpWeights(ctypes.Structure):
    _fields_ = [("norm_h", c_void_p), ("norm_e", c_void_p), ("w_proj", c_void_p), ("final_norm", c_void_p),
                ("layer", LayerWeights)]


class KVCacheDesc(ctypes.Structure):
    _fields_ = [("k_pages", ctypes.POINTER(c_void_p)), ("v_pages", ctypes.POINTER(c_void_p)),
                ("n_layers", c_int), ("page_size", c_int), ("num_pages", c_int), ("max_pages_per_seq", c_int),
                ("block_table", c_void_p), ("seq_lens", c_void_p), ("max_ctx", c_int)]


_lib = None

EXPORTS = ["gm_workspace_size", "gm_verify_forward", "gm_verify_attention", "gm_spec_accept", "gm_kv_commit",
           "gm_mtp_draft", "gm_mtp_reconstruct", "gm_dca_loss", "gm_last_error", "gm_trace_every", "gm_trace_start", "gm_trace_stop", "gm_trace_count", "gm_trace_get", "gm_spec_accept_noalloc"]


def lib() -> ctypes.CDLL:
    """Load libgm.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libgm.so not found at %s: build it with `python -m paper_2609_16648_amd.build`" % LIB_PATH)
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    L.gm_workspace_size.restype = c_size_t
    L.gm_workspace_size.argtypes = [c_int, P(ModelConfig), c_int, c_int, c_int]
    L.gm_verify_forward.restype = c_int
    L.gm_verify_forward.argtypes = [P(ModelConfig), P(ModelWeights), P(KVCacheDesc), c_int, c_int, c_void_p,
                                    c_void_p, c_void_p, c_float, c_void_p, c_void_p, c_size_t, c_void_p, c_void_p]
    L.gm_verify_attention.restype = c_int
    L.gm_verify_attention.argtypes = [P(ModelConfig), P(KVCacheDesc), c_int, c_int, c_int, c_void_p, c_void_p,
                                      c_void_p, c_size_t, c_void_p, c_void_p]
    L.gm_spec_accept.restype = c_int
    L.gm_spec_accept.argtypes = [c_int, c_int, c_int, c_int, c_float, c_float, c_void_p, c_void_p, c_void_p,
                                 c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                 c_void_p, c_size_t, c_void_p]
    L.gm_spec_accept_noalloc.restype = c_int
    L.gm_spec_accept_noalloc.argtypes = [c_int, c_int, c_int, c_int, c_float, c_float, c_void_p, c_void_p, c_void_p,
                                         c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                         c_void_p]
    L.gm_kv_commit.restype = c_int
    L.gm_kv_commit.argtypes = [P(KVCacheDesc), c_int, c_int, c_void_p, c_void_p, c_void_p]
    L.gm_mtp_draft.restype = c_int
    L.gm_mtp_draft.argtypes = [P(ModelConfig), P(MtpWeights), P(ModelWeights), P(KVCacheDesc), c_int, c_int,
                               c_int, c_float, c_float, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                               c_void_p, c_void_p, c_size_t, c_void_p, c_void_p]
    L.gm_mtp_reconstruct.restype = c_int
    L.gm_mtp_reconstruct.argtypes = [P(ModelConfig), P(MtpWeights), P(ModelWeights), P(KVCacheDesc), c_int, c_int,
                                     c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p, c_void_p]
    L.gm_dca_loss.restype = c_int
    L.gm_dca_loss.argtypes = [c_int, c_int, c_int, c_int, c_void_p, c_void_p, c_void_p, c_void_p, c_int, c_void_p,
                              c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
    L.gm_last_error.restype = ctypes.c_char_p
    L.gm_last_error.argtypes = []
    L.gm_trace_every.restype = c_int
    L.gm_trace_every.argtypes = [c_int]
    L.gm_trace_start.restype = c_int
    L.gm_trace_start.argtypes = [ctypes.c_char_p]
    L.gm_trace_stop.restype = c_int
    L.gm_trace_stop.argtypes = []
    L.gm_trace_count.restype = c_int
    L.gm_trace_count.argtypes = []
    L.gm_trace_get.restype = c_int
    L.gm_trace_get.argtypes = [c_int, P(ctypes.c_char_p), P(c_int), P(c_double)]
    _lib = L
    return L


def last_error() -> str:
    return lib().gm_last_error().decode()


def _check(st: int):
    if st != GM_OK:
        raise GMError(st, last_error())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to libgm must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _need(t: torch.Tensor, dtype, shape, name: str):
    if t.dtype != dtype or tuple(t.shape) != tuple(shape):
        raise ValueError("%s: expected %s %s, got %s %s" % (name, dtype, tuple(shape), t.dtype, tuple(t.shape)))
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)


# ------------------------------------------------------------------------ configs and weights
def model_config(shape) -> ModelConfig:
    """ModelConfig from an object with the fields of synth.ModelShape."""
    return ModelConfig(shape.n_layers, shape.hidden, shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.ffn,
                       shape.vocab, float(shape.rope_base), float(shape.rms_eps),
                       GM_BF16 if shape.dtype == "bf16" else GM_F32, int(shape.qk_norm), int(shape.tie_embed))


def torch_dtype(shape):
    return torch.bfloat16 if shape.dtype == "bf16" else torch.float32


def _dev(a: np.ndarray, dtype, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device=device, dtype=dtype)


def _dev_linear(a: np.ndarray, dtype, device) -> torch.Tensor:
    """A linear weight in the layout gm.h gives its dtype: tiled for bf16, row-major for float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return _dev(layout.tile_weight(a) if dtype == torch.bfloat16 else a, dtype, device)


class DeviceLayer:
    """One decoder layer's weights on the device, packed as gm.h lays them out."""

    def __init__(self, shape, w: Dict[str, np.ndarray], device):
        dt = torch_dtype(shape)
        self.t = {
            "attn_norm": _dev(w["attn_norm"], dt, device),
            "w_qkv": _dev_linear(np.concatenate([w["wq"], w["wk"], w["wv"]], 0), dt, device),
            "w_o": _dev_linear(w["wo"], dt, device),
            "ffn_norm": _dev(w["ffn_norm"], dt, device),
            "w_gate_up": _dev_linear(np.concatenate([w["w_gate"], w["w_up"]], 0), dt, device),
            "w_down": _dev_linear(w["w_down"], dt, device),
        }
        if shape.qk_norm:
            self.t["q_norm"] = _dev(w["q_norm"], dt, device)
            self.t["k_norm"] = _dev(w["k_norm"], dt, device)

    def struct(self) -> LayerWeights:
        g = lambda n: _ptr(self.t[n]) if n in self.t else None
        return LayerWeights(g("attn_norm"), g("w_qkv"), g("q_norm"), g("k_norm"), g("w_o"), g("ffn_norm"),
                            g("w_gate_up"), g("w_down"))


class DeviceModel:
    """Backbone weights on the device (from synth.model_weights)."""

    def __init__(self, shape, w: Dict[str, object], device="cuda"):
        self.shape = shape
        self.cfg = model_config(shape)
        dt = torch_dtype(shape)
        self.embed = _dev(w["embed"], dt, device)
        # the LM head is a linear weight (tiled for bf16), the embedding a row-major table
        if w["lm_head"] is w["embed"] and dt != torch.bfloat16:
            self.lm_head = self.embed
        else:
            self.lm_head = _dev_linear(w["lm_head"], dt, device)
        self.final_norm = _dev(w["final_norm"], dt, device)
        self.layers = [DeviceLayer(shape, L, device) for L in w["layers"]]
        self._layer_arr = (LayerWeights * len(self.layers))(*[L.struct() for L in self.layers])
        self.struct = ModelWeights(_ptr(self.embed), _ptr(self.final_norm), _ptr(self.lm_head),
                                   ctypes.cast(self._layer_arr, ctypes.POINTER(LayerWeights)))


class DeviceMtp:
    """Draft-head weights on the device (from synth.mtp_weights)."""

    def __init__(self, shape, w: Dict[str, object], device="cuda"):
        dt = torch_dtype(shape)
        self.norm_h = _dev(w["norm_h"], dt, device)
        self.norm_e = _dev(w["norm_e"], dt, device)
        self.w_proj = _dev_linear(w["w_proj"], dt, device)
        self.final_norm = _dev(w["final_norm"], dt, device)
        self.layer = DeviceLayer(shape, w["layer"], device)
        self.struct = MtpWeights(_ptr(self.norm_h), _ptr(self.norm_e), _ptr(self.w_proj), _ptr(self.final_norm),
                                 self.layer.struct())


class PagedCache:
    """A paged KV cache on the device (gm_kv_cache) with its page table.

    pages_needed[b] pages are dealt to sequence b from a shuffled pool, or the
    rows of an explicit page table (pages may then be shared between rows);
    max_ctx is the host bound on the committed lengths."""

    def __init__(self, shape, n_layers: int, lens: Sequence[int], capacity: Sequence[int], page_size: int = 16,
                 max_ctx: Optional[int] = None, device="cuda", seed: int = 0, fill: str = "zero",
                 table: Optional[np.ndarray] = None):
        self.shape, self.n_layers, self.page_size = shape, n_layers, page_size
        self.dtype = torch_dtype(shape)
        lens = np.asarray(lens, dtype=np.int64)
        capacity = np.asarray(capacity, dtype=np.int64)
        self.B = len(lens)
        need = (capacity + page_size - 1) // page_size
        if table is None:
            self.max_pages = int(need.max())
            table, self.num_pages = layout.block_table(need, self.max_pages, seed)
        else:
            table = np.ascontiguousarray(table, dtype=np.int32)
            if table.shape[0] != self.B or any((table[b, :need[b]] < 0).any() for b in range(self.B)):
                raise ValueError("the page table must give every sequence pages_needed pages")
            self.max_pages, self.num_pages = table.shape[1], int(table.max()) + 1
        self.block_table_host = table
        self.block_table = torch.from_numpy(table).to(device)
        self.seq_lens = torch.from_numpy(lens.astype(np.int32)).to(device)
        self.max_ctx = int(lens.max()) if max_ctx is None else int(max_ctx)
        blk = shape.n_kv_heads * page_size * shape.head_dim
        make = torch.zeros if fill == "zero" else torch.empty
        self.k = [make((self.num_pages, blk), dtype=self.dtype, device=device) for _ in range(n_layers)]
        self.v = [make((self.num_pages, blk), dtype=self.dtype, device=device) for _ in range(n_layers)]
        self._kp = (c_void_p * n_layers)(*[t.data_ptr() for t in self.k])
        self._vp = (c_void_p * n_layers)(*[t.data_ptr() for t in self.v])

    def struct(self) -> KVCacheDesc:
        return KVCacheDesc(self._kp, self._vp, self.n_layers, self.page_size, self.num_pages, self.max_pages,
                           _ptr(self.block_table), _ptr(self.seq_lens), self.max_ctx)

    def _pool(self, layer: int, which: str) -> np.ndarray:
        t = (self.k if which == "k" else self.v)[layer]
        return t.view(self.num_pages, self.shape.n_kv_heads, -1)

    def write(self, layer: int, b: int, positions, k: np.ndarray, v: np.ndarray):
        """Store logical entries [T, n_kv, head_dim] at the given positions of sequence b."""
        positions = np.asarray(positions, dtype=np.int64)
        for which, ent in (("k", k), ("v", v)):
            page, elem = layout.element_index(positions, self.block_table_host[b], self.page_size,
                                              self.shape.head_dim, which)
            pool = self._pool(layer, which)
            idx_p = torch.from_numpy(page).to(pool.device)[:, None, None]
            idx_h = torch.arange(self.shape.n_kv_heads, device=pool.device)[None, :, None]
            idx_e = torch.from_numpy(elem).to(pool.device)[:, None, :]
            pool[idx_p, idx_h, idx_e] = torch.from_numpy(np.ascontiguousarray(ent, np.float32)).to(
                device=pool.device, dtype=self.dtype)

    def read(self, layer: int, b: int, positions):
        """Logical entries (K, V) [T, n_kv, head_dim] float32 at the given positions of sequence b."""
        positions = np.asarray(positions, dtype=np.int64)
        out = []
        for which in ("k", "v"):
            page, elem = layout.element_index(positions, self.block_table_host[b], self.page_size,
                                              self.shape.head_dim, which)
            pool = self._pool(layer, which)
            idx_p = torch.from_numpy(page).to(pool.device)[:, None, None]
            idx_h = torch.arange(self.shape.n_kv_heads, device=pool.device)[None, :, None]
            idx_e = torch.from_numpy(elem).to(pool.device)[:, None, :]
            out.append(pool[idx_p, idx_h, idx_e].float().cpu().numpy())
        return out[0], out[1]


class Workspace:
    """A growable device scratch buffer (allocated outside the step)."""

    def __init__(self, device="cuda"):
        self.device = device
        self.buf = None

    def get(self, nbytes: int) -> torch.Tensor:
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        return self.buf


def workspace_size(op: int, cfg: ModelConfig, B: int, k: int, max_ctx: int) -> int:
    return int(lib().gm_workspace_size(op, ctypes.byref(cfg), B, k, max_ctx))


# ------------------------------------------------------------------------ entry points
def verify_forward(model: DeviceModel, cache: PagedCache, tokens: torch.Tensor, logits: torch.Tensor,
                   hidden: torch.Tensor, ws: Workspace, dev_err: Optional[torch.Tensor] = None, stream=None,
                   target_stats: Optional[torch.Tensor] = None, temperature: float = 1.0):
    """target_stats: optional [B, k+1] row statistics (new_row_stats) of the logits at `temperature`,
    taken in the LM head's epilogue, for spec_accept(target_stats=...)."""
    B, k1 = tokens.shape
    s = model.shape
    _need(tokens, torch.int32, (B, k1), "tokens")
    _need(logits, torch.float32, (B, k1, s.vocab), "logits")
    _need(hidden, torch.float32, (B, k1, s.hidden), "hidden")
    if target_stats is not None:
        _need(target_stats, torch.uint8, (B, k1, ROW_STATS_BYTES), "target_stats")
    cs = cache.struct()
    n = workspace_size(GM_OP_VERIFY_FORWARD, model.cfg, B, k1 - 1, cache.max_ctx)
    buf = ws.get(n)
    _check(lib().gm_verify_forward(ctypes.byref(model.cfg), ctypes.byref(model.struct), ctypes.byref(cs), B, k1 - 1,
                                   _ptr(tokens), _ptr(logits), _ptr(hidden), float(temperature), _ptr(target_stats),
                                   _ptr(buf), buf.numel(), _ptr(dev_err), _stream(stream)))


def verify_attention(cfg: ModelConfig, cache: PagedCache, layer: int, q: torch.Tensor, out: torch.Tensor,
                     ws: Workspace, dev_err: Optional[torch.Tensor] = None, stream=None):
    B, k1 = q.shape[0], q.shape[1]
    _need(q, cache.dtype, (B, k1, cfg.n_heads, cfg.head_dim), "q")
    _need(out, cache.dtype, (B, k1, cfg.n_heads, cfg.head_dim), "out")
    cs = cache.struct()
    n = workspace_size(GM_OP_VERIFY_ATTENTION, cfg, B, k1 - 1, cache.max_ctx)
    buf = ws.get(n)
    _check(lib().gm_verify_attention(ctypes.byref(cfg), ctypes.byref(cs), layer, B, k1 - 1, _ptr(q), _ptr(out),
                                     _ptr(buf), buf.numel(), _ptr(dev_err), _stream(stream)))


ROW_STATS_BYTES = 16   # gm_row_stats: float max, int32 argmax, double sum
RECORD_MAX_TOPK = 64


class Record(ctypes.Structure):
    """gm_record: the cycle record's top-k log-probabilities (bf16) and ids."""
    _fields_ = [("topk", ctypes.c_int), ("logp", ctypes.c_void_p), ("ids", ctypes.c_void_p)]


NUCLEUS_BYTES = 24   # gm_nucleus: float64 m, float64 mass, uint32 key, int32 last_id


def new_nuclei(B: int, k: int, device="cuda") -> torch.Tensor:
    """Device buffer for gm_nucleus [B][k] (the top-p handoff from mtp_draft to spec_accept)."""
    return torch.zeros((B, k, NUCLEUS_BYTES), dtype=torch.uint8, device=device)


def new_row_stats(B: int, k: int, device="cuda") -> torch.Tensor:
    """Storage for [B][k] gm_row_stats (as bytes)."""
    return torch.zeros((B, k, ROW_STATS_BYTES), dtype=torch.uint8, device=device)


def decode_row_stats(t: torch.Tensor):
    """(max float32, argmax int32, sum float64) arrays of a gm_row_stats tensor."""
    h = t.detach().cpu().contiguous()
    return (h[..., 0:4].contiguous().view(torch.float32)[..., 0].numpy(),
            h[..., 4:8].contiguous().view(torch.int32)[..., 0].numpy(),
            h[..., 8:16].contiguous().view(torch.float64)[..., 0].numpy())


def spec_accept(target_logits: torch.Tensor, draft_logits: Optional[torch.Tensor], draft_tokens: torch.Tensor,
                u_accept: Optional[torch.Tensor], u_final: Optional[torch.Tensor], n_accept: torch.Tensor,
                out_tokens: torch.Tensor, mode: int, ws: Workspace, temperature: float = 1.0, stream=None,
                draft_stats: Optional[torch.Tensor] = None, record=None, top_p: float = 1.0,
                draft_nucleus: Optional[torch.Tensor] = None, target_stats: Optional[torch.Tensor] = None):
    """record: optional (logp [B, k, topk] bfloat16, ids [B, k, topk] int32) for the cycle record;
    top_p < 1: the accept rule on the nuclei of p and q (see gm.h); draft_nucleus: the draft
    rows' nuclei as mtp_draft wrote them (new_nuclei); target_stats: the target rows' statistics
    as verify_forward wrote them."""
    B, k1, V = target_logits.shape
    k = k1 - 1
    _need(target_logits, torch.float32, (B, k1, V), "target_logits")
    if draft_logits is not None:
        _need(draft_logits, torch.float32, (B, k, V), "draft_logits")
    _need(draft_tokens, torch.int32, (B, k), "draft_tokens")
    _need(n_accept, torch.int32, (B,), "n_accept")
    _need(out_tokens, torch.int32, (B, k1), "out_tokens")
    if draft_stats is not None:
        _need(draft_stats, torch.uint8, (B, k, ROW_STATS_BYTES), "draft_stats")
    if draft_nucleus is not None:
        _need(draft_nucleus, torch.uint8, (B, k, NUCLEUS_BYTES), "draft_nucleus")
    if target_stats is not None:
        _need(target_stats, torch.uint8, (B, k1, ROW_STATS_BYTES), "target_stats")
    rec = None
    if record is not None:
        logp, ids = record
        topk = logp.shape[-1] if logp.dim() == 3 else 0
        _need(logp, torch.bfloat16, (B, k, topk), "record logp")
        _need(ids, torch.int32, (B, k, topk), "record ids")
        rec = Record(topk, _ptr(logp), _ptr(ids))
    cfg = ModelConfig()
    cfg.vocab = V
    n = workspace_size(GM_OP_SPEC_ACCEPT, cfg, B, k, 0)
    buf = ws.get(n)
    _check(lib().gm_spec_accept(B, k, V, mode, float(temperature), float(top_p), _ptr(target_logits),
                                _ptr(draft_logits), _ptr(target_stats),
                                _ptr(draft_stats), _ptr(draft_nucleus), _ptr(draft_tokens), _ptr(u_accept), _ptr(u_final), _ptr(n_accept),
                                _ptr(out_tokens), ctypes.byref(rec) if rec is not None else None, _ptr(buf),
                                buf.numel(), _stream(stream)))


def spec_accept_noalloc(target_logits: torch.Tensor, draft_logits: Optional[torch.Tensor], draft_tokens: torch.Tensor,
                        u_accept: Optional[torch.Tensor], u_final: Optional[torch.Tensor], n_accept: torch.Tensor,
                        out_tokens: torch.Tensor, mode: int, temperature: float = 1.0, stream=None,
                        draft_stats: Optional[torch.Tensor] = None, top_p: float = 1.0,
                        target_stats: Optional[torch.Tensor] = None):
    """spec_accept on the library's fixed device scratch (no workspace, nothing allocated)."""
    B, k1, V = target_logits.shape
    k = k1 - 1
    _need(target_logits, torch.float32, (B, k1, V), "target_logits")
    if draft_logits is not None:
        _need(draft_logits, torch.float32, (B, k, V), "draft_logits")
    _need(draft_tokens, torch.int32, (B, k), "draft_tokens")
    _need(n_accept, torch.int32, (B,), "n_accept")
    _need(out_tokens, torch.int32, (B, k1), "out_tokens")
    _check(lib().gm_spec_accept_noalloc(B, k, V, mode, float(temperature), float(top_p), _ptr(target_logits),
                                        _ptr(draft_logits), _ptr(target_stats), _ptr(draft_stats), None,
                                        _ptr(draft_tokens), _ptr(u_accept), _ptr(u_final), _ptr(n_accept),
                                        _ptr(out_tokens), None, _stream(stream)))


def kv_commit(cache: PagedCache, k: int, n_accept: torch.Tensor, committed_slots: Optional[torch.Tensor] = None,
              stream=None):
    cs = cache.struct()
    _check(lib().gm_kv_commit(ctypes.byref(cs), cache.B, k, _ptr(n_accept), _ptr(committed_slots), _stream(stream)))


def mtp_draft(model: DeviceModel, mtp: DeviceMtp, mtp_cache: PagedCache, k: int, mode: int,
              verify_hidden: torch.Tensor, n_accept: torch.Tensor, out_tokens: torch.Tensor,
              u_draft: Optional[torch.Tensor], drafts: torch.Tensor, draft_logits: torch.Tensor, ws: Workspace,
              temperature: float = 1.0, dev_err: Optional[torch.Tensor] = None, stream=None,
              draft_stats: Optional[torch.Tensor] = None, top_p: float = 1.0,
              draft_nucleus: Optional[torch.Tensor] = None):
    """top_p < 1 (sample mode): each draft is drawn from its row's nucleus (see gm.h), written
    to draft_nucleus (new_nuclei) when given."""
    B = mtp_cache.B
    s = model.shape
    _need(verify_hidden, torch.float32, (B, k + 1, s.hidden), "verify_hidden")
    _need(drafts, torch.int32, (B, k), "drafts")
    _need(draft_logits, torch.float32, (B, k, s.vocab), "draft_logits")
    if draft_stats is not None:
        _need(draft_stats, torch.uint8, (B, k, ROW_STATS_BYTES), "draft_stats")
    if draft_nucleus is not None:
        _need(draft_nucleus, torch.uint8, (B, k, NUCLEUS_BYTES), "draft_nucleus")
    cs = mtp_cache.struct()
    n = workspace_size(GM_OP_MTP_DRAFT, model.cfg, B, k, mtp_cache.max_ctx)
    buf = ws.get(n)
    _check(lib().gm_mtp_draft(ctypes.byref(model.cfg), ctypes.byref(mtp.struct), ctypes.byref(model.struct),
                              ctypes.byref(cs), B, k, mode, float(temperature), float(top_p), _ptr(verify_hidden),
                              _ptr(n_accept),
                              _ptr(out_tokens), _ptr(u_draft), _ptr(drafts), _ptr(draft_logits), _ptr(draft_stats), _ptr(draft_nucleus),
                              _ptr(buf),
                              buf.numel(), _ptr(dev_err), _stream(stream)))


def mtp_reconstruct(model: DeviceModel, mtp: DeviceMtp, mtp_cache: PagedCache, K: int,
                    start_hidden: torch.Tensor, start_tokens: torch.Tensor, drafts: Optional[torch.Tensor],
                    head_logits: torch.Tensor, ws: Workspace, dev_err: Optional[torch.Tensor] = None, stream=None):
    """Draft-path reconstruction of mtp_cache.B recorded cycles over K depths (see gm.h)."""
    R = mtp_cache.B
    s = model.shape
    _need(start_hidden, torch.float32, (R, s.hidden), "start_hidden")
    _need(start_tokens, torch.int32, (R,), "start_tokens")
    if drafts is not None:
        _need(drafts, torch.int32, (R, K), "drafts")
    _need(head_logits, torch.float32, (R, K, s.vocab), "head_logits")
    cs = mtp_cache.struct()
    n = workspace_size(GM_OP_MTP_RECONSTRUCT, model.cfg, R, K, mtp_cache.max_ctx)
    buf = ws.get(n)
    _check(lib().gm_mtp_reconstruct(ctypes.byref(model.cfg), ctypes.byref(mtp.struct), ctypes.byref(model.struct),
                                    ctypes.byref(cs), R, K, _ptr(start_hidden), _ptr(start_tokens), _ptr(drafts),
                                    _ptr(head_logits), _ptr(buf), buf.numel(), _ptr(dev_err), _stream(stream)))


def dca_loss(head_logits: torch.Tensor, rec_logp: torch.Tensor, rec_ids: torch.Tensor,
             n_accept: Optional[torch.Tensor], loss: torch.Tensor, alpha: torch.Tensor,
             grad: Optional[torch.Tensor], ws: Workspace, vgm: bool = True, stream=None):
    """DCA loss (with verify-gated masking when vgm) over the cycle record; see gm.h."""
    N, K, V = head_logits.shape
    topk = rec_ids.shape[-1]
    _need(head_logits, torch.float32, (N, K, V), "head_logits")
    _need(rec_logp, torch.bfloat16, (N, K, topk), "rec_logp")
    _need(rec_ids, torch.int32, (N, K, topk), "rec_ids")
    if n_accept is not None:
        _need(n_accept, torch.int32, (N,), "n_accept")
    _need(loss, torch.float32, (N,), "loss")
    _need(alpha, torch.float32, (N, K), "alpha")
    if grad is not None:
        _need(grad, torch.float32, (N, K, V), "grad")
    cfg = ModelConfig()
    cfg.vocab = V
    buf = ws.get(workspace_size(GM_OP_DCA_LOSS, cfg, N, K, 0))
    _check(lib().gm_dca_loss(N, K, V, topk, _ptr(head_logits), _ptr(rec_logp), _ptr(rec_ids), _ptr(n_accept),
                             int(bool(vgm)), _ptr(loss), _ptr(alpha), _ptr(grad), _ptr(buf), buf.numel(),
                             _stream(stream)))


# ------------------------------------------------------------------------ kernel timing
def trace_start(filter_name: Optional[str] = None, every: int = 1):
    """Starts tracing the launches of `filter_name` (all kernels when None), every `every`-th
    matching launch."""
    _check(lib().gm_trace_every(every))
    _check(lib().gm_trace_start(filter_name.encode() if filter_name else None))


def trace_stop() -> Dict[str, tuple]:
    """Stops tracing; returns {kernel name: (launches, total ms)}."""
    _check(lib().gm_trace_stop())
    out = {}
    for i in range(lib().gm_trace_count()):
        name, n, ms = ctypes.c_char_p(), c_int(), c_double()
        _check(lib().gm_trace_get(i, ctypes.byref(name), ctypes.byref(n), ctypes.byref(ms)))
        out[name.value.decode()] = (n.value, ms.value)
    return out
