"""Seeded synthetic inputs for the speculative rollout step.

This module is shared by the CPU oracle's tests, the GPU tests and the
benchmark.  It holds random draws and storage-format quantisation only: no
arithmetic of the method (no norm, projection, attention, softmax or
acceptance step) lives here.

The paper trains on rollouts of real checkpoints over DAPO-Math-17K /
TACO-Verified prompts (Section 4 setup; App. "RL Training Configuration").
Neither the datasets nor the weights exist here, so every workload below is a
random-init model with the shapes of the paper's backbones and the paper's
sampling settings (temperature 1.0, top-p 1.0), with the recipes:

* every linear weight N(0, 0.02) and every RMSNorm weight 1, the draft-head
  initialisation of App. "Models and Draft Heads" (seed 0);
* context lengths and token ids uniform (seed 1);
* prefix K/V entries N(0, 1) (seed 2);
* draft logits N(0, 1) and the draft-mixing draws (seed 3);
* the uniforms consumed by the accept rule and by sampling (seed 4).

Every tensor is drawn from its own PCG64 stream keyed by (seed, name), so the
value of one tensor does not depend on which other tensors were drawn.
"""
from __future__ import annotations

import dataclasses
import zlib
from typing import Dict, List, Optional

import numpy as np

SEED_WEIGHTS = 0
SEED_TOKENS = 1
SEED_KV = 2
SEED_DRAFT = 3
SEED_UNIFORM = 4


# --------------------------------------------------------------------------
# random streams and storage quantisation
# --------------------------------------------------------------------------
def stream(seed: int, *tags) -> np.random.Generator:
    """A PCG64 generator keyed by an integer seed and a tuple of tags."""
    key = [int(seed)] + [zlib.crc32(str(t).encode()) for t in tags]
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even.

    Storage conversion for synthetic tensors (inputs are finite)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return ((b + bias) >> np.uint32(16)).astype(np.uint16)


def bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def quantise(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round a float32 array to the storage dtype, returned as float32."""
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return bits_to_f32(bf16_bits(x))
    raise ValueError(dtype)


# --------------------------------------------------------------------------
# model shapes and workloads
# --------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class ModelShape:
    n_layers: int
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    dtype: str = "bf16"          # storage dtype of weights and KV: "f32" | "bf16"
    qk_norm: bool = False
    tie_embed: bool = False


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    batch: int
    k: int
    ctx_lo: int                  # committed prefix length m_b ~ U{ctx_lo..ctx_hi}
    ctx_hi: int
    mix_prob: Optional[float]    # draft = target top-1 with this probability (None: not mixing)
    with_mtp: bool = False
    page_size: int = 16


TINY = ModelShape(n_layers=2, hidden=256, n_heads=4, n_kv_heads=4, head_dim=64,
                  ffn=1024, vocab=1024, dtype="f32")
QWEN3_4B_LAYER = ModelShape(n_layers=1, hidden=2560, n_heads=32, n_kv_heads=8,
                            head_dim=128, ffn=9728, vocab=151936)
QWEN3_4B = dataclasses.replace(QWEN3_4B_LAYER, n_layers=36)
MIMO_7B = ModelShape(n_layers=36, hidden=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                     ffn=11008, vocab=151680)

WORKLOADS: Dict[str, Workload] = {
    # tiny fp32 decoder, 128-token prefill, k=3 uniform drafts
    "tiny": Workload("tiny", TINY, batch=4, k=3, ctx_lo=128, ctx_hi=128, mix_prob=None),
    # one Qwen3-4B-shaped layer + LM head, 64 sequences, contexts 1K..4K, 0.7 top-1 mixing
    "qwen3_4b_layer": Workload("qwen3_4b_layer", QWEN3_4B_LAYER, batch=64, k=3,
                               ctx_lo=1024, ctx_hi=4096, mix_prob=0.7, with_mtp=True),
    # full 36-layer Qwen3-4B shape, 256 rollouts of 512 + U{0..8192} tokens, MTP chain drafts
    "qwen3_4b_full": Workload("qwen3_4b_full", QWEN3_4B, batch=256, k=3,
                              ctx_lo=512, ctx_hi=512 + 8192, mix_prob=None, with_mtp=True),
    # MiMo-7B shape, 128 rollouts of 2K..16K tokens, k=1, 0.5 top-1 mixing
    "mimo_7b": Workload("mimo_7b", MIMO_7B, batch=128, k=1, ctx_lo=2048, ctx_hi=16384,
                        mix_prob=0.5, with_mtp=True),
    # the qwen3_4b_layer workload at the depth study's deepest chain (k=7)
    "qwen3_4b_layer_k7": Workload("qwen3_4b_layer_k7", QWEN3_4B_LAYER, batch=64, k=7,
                                  ctx_lo=1024, ctx_hi=4096, mix_prob=0.7, with_mtp=True),
    # long-context attention + accept stress, 32 sequences of 16K..32K, k=7
    "long_ctx": Workload("long_ctx", QWEN3_4B_LAYER, batch=32, k=7, ctx_lo=16384,
                         ctx_hi=32768, mix_prob=None),
}


# --------------------------------------------------------------------------
# weights
# --------------------------------------------------------------------------
def _linear(seed, name, rows, cols, dtype):
    w = stream(seed, name).standard_normal((rows, cols), dtype=np.float32)
    w *= np.float32(0.02)
    return quantise(w, dtype)


def _ones(n, dtype):
    return quantise(np.ones(n, np.float32), dtype)


def layer_weights(s: ModelShape, seed: int, prefix: str) -> Dict[str, np.ndarray]:
    H, d = s.hidden, s.head_dim
    w = {
        "attn_norm": _ones(H, s.dtype),
        "wq": _linear(seed, prefix + "wq", s.n_heads * d, H, s.dtype),
        "wk": _linear(seed, prefix + "wk", s.n_kv_heads * d, H, s.dtype),
        "wv": _linear(seed, prefix + "wv", s.n_kv_heads * d, H, s.dtype),
        "wo": _linear(seed, prefix + "wo", H, s.n_heads * d, s.dtype),
        "ffn_norm": _ones(H, s.dtype),
        "w_gate": _linear(seed, prefix + "w_gate", s.ffn, H, s.dtype),
        "w_up": _linear(seed, prefix + "w_up", s.ffn, H, s.dtype),
        "w_down": _linear(seed, prefix + "w_down", H, s.ffn, s.dtype),
    }
    if s.qk_norm:
        w["q_norm"] = _ones(d, s.dtype)
        w["k_norm"] = _ones(d, s.dtype)
    return w


def model_weights(s: ModelShape, seed: int = SEED_WEIGHTS, threads: int = 1) -> Dict[str, object]:
    """Backbone weights, all row-major [out, in] as nn.Linear stores them.

    threads > 1 draws the tensors concurrently; every tensor has its own
    stream, so the values do not depend on it."""
    def job(i):
        if i == s.n_layers:
            return _linear(seed, "embed", s.vocab, s.hidden, s.dtype)
        if i == s.n_layers + 1:
            return None if s.tie_embed else _linear(seed, "lm_head", s.vocab, s.hidden, s.dtype)
        return layer_weights(s, seed, "layer%d." % i)
    if threads > 1:
        import concurrent.futures
        with concurrent.futures.ThreadPoolExecutor(threads) as ex:
            parts = list(ex.map(job, range(s.n_layers + 2)))
    else:
        parts = [job(i) for i in range(s.n_layers + 2)]
    w: Dict[str, object] = {
        "embed": parts[s.n_layers],
        "final_norm": _ones(s.hidden, s.dtype),
        "layers": parts[:s.n_layers],
    }
    w["lm_head"] = w["embed"] if s.tie_embed else parts[s.n_layers + 1]
    return w


def mtp_weights(s: ModelShape, seed: int = SEED_WEIGHTS) -> Dict[str, object]:
    """Draft-head weights: two input RMSNorms, the bias-free 2H -> H projection,
    one decoder layer of the backbone's shape and a final RMSNorm."""
    H = s.hidden
    return {
        "norm_h": _ones(H, s.dtype),
        "norm_e": _ones(H, s.dtype),
        "w_proj": _linear(seed, "mtp.w_proj", H, 2 * H, s.dtype),
        "final_norm": _ones(H, s.dtype),
        "layer": layer_weights(s, seed, "mtp.layer."),
    }


# --------------------------------------------------------------------------
# sequences, KV contents, logits and uniforms
# --------------------------------------------------------------------------
def context_lengths(w: Workload, seed: int = SEED_TOKENS) -> np.ndarray:
    return stream(seed, w.name, "ctx").integers(w.ctx_lo, w.ctx_hi + 1, size=w.batch).astype(np.int32)


def token_ids(n, vocab, seed: int, *tags) -> np.ndarray:
    return stream(seed, "tokens", *tags).integers(0, vocab, size=n).astype(np.int32)


def kv_prefix(shape: ModelShape, lens: np.ndarray, layer: int, seed: int = SEED_KV,
              seqs: Optional[List[int]] = None):
    """N(0,1) K and V entries of the committed prefix of each sequence.

    Returns two lists (K, V) of float32 arrays [m_b, n_kv, head_dim], values
    exact in the storage dtype."""
    ks, vs = [], []
    for b in (range(len(lens)) if seqs is None else seqs):
        shp = (int(lens[b]), shape.n_kv_heads, shape.head_dim)
        ks.append(quantise(stream(seed, "k", layer, b).standard_normal(shp, dtype=np.float32), shape.dtype))
        vs.append(quantise(stream(seed, "v", layer, b).standard_normal(shp, dtype=np.float32), shape.dtype))
    return ks, vs


def normal_logits(shape, seed: int, *tags) -> np.ndarray:
    return stream(seed, "logits", *tags).standard_normal(shape, dtype=np.float32)


def normal_tensor(shape, seed: int, dtype: str, *tags) -> np.ndarray:
    return quantise(stream(seed, "normal", *tags).standard_normal(shape, dtype=np.float32), dtype)


def uniforms(batch: int, k: int, seed: int = SEED_UNIFORM, *tags):
    """u_accept [B,k], u_final [B], u_draft [B,k]: float32 in [0, 1)."""
    g = stream(seed, "uniform", *tags)
    u_accept = g.random((batch, k), dtype=np.float32)
    u_final = g.random(batch, dtype=np.float32)
    u_draft = g.random((batch, k), dtype=np.float32)
    return u_accept, u_final, u_draft


def mixing_draws(batch: int, k: int, vocab: int, prob: float, seed: int = SEED_DRAFT, *tags):
    """The random part of the top-1 mixing draft rule: per position, whether the
    draft takes the target's top-1 token (probability `prob`), and the uniform
    token used otherwise."""
    g = stream(seed, "mixing", *tags)
    take_top1 = g.random((batch, k)) < prob
    alt = g.integers(0, vocab, size=(batch, k)).astype(np.int32)
    return take_top1, alt
