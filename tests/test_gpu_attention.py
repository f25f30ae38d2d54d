"""GPU parity of gm_verify_attention against the oracle's grouped causal
attention on the same seeded Q and KV (bf16 within 2e-2 relative error,
float32 within 1e-4), across ragged contexts, block lengths and page sizes."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import need_gpu, rel_err, t32, i32
from paper_2609_16648_amd import gm

pytestmark = pytest.mark.gpu


def _case(shape, lens, k, page_size, seed):
    B, R = len(lens), k + 1
    ctx = np.asarray(lens) + R
    ks, vs = synth.kv_prefix(shape, ctx, layer=seed, seed=2)
    q = synth.normal_tensor((B, R, shape.n_heads, shape.head_dim), 5, shape.dtype, "q", seed)
    cache = gm.PagedCache(shape, 1, lens, ctx, page_size=page_size, seed=seed, fill="empty")
    for b in range(B):
        cache.write(0, b, np.arange(ctx[b]), ks[b], vs[b])
    dt = gm.torch_dtype(shape)
    qd = t32(q, dt)
    out = torch.empty_like(qd)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    gm.verify_attention(gm.model_config(shape), cache, 0, qd, out, gm.Workspace(), err)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    ref = np.stack([oracle.attention(q[b].astype(np.float64), ks[b].astype(np.float64), vs[b].astype(np.float64),
                                     lens[b] + np.arange(R) + 1) for b in range(B)])
    assert int(err.item()) == 0
    return got, ref, cache


@pytest.mark.parametrize("lens,k,page_size", [
    ([1, 15, 16, 17, 100, 1023, 2500, 4096], 3, 16),
    ([5, 333, 2049, 4000], 3, 64),
    ([7, 300, 3001], 0, 16),
    ([1, 64, 1000], 15, 32),
    ([0, 3, 40], 1, 16),
])
def test_bf16_attention_matches_oracle(lens, k, page_size):
    need_gpu()
    shape = synth.QWEN3_4B_LAYER
    got, ref, _ = _case(shape, np.array(lens), k, page_size, seed=len(lens) + k)
    e = rel_err(got, ref)
    print("[attention bf16 k=%d] rel err %.3e" % (k, e), flush=True)
    assert e < 2e-2
    # the only bf16 rounding left is the output's: agreement to one bf16 step
    assert np.abs(got - oracle.round_bf16(ref)).max() <= 2.0 ** -7 * np.abs(ref).max()


def test_bf16_attention_long_context():
    need_gpu()
    shape = synth.QWEN3_4B_LAYER
    lens = synth.context_lengths(synth.WORKLOADS["long_ctx"])[:3]
    got, ref, _ = _case(shape, lens, 7, 16, seed=11)
    e = rel_err(got, ref)
    print("[attention bf16 long] lens %s rel err %.3e" % (list(lens), e), flush=True)
    assert e < 2e-2


def test_f32_attention_matches_oracle():
    need_gpu()
    shape = synth.TINY
    got, ref, _ = _case(shape, np.array([1, 20, 128, 131]), 3, 16, seed=4)
    e = rel_err(got, ref)
    print("[attention f32] rel err %.3e" % e, flush=True)
    assert e < 1e-4


def test_gqa_group_of_eight_and_odd_rows():
    # 32 query heads on 4 KV heads with k = 2: 24 rows in two 16-row tiles
    need_gpu()
    shape = dataclasses.replace(synth.QWEN3_4B_LAYER, n_kv_heads=4)
    got, ref, _ = _case(shape, np.array([9, 700, 1600]), 2, 16, seed=21)
    assert rel_err(got, ref) < 2e-2


def test_bad_page_sets_device_error():
    need_gpu()
    shape = synth.QWEN3_4B_LAYER
    lens = np.array([40, 40])
    cache = gm.PagedCache(shape, 1, lens, lens + 4, page_size=16, seed=1)
    bt = cache.block_table_host.copy()
    bt[1, 1] = -1                                  # a hole inside sequence 1's context
    cache.block_table.copy_(torch.from_numpy(bt))
    q = torch.zeros((2, 4, shape.n_heads, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    gm.verify_attention(gm.model_config(shape), cache, 0, q, out, gm.Workspace(), err)
    torch.cuda.synchronize()
    assert int(err.item()) & gm.GM_DEVERR_PAGE
    assert torch.isfinite(out.float()).all()
