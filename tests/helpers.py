"""Shared set-up of the GPU parity tests: device caches filled from the
oracle's logical KV, comparisons and flags."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2609_16648_amd import gm

CONTRACT = oracle.Rounding("contract")
EXACT = oracle.Rounding("exact")


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gm.lib()          # fails loudly if the HIP library is missing


def rel_err(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-30))


def device_cache(shape, caches, lens, extra: int, page_size: int = 16, seed: int = 0) -> gm.PagedCache:
    """A PagedCache holding the logical prefix entries caches[l] = (K list, V list)."""
    lens = np.asarray(lens)
    cache = gm.PagedCache(shape, len(caches), lens, lens + extra, page_size=page_size, seed=seed)
    for l, (ks, vs) in enumerate(caches):
        for b in range(len(lens)):
            if lens[b]:
                cache.write(l, b, np.arange(lens[b]), ks[b], vs[b])
    return cache


def synth_caches(shape, lens, n_layers):
    out = []
    for l in range(n_layers):
        ks, vs = synth.kv_prefix(shape, lens, l)
        out.append((ks, vs))
    return out


def t32(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


def i32(a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).cuda()


def flag_report(name: str, flagged: np.ndarray, total: int):
    print("[%s] flagged %d of %d" % (name, int(np.sum(flagged)), total), flush=True)
