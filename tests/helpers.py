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



def row_window(z, temperature):
    """The part of the final-draw window that one row of logits contributes (probability units).

    The kernels build each per-id mass from the float32 term expf(y_i - m), y_i = z_i * t with
    t = float32(1 / T) and m the row's max of y, then normalise and sum in float64.  Against
    exp(z_i / T - max) that term carries a relative error eps_i of two kinds:
      * systematic: t differs from 1 / T by |dt| <= 2^-24 / T, which tilts the row like a change
        of temperature; a running sum of p moves by at most |dt| E_p|z - E_p z| under it;
      * rounding: the exponential's own error (taken as 2 ulp) and the rounding of the product
        (none when t = 1) and of the subtraction, |eps_i| <= b_i = 2^-23 + 2^-24 (|y_i| + |y_i - m|).
    The rounding errors of different ids are independent; a bias of the exponential common to all
    terms cancels in the normalisation.  A running sum of p_i eps_i, and the normaliser's own
    relative error, then exceed 6 sqrt(sum_i p_i^2 b_i^2) with probability below 2e-8 each
    (Hoeffding), hence 12 of them.  A row whose mass sits on one id (sqrt(sum p^2) ~ 1) gets a
    window of a few 1e-6; a row spread over 1e5 ids one of ~1e-9."""
    t = np.float32(1.0 / temperature)
    y = (np.asarray(z, dtype=np.float32) * t).astype(np.float64)
    m = y.max(-1, keepdims=True)
    p = np.exp(y - m)
    p /= p.sum(-1, keepdims=True)
    b = 2.0 ** -23 + 2.0 ** -24 * ((0.0 if t == 1 else 1.0) * np.abs(y) + (m - y))
    zz = np.asarray(z, dtype=np.float64)
    mean = (p * zz).sum(-1, keepdims=True)
    tilt = abs(float(t) - 1.0 / temperature) * (p * np.abs(zz - mean)).sum(-1)
    return tilt + 12.0 * np.sqrt((p * p * b * b).sum(-1))


def draw_window(target_logits, draft_logits=None, temperature=1.0, top_p=1.0):
    """Per sequence, the window (probability units) around the edges of the oracle's chosen
    interval inside which the kernel's final draw may differ from the float64 one.

    W_p, W_q: the largest ``row_window`` over the sequence's target and draft rows.  Every
    running sum of the residual max(0, p - q) (a sum over part of the ids of p minus the same of
    q) moves by at most W_p + W_q, and so does u * Z: the distance of u * Z from an edge moves by
    at most 2 (W_p + W_q).  Under top-p the masses are divided by their kept total P >= top_p,
    whose own relative error is within the same sums: the window doubles and is divided by
    top_p.  float64 accumulation adds ~1e-16 per term; 1e-12 is added on top."""
    zt = np.asarray(target_logits)
    B = zt.shape[0]
    out = np.zeros(B)
    for b in range(B):
        w = row_window(zt[b], temperature).max()
        if draft_logits is not None and np.asarray(draft_logits).shape[1]:
            w += row_window(np.asarray(draft_logits)[b], temperature).max()
        out[b] = (2.0 if top_p >= 1.0 else 4.0 / top_p) * w + 1e-12
    return out
