"""Pins of the oracle's cycle-record capture (App. "Implementing Draft-Path
Reconstruction in verl": the target's top-64 log-probabilities per draft
position, full-vocabulary normalised, stored in bf16)."""
import math

import numpy as np
import pytest
import torch

import oracle


def _brute(row, T, topk):
    """A full sort by (decreasing logit, increasing id) and math.fsum's log-sum-exp."""
    order = sorted(range(len(row)), key=lambda x: (-float(row[x]), x))[:topk]
    s = [float(v) / T for v in row]
    m = max(s)
    lse = m + math.log(math.fsum(math.exp(v - m) for v in s))
    lp = torch.tensor([s[x] - lse for x in order], dtype=torch.float64).to(torch.float32).to(torch.bfloat16)
    return order, lp.to(torch.float64).numpy()


@pytest.mark.parametrize("V,topk,T", [(40, 8, 1.0), (300, 64, 1.0), (300, 64, 0.7), (64, 64, 1.0)])
def test_record_matches_brute_force(V, topk, T):
    g = np.random.default_rng(V + topk)
    z = g.standard_normal((3, 4, V)).astype(np.float32) * 2
    ids, logp = oracle.record_topk(z, 3, T, topk)
    for b in range(3):
        for i in range(3):
            order, lp = _brute(z[b, i], T, topk)
            assert list(ids[b, i]) == order
            np.testing.assert_array_equal(logp[b, i], lp)


def test_record_reads_the_rows_that_verify_the_drafts():
    # block rows 0..k-1 verify d_1..d_k; row k (the bonus row) is not recorded
    z = np.zeros((1, 3, 10), dtype=np.float32)
    z[0, 0, 7] = 5
    z[0, 1, 2] = 5
    z[0, 2, 9] = 5
    ids, _ = oracle.record_topk(z, 2, 1.0, 1)
    assert ids[0, :, 0].tolist() == [7, 2]


def test_record_keeps_full_vocabulary_normalisation():
    # kept mass is below one when the vocabulary is larger than the record, one when it is not
    g = np.random.default_rng(5)
    z = g.standard_normal((1, 2, 200)).astype(np.float32)
    _, lp = oracle.record_topk(z, 1, 1.0, 64)
    kept = np.exp(lp[0, 0]).sum()
    p = oracle.softmax(z[0, 0].astype(np.float64))
    assert kept < 0.99 and abs(kept - np.sort(p)[::-1][:64].sum()) < 64 * 2 ** -8
    _, lp_all = oracle.record_topk(z[:, :, :64], 1, 1.0, 64)
    assert abs(np.exp(lp_all[0, 0]).sum() - 1) < 64 * 2 ** -8


def test_record_ties_go_to_lower_ids_and_order_is_descending():
    z = np.zeros((1, 2, 50), dtype=np.float32)
    z[0, 0, [3, 17, 40]] = 2.0          # a three-way tie at the top
    z[0, 0, [10, 20]] = 1.0
    ids, lp = oracle.record_topk(z, 1, 1.0, 6)
    assert ids[0, 0].tolist() == [3, 17, 40, 10, 20, 0]
    assert np.all(np.diff(lp[0, 0]) <= 0)


def test_record_temperature_scales_the_logits():
    g = np.random.default_rng(9)
    z = g.standard_normal((2, 3, 128)).astype(np.float32)
    i1, l1 = oracle.record_topk(z, 2, 0.5, 16)
    i2, l2 = oracle.record_topk((2 * z.astype(np.float64)).astype(np.float32), 2, 1.0, 16)
    np.testing.assert_array_equal(i1, i2)
    np.testing.assert_array_equal(l1, l2)
