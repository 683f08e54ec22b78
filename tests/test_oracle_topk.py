"""Pins for the oracle's log-softmax + top-k stage (no GPU).

The top-k set and order are checked against NumPy's full stable sort of the
row (value descending, id ascending); log q against scipy's fp64
log-sum-exp.  bf16 rows at Qwen3 vocabulary size have frequent ties, so
the id tie-break is exercised.
"""
import numpy as np
import pytest
from scipy.special import logsumexp

import oracle
import synthetic as sy


def _ref(rows_f32, k):
    ids, lp = [], []
    for row in rows_f32:
        order = np.lexsort((np.arange(row.size), -row.astype(np.float64)))[:k]
        l = logsumexp(row.astype(np.float64))
        ids.append(order)
        lp.append(row[order].astype(np.float64) - l)
    return np.array(ids), np.array(lp)


@pytest.mark.parametrize("dtype,V,k", [("f32", 1024, 2), ("bf16", 151936, 4), ("bf16", 151936, 16),
                                       ("bf16", 4099, 8), ("f32", 37, 37)])
def test_topk_matches_full_sort(dtype, V, k):
    rng = np.random.default_rng([7, V, k])
    x = (rng.standard_normal((6, V), dtype=np.float32) * 4).astype(np.float32)
    x[1, rng.choice(V, 3, replace=False)] = x[1].max() + 8  # tied planted peaks
    x[2, :] = np.round(x[2])                                 # heavy ties
    x[3, ::3] = -np.inf
    store = sy.cast(x, dtype)
    ids, lp, lse, nan_rows = oracle.topk(store, k, dtype)
    xf = sy.as_f32(store, dtype)
    rid, rlp = _ref(xf, k)
    assert nan_rows == 0
    np.testing.assert_array_equal(ids, rid)
    np.testing.assert_allclose(lp, rlp, rtol=0, atol=1e-6 * np.maximum(1, np.abs(rlp)).max())
    np.testing.assert_allclose(lse, logsumexp(xf.astype(np.float64), axis=1), rtol=1e-7)


def test_topk_negative_zero_ties_positive_zero():
    x = np.zeros((1, 8), np.float32)
    x[0, 2] = -0.0
    x[0, 5] = 1.0
    ids, lp, lse, _ = oracle.topk(x, 3, "f32")
    assert ids.tolist() == [[5, 0, 1]]


@pytest.mark.parametrize("offset", [-1e30, -3e8, 1e20, 300.0])
def test_topk_constant_row_far_from_zero(offset):
    """A constant row is uniform whatever its offset: log q = -log V exactly,
    even where fp64 cannot hold offset + log V."""
    V = 1000
    x = np.full((1, V), offset, np.float32)
    ids, lp, lse, _ = oracle.topk(x, 3, "f32")
    assert ids.tolist() == [[0, 1, 2]]
    np.testing.assert_array_equal(lp, np.float32(-np.log(V)))


def test_topk_all_neg_inf_row():
    x = np.full((1, 16), -np.inf, np.float32)
    ids, lp, lse, _ = oracle.topk(x, 2, "f32")
    assert ids.tolist() == [[0, 1]]
    assert np.all(np.isneginf(lp)) and np.isneginf(lse[0])


def test_topk_nan_is_flagged():
    x = np.zeros((3, 16), np.float32)
    x[1, 4] = np.nan
    *_, nan_rows = oracle.topk(x, 2, "f32")
    assert nan_rows == 1


def test_threads_do_not_change_results():
    rng = np.random.default_rng(3)
    x = sy.to_bf16_bits(rng.standard_normal((32, 5000), dtype=np.float32) * 4)
    oracle.set_threads(1)
    a = oracle.topk(x, 8, "bf16")
    oracle.set_threads(4)
    b = oracle.topk(x, 8, "bf16")
    for u, v in zip(a[:3], b[:3]):
        np.testing.assert_array_equal(u, v)
