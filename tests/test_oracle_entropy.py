"""Pins for the oracle's entropy-adaptive prefix weight (Appendix F), no GPU.

H_d = -sum_w q_d(w) log q_d(w) is pinned to closed forms (uniform rows give
log V, a one-hot row 0, two-point rows the binary entropy), to the identity
H = LSE - E_q[z] evaluated with scipy's log-sum-exp, and to
scipy.stats.entropy of the softmax.  lambda(H) = beta H / (H + C) is pinned
to its limits and fixed points.  The per-sequence weight of the tree oracle
is pinned by splitting a batch into one-sequence calls.
"""
import numpy as np
import pytest
from scipy.special import logsumexp, softmax
from scipy.stats import entropy as scipy_entropy

import oracle
import synthetic as sy


@pytest.mark.parametrize("V", [1, 2, 37, 1024, 151936])
def test_uniform_row_has_entropy_log_v(V):
    x = np.full((4, V), 3.25, np.float32)
    x[1] = -7.0
    x[2] = -1e30    # offsets fp64 cannot add log V to
    x[3] = 3e20
    h = oracle.entropy(x, "f32")
    np.testing.assert_allclose(h, np.log(V), rtol=1e-12, atol=1e-12)


def test_one_hot_and_empty_rows_have_zero_entropy():
    x = np.full((3, 64), -np.inf, np.float32)
    x[0, 17] = 5.0          # one finite logit: q is a point mass
    x[1, 3] = -1e30         # very negative but finite: still a point mass
    h = oracle.entropy(x, "f32")
    assert h[0] == 0.0 and h[1] == 0.0
    assert h[2] == 0.0      # only -inf: no distribution, defined as 0


@pytest.mark.parametrize("p", [0.5, 0.1, 1e-3, 0.999])
def test_two_point_rows_give_binary_entropy(p):
    x = np.full((1, 16), -np.inf, np.float32)
    x[0, 4] = 0.0
    x[0, 9] = np.float32(np.log(p / (1 - p)))
    pf = 1.0 / (1.0 + np.exp(-np.float64(x[0, 9])))  # the p the fp32 logit encodes
    want = -(pf * np.log(pf) + (1 - pf) * np.log(1 - pf))
    np.testing.assert_allclose(oracle.entropy(x, "f32"), [want], rtol=1e-12)


@pytest.mark.parametrize("dtype,V,scale", [("f32", 1024, 1.0), ("f32", 4099, 6.0),
                                           ("bf16", 151936, 4.0), ("bf16", 257, 30.0)])
def test_entropy_matches_lse_identity_and_scipy(dtype, V, scale):
    rng = np.random.default_rng([11, V])
    x = (rng.standard_normal((5, V)) * scale).astype(np.float32)
    x[2, ::5] = -np.inf                 # zero-probability entries contribute nothing
    x[3] = np.round(x[3])               # many equal logits
    store = sy.cast(x, dtype)
    xf = sy.as_f32(store, dtype).astype(np.float64)
    h = oracle.entropy(store, dtype)
    # H = log Z - sum_w q(w) z(w): a different arrangement of the same sum
    lse = logsumexp(xf, axis=1)
    qz = np.array([np.sum(softmax(r)[np.isfinite(r)] * r[np.isfinite(r)]) for r in xf])
    np.testing.assert_allclose(h, lse - qz, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(h, scipy_entropy(softmax(xf, axis=1), axis=1), rtol=1e-10,
                               atol=1e-12)
    assert np.all(h >= 0) and np.all(h <= np.log(V) + 1e-12)


def test_entropy_lambda_limits_and_fixed_points():
    beta, c = 0.7, 1.5
    h = np.array([0.0, c, 3 * c, 1e30, 1e-300])
    lam = oracle.entropy_lambda(h, beta, c)
    assert lam[0] == 0.0                      # a certain drafter: no prefix correction
    assert lam[1] == pytest.approx(beta / 2, rel=1e-15)
    assert lam[2] == pytest.approx(beta * 3 / 4, rel=1e-15)
    assert lam[3] == pytest.approx(beta, rel=1e-15)   # bounded by beta
    assert 0 < lam[4] < 1e-299
    grid = np.linspace(0, 12, 1001)
    assert np.all(np.diff(oracle.entropy_lambda(grid, beta, c)) > 0)  # increasing in H


def test_per_sequence_lambda_equals_one_sequence_calls():
    w = sy.workload(1, batch=4, budget=24)
    rin = sy.round_inputs(w)
    ids, lp, _, _ = oracle.topk(rin["drafter_logits"], w.k, w.dtype)
    ids = ids.reshape(w.batch, w.depth, w.k)
    lp = lp.reshape(w.batch, w.depth, w.k)
    rho = rin["rho"]
    rng = np.random.default_rng(5)
    lam2 = rng.uniform(0, 2, (w.batch, w.depth)).astype(np.float32)
    lam2[1] = 0.0                                   # one sequence without the prefix term
    full = oracle.build_tree(ids, lp, rho, lam2, rin["root_token"], w.depth, w.k, w.budget)
    for b in range(w.batch):
        one = oracle.build_tree(ids[b:b + 1], lp[b:b + 1], rho[b:b + 1], lam2[b],
                                rin["root_token"][b:b + 1], w.depth, w.k, w.budget)
        for key in one:
            np.testing.assert_array_equal(full[key][b], one[key][0], err_msg=f"{key} b={b}")
    # a zero weight is the same as no lattice at all
    plain = oracle.build_tree(ids[1:2], lp[1:2], None, lam2[1], rin["root_token"][1:2], w.depth,
                              w.k, w.budget)
    for key in plain:
        np.testing.assert_array_equal(full[key][1], plain[key][0], err_msg=key)
