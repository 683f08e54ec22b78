"""Pins for the oracle's greedy acceptance walk (no GPU).

* Brute force (Eq. 1 at temperature 0): every root-to-node path is checked
  token by token against np.argmax of its parent's target logits; the
  longest accepted path wins and the bonus is the prediction after it.
* Position-wise coverage (Observation 1): with a complete candidate tree and
  target predictions that depend only on depth, the accepted length is the
  longest run of depths whose predicted token is among that depth's
  candidates.
* The symbolic example of Appendix C (D->E, D->F->G, F accepted).
"""
import json
import os

import numpy as np
import pytest

import oracle
import synthetic as sy
from brute import brute_accept

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _tree_with_distinct_siblings(rng, N, V, depth_cap):
    parent = np.full(N, -1, np.int32)
    token = np.full(N, -1, np.int32)
    depth = np.zeros(N, np.int32)
    token[0] = rng.integers(V)
    used = {0: set()}
    for n in range(1, N):
        while True:
            p = int(rng.integers(0, n))
            if depth[p] < depth_cap:
                break
        t = int(rng.integers(V))
        while t in used[p]:
            t = int(rng.integers(V))
        used[p].add(t)
        used[n] = set()
        parent[n], token[n], depth[n] = p, t, depth[p] + 1
    return parent, token, depth


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seed", range(12))
def test_accept_matches_brute_force(dtype, seed):
    rng = np.random.default_rng([seed, 17])
    b, N, V, D = 3, 24, 40, 6
    parents, tokens, nn = [], [], []
    T = rng.standard_normal((b, N, V), dtype=np.float32)
    for s in range(b):
        p, t, dep = _tree_with_distinct_siblings(rng, N, V, D)
        n_live = N if s == 0 else int(rng.integers(1, N + 1))
        p[n_live:] = -1
        t[n_live:] = -1
        # make the target agree with one child most of the time
        for n in range(n_live):
            kids = [c for c in range(1, n_live) if p[c] == n]
            if kids and rng.random() < 0.8:
                T[s, n, t[rng.choice(kids)]] = 10.0
        if seed % 3 == 0:
            T[s, :, :5] = np.round(T[s, :, :5])  # ties among low ids
        parents.append(p)
        tokens.append(t)
        nn.append(n_live)
    parent, token, n_nodes = np.stack(parents), np.stack(tokens), np.array(nn, np.int32)
    store = sy.cast(T, dtype)
    r = oracle.accept(dtype, store, parent, token, n_nodes, D)
    Tf = sy.as_f32(store, dtype)
    for s in range(b):
        L, chain, bonus, a = brute_accept(Tf, parent, token, n_nodes, s)
        assert r["accept_len"][s] == L
        assert r["path"][s].tolist() == chain + [-1] * (D + 1 - len(chain))
        assert r["bonus"][s] == bonus
        assert r["target_argmax"][s, :n_nodes[s]].tolist() == a
        assert (r["target_argmax"][s, n_nodes[s]:] == -1).all()
    assert r["nan_rows"] == 0


def test_complete_tree_accepts_the_coverage_length():
    rng = np.random.default_rng(4)
    D, k, V = 4, 2, 30
    ids = np.stack([rng.choice(V, k, replace=False) for _ in range(D)]).astype(np.int32)
    lp = np.log(np.full((D, k), 0.3, np.float32))
    full = sum(k ** d for d in range(1, D + 1))
    t = oracle.build_tree(ids[None], lp[None], None, np.zeros(D, np.float32),
                          np.array([1], np.int32), D, k, full)
    depth = t["depth"][0]
    for trial in range(20):
        # prediction at depth delta is a fixed token per depth (position-wise)
        pred = [int(ids[d, rng.integers(k)]) if rng.random() < 0.75 else int(rng.integers(V))
                for d in range(D)] + [int(rng.integers(V))]
        T = np.zeros((1, full + 1, V), np.float32)
        for n in range(full + 1):
            T[0, n, pred[min(depth[n], D)]] = 1.0
        r = oracle.accept("f32", T, t["parent"], t["token"], t["n_nodes"], D)
        cover = 0
        while cover < D and pred[cover] in ids[cover]:
            cover += 1
        assert r["accept_len"][0] == cover
        assert r["bonus"][0] == pred[cover]


def test_golden_fig3():
    g = json.load(open(os.path.join(GOLD, "fig3_accept.json")))
    N, V = len(g["parent"]), g["vocab"]
    T = np.zeros((1, N, V), np.float32)
    for n, a in enumerate(g["target_argmax_per_node"]):
        T[0, n, a] = 1.0
    r = oracle.accept("f32", T, np.array([g["parent"]], np.int32), np.array([g["token"]], np.int32),
                      np.array([N], np.int32), g["depth"])
    assert r["accept_len"][0] == g["expected"]["accept_len"]
    assert r["path"][0].tolist() == g["expected"]["path"]
    assert r["bonus"][0] == g["expected"]["bonus"]


def test_nan_is_flagged():
    T = np.zeros((1, 3, 8), np.float32)
    T[0, 1, 2] = np.nan
    r = oracle.accept("f32", T, np.array([[-1, 0, 0]], np.int32), np.array([[1, 2, 3]], np.int32),
                      np.array([3], np.int32), 1)
    assert r["nan_rows"] == 1
