"""Pins for the oracle's prefix-aligned scoring and tree construction (no GPU).

* Closed form (Sec. 4.2 with Eq. 3 / Appendix A): the best-first tree equals
  the B best prefixes of the fully enumerated candidate tree, in order.
* Objective (Eq. 3): its surrogate mass sum exp(S) is the maximum over every
  prefix-closed set of B nodes (exhaustive, no ranking rule involved).
* lambda = 0 reduces to the marginal surrogate (Eq. 6): exp(S) is the
  product of softmax probabilities, and rho is ignored.
* k = 1 gives the linear chain of the dFlash baseline (Sec. 1).
* Hand-worked fixtures for rho re-ranking and for literal Alg. 2.
* Beam search with global retention (Alg. 1): a literal Python simulation on
  the enumerated candidate tree; with a beam wide enough to hold every node
  it reduces to the B best prefixes of the depths it explored; with width 1
  and one child per node it is the greedy chain.
"""
import json
import os

import numpy as np
import pytest
from scipy.special import softmax

import oracle
from brute import full_tree, max_prefix_mass, paths_of, top_b

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _instance(seed, D, k, quant=True, lam=0.2, with_rho=True):
    rng = np.random.default_rng(seed)
    lp = -rng.exponential(1.5, size=(D, k))
    R = -rng.exponential(2.0, size=(D, k, k, k))
    if quant:
        lp = np.round(lp * 4) / 4
        R = np.round(R * 2) / 2
    R[rng.random(R.shape) < 0.3] = np.log(np.float32(1e-4))
    lp = -np.sort(-lp, axis=1)  # ranks are ordered by log q, as top-k produces them
    ids = np.stack([rng.choice(1000, k, replace=False) for _ in range(D)])
    return (ids.astype(np.int32), lp.astype(np.float32),
            R.astype(np.float32) if with_rho else None, np.full(D, lam, np.float32))


def _build(ids, lp, R, lam, D, k, B, branch=None, mode=oracle.BEST_FIRST, root=7, beam_width=0):
    return oracle.build_tree(ids[None], lp[None], None if R is None else R[None], lam,
                             np.array([root], np.int32), D, k, B, branch=branch, mode=mode,
                             beam_width=beam_width)


def _check_structure(t, ids, s=0):
    n = int(t["n_nodes"][s])
    N = t["parent"].shape[1]
    paths = paths_of(t, s)
    index = {p: i for i, p in enumerate(paths)}
    for i in range(1, n):
        p = paths[i]
        assert t["depth"][s, i] == len(p)
        assert t["parent"][s, i] == index[p[:-1]]
        assert t["token"][s, i] == ids[len(p) - 1, p[-1]]
        bits = [j for j in range(N) if (int(t["anc"][s, i, j // 64]) >> (j % 64)) & 1]
        assert bits == sorted(index[p[:m]] for m in range(len(p) + 1))
    for i in range(n, N):
        assert t["parent"][s, i] == -1 and t["token"][s, i] == -1 and np.isneginf(t["score"][s, i])
        assert not t["anc"][s, i].any()
    return paths


@pytest.mark.parametrize("seed", range(60))
def test_best_first_is_top_b_of_full_tree(seed):
    rng = np.random.default_rng(1000 + seed)
    D, k = int(rng.integers(1, 6)), int(rng.integers(1, 4))
    branch = int(rng.integers(1, k + 1))
    lam = [0.0, 0.2, 1.0][seed % 3]
    ids, lp, R, lamv = _instance(seed, D, k, quant=seed % 2 == 0, lam=lam, with_rho=seed % 5 != 0)
    nodes = full_tree(lp, lamv, R, D, k, branch)
    total = len(nodes) - 1
    for B in sorted({1, 2, max(1, total // 2), total, total + 3}):
        t = _build(ids, lp, R, lamv, D, k, B, branch=branch)
        paths = _check_structure(t, ids)
        want = top_b(nodes, B)
        assert paths[1:] == want
        assert t["n_nodes"][0] == 1 + min(B, total)
        np.testing.assert_array_equal(t["score"][0, 1:1 + len(want)],
                                      np.array([nodes[u] for u in want], np.float32))


@pytest.mark.parametrize("seed", range(25))
def test_prefix_mass_is_maximal(seed):
    rng = np.random.default_rng(5000 + seed)
    D, k = int(rng.integers(2, 4)), 2
    ids, lp, R, lam = _instance(seed + 77, D, k, quant=False)
    nodes = full_tree(lp, lam, R, D, k)
    if len(nodes) - 1 > 14:
        pytest.skip("tree too large for exhaustive subsets")
    for B in range(1, len(nodes)):
        t = _build(ids, lp, R, lam, D, k, B)
        mass = np.exp(t["score"][0, 1:1 + B].astype(np.float64)).sum()
        assert mass == pytest.approx(max_prefix_mass(nodes, B), rel=1e-12)


def test_lambda_zero_is_marginal_product():
    rng = np.random.default_rng(11)
    D, k, V = 4, 3, 50
    logits = rng.standard_normal((D, V)) * 3
    q = softmax(logits.astype(np.float64), axis=1)
    ids = np.argsort(-q, axis=1, kind="stable")[:, :k].astype(np.int32)
    lp = np.log(np.take_along_axis(q, ids, 1)).astype(np.float32)
    garbage = -np.abs(rng.standard_normal((D, k, k, k))).astype(np.float32) * 50
    lam0 = np.zeros(D, np.float32)
    t0 = _build(ids, lp, garbage, lam0, D, k, 20)
    t1 = _build(ids, lp, None, lam0, D, k, 20)
    for key in ("parent", "token", "rank", "score"):
        np.testing.assert_array_equal(t0[key], t1[key])
    for i, p in enumerate(paths_of(t0)):
        prod = np.prod([q[d, ids[d, r]] for d, r in enumerate(p)])
        assert np.exp(np.float64(t0["score"][0, i])) == pytest.approx(prod, rel=1e-5)


def test_k1_is_linear_chain():
    D = 6
    ids, lp, R, lam = _instance(3, D, 1)
    for B in (3, 6, 10):
        t = _build(ids, lp, R, lam, D, 1, B)
        n = min(B, D)
        assert t["n_nodes"][0] == n + 1
        assert t["parent"][0, 1:n + 1].tolist() == list(range(n))
        assert t["token"][0, 1:n + 1].tolist() == ids[:n, 0].tolist()


def _gold_inputs(g):
    D, k = g["depth"], g["k"]
    ids = np.array(g["ids"], np.int32)
    lp = np.array(g["logprob"], np.float32)
    R = np.zeros((D, k, k, k), np.float32)
    for d, a, b, r, v in g.get("rho_nonzero", []):
        R[d, a, b, r] = v
    return ids, lp, R


def test_golden_rho_reranks_tree():
    g = json.load(open(os.path.join(GOLD, "rho_reranks_tree.json")))
    ids, lp, R = _gold_inputs(g)
    for lam, want in g["expected"].items():
        t = _build(ids, lp, R, np.full(g["depth"], float(lam), np.float32), g["depth"], g["k"],
                   g["budget"], root=g["root_token"])
        paths = paths_of(t)
        assert [list(p) for p in paths[1:]] == want["paths"]
        assert t["token"][0, 1:].tolist() == want["tokens"]
        assert t["parent"][0, 1:].tolist() == want["parents"]
        np.testing.assert_allclose(t["score"][0, 1:], want["scores"], atol=1e-6)
        assert t["token"][0, 0] == g["root_token"] and t["parent"][0, 0] == -1


def test_golden_alg2_differs_from_top_b():
    g = json.load(open(os.path.join(GOLD, "alg2_vs_top_b.json")))
    ids, lp, _ = _gold_inputs(g)
    lam = np.zeros(g["depth"], np.float32)
    for mode, want in ((oracle.BEST_FIRST_ALG2, g["expected_alg2"]),
                       (oracle.BEST_FIRST, g["expected_best_first"])):
        t = _build(ids, lp, None, lam, g["depth"], g["k"], g["budget"], mode=mode,
                   root=g["root_token"])
        assert [list(p) for p in paths_of(t)[1:]] == want["paths"]
        assert t["token"][0, 1:].tolist() == want["tokens"]
        assert t["parent"][0, 1:].tolist() == want["parents"]


def _alg2_literal(lp, lam, R, D, k, branch, B):
    nodes = full_tree(lp, lam, R, D, k, branch)
    frontier, T = [()], []
    while len(T) < B and frontier:
        v = min(frontier, key=lambda u: (-float(nodes[u]), u))
        frontier.remove(v)
        kids = [u for u in nodes if len(u) == len(v) + 1 and u[:-1] == v]
        kids.sort(key=lambda u: (-float(nodes[u]), u))
        frontier += kids
        T += kids
    T.sort(key=lambda u: (-float(nodes[u]), u))
    return T[:B], nodes


@pytest.mark.parametrize("seed", range(40))
def test_alg2_literal_and_invariants(seed):
    rng = np.random.default_rng(9000 + seed)
    D, k = int(rng.integers(1, 5)), int(rng.integers(1, 4))
    branch = int(rng.integers(1, k + 1))
    ids, lp, R, lam = _instance(seed + 300, D, k, quant=seed % 2 == 1)
    full = full_tree(lp, lam, R, D, k, branch)
    for B in sorted({1, 2, 3, max(1, (len(full) - 1) // 2), len(full) + 1}):
        want, nodes = _alg2_literal(lp, lam, R, D, k, branch, B)
        t = _build(ids, lp, R, lam, D, k, B, branch=branch, mode=oracle.BEST_FIRST_ALG2)
        paths = _check_structure(t, ids)
        assert paths[1:] == want
        # prefix closed, and never more surrogate mass than the top-B tree
        assert all(len(p) == 1 or p[:-1] in set(paths) for p in paths[1:])
        best = _build(ids, lp, R, lam, D, k, B, branch=branch)
        n = int(t["n_nodes"][0])
        assert n == int(best["n_nodes"][0])
        m_alg2 = np.exp(t["score"][0, 1:n].astype(np.float64)).sum()
        m_best = np.exp(best["score"][0, 1:n].astype(np.float64)).sum()
        assert m_alg2 <= m_best * (1 + 1e-12)


def test_batch_sequences_are_independent():
    D, k, B = 3, 3, 9
    seqs = [_instance(s, D, k) for s in range(4)]
    ids = np.stack([s[0] for s in seqs])
    lp = np.stack([s[1] for s in seqs])
    R = np.stack([s[2] for s in seqs])
    lam = seqs[0][3]
    roots = np.arange(4, dtype=np.int32) + 100
    tb = oracle.build_tree(ids, lp, R, lam, roots, D, k, B)
    for s in range(4):
        t1 = _build(ids[s], lp[s], R[s], lam, D, k, B, root=int(roots[s]))
        for key in ("parent", "token", "rank", "score", "anc", "depth"):
            np.testing.assert_array_equal(tb[key][s], t1[key][0])


def _beam_literal(nodes, D, W, B):
    """Alg. 1 on the enumerated candidate tree: per depth, every beam node's
    children join T; the W best of them (total order) are the next beam."""
    order = lambda u: (-float(nodes[u]), u)
    beam, T = [()], []
    for d in range(1, D + 1):
        if len(T) >= B or not beam:
            break
        kids = [u for u in nodes if len(u) == d and u[:-1] in set(beam)]
        T += kids
        beam = sorted(kids, key=order)[:W]
    return sorted(T, key=order)[:B]


@pytest.mark.parametrize("seed", range(40))
def test_beam_literal_and_invariants(seed):
    rng = np.random.default_rng(7000 + seed)
    D, k = int(rng.integers(1, 6)), int(rng.integers(1, 4))
    branch = int(rng.integers(1, k + 1))
    ids, lp, R, lam = _instance(seed + 500, D, k, quant=seed % 2 == 0,
                                lam=[0.0, 0.2, 1.0][seed % 3])
    nodes = full_tree(lp, lam, R, D, k, branch)
    for W in (1, 2, 3, 5):
        for B in sorted({1, 2, 4, max(1, (len(nodes) - 1) // 2), len(nodes) + 2}):
            want = _beam_literal(nodes, D, W, B)
            t = _build(ids, lp, R, lam, D, k, B, branch=branch, mode=oracle.BEAM, beam_width=W)
            paths = _check_structure(t, ids)
            assert paths[1:] == want
            assert all(len(p) == 1 or p[:-1] in set(paths) for p in paths[1:])
            # never more surrogate mass than the B best prefixes (Eq. 3)
            best = _build(ids, lp, R, lam, D, k, B, branch=branch)
            n = int(t["n_nodes"][0])
            m_beam = np.exp(t["score"][0, 1:n].astype(np.float64)).sum()
            m_best = np.exp(best["score"][0, 1:int(best["n_nodes"][0])].astype(np.float64)).sum()
            assert m_beam <= m_best * (1 + 1e-12)


@pytest.mark.parametrize("seed", range(12))
def test_beam_full_width_is_top_b_of_explored_depths(seed):
    """With a beam that holds every node, T is the whole candidate tree down
    to the first depth at which it reaches B nodes (or D): TopB(T) is then
    the B best prefixes of that depth-truncated tree."""
    rng = np.random.default_rng(7500 + seed)
    D, k = int(rng.integers(1, 6)), int(rng.integers(1, 4))
    ids, lp, R, lam = _instance(seed + 800, D, k)
    nodes = full_tree(lp, lam, R, D, k)
    W = k ** D
    for B in (1, 3, 7, len(nodes) + 1):
        count, stop = 0, 0
        for d in range(1, D + 1):
            if count >= B:
                break
            count += sum(1 for u in nodes if len(u) == d)
            stop = d
        truncated = {u: v for u, v in nodes.items() if len(u) <= stop}
        t = _build(ids, lp, R, lam, D, k, B, mode=oracle.BEAM, beam_width=W)
        assert paths_of(t)[1:] == top_b(truncated, B)


def test_beam_width_one_single_child_is_greedy_chain():
    D, k = 6, 3
    ids, lp, R, lam = _instance(11, D, k)
    t = _build(ids, lp, R, lam, D, k, 10, branch=1, mode=oracle.BEAM, beam_width=1)
    paths = paths_of(t)
    # every node has the best-scoring child of its parent's context
    for i in range(1, len(paths)):
        p = paths[i]
        d = len(p) - 1
        a = p[-3] if len(p) >= 3 else 0
        b = p[-2] if len(p) >= 2 else 0
        from brute import token_score
        s = [token_score(lp, lam, R, d, a, b, r) for r in range(k)]
        assert p[-1] == min(range(k), key=lambda r: (-float(s[r]), r))
    assert [len(p) for p in paths] == list(range(D + 1))


def test_beam_rejects_zero_width():
    D, k = 3, 2
    ids, lp, R, lam = _instance(3, D, k)
    with pytest.raises(ValueError):
        _build(ids, lp, R, lam, D, k, 4, mode=oracle.BEAM, beam_width=0)

