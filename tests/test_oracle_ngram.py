"""Pins for the oracle's n-gram lattice gather (Sec. 5.1: rho is a trigram
model; Eq. 9 reads log rho(t | two preceding path tokens)), no GPU.

* a hand-worked fixture (tests/golden/ngram_gather_small.json);
* a path walk: for every node of the candidate tree, the two tokens before
  it are read off its rank path and looked up by a linear scan of the raw
  entries, which must equal the lattice slot the tree stage reads;
* end to end: the oracle tree built from the gathered lattice equals the
  B best prefixes of a candidate tree scored straight from path tokens.
"""
import json
import os

import numpy as np
import pytest

import brute
import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _scan(entries, a, b, c, floor):
    """log rho of (a, b, c) by a linear scan: the largest valid value given."""
    best = None
    for t2, t1, t, v in entries:
        if (t2, t1, t) == (a, b, c) and np.isfinite(v) and v <= 0 and \
                all(0 <= x < oracle.NGRAM_TOKEN_LIMIT for x in (t2, t1, t)):
            best = v if best is None else max(best, v)
    return np.float32(floor if best is None else best)


def _unzip(entries):
    e = list(zip(*entries))
    return (np.array(e[0], np.int64), np.array(e[1], np.int64), np.array(e[2], np.int64),
            np.array(e[3], np.float32))


def test_ngram_golden_fixture():
    g = json.load(open(os.path.join(GOLD, "ngram_gather_small.json")))
    table = oracle.ngram_table(*_unzip(g["entries"]))
    ids = np.array([g["ids"]], np.int32)
    lat = oracle.ngram_lattice(table, g["floor"], ids, [g["prev_token"]], [g["root_token"]])[0]
    exp = g["expected_by_depth"]
    for r2 in range(2):
        for r1 in range(2):
            np.testing.assert_array_equal(lat[0, r2, r1], np.float32(exp["0"]["any_r2_r1"]))
        np.testing.assert_array_equal(lat[1, r2], np.float32(exp["1"]["any_r2"]))
    np.testing.assert_array_equal(lat[2], np.float32(exp["2"]))


def _random_case(seed, B, D, k, vocab=40, n_entries=600):
    rng = np.random.default_rng(seed)
    ids = np.stack([[rng.choice(vocab, k, replace=False) for _ in range(D)] for _ in range(B)])
    prev = rng.integers(-1, vocab, B)
    root = rng.integers(0, vocab, B)
    t2, t1, t = (rng.integers(0, vocab, n_entries) for _ in range(3))
    v = np.log(rng.uniform(1e-3, 1.0, n_entries)).astype(np.float32)
    v[::17] = 0.0
    v[::23] = -0.0
    v[5::31] = 0.25                   # invalid: positive
    t[7::29] = 1 << 21                # invalid: token out of range
    entries = list(zip(t2.tolist(), t1.tolist(), t.tolist(), v.tolist()))
    entries += entries[::5]           # duplicates
    return ids.astype(np.int32), prev, root, entries


@pytest.mark.parametrize("B,D,k", [(1, 1, 1), (2, 3, 2), (3, 5, 3), (1, 4, 4)])
def test_ngram_lattice_matches_path_walk(B, D, k):
    ids, prev, root, entries = _random_case([B, D, k], B, D, k)
    floor = np.float32(np.log(1e-4))
    lat = oracle.ngram_lattice(oracle.ngram_table(*_unzip(entries)), floor, ids, prev, root)
    for b in range(B):
        nodes = brute.full_tree(np.zeros((D, k), np.float32), None, None, D, k)
        for u in nodes:
            if not u:
                continue
            d = len(u) - 1                      # the node reads drafter row d
            toks = [int(prev[b]), int(root[b])] + [int(ids[b, i, r]) for i, r in enumerate(u)]
            want = _scan(entries, toks[-3], toks[-2], toks[-1], floor)
            r1 = u[-2] if d >= 1 else 0         # rank of the parent (0: outside the block)
            r2 = u[-3] if d >= 2 else 0         # rank of the grandparent
            got = lat[b, d, r2, r1, u[-1]]
            assert got.view(np.uint32) == want.view(np.uint32), (b, u)


def test_ngram_tree_equals_top_b_of_token_scored_tree():
    B, D, k, budget = 2, 4, 3, 20
    ids, prev, root, entries = _random_case(99, B, D, k, vocab=12, n_entries=500)
    rng = np.random.default_rng(4)
    lp = -np.sort(rng.exponential(1.0, (B, D, k)), axis=2).astype(np.float32)
    lam = np.full(D, 0.6, np.float32)
    floor = np.float32(np.log(1e-4))
    lat = oracle.ngram_lattice(oracle.ngram_table(*_unzip(entries)), floor, ids, prev, root)
    tree = oracle.build_tree(ids, lp, lat, lam, root.astype(np.int32), D, k, budget)
    for b in range(B):
        # score every candidate-tree node from its own path tokens
        S = {(): np.float32(0.0)}
        for u in sorted(brute.full_tree(lp[b], None, None, D, k), key=len):
            if not u:
                continue
            toks = [int(prev[b]), int(root[b])] + [int(ids[b, i, r]) for i, r in enumerate(u)]
            lr = _scan(entries, toks[-3], toks[-2], toks[-1], floor)
            s = np.float32(lp[b, len(u) - 1, u[-1]] + np.float32(lam[len(u) - 1] * lr))
            S[u] = np.float32(S[u[:-1]] + s)
        want = brute.top_b(S, budget)
        got = brute.paths_of(tree, b)[1:]
        assert got == want
