"""Pins for the oracle's bookkeeping between rounds (no GPU).

* commit: after appending the accepted path, attention of the last
  accepted node over the new cache alone equals its tree attention over the
  old cache plus its root path (recomputed from parent pointers); the new
  rows are that root path in depth order; nothing else moves; an overflow
  leaves the sequence as it was.
* slot selection and flattening: the Appendix C walk-through worked by hand
  (tests/golden/self_spec_round.json); the node rows of the flattened mask
  equal the tree's own ancestor mask; node rows of the composite attention
  equal plain tree attention (they never see a slot).
"""
import json
import os

import numpy as np
import pytest
from scipy.special import softmax

import brute
import oracle
import synthetic as sy

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _tree_and_accept(seed, B=3, D=5, k=3, budget=20, V=50):
    rng = np.random.default_rng(seed)
    lp = -np.sort(rng.exponential(1.0, (B, D, k)), axis=2).astype(np.float32)
    ids = np.stack([[rng.choice(V, k, replace=False) for _ in range(D)] for _ in range(B)])
    root = rng.integers(0, V, B).astype(np.int32)
    tree = oracle.build_tree(ids.astype(np.int32), lp, None, np.zeros(D, np.float32), root, D, k,
                             budget)
    N = budget + 1
    T = rng.standard_normal((B, N, V)).astype(np.float32)
    for b in range(B):  # make a random chain acceptable
        n = 0
        while rng.random() < 0.8:
            kids = [c for c in range(1, int(tree["n_nodes"][b])) if tree["parent"][b, c] == n]
            if not kids:
                break
            c = int(rng.choice(kids))
            T[b, n, tree["token"][b, c]] = 50.0
            n = c
    acc = oracle.accept("f32", T, tree["parent"], tree["token"], tree["n_nodes"], D)
    return tree, acc, N


def test_commit_attention_invariant_and_path_order():
    B, hq, hkv, d = 3, 4, 2, 64
    tree, acc, N = _tree_and_accept(1, B=B)
    rng = np.random.default_rng(2)
    cap = np.array([40, 60, 35], np.int32)
    start = np.array([5, 50, 120], np.int32)
    ln = np.array([10, 0, 20], np.int32)
    rows = 200
    kc = rng.standard_normal((rows, hkv, d)).astype(np.float32)
    vc = rng.standard_normal((rows, hkv, d)).astype(np.float32)
    kt = rng.standard_normal((B, N, hkv, d)).astype(np.float32)
    vt = rng.standard_normal((B, N, hkv, d)).astype(np.float32)
    q = rng.standard_normal((B, N, hq, d)).astype(np.float32)
    ctx = np.stack([start, ln], 1)
    kc2, vc2, ctx2, skipped = oracle.commit_kv(kt, vt, acc["path"], acc["accept_len"], kc, vc, ctx,
                                               cap)
    assert not skipped.any()
    np.testing.assert_array_equal(ctx2[:, 1], ln + acc["accept_len"] + 1)
    touched = np.zeros(rows, bool)
    scale = d ** -0.5
    for b in range(B):
        m = int(acc["accept_len"][b]) + 1
        new = slice(start[b] + ln[b], start[b] + ln[b] + m)
        touched[new] = True
        # the new rows are the root path of the last accepted node, in depth order
        src = [int(np.flatnonzero((kt[b] == kc2[r]).all(axis=(1, 2)))[0]) for r in range(new.start,
                                                                                     new.stop)]
        assert src[0] == 0 and all(tree["parent"][b, src[i + 1]] == src[i] for i in range(m - 1))
        assert all(tree["depth"][b, s] == i for i, s in enumerate(src))
        last = src[-1]
        for h in range(hq):
            # old cache rows of b followed by the root path, attended by the last node
            g = h // (hq // hkv)
            K = np.concatenate([kc[start[b]:start[b] + ln[b], g], kt[b, src, g]]).astype(np.float64)
            V_ = np.concatenate([vc[start[b]:start[b] + ln[b], g], vt[b, src, g]]).astype(np.float64)
            ref = softmax(K @ q[b, last, h].astype(np.float64) * scale) @ V_
            Kn = kc2[start[b]:start[b] + ctx2[b, 1], g].astype(np.float64)
            Vn = vc2[start[b]:start[b] + ctx2[b, 1], g].astype(np.float64)
            got = softmax(Kn @ q[b, last, h].astype(np.float64) * scale) @ Vn
            np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(kc2[~touched], kc[~touched])
    np.testing.assert_array_equal(vc2[~touched], vc[~touched])


def test_commit_attention_matches_brute_path_attention():
    """Single sequence at cache offset 0: the brute recomputation from parent
    pointers over [old cache ; root .. last] equals attention over the new cache."""
    B, hq, hkv, d = 1, 2, 1, 64
    tree, acc, N = _tree_and_accept(7, B=B)
    rng = np.random.default_rng(8)
    kc = rng.standard_normal((64, hkv, d)).astype(np.float32)
    vc = rng.standard_normal((64, hkv, d)).astype(np.float32)
    kt = rng.standard_normal((B, N, hkv, d)).astype(np.float32)
    vt = rng.standard_normal((B, N, hkv, d)).astype(np.float32)
    q = rng.standard_normal((B, N, hq, d)).astype(np.float32)
    ctx = np.array([[0, 30]], np.int32)
    kc2, vc2, ctx2, _ = oracle.commit_kv(kt, vt, acc["path"], acc["accept_len"], kc, vc, ctx,
                                         np.array([64], np.int32))
    last = int(acc["path"][0, acc["accept_len"][0]])
    for h in range(hq):
        ref = brute.path_attention(q, kc, vc, np.array([0, 30]), kt, vt, tree["parent"], 0, last, h,
                                   d ** -0.5)
        K = kc2[:ctx2[0, 1], 0].astype(np.float64)
        V_ = vc2[:ctx2[0, 1], 0].astype(np.float64)
        got = softmax(K @ q[0, last, h].astype(np.float64) * d ** -0.5) @ V_
        np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_commit_overflow_and_bad_path_leave_sequence_unchanged():
    tree, acc, N = _tree_and_accept(3, B=2)
    kt = np.ones((2, N, 1, 64), np.float32)
    kc = np.zeros((40, 1, 64), np.float32)
    al = np.maximum(acc["accept_len"], 1)
    path = acc["path"].copy()
    path[:, 1] = np.where(acc["accept_len"] >= 1, path[:, 1], 1)
    ctx = np.array([[0, 19 - int(al[0])], [20, 3]], np.int32)      # seq 0 exactly fills, seq 1 below
    cap = np.array([20, 20], np.int32)
    kc2, _, ctx2, sk = oracle.commit_kv(kt, kt, path, al, kc, kc, ctx, cap)
    assert not sk.any() and ctx2[0, 1] == 20
    ctx = np.array([[0, 20 - int(al[0])], [20, 3]], np.int32)      # seq 0 one row short
    kc2, _, ctx2, sk = oracle.commit_kv(kt, kt, path, al, kc, kc, ctx, cap)
    assert sk.tolist() == [True, False] and ctx2[0, 1] == ctx[0, 1]
    assert not kc2[:20].any()
    bad = path.copy()
    bad[1, 0] = 3                                                   # path must start at the root
    _, _, ctx3, sk = oracle.commit_kv(kt, kt, bad, al, kc, kc, np.array([[0, 0], [20, 0]], np.int32),
                                      cap)
    assert sk.tolist() == [False, True] and ctx3[1, 1] == 0


def test_select_and_flatten_golden():
    g = json.load(open(os.path.join(GOLD, "self_spec_round.json")))
    path = np.array([g["path"]], np.int32)
    al = np.array([g["accept_len"]], np.int32)
    sel = oracle.select_slots(path, al, g["n_max"], g["select"]["slots"], g["select"]["first_slot"])
    assert sel[0].tolist() == g["select"]["expected_rows"]
    f = g["flatten"]
    out = oracle.flatten_slots(np.array([g["parent"]]), np.array([g["depth"]]),
                               np.array([len(g["parent"])]), np.array([f["root_pos"]]), f["slots"])
    assert out["pos"][0].tolist() == f["expected_pos"]
    assert int(out["n_rows"][0]) == 12
    for r, vis in enumerate(f["expected_visible"]):
        bits = [c for c in range(12) if (int(out["anc"][0, r, 0]) >> c) & 1]
        assert bits == vis, r


@pytest.mark.parametrize("slots", [1, 3, 7])
def test_flatten_node_rows_are_the_tree_mask(slots):
    tree, _, N = _tree_and_accept(11, B=3, budget=40)
    out = oracle.flatten_slots(tree["parent"], tree["depth"], tree["n_nodes"],
                               np.array([0, 5, 100]), slots)
    blk = 1 + slots
    for b in range(3):
        nn = int(tree["n_nodes"][b])
        for n in range(N):
            r = n * blk
            cols = [c for c in range(N * blk) if (int(out["anc"][b, r, c // 64]) >> (c % 64)) & 1]
            tcols = [m * blk for m in range(N) if (int(tree["anc"][b, n, m // 64]) >> (m % 64)) & 1]
            assert cols == (tcols if n < nn else []), (b, n)
            if n < nn:
                assert out["pos"][b, r] == [0, 5, 100][b] + tree["depth"][b, n]


def test_flatten_composite_attention_node_rows_equal_tree_attention():
    B, hq, hkv, d, slots = 2, 2, 1, 64, 3
    tree, _, N = _tree_and_accept(13, B=B, budget=12)
    blk = 1 + slots
    R = N * blk
    rng = np.random.default_rng(14)
    ctx = np.array([0, 17, 40], np.int32)
    kc = rng.standard_normal((40, hkv, d)).astype(np.float32)
    vc = rng.standard_normal((40, hkv, d)).astype(np.float32)
    q = rng.standard_normal((B, R, hq, d)).astype(np.float32)
    kt = rng.standard_normal((B, R, hkv, d)).astype(np.float32)
    vt = rng.standard_normal((B, R, hkv, d)).astype(np.float32)
    f = oracle.flatten_slots(tree["parent"], tree["depth"], tree["n_nodes"], np.zeros(B), slots)
    comp = oracle.tree_attention("f32", q, kc, vc, ctx, kt, vt, f["anc"], f["n_rows"])
    node = np.arange(N) * blk
    plain = oracle.tree_attention("f32", np.ascontiguousarray(q[:, node]), kc, vc, ctx,
                                  np.ascontiguousarray(kt[:, node]), np.ascontiguousarray(vt[:, node]),
                                  tree["anc"], tree["n_nodes"])
    np.testing.assert_array_equal(comp[:, node], plain)
