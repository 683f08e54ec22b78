"""GPU parity of presto_accept: per-node target argmax, accepted length,
path and bonus token equal the oracle's exactly (both sides take the
oracle's tree of the workload, or random trees)."""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2607_22634_amd as P
import synthetic as sy
from gpu_util import oracle_tree, round_data, to_dev, to_host, tree_to_dev, tree_to_host

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _check(w, T_store, th, tree_dev):
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    g = P.presto_accept(to_dev(T_store, w.dtype), tree_dev["parent"], tree_dev["token"],
                        tree_dev["n_nodes"], w.depth, flags=flags)
    torch.cuda.synchronize()
    o = oracle.accept(w.dtype, T_store, th["parent"], th["token"], th["n_nodes"], w.depth)
    for key in ("accept_len", "path", "bonus", "target_argmax"):
        np.testing.assert_array_equal(to_host(g[key]), o[key], err_msg=key)
    assert int(flags.item()) == 0
    return o


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_accept_matches_oracle_on_workload(cfg):
    w, rin = round_data(cfg)
    print(f"accept cfg={cfg}", flush=True)
    th = oracle_tree(cfg)
    T = sy.target_logits(w, rin["field"], th["parent"], th["rank"], th["n_nodes"])
    o = _check(w, T, th, tree_to_dev(th))
    print("accept_len", o["accept_len"].tolist(), flush=True)


def test_accept_fig3_golden():
    g = json.load(open(os.path.join(GOLD, "fig3_accept.json")))
    N, V = len(g["parent"]), g["vocab"]
    T = np.zeros((1, N, V), np.float32)
    for n, a in enumerate(g["target_argmax_per_node"]):
        T[0, n, a] = 1.0
    par = to_dev(np.array([g["parent"]], np.int32))
    tok = to_dev(np.array([g["token"]], np.int32))
    nn = to_dev(np.array([N], np.int32))
    r = P.presto_accept(to_dev(T), par, tok, nn, g["depth"])
    torch.cuda.synchronize()
    assert int(to_host(r["accept_len"])[0]) == g["expected"]["accept_len"]
    assert to_host(r["path"])[0].tolist() == g["expected"]["path"]
    assert int(to_host(r["bonus"])[0]) == g["expected"]["bonus"]


@pytest.mark.parametrize("dtype,V", [("f32", 1000), ("bf16", 4099), ("bf16", 151936)])
def test_accept_random_trees_with_ties(dtype, V):
    rng = np.random.default_rng([V, 3])
    b, N, D = 6, 40, 8
    parent = np.full((b, N), -1, np.int32)
    token = np.full((b, N), -1, np.int32)
    n_nodes = np.array([40, 1, 2, 17, 40, 33], np.int32)
    T = (rng.standard_normal((b, N, V)) * 2).astype(np.float32)
    for s in range(b):
        depth = np.zeros(N, int)
        used = {0: set()}
        token[s, 0] = rng.integers(V)
        for n in range(1, int(n_nodes[s])):
            p = int(rng.integers(0, n))
            while depth[p] >= D:
                p = int(rng.integers(0, n))
            t = int(rng.integers(V))
            while t in used[p]:
                t = int(rng.integers(V))
            used[p].add(t)
            used[n] = set()
            parent[s, n], token[s, n], depth[n] = p, t, depth[p] + 1
        for n in range(int(n_nodes[s])):
            kids = [c for c in range(1, int(n_nodes[s])) if parent[s, c] == n]
            if kids and rng.random() < 0.85:
                c = int(rng.choice(kids))
                T[s, n, token[s, c]] = 9.0
                if rng.random() < 0.3:
                    T[s, n, rng.integers(V)] = 9.0  # a tie: the lower id wins
    w = sy.workload(1).with_(dtype=dtype, depth=D, vocab=V)
    store = sy.cast(T, dtype)
    th = {"parent": parent, "token": token, "n_nodes": n_nodes}
    tree_dev = {k: to_dev(v) for k, v in th.items()}
    _check(w, store, th, tree_dev)


def test_accept_nan_flag():
    T = np.zeros((1, 3, 64), np.float32)
    T[0, 1, 5] = np.nan
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    P.presto_accept(to_dev(T), to_dev(np.array([[-1, 0, 0]], np.int32)),
                    to_dev(np.array([[1, 2, 3]], np.int32)), to_dev(np.array([3], np.int32)), 1,
                    flags=flags)
    torch.cuda.synchronize()
    assert int(flags.item()) & P.PRESTO_FLAG_NAN_TARGET


def test_accept_workspace_reuse_keeps_results():
    w, rin = round_data(2)
    ids, lp, _ = P.presto_topk(to_dev(rin["drafter_logits"], w.dtype), w.k)
    t = P.presto_build_tree(ids, lp, to_dev(rin["rho"]), to_dev(rin["lam"]),
                            to_dev(rin["root_token"]), w.depth, w.k, w.budget)
    th = tree_to_host(t)
    T = to_dev(sy.target_logits(w, rin["field"], th["parent"], th["rank"], th["n_nodes"]), w.dtype)
    ws = torch.zeros(P.lib().presto_accept_workspace(w.batch, w.n_max, w.vocab), dtype=torch.uint8,
                     device="cuda")
    ref = {k: to_host(v) for k, v in P.presto_accept(T, t["parent"], t["token"], t["n_nodes"],
                                                       w.depth, workspace=ws).items()}
    for _ in range(3):
        r = P.presto_accept(T, t["parent"], t["token"], t["n_nodes"], w.depth, workspace=ws)
        for key in ref:
            np.testing.assert_array_equal(to_host(r[key]), ref[key])
