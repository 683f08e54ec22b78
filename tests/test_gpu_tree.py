"""GPU parity of presto_build_tree: fed the same candidate tables (the
oracle's top-k of the workload, or random tables), the GPU tree equals the
oracle's bit for bit (topology, tokens, depths, ranks, fp32 scores, ancestor
masks, node counts)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_22634_amd as P
import synthetic as sy
from gpu_util import oracle_candidates, round_data, to_dev, to_host, tree_to_host

pytestmark = pytest.mark.gpu

KEYS = ("n_nodes", "parent", "token", "depth", "rank", "score", "anc")


def _gpu_and_oracle(ids, lp, rho, lam, root, D, k, B, branch=None, beam_width=0, alg2=False):
    mode = P.PRESTO_TREE_BEAM if beam_width else P.PRESTO_TREE_BEST_FIRST
    omode = oracle.BEAM if beam_width else oracle.BEST_FIRST
    if alg2:
        mode, omode = P.PRESTO_TREE_BEST_FIRST_ALG2, oracle.BEST_FIRST_ALG2
    g = P.presto_build_tree(to_dev(ids), to_dev(lp), None if rho is None else to_dev(rho),
                            to_dev(lam), to_dev(root), D, k, B, branch=branch, mode=mode,
                            beam_width=beam_width)
    torch.cuda.synchronize()
    g = tree_to_host(g)
    o = oracle.build_tree(ids, lp, rho, lam, root, D, k, B, branch=branch, mode=omode,
                          beam_width=beam_width)
    return g, o


def _assert_same(g, o):
    for key in KEYS:
        if key == "score":
            np.testing.assert_array_equal(g[key].view(np.uint32), o[key].view(np.uint32), err_msg=key)
        else:
            np.testing.assert_array_equal(g[key], o[key], err_msg=key)


@pytest.mark.parametrize("cfg,lam", [(1, None), (2, None), (3, None), (4, None), (5, None), (5, 0.2)])
def test_tree_matches_oracle_on_workload(cfg, lam):
    over = {} if lam is None else {"lam": lam}
    w, rin = round_data(cfg, **over)
    print(f"tree cfg={cfg} batch={w.batch} B={w.budget} k={w.k}", flush=True)
    ids, lp = oracle_candidates(cfg)
    g, o = _gpu_and_oracle(ids, lp, rin["rho"], rin["lam"], rin["root_token"], w.depth, w.k,
                           w.budget)
    _assert_same(g, o)
    assert (g["n_nodes"] == w.budget + 1).all()


def _random_batch(seed, b, D, k, quant):
    rng = np.random.default_rng(seed)
    lp = -rng.exponential(1.5, size=(b, D, k))
    R = -rng.exponential(2.0, size=(b, D, k, k, k))
    if quant:
        lp = np.round(lp * 4) / 4
        R = np.round(R * 2) / 2
    R[rng.random(R.shape) < 0.3] = np.log(np.float32(1e-4))
    lp = -np.sort(-lp, axis=2)
    ids = np.stack([[rng.choice(5000, k, replace=False) for _ in range(D)] for _ in range(b)])
    root = rng.integers(0, 5000, size=b)
    return (ids.astype(np.int32), lp.astype(np.float32), R.astype(np.float32),
            root.astype(np.int32))


@pytest.mark.parametrize("D,k,branch,B", [(1, 1, 1, 1), (3, 2, 2, 4), (4, 3, 2, 40), (5, 3, 3, 200),
                                          (6, 2, 1, 9), (16, 8, 8, 256), (32, 4, 3, 128),
                                          (8, 16, 16, 255), (2, 16, 5, 63), (12, 5, 5, 130),
                                          (10, 4, 4, 511), (20, 5, 5, 300), (7, 5, 5, 100)])
@pytest.mark.parametrize("quant", [False, True])
def test_tree_matches_oracle_random(D, k, branch, B, quant):
    ids, lp, R, root = _random_batch([D, k, B, int(quant)], 24, D, k, quant)
    for lam_v, rho in ((0.2, R), (0.0, R), (1.0, None)):
        lam = np.full(D, lam_v, np.float32)
        g, o = _gpu_and_oracle(ids, lp, rho, lam, root, D, k, B, branch=branch)
        _assert_same(g, o)


def test_tree_is_deterministic():
    ids, lp, R, root = _random_batch(3, 8, 16, 8, True)
    lam = np.full(16, 0.2, np.float32)
    a = tree_to_host(P.presto_build_tree(to_dev(ids), to_dev(lp), to_dev(R), to_dev(lam),
                                         to_dev(root), 16, 8, 256))
    b = tree_to_host(P.presto_build_tree(to_dev(ids), to_dev(lp), to_dev(R), to_dev(lam),
                                         to_dev(root), 16, 8, 256))
    for key in KEYS:
        np.testing.assert_array_equal(a[key], b[key])


@pytest.mark.parametrize("cfg,W", [(2, 10), (3, 4), (4, 10), (5, 10)])
def test_beam_tree_matches_oracle_on_workload(cfg, W):
    w, rin = round_data(cfg)
    print(f"beam cfg={cfg} W={W}", flush=True)
    ids, lp = oracle_candidates(cfg)
    g, o = _gpu_and_oracle(ids, lp, rin["rho"], rin["lam"], rin["root_token"], w.depth, w.k,
                           w.budget, beam_width=W)
    _assert_same(g, o)


@pytest.mark.parametrize("D,k,branch,B,W", [(1, 1, 1, 1, 1), (3, 2, 2, 4, 1), (4, 3, 2, 40, 3),
                                            (5, 3, 3, 200, 64), (6, 2, 1, 9, 2), (16, 8, 8, 256, 10),
                                            (32, 4, 3, 128, 16), (8, 16, 16, 255, 16),
                                            (12, 5, 5, 130, 51), (10, 4, 4, 511, 64)])
@pytest.mark.parametrize("quant", [False, True])
def test_beam_tree_matches_oracle_random(D, k, branch, B, W, quant):
    ids, lp, R, root = _random_batch([D, k, B, W, int(quant)], 12, D, k, quant)
    for lam_v, rho in ((0.2, R), (1.0, None)):
        lam = np.full(D, lam_v, np.float32)
        g, o = _gpu_and_oracle(ids, lp, rho, lam, root, D, k, B, branch=branch, beam_width=W)
        _assert_same(g, o)



@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_alg2_tree_matches_oracle_on_workload(cfg):
    """Literal Alg. 2 (whole expansions, then TopB(T)) at the workloads' shapes."""
    w, rin = round_data(cfg)
    print(f"alg2 cfg={cfg}", flush=True)
    ids, lp = oracle_candidates(cfg)
    g, o = _gpu_and_oracle(ids, lp, rin["rho"], rin["lam"], rin["root_token"], w.depth, w.k,
                           w.budget, alg2=True)
    _assert_same(g, o)


@pytest.mark.parametrize("D,k,branch,B", [(1, 1, 1, 1), (3, 2, 2, 4), (4, 3, 2, 40), (5, 3, 3, 200),
                                          (6, 2, 1, 9), (16, 8, 8, 256), (32, 4, 3, 128),
                                          (8, 16, 16, 255), (2, 16, 5, 63), (12, 5, 5, 130),
                                          (10, 4, 4, 511), (2, 3, 3, 500), (7, 16, 16, 511)])
@pytest.mark.parametrize("quant", [False, True])
def test_alg2_tree_matches_oracle_random(D, k, branch, B, quant):
    """Random tables, quantised ones full of ties; (2, 3, 3, 500): the whole
    candidate tree (12 nodes) is smaller than the budget."""
    ids, lp, R, root = _random_batch([D, k, B, int(quant), 2], 12, D, k, quant)
    for lam_v, rho in ((0.2, R), (1.0, None)):
        lam = np.full(D, lam_v, np.float32)
        g, o = _gpu_and_oracle(ids, lp, rho, lam, root, D, k, B, branch=branch, alg2=True)
        _assert_same(g, o)


@pytest.mark.parametrize("cfg,beam_width", [(2, 0), (3, 0), (4, 0), (3, 4)])
def test_tree_with_entropy_adaptive_lambda(cfg, beam_width):
    """Per-sequence, per-position weights lambda_d(H_d) (Appendix F): the
    weights come from the oracle's entropies and enter both sides as the
    same fp32 [batch, depth] table."""
    w, rin = round_data(cfg)
    print(f"tree entropy-lambda cfg={cfg} W={beam_width}", flush=True)
    ids, lp = oracle_candidates(cfg)
    h = oracle.entropy(rin["drafter_logits"], w.dtype)
    lam = oracle.entropy_lambda(h, 0.6, 2.0).astype(np.float32).reshape(w.batch, w.depth)
    assert np.ptp(lam) > 0  # the weights really vary
    g, o = _gpu_and_oracle(ids, lp, rin["rho"], lam, rin["root_token"], w.depth, w.k, w.budget,
                           beam_width=beam_width)
    _assert_same(g, o)


def test_tree_per_sequence_lambda_random():
    D, k, B, b = 12, 5, 130, 24
    ids, lp, R, root = _random_batch([D, k, B, 77], b, D, k, False)
    lam = np.random.default_rng(3).uniform(0, 1.5, (b, D)).astype(np.float32)
    lam[::5] = 0.0
    g, o = _gpu_and_oracle(ids, lp, R, lam, root, D, k, B, branch=4)
    _assert_same(g, o)


@pytest.mark.parametrize("B", [128, 256, 512, 1023])
@pytest.mark.parametrize("mode", ["best_first", "beam10", "alg2"])
def test_tree_paper_operating_point(B, mode):
    """Sec. 5.1's operating point: k = 10 candidates per position from the
    16-position block of the single-sequence workload, beam width 10, budgets
    128, 256, 512 (and 1023: N = 1024 rows, the largest tree Table 1's budget
    range reaches).  The 64,000-byte trigram lattice of k = 10 is read from
    LDS at every budget."""
    w, rin = round_data(2)
    k, D = 10, w.depth
    ids, lp, _, _ = oracle.topk(rin["drafter_logits"], k, w.dtype)
    ids, lp = ids.reshape(1, D, k), lp.reshape(1, D, k)
    rho = sy.rho_lattice(w.with_(k=k))
    print(f"paper point mode={mode} B={B}", flush=True)
    g, o = _gpu_and_oracle(ids, lp, rho, rin["lam"], rin["root_token"], D, k, B,
                           beam_width=10 if mode == "beam10" else 0, alg2=mode == "alg2")
    _assert_same(g, o)
    assert int(g["n_nodes"][0]) == B + 1


@pytest.mark.parametrize("D,k,branch,B", [(16, 10, 10, 1023), (24, 16, 16, 1023), (9, 3, 3, 700),
                                          (16, 10, 6, 777)])
@pytest.mark.parametrize("mode", ["best_first", "beam10", "alg2"])
def test_tree_large_budgets_random(D, k, branch, B, mode):
    """Budgets above 511 on random and tie-heavy tables, every mode, with
    k = 16 (the lattice is read from global memory: 393 KB per sequence) and
    branch < k among them."""
    for quant in (False, True):
        ids, lp, R, root = _random_batch([D, k, B, int(quant), 9], 6, D, k, quant)
        for lam_v, rho in ((0.2, R), (1.0, None)):
            lam = np.full(D, lam_v, np.float32)
            g, o = _gpu_and_oracle(ids, lp, rho, lam, root, D, k, B, branch=branch,
                                   beam_width=10 if mode == "beam10" else 0, alg2=mode == "alg2")
            _assert_same(g, o)


@pytest.mark.parametrize("D,k,B", [(32, 3, 700), (32, 2, 1023), (20, 5, 400), (32, 3, 200), (32, 2, 255),
                                   (20, 5, 100), (24, 8, 64)])
@pytest.mark.parametrize("mode", ["best_first", "beam10", "alg2"])
def test_tree_deep_ties(D, k, B, mode):
    """Whole tied subtrees: lambda = 0 and log q on a coarse grid with equal
    candidates in most rows, so siblings with equal log q root score-identical
    subtrees and most pops break a tie of S by rank-path keys, deep in the
    tree and several times under the same ancestors."""
    rng = np.random.default_rng([D, k, B, 31])
    b = 8
    lp = -np.round(rng.exponential(1.0, size=(b, D, k)) * 2) / 2
    lp[:, :, 1] = lp[:, :, 0]  # the two best candidates of every row tie
    lp = -np.sort(-lp, axis=2).astype(np.float32)
    ids = np.stack([[rng.choice(5000, k, replace=False) for _ in range(D)] for _ in range(b)]).astype(np.int32)
    root = rng.integers(0, 5000, size=b).astype(np.int32)
    lam = np.zeros(D, np.float32)
    g, o = _gpu_and_oracle(ids, lp, None, lam, root, D, k, B, beam_width=10 if mode == "beam10" else 0,
                           alg2=mode == "alg2")
    _assert_same(g, o)
    ties = sum(int((np.diff(np.sort(row[np.isfinite(row)])) == 0).sum()) for row in o["score"][:, 1:])
    assert ties > b * 10  # ties really occur
