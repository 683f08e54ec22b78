"""GPU parity of presto_topk against the oracle (ids bit-exact, log q within
1e-5 * max(1, |ref|)), at the five workloads' full sizes and on edge cases;
the entropy output and the entropy-adaptive weight (Appendix F) against the
oracle's fp64 values."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_22634_amd as P
import synthetic as sy
from gpu_util import round_data, to_dev, to_host

pytestmark = pytest.mark.gpu


def _compare(logits_store, dtype, k, ids, lp, lse):
    rid, rlp, rlse, _ = oracle.topk(logits_store, k, dtype)
    np.testing.assert_array_equal(to_host(ids), rid)
    lp = to_host(lp)
    fin = np.isfinite(rlp)
    assert (np.isneginf(lp) == np.isneginf(rlp)).all()
    err = np.abs(lp[fin] - rlp[fin]) / np.maximum(1.0, np.abs(rlp[fin]))
    assert err.max(initial=0) <= 1e-5, err.max()
    lse = to_host(lse)
    fl = np.isfinite(rlse)
    np.testing.assert_allclose(lse[fl], rlse[fl], rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_topk_matches_oracle_on_workload(cfg):
    w, rin = round_data(cfg)
    logits = rin["drafter_logits"]
    print(f"topk cfg={cfg} rows={logits.shape[0]} k={w.k}", flush=True)
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    ids, lp, lse = P.presto_topk(to_dev(logits, w.dtype), w.k, flags=flags)
    torch.cuda.synchronize()
    assert int(flags.item()) == 0
    _compare(logits, w.dtype, w.k, ids, lp, lse)


EDGE = [
    ("f32", 1000, 1), ("bf16", 1000, 3), ("bf16", 4099, 16), ("f32", 37, 16),
    ("bf16", 151936, 8), ("f32", 151936, 2), ("bf16", 16, 16), ("bf16", 2048, 5),
]


@pytest.mark.parametrize("dtype,V,k", EDGE)
def test_topk_edge_rows(dtype, V, k):
    rng = np.random.default_rng([V, k, 11])
    rows = 9
    x = (rng.standard_normal((rows, V)) * 4).astype(np.float32)
    x[1, :] = 1.5                                   # one giant tie: exact fallback path
    x[2, :] = np.round(x[2])                        # heavy ties
    x[3, ::2] = -np.inf                             # masked vocabulary
    x[4, :] = -np.inf                               # fully masked row
    x[5, : min(V, 40)] = 0.0
    x[5, 1:min(V, 40):2] = -0.0                     # signed zeros tie
    x[6, rng.choice(V, min(V, 3), replace=False)] = x[6].max() + 8
    x[7, -1] = x[7].max() + 1                       # best entry in the ragged tail
    x[8, :] = -1e30
    store = sy.cast(x, dtype)
    ids, lp, lse = P.presto_topk(to_dev(store, dtype), k)
    torch.cuda.synchronize()
    _compare(store, dtype, k, ids, lp, lse)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_topk_unaligned_row_stride(dtype):
    rng = np.random.default_rng(5)
    V, stride, rows, k = 3001, 3005, 6, 4
    big = (rng.standard_normal((rows, stride)) * 4).astype(np.float32)
    store = sy.cast(big, dtype)
    t = to_dev(store, dtype)[:, :V]
    ids, lp, lse = P.presto_topk(t, k)
    torch.cuda.synchronize()
    _compare(np.ascontiguousarray(store[:, :V]), dtype, k, ids, lp, lse)


def test_topk_nan_sets_flag_only_for_nan():
    x = np.random.default_rng(1).standard_normal((4, 5000)).astype(np.float32)
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    P.presto_topk(to_dev(x), 4, flags=flags)
    torch.cuda.synchronize()
    assert int(flags.item()) == 0
    x[2, 77] = np.nan
    P.presto_topk(to_dev(x), 4, flags=flags)
    torch.cuda.synchronize()
    assert int(flags.item()) & P.PRESTO_FLAG_NAN_DRAFTER


def test_topk_is_deterministic():
    w, rin = round_data(2)
    t = to_dev(rin["drafter_logits"], w.dtype)
    a = [to_host(x) for x in P.presto_topk(t, w.k)]
    b = [to_host(x) for x in P.presto_topk(t, w.k)]
    for u, v in zip(a, b):
        np.testing.assert_array_equal(u, v)


def test_topk_workspace_reuse_keeps_results():
    """Counters in the workspace are re-armed by every call: reuse is safe."""
    w, rin = round_data(3)
    t = to_dev(rin["drafter_logits"], w.dtype)
    rows = t.shape[0]
    ws = torch.zeros(P.lib().presto_topk_workspace(rows, w.vocab, w.k), dtype=torch.uint8,
                     device="cuda")
    first = [to_host(x) for x in P.presto_topk(t, w.k, workspace=ws)]
    for _ in range(3):
        again = [to_host(x) for x in P.presto_topk(t, w.k, workspace=ws)]
        for u, v in zip(first, again):
            np.testing.assert_array_equal(u, v)


def _compare_entropy(store, dtype, h):
    """The kernel forms H = log S - X / S with S = sum e^(z-M) and
    X = sum e^(z-M) (z-M), M the row max.  log S is the min-entropy, so
    0 <= log S <= H and -X / S = E_q[M - z] = H - log S lies in [0, H]: each
    term is at most H and carries a relative error of a few hundred fp32
    ulps after the sums over V terms, giving the bound 2e-5 * (1 + H)."""
    rh = oracle.entropy(store, dtype)
    h = to_host(h).astype(np.float64)
    tol = 2e-5 * (1.0 + rh)
    err = np.abs(h - rh)
    assert (err <= tol).all(), (err / tol).max()


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_topk_entropy_matches_oracle_on_workload(cfg):
    """With the entropy output on, ids/log q/LSE stay as before and H_d
    (Appendix F) matches the oracle's fp64 entropy."""
    w, rin = round_data(cfg)
    logits = rin["drafter_logits"]
    print(f"topk+entropy cfg={cfg} rows={logits.shape[0]}", flush=True)
    ids, lp, lse, h = P.presto_topk(to_dev(logits, w.dtype), w.k, entropy=True)
    torch.cuda.synchronize()
    _compare(logits, w.dtype, w.k, ids, lp, lse)
    _compare_entropy(logits, w.dtype, h)


@pytest.mark.parametrize("dtype,V,k", EDGE)
def test_topk_entropy_edge_rows(dtype, V, k):
    rng = np.random.default_rng([V, k, 12])
    x = (rng.standard_normal((8, V)) * 4).astype(np.float32)
    x[1, :] = 1.5                                   # uniform: H = log V
    x[2, :] = -np.inf
    x[2, V // 2] = 3.0                              # point mass: H = 0
    x[3, ::2] = -np.inf                             # zero-probability entries
    x[4, :] = -np.inf                               # no distribution: H = 0
    x[5, :] = -1e30                                 # uniform far below zero
    x[6, :] = x[6] * 60                             # nearly one-hot
    x[7, :] = 300.0 + x[7]                          # large offsets
    store = sy.cast(x, dtype)
    ids, lp, lse, h = P.presto_topk(to_dev(store, dtype), k, entropy=True)
    torch.cuda.synchronize()
    _compare(store, dtype, k, ids, lp, lse)
    _compare_entropy(store, dtype, h)
    hh = to_host(h)
    assert hh[2] == 0.0 and hh[4] == 0.0


def test_entropy_lambda_matches_oracle():
    rng = np.random.default_rng(21)
    h = np.concatenate([[0.0, 1e-30, 1.5, 12.0, 1e6], rng.uniform(0, 12, 4091)]).astype(np.float32)
    for beta, c in [(1.0, 1.0), (0.35, 2.5), (4.0, 0.01)]:
        lam = to_host(P.presto_entropy_lambda(to_dev(h), beta, c))
        want = oracle.entropy_lambda(h.astype(np.float64), np.float32(beta), np.float32(c))
        # three fp32 roundings (H + C, the quotient, the product)
        np.testing.assert_allclose(lam, want, rtol=4e-7, atol=0)
        assert lam[0] == 0.0


@pytest.mark.parametrize("cfg,k", [(2, 8), (2, 10), (2, 16), (4, 10), (5, 10), (3, 12)])
def test_topk_large_k_on_workload(cfg, k):
    """k above 8 (the paper's k = 10, Sec. 5.1) at the workloads' shapes: ids
    bit-exact, and the fast path holds every chunk (no exact-pass fallback
    on continuous logits: at most one group per lane reaches the bound)."""
    w, rin = round_data(cfg)
    logits = rin["drafter_logits"]
    print(f"topk large-k cfg={cfg} rows={logits.shape[0]} k={k}", flush=True)
    dev_logits = to_dev(logits, w.dtype)
    ws = P.topk_workspace(logits.shape[0], w.vocab, k, dev_logits.device)
    ids, lp, lse = P.presto_topk(dev_logits, k, workspace=ws)
    torch.cuda.synchronize()
    _compare(logits, w.dtype, k, ids, lp, lse)
    assert P.topk_fallback_chunks(ws) == 0


def test_topk_fallback_count_on_ties():
    """Rows made of one repeated value send every chunk through the exact
    pass; the workspace counter says how many chunks that was, and a later
    call without ties resets it."""
    rng = np.random.default_rng(8)
    rows, V, k = 6, 151936, 10
    x = (rng.standard_normal((rows, V)) * 4).astype(np.float32)
    x[1, :] = 2.0
    x[4, :] = np.round(x[4] / 64) * 64  # a handful of distinct values
    store = sy.cast(x, "bf16")
    dl = to_dev(store, "bf16")
    ws = P.topk_workspace(rows, V, k, dl.device)
    ids, lp, lse = P.presto_topk(dl, k, workspace=ws)
    torch.cuda.synchronize()
    _compare(store, "bf16", k, ids, lp, lse)
    n_fb = P.topk_fallback_chunks(ws)
    assert n_fb > 0
    ids, lp, lse = P.presto_topk(dl[:1].contiguous(), k, workspace=ws)
    torch.cuda.synchronize()
    _compare(np.ascontiguousarray(store[:1]), "bf16", k, ids, lp, lse)
    assert P.topk_fallback_chunks(ws) == 0


@pytest.mark.parametrize("k", [1, 5, 8, 10])
def test_topk_tie_runs_around_a_wave_of_candidates(k):
    """Runs of 63, 64 and 65 equal maxima in one chunk (in the first and in
    a later chunk): up to 64 entries at or above the chunk's bound each
    lane takes one and is placed by rank, above 64 the chunk takes the
    wave-maximum selection; a run spread one per group over more groups
    than the candidate list holds takes the exact pass.  The winners are
    the run's lowest ids (value desc, id asc)."""
    rng = np.random.default_rng([k, 64])
    V = 151936
    runs = [(0, 63), (0, 64), (0, 65), (4096 + 8, 64), (4096 + 8, 65), (2 * 4096 + 3, 64)]
    x = np.clip(rng.standard_normal((len(runs) + 1, V)) * 2, -8, 8).astype(np.float32)
    for r, (start, n) in enumerate(runs):
        x[r, start:start + n] = 12.0
    x[len(runs), 0:64 * 8:8] = 12.0  # one entry in each of 64 groups
    store = sy.cast(x, "bf16")
    ids, lp, lse = P.presto_topk(to_dev(store, "bf16"), k)
    torch.cuda.synchronize()
    _compare(store, "bf16", k, ids, lp, lse)
    got = to_host(ids)
    for r, (start, n) in enumerate(runs):
        np.testing.assert_array_equal(got[r], np.arange(start, start + k))
