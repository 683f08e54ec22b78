"""GPU parity of presto_tree_attention against the oracle.

Per (b, n, h) row: ||o - o_ref||_2 <= tol * ||o_ref||_2 with tol = 2e-2 for
bf16 (matrix cores, fp32 accumulation, bf16 probabilities) and 1e-4 for the
fp32 path; padding rows must be exactly zero.  The small workloads are
compared in full, the large ones on sampled rows that the oracle computes
one by one, in the launch configuration the bench uses.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_22634_amd as P
import synthetic as sy
from brute import anc_from_parent
from gpu_util import attn_data, oracle_tree, round_data, to_dev, to_host, tree_to_dev, tree_to_host

pytestmark = pytest.mark.gpu


def _tree_for(cfg):
    """The oracle's tree of the workload, on the device (both sides use it)."""
    w, _ = round_data(cfg)
    return w, tree_to_dev(oracle_tree(cfg))


def _run(w, att, tree_dev, total_ctx=0):
    return P.presto_tree_attention(
        to_dev(att["q"], w.dtype), to_dev(att["k_cache"], w.dtype), to_dev(att["v_cache"], w.dtype),
        to_dev(att["ctx_offsets"]), to_dev(att["k_tree"], w.dtype), to_dev(att["v_tree"], w.dtype),
        tree_dev["anc"], tree_dev["n_nodes"], int(np.diff(att["ctx_offsets"]).max()), w.scale,
        total_ctx=total_ctx)


def _row_errors(got, ref):
    num = np.linalg.norm(got - ref, axis=-1)
    den = np.linalg.norm(ref, axis=-1)
    return num / np.maximum(den, 1e-30)


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_attention_matches_oracle_full(cfg):
    w, tree = _tree_for(cfg)
    _, att = attn_data(cfg)
    print(f"attn cfg={cfg} full compare", flush=True)
    out = _run(w, att, tree)
    torch.cuda.synchronize()
    th = tree_to_host(tree)
    ref = oracle.tree_attention(w.dtype, att["q"], att["k_cache"], att["v_cache"],
                                att["ctx_offsets"], att["k_tree"], att["v_tree"], th["anc"],
                                th["n_nodes"], w.scale)
    got = sy.as_f32(to_host(out), w.dtype).astype(np.float64)
    reff = sy.as_f32(ref, w.dtype).astype(np.float64)
    tol = 2e-2 if w.dtype == "bf16" else 1e-4
    for s in range(w.batch):
        nn = int(th["n_nodes"][s])
        err = _row_errors(got[s, :nn], reff[s, :nn])
        assert err.max() <= tol, (s, err.max())
        assert not got[s, nn:].any()


@pytest.mark.parametrize("cfg", [4, 5])
def test_attention_matches_oracle_sampled(cfg):
    w, tree = _tree_for(cfg)
    _, att = attn_data(cfg)
    print(f"attn cfg={cfg} sampled compare", flush=True)
    out = _run(w, att, tree)
    torch.cuda.synchronize()
    th = tree_to_host(tree)
    rng = np.random.default_rng(cfg)
    rows = []
    for s in range(w.batch):
        nn = int(th["n_nodes"][s])
        nodes = {0, nn - 1} | set(rng.integers(0, nn, size=6).tolist())
        for n in nodes:
            for h in rng.choice(w.hq, size=4, replace=False):
                rows.append((s, n, int(h)))
    rows = np.array(rows, np.int32)
    ref = oracle.tree_attention_rows(w.dtype, att["q"], att["k_cache"], att["v_cache"],
                                     att["ctx_offsets"], att["k_tree"], att["v_tree"], th["anc"],
                                     th["n_nodes"], rows, w.scale)
    got = sy.as_f32(to_host(out), w.dtype)[rows[:, 0], rows[:, 1], rows[:, 2]].astype(np.float64)
    err = _row_errors(got, ref)
    assert err.max() <= 2e-2, err.max()


def _edge_inputs(rng, b, N, hq, hkv, d, ctx, dtype, parent, n_nodes):
    offs = np.zeros(b + 1, np.int32)
    offs[1:] = np.cumsum(ctx)
    f = lambda *s: sy.cast(rng.standard_normal(s, dtype=np.float32), dtype)
    att = {"q": f(b, N, hq, d), "k_cache": f(max(int(offs[-1]), 1), hkv, d),
           "v_cache": f(max(int(offs[-1]), 1), hkv, d), "ctx_offsets": offs,
           "k_tree": f(b, N, hkv, d), "v_tree": f(b, N, hkv, d)}
    anc = anc_from_parent(parent, n_nodes, N)
    return att, anc


@pytest.mark.parametrize("dtype,hq,hkv,d", [("bf16", 32, 8, 128), ("bf16", 8, 8, 64),
                                            ("bf16", 16, 2, 128), ("f32", 4, 2, 128)])
def test_attention_edges(dtype, hq, hkv, d):
    rng = np.random.default_rng([hq, hkv, d])
    b, N = 5, 70
    ctx = np.array([0, 1, 63, 64, 3000], np.int32)
    parent = np.full((b, N), -1, np.int32)
    n_nodes = np.array([1, 70, 37, 2, 70], np.int32)
    for s in range(b):
        for n in range(1, int(n_nodes[s])):
            parent[s, n] = n - 1 if s == 3 else rng.integers(0, n)  # chain or random tree
    att, anc = _edge_inputs(rng, b, N, hq, hkv, d, ctx, dtype, parent, n_nodes)
    w = sy.workload(1).with_(dtype=dtype, head_dim=d)
    scale = 1 / np.sqrt(d)
    out = P.presto_tree_attention(
        to_dev(att["q"], dtype), to_dev(att["k_cache"], dtype), to_dev(att["v_cache"], dtype),
        to_dev(att["ctx_offsets"]), to_dev(att["k_tree"], dtype), to_dev(att["v_tree"], dtype),
        to_dev(anc), to_dev(n_nodes), int(ctx.max()), scale)
    torch.cuda.synchronize()
    ref = oracle.tree_attention(dtype, att["q"], att["k_cache"], att["v_cache"],
                                att["ctx_offsets"], att["k_tree"], att["v_tree"], anc, n_nodes,
                                scale)
    got = sy.as_f32(to_host(out), dtype).astype(np.float64)
    reff = sy.as_f32(ref, dtype).astype(np.float64)
    tol = 2e-2 if dtype == "bf16" else 1e-4
    for s in range(b):
        nn = int(n_nodes[s])
        assert _row_errors(got[s, :nn], reff[s, :nn]).max() <= tol
        assert not got[s, nn:].any()


def test_attention_is_deterministic():
    w, tree = _tree_for(2)
    _, att = attn_data(2)
    a = to_host(_run(w, att, tree))
    b = to_host(_run(w, att, tree))
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("hint", ["actual", "tiny", "half", "uniform"])
def test_attention_ragged_total_ctx_hint(hint):
    """Ragged contexts (workload 3): the total-context hint only changes how
    the context is split and dealt to workgroups, never the result; a hint
    below the real total (down to 1) or at batch x max_ctx (no compaction)
    must match the oracle just the same."""
    w, tree = _tree_for(3)
    _, att = attn_data(3)
    ctx = np.diff(att["ctx_offsets"]).astype(np.int64)
    total = {"actual": int(ctx.sum()), "tiny": 1, "half": int(ctx.sum()) // 2,
             "uniform": int(w.batch * ctx.max())}[hint]
    print(f"attn ragged hint={hint} total_ctx={total}", flush=True)
    out = _run(w, att, tree, total_ctx=total)
    torch.cuda.synchronize()
    th = tree_to_host(tree)
    ref = oracle.tree_attention(w.dtype, att["q"], att["k_cache"], att["v_cache"],
                                att["ctx_offsets"], att["k_tree"], att["v_tree"], th["anc"],
                                th["n_nodes"], w.scale)
    got = sy.as_f32(to_host(out), w.dtype).astype(np.float64)
    reff = sy.as_f32(ref, w.dtype).astype(np.float64)
    for s in range(w.batch):
        nn = int(th["n_nodes"][s])
        err = _row_errors(got[s, :nn], reff[s, :nn])
        assert err.max() <= 2e-2, (s, err.max())
        assert not got[s, nn:].any()


@pytest.mark.parametrize("layout", ["packed", "slots"])
def test_attention_many_ragged_sequences_compact(layout):
    """More sequences than a wave has lanes (70), ragged contexts including
    empty ones, with the total-context hint: the workgroups' pair search runs
    over several 64-sequence groups.  The slots layout leaves gaps of large
    values between the sequences' cache rows, which must never be read."""
    rng = np.random.default_rng(77 if layout == "packed" else 78)
    b, N, hq, hkv, d, dtype = 70, 9, 8, 2, 64, "bf16"
    ctx = rng.integers(0, 600, b).astype(np.int32)
    ctx[[3, 40]] = 0
    ctx[65] = 3000
    parent = np.full((b, N), -1, np.int32)
    n_nodes = rng.integers(1, N + 1, b).astype(np.int32)
    for s in range(b):
        for n in range(1, int(n_nodes[s])):
            parent[s, n] = rng.integers(0, n)
    att, anc = _edge_inputs(rng, b, N, hq, hkv, d, ctx, dtype, parent, n_nodes)
    scale = 1 / np.sqrt(d)
    total = int(ctx.sum())
    kc, vc, offs = att["k_cache"], att["v_cache"], att["ctx_offsets"]
    ctx_arg, lay = offs, P.PRESTO_CTX_PACKED
    if layout == "slots":
        gap = 5
        start = (offs[:-1] + gap * np.arange(1, b + 1)).astype(np.int32)
        rows = int(start[-1] + ctx[-1]) + gap
        big = sy.cast(np.full((rows, hkv, d), 300.0, np.float32), dtype)
        ks, vs = big.copy(), big.copy()
        for s in range(b):
            ks[start[s]:start[s] + ctx[s]] = kc[offs[s]:offs[s + 1]]
            vs[start[s]:start[s] + ctx[s]] = vc[offs[s]:offs[s + 1]]
        kc_dev, vc_dev = to_dev(ks, dtype), to_dev(vs, dtype)
        ctx_arg, lay = np.stack([start, ctx], axis=1).astype(np.int32), P.PRESTO_CTX_SLOTS
    else:
        kc_dev, vc_dev = to_dev(kc, dtype), to_dev(vc, dtype)
    print(f"attn compact layout={layout} batch={b} total_ctx={total}", flush=True)
    out = P.presto_tree_attention(
        to_dev(att["q"], dtype), kc_dev, vc_dev, to_dev(ctx_arg), to_dev(att["k_tree"], dtype),
        to_dev(att["v_tree"], dtype), to_dev(anc), to_dev(n_nodes), int(ctx.max()), scale,
        ctx_layout=lay, total_ctx=total)
    torch.cuda.synchronize()
    ref = oracle.tree_attention(dtype, att["q"], kc, vc, offs, att["k_tree"], att["v_tree"], anc,
                                n_nodes, scale)
    got = sy.as_f32(to_host(out), dtype).astype(np.float64)
    reff = sy.as_f32(ref, dtype).astype(np.float64)
    for s in range(b):
        nn = int(n_nodes[s])
        assert _row_errors(got[s, :nn], reff[s, :nn]).max() <= 2e-2, s
        assert not got[s, nn:].any()
