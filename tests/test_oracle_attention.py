"""Pins for the oracle's tree-masked attention (no GPU).

* Per-path recomputation (Appendix C stage I: a draft token attends to the
  committed prefix and its ancestors): each node's output equals ordinary
  attention of its query over the explicit sequence [cache ; root .. node],
  rebuilt from parent pointers, not from the mask.
* A chain tree is causal attention: torch's scaled_dot_product_attention
  with is_causal over [cache ; chain], with GQA head grouping.
* Root-only trees are plain decode attention over [cache ; root].
"""
import numpy as np
import pytest
import torch

import oracle
import synthetic as sy
from brute import anc_from_parent, path_attention


def _random_tree(rng, b, N):
    parent = np.full((b, N), -1, np.int32)
    n_nodes = rng.integers(1, N + 1, size=b).astype(np.int32)
    n_nodes[0] = N
    for s in range(b):
        for n in range(1, int(n_nodes[s])):
            parent[s, n] = rng.integers(0, n)
    return parent, n_nodes


def _inputs(rng, dtype, b, N, hq, hkv, d, ctx):
    offs = np.zeros(b + 1, np.int32)
    offs[1:] = np.cumsum(ctx)
    f = lambda *s: sy.cast(rng.standard_normal(s, dtype=np.float32), dtype)
    return f(b, N, hq, d), f(int(offs[-1]), hkv, d), f(int(offs[-1]), hkv, d), offs, \
        f(b, N, hkv, d), f(b, N, hkv, d)


@pytest.mark.parametrize("dtype,hq,hkv,d", [("f32", 2, 1, 64), ("bf16", 8, 2, 128), ("f32", 4, 4, 64)])
def test_attention_equals_per_path_recompute(dtype, hq, hkv, d):
    rng = np.random.default_rng([hq, hkv, d])
    b, N = 3, 21
    ctx = np.array([5, 1, 17], np.int32)
    q, kc, vc, offs, kt, vt = _inputs(rng, dtype, b, N, hq, hkv, d, ctx)
    parent, n_nodes = _random_tree(rng, b, N)
    anc = anc_from_parent(parent, n_nodes, N)
    scale = 1 / np.sqrt(d)
    out = oracle.tree_attention(dtype, q, kc, vc, offs, kt, vt, anc, n_nodes)
    rows = np.array([(s, n, h) for s in range(b) for n in range(N) for h in range(hq)], np.int32)
    exact = oracle.tree_attention_rows(dtype, q, kc, vc, offs, kt, vt, anc, n_nodes, rows)
    qf, kcf, vcf, ktf, vtf = (sy.as_f32(x, dtype) for x in (q, kc, vc, kt, vt))
    outf = sy.as_f32(out, dtype)
    for i, (s, n, h) in enumerate(rows):
        if n >= n_nodes[s]:
            assert not exact[i].any() and not outf[s, n, h].any()
            continue
        ref = path_attention(qf, kcf, vcf, offs, ktf, vtf, parent, s, n, h, scale)
        np.testing.assert_allclose(exact[i], ref, rtol=1e-10, atol=1e-12)
        # rounded output is the exact value rounded once to the storage type
        tol = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -23
        np.testing.assert_allclose(outf[s, n, h], ref, rtol=tol, atol=1e-30)


def test_chain_tree_is_causal_sdpa_with_gqa():
    rng = np.random.default_rng(5)
    b, N, hq, hkv, d, ctx = 1, 9, 6, 2, 64, 13
    q, kc, vc, offs, kt, vt = _inputs(rng, "f32", b, N, hq, hkv, d, np.array([ctx], np.int32))
    parent = np.arange(-1, N - 1, dtype=np.int32)[None]
    n_nodes = np.array([N], np.int32)
    anc = anc_from_parent(parent, n_nodes, N)
    out = oracle.tree_attention("f32", q, kc, vc, offs, kt, vt, anc, n_nodes)
    K = torch.from_numpy(np.concatenate([kc, kt[0]], 0)).double().permute(1, 0, 2)[None]
    V = torch.from_numpy(np.concatenate([vc, vt[0]], 0)).double().permute(1, 0, 2)[None]
    # queries sit at the last N positions of a causal sequence of length ctx + N
    Q = torch.zeros(1, hq, ctx + N, d, dtype=torch.float64)
    Q[0, :, ctx:] = torch.from_numpy(q[0]).double().permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(Q, K, V, is_causal=True, enable_gqa=True)
    ref = ref[0, :, ctx:].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(out[0], ref, rtol=2e-6, atol=1e-7)


def test_root_only_is_decode_attention():
    rng = np.random.default_rng(6)
    b, N, hq, hkv, d = 2, 4, 4, 1, 64
    ctx = np.array([30, 3], np.int32)
    q, kc, vc, offs, kt, vt = _inputs(rng, "f32", b, N, hq, hkv, d, ctx)
    parent = np.full((b, N), -1, np.int32)
    n_nodes = np.ones(b, np.int32)
    anc = anc_from_parent(parent, n_nodes, N)
    out = oracle.tree_attention("f32", q, kc, vc, offs, kt, vt, anc, n_nodes)
    for s in range(b):
        K = torch.from_numpy(np.concatenate([kc[offs[s]:offs[s + 1]], kt[s, :1]], 0)).double()
        V = torch.from_numpy(np.concatenate([vc[offs[s]:offs[s + 1]], vt[s, :1]], 0)).double()
        Q = torch.from_numpy(q[s, 0]).double()
        ref = torch.nn.functional.scaled_dot_product_attention(
            Q[:, None], K.permute(1, 0, 2).expand(hq, -1, -1), V.permute(1, 0, 2).expand(hq, -1, -1))
        np.testing.assert_allclose(out[s, 0], ref[:, 0].numpy(), rtol=2e-6, atol=1e-7)
        assert not out[s, 1:].any()
