"""GPU parity of the bookkeeping between rounds: tree attention over a
slotted cache (start, len per sequence), the KV commit after acceptance,
slot selection with row-gathered top-k, and the flattened slot-block layout
of quadratic self-speculation (Appendix C stages I, II and IV).  Every
input the oracle sees comes from the oracle or the synthetic generators."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_22634_amd as P
import synthetic as sy
from gpu_util import attn_data, oracle_tree, round_data, to_dev, to_host, tree_to_dev

pytestmark = pytest.mark.gpu


def _slotted(att, caps, gap_seed):
    """The packed cache of `att` re-laid into per-sequence slots of `caps`
    rows with random gaps; returns (k, v, ctx [b, 2], starts)."""
    offs = att["ctx_offsets"]
    B = len(offs) - 1
    rng = np.random.default_rng(gap_seed)
    starts, pos = [], 0
    for b in range(B):
        pos += int(rng.integers(0, 40))
        starts.append(pos)
        pos += int(caps[b])
    rows = pos + 8
    k = np.zeros((rows,) + att["k_cache"].shape[1:], att["k_cache"].dtype)
    v = np.zeros_like(k)
    ctx = np.zeros((B, 2), np.int32)
    for b in range(B):
        n = offs[b + 1] - offs[b]
        k[starts[b]:starts[b] + n] = att["k_cache"][offs[b]:offs[b + 1]]
        v[starts[b]:starts[b] + n] = att["v_cache"][offs[b]:offs[b + 1]]
        ctx[b] = (starts[b], n)
    return k, v, ctx, np.array(starts)


def _rel_err(got, ref):
    num = np.linalg.norm(got - ref, axis=-1)
    return num / np.maximum(np.linalg.norm(ref, axis=-1), 1e-30)


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_attention_slotted_cache_equals_packed(cfg):
    w, _ = round_data(cfg)
    _, att = attn_data(cfg)
    th = oracle_tree(cfg)
    td = tree_to_dev(th)
    caps = (np.diff(att["ctx_offsets"]) + 64).astype(np.int32)
    k, v, ctx, _ = _slotted(att, caps, cfg)
    max_ctx = int(np.diff(att["ctx_offsets"]).max())
    print(f"slotted attention cfg={cfg}", flush=True)
    out = P.presto_tree_attention(to_dev(att["q"], w.dtype), to_dev(k, w.dtype), to_dev(v, w.dtype),
                                  to_dev(ctx), to_dev(att["k_tree"], w.dtype),
                                  to_dev(att["v_tree"], w.dtype), td["anc"], td["n_nodes"],
                                  max_ctx, w.scale, ctx_layout=P.PRESTO_CTX_SLOTS)
    torch.cuda.synchronize()
    ref = oracle.tree_attention(w.dtype, att["q"], att["k_cache"], att["v_cache"],
                                att["ctx_offsets"], att["k_tree"], att["v_tree"], th["anc"],
                                th["n_nodes"], w.scale)
    got = sy.as_f32(to_host(out), w.dtype).astype(np.float64)
    reff = sy.as_f32(ref, w.dtype).astype(np.float64)
    tol = 2e-2 if w.dtype == "bf16" else 1e-4
    for s in range(w.batch):
        nn = int(th["n_nodes"][s])
        assert _rel_err(got[s, :nn], reff[s, :nn]).max() <= tol
        assert not got[s, nn:].any()


def _accept_for(cfg):
    w, rin = round_data(cfg)
    th = oracle_tree(cfg)
    T = sy.target_logits(w, rin["field"], th["parent"], th["rank"], th["n_nodes"])
    return w, th, oracle.accept(w.dtype, T, th["parent"], th["token"], th["n_nodes"], w.depth)


@pytest.mark.parametrize("cfg", [1, 2, 3, 5])
def test_commit_kv_matches_oracle(cfg):
    w, th, acc = _accept_for(cfg)
    _, att = attn_data(cfg)
    caps = (np.diff(att["ctx_offsets"]) + w.depth + 1).astype(np.int32)
    caps[0] = np.diff(att["ctx_offsets"])[0] + int(acc["accept_len"][0])  # one row short
    k, v, ctx, _ = _slotted(att, caps, 100 + cfg)
    kd, vd, cd = to_dev(k, w.dtype), to_dev(v, w.dtype), to_dev(ctx)
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    print(f"commit cfg={cfg} accept_len={acc['accept_len'].tolist()[:4]}", flush=True)
    P.presto_commit_kv(to_dev(att["k_tree"], w.dtype), to_dev(att["v_tree"], w.dtype),
                       to_dev(acc["path"]), to_dev(acc["accept_len"]), kd, vd, cd, to_dev(caps),
                       flags=flags)
    torch.cuda.synchronize()
    ok, ov, octx, skipped = oracle.commit_kv(att["k_tree"], att["v_tree"], acc["path"],
                                             acc["accept_len"], k, v, ctx, caps)
    assert skipped[0] and not skipped[1:].any()
    assert int(flags.item()) == P.PRESTO_FLAG_KV_COMMIT
    np.testing.assert_array_equal(to_host(cd), octx)
    np.testing.assert_array_equal(to_host(kd), ok)
    np.testing.assert_array_equal(to_host(vd), ov)


def test_two_rounds_through_a_slotted_cache():
    """Round 1 attention -> accept -> commit; round 2 attends over the grown
    cache with a fresh tree.  The GPU chain and the oracle chain start from
    the same inputs and must agree."""
    cfg = 3
    w, th, acc = _accept_for(cfg)
    _, att = attn_data(cfg)
    caps = (np.diff(att["ctx_offsets"]) + 4 * (w.depth + 1)).astype(np.int32)
    k, v, ctx, starts = _slotted(att, caps, 7)
    kd, vd, cd, capd = to_dev(k, w.dtype), to_dev(v, w.dtype), to_dev(ctx), to_dev(caps)
    P.presto_commit_kv(to_dev(att["k_tree"], w.dtype), to_dev(att["v_tree"], w.dtype),
                       to_dev(acc["path"]), to_dev(acc["accept_len"]), kd, vd, cd, capd)
    ok, ov, octx, _ = oracle.commit_kv(att["k_tree"], att["v_tree"], acc["path"], acc["accept_len"],
                                       k, v, ctx, caps)
    # round 2: the next layer's draws as the new tree's Q/K/V, the same tree shape
    _, att2 = attn_data(cfg, 1) if w.layers > 1 else (None, sy.attention_inputs(w.with_(seed=99)))
    td = tree_to_dev(th)
    max_ctx = int(octx[:, 1].max())
    out = P.presto_tree_attention(to_dev(att2["q"], w.dtype), kd, vd, cd,
                                  to_dev(att2["k_tree"], w.dtype), to_dev(att2["v_tree"], w.dtype),
                                  td["anc"], td["n_nodes"], max_ctx, w.scale,
                                  ctx_layout=P.PRESTO_CTX_SLOTS)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_host(cd), octx)
    # the oracle attends over its own committed cache, repacked
    packed_k = np.concatenate([ok[s:s + n] for s, n in octx])
    packed_v = np.concatenate([ov[s:s + n] for s, n in octx])
    offs = np.concatenate([[0], np.cumsum(octx[:, 1])]).astype(np.int32)
    ref = oracle.tree_attention(w.dtype, att2["q"], packed_k, packed_v, offs, att2["k_tree"],
                                att2["v_tree"], th["anc"], th["n_nodes"], w.scale)
    got = sy.as_f32(to_host(out), w.dtype).astype(np.float64)
    reff = sy.as_f32(ref, w.dtype).astype(np.float64)
    for s in range(w.batch):
        nn = int(th["n_nodes"][s])
        assert _rel_err(got[s, :nn], reff[s, :nn]).max() <= 2e-2


@pytest.mark.parametrize("slots,first", [(16, 1), (17, 1), (5, 0)])
def test_select_slots_and_topk_rows_match_oracle(slots, first):
    cfg = 3
    w, th, acc = _accept_for(cfg)
    rng = np.random.default_rng([slots, first])
    V = 4099
    logits = sy.cast((rng.standard_normal((w.batch * w.n_max * slots, V)) * 4).astype(np.float32),
                     "bf16")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    ri = P.presto_select_slots(to_dev(acc["path"]), to_dev(acc["accept_len"]), w.n_max, slots,
                               first, flags=flags)
    ids, lp, lse = P.presto_topk_rows(to_dev(logits, "bf16"), ri.view(-1), w.k, flags=flags)
    torch.cuda.synchronize()
    assert int(flags.item()) == 0
    want_rows = oracle.select_slots(acc["path"], acc["accept_len"], w.n_max, slots, first)
    np.testing.assert_array_equal(to_host(ri), want_rows)
    rid, rlp, rlse, _ = oracle.topk(np.ascontiguousarray(logits[want_rows.reshape(-1)]), w.k, "bf16")
    np.testing.assert_array_equal(to_host(ids), rid)
    np.testing.assert_allclose(to_host(lp), rlp, rtol=0, atol=1e-5 * max(1.0, np.abs(rlp).max()))
    np.testing.assert_allclose(to_host(lse), rlse, rtol=1e-6, atol=1e-6)


def test_topk_rows_bad_index_is_flagged():
    x = np.random.default_rng(3).standard_normal((6, 3000)).astype(np.float32)
    idx = torch.tensor([5, -1, 0, 6, 2], dtype=torch.int64, device="cuda")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")
    ids, lp, lse = P.presto_topk_rows(to_dev(x), idx, 3, flags=flags)
    torch.cuda.synchronize()
    assert int(flags.item()) & P.PRESTO_FLAG_BAD_INDEX
    lp, lse = to_host(lp), to_host(lse)
    for r in (1, 3):
        assert np.isneginf(lse[r]) and np.isneginf(lp[r]).all()
    rid, rlp, _, _ = oracle.topk(np.ascontiguousarray(x[[5, 0, 2]]), 3, "f32")
    np.testing.assert_array_equal(to_host(ids)[[0, 2, 4]], rid)


@pytest.mark.parametrize("cfg,slots", [(1, 3), (2, 1), (2, 14), (3, 4), (4, 2), (5, 3), (1, 64), (2, 64), (2, 63)])
def test_flatten_slots_matches_oracle(cfg, slots):
    w, th, _ = _accept_for(cfg)
    root_pos = np.random.default_rng(cfg).integers(0, 9000, w.batch).astype(np.int32)
    td = tree_to_dev(th)
    g = P.presto_flatten_slots(td["depth"], td["anc"], td["n_nodes"], to_dev(root_pos), slots)
    torch.cuda.synchronize()
    o = oracle.flatten_slots(th["parent"], th["depth"], th["n_nodes"], root_pos, slots)
    np.testing.assert_array_equal(to_host(g["pos"]), o["pos"])
    np.testing.assert_array_equal(to_host(g["anc"]).view(np.uint64), o["anc"])
    np.testing.assert_array_equal(to_host(g["n_rows"]), o["n_rows"])


def test_composite_attention_over_flattened_slots():
    """The flattened mask drives presto_tree_attention over the composite
    rows (65 nodes x (1 + 14 slots) = 975 rows)."""
    cfg, slots = 2, 14
    w, th, _ = _accept_for(cfg)
    R = w.n_max * (1 + slots)
    f = oracle.flatten_slots(th["parent"], th["depth"], th["n_nodes"], np.zeros(w.batch), slots)
    wc = w.with_(budget=R - 1)
    att = sy.attention_inputs(wc)
    out = P.presto_tree_attention(to_dev(att["q"], w.dtype), to_dev(att["k_cache"], w.dtype),
                                  to_dev(att["v_cache"], w.dtype), to_dev(att["ctx_offsets"]),
                                  to_dev(att["k_tree"], w.dtype), to_dev(att["v_tree"], w.dtype),
                                  to_dev(f["anc"]), to_dev(f["n_rows"]),
                                  int(np.diff(att["ctx_offsets"]).max()), w.scale)
    torch.cuda.synchronize()
    rows = [(0, r, h) for r in (0, 1, 7, 15, 16, 30, 31, 500, 974) for h in (0, 5, 31)]
    ref = oracle.tree_attention_rows(w.dtype, att["q"], att["k_cache"], att["v_cache"],
                                     att["ctx_offsets"], att["k_tree"], att["v_tree"], f["anc"],
                                     f["n_rows"], rows, w.scale)
    got = sy.as_f32(to_host(out), w.dtype).astype(np.float64)
    for i, (b, r, h) in enumerate(rows):
        if r < int(f["n_rows"][0]):
            assert _rel_err(got[b, r, h][None], ref[i][None])[0] <= 2e-2, (r, h)
