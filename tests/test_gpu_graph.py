"""A whole round (top-k -> tree build -> tree attention -> accept) captured
once into a HIP graph and replayed gives the eager result, bit for bit, on
every replay, with other eager rounds (on other inputs, into the same output
buffers) and host synchronisations between the replays.  The library only
launches kernels (no memset nodes, no host calls), which is what makes the
round capturable; this is the check that it stays so."""
import numpy as np
import pytest
import torch

import paper_2607_22634_amd as P
import synthetic as sy
from gpu_util import oracle_tree, round_data, to_dev, to_host

pytestmark = pytest.mark.gpu


def _setup(cfg):
    w, rin = round_data(cfg)
    tree = oracle_tree(cfg)
    target = sy.target_logits(w, rin["field"], tree["parent"], tree["rank"], tree["n_nodes"])
    att = sy.attention_inputs(w, 0, rin["ctx"])
    inp = {
        "drafter": to_dev(rin["drafter_logits"], w.dtype),
        "rho": to_dev(rin["rho"]), "lam": to_dev(rin["lam"]), "root": to_dev(rin["root_token"]),
        "target": to_dev(target, w.dtype),
        "att": {k: to_dev(v, w.dtype if v.dtype == np.uint16 else None) for k, v in att.items()},
    }
    return w, rin, inp


def _outputs(w, inp):
    dev = inp["drafter"].device
    i32 = dict(dtype=torch.int32, device=dev)
    rows, N = w.batch * w.depth, w.n_max
    W = (N + 63) // 64
    return {
        "ids": torch.empty(rows, w.k, **i32),
        "logprob": torch.empty(rows, w.k, dtype=torch.float32, device=dev),
        "lse": torch.empty(rows, dtype=torch.float32, device=dev),
        "tree": {"n_nodes": torch.empty(w.batch, **i32), "parent": torch.empty(w.batch, N, **i32),
                 "token": torch.empty(w.batch, N, **i32), "depth": torch.empty(w.batch, N, **i32),
                 "rank": torch.empty(w.batch, N, **i32),
                 "score": torch.empty(w.batch, N, dtype=torch.float32, device=dev),
                 "anc": torch.empty(w.batch, N, W, dtype=torch.int64, device=dev)},
        "attn": torch.empty_like(inp["att"]["q"]),
        "acc": {"accept_len": torch.empty(w.batch, **i32), "path": torch.empty(w.batch, w.depth + 1, **i32),
                "bonus": torch.empty(w.batch, **i32), "target_argmax": torch.empty(w.batch, N, **i32)},
        "flags": torch.zeros(1, **i32),
    }


def _round(w, rin, inp, out, ws):
    a = inp["att"]
    P.presto_topk(inp["drafter"], w.k, ids=out["ids"], logprob=out["logprob"], lse=out["lse"],
                  flags=out["flags"], workspace=ws["topk"])
    P.presto_build_tree(out["ids"], out["logprob"], inp["rho"], inp["lam"], inp["root"], w.depth, w.k,
                        w.budget, out=out["tree"], workspace=ws["tree"])
    P.presto_tree_attention(a["q"], a["k_cache"], a["v_cache"], a["ctx_offsets"], a["k_tree"],
                            a["v_tree"], out["tree"]["anc"], out["tree"]["n_nodes"],
                            int(rin["ctx"].max()), w.scale, out=out["attn"], workspace=ws["attn"])
    P.presto_accept(inp["target"], out["tree"]["parent"], out["tree"]["token"],
                    out["tree"]["n_nodes"], w.depth, out=out["acc"], flags=out["flags"],
                    workspace=ws["acc"])


def _snapshot(out):
    snap = {}
    for k, v in out.items():
        if isinstance(v, dict):
            for kk, vv in v.items():
                snap[f"{k}.{kk}"] = to_host(vv).copy()
        else:
            snap[k] = to_host(v).copy()
    return snap


def _workspaces(w, rin, inp):
    import ctypes

    lib = P.lib()
    dev = inp["drafter"].device

    def buf(n):
        return torch.empty(max(1, n), dtype=torch.uint8, device=dev)

    N = w.n_max
    desc = P.AttnDesc(w.batch, N, w.hq, w.hkv, w.head_dim, int(rin["ctx"].max()), w.scale,
                      P.PRESTO_DT_BF16 if w.dtype == "bf16" else P.PRESTO_DT_F32)
    tdesc = P.TreeDesc(w.batch, w.depth, w.k, w.k, w.budget, P.PRESTO_TREE_BEST_FIRST, 0,
                       int(np.asarray(rin["lam"]).ndim == 2))
    return {"topk": buf(lib.presto_topk_workspace(w.batch * w.depth, w.vocab, w.k)),
            "tree": buf(lib.presto_build_tree_workspace(ctypes.byref(tdesc))),
            "attn": buf(lib.presto_tree_attention_workspace(ctypes.byref(desc))),
            "acc": buf(lib.presto_accept_workspace(w.batch, N, w.vocab))}


@pytest.mark.parametrize("cfg", [2, 3])
def test_round_graph_replays_match_eager(cfg):
    w, rin, inp = _setup(cfg)
    out = _outputs(w, inp)
    ws = _workspaces(w, rin, inp)
    print(f"graph round cfg={cfg}: eager reference", flush=True)
    _round(w, rin, inp, out, ws)
    torch.cuda.synchronize()
    ref = _snapshot(out)
    assert int(out["flags"].item()) == 0

    # other inputs for the eager rounds between replays (same shapes)
    other = dict(inp)
    other["drafter"] = inp["drafter"].flip(-1).contiguous()
    other["target"] = inp["target"].roll(1, dims=-1).contiguous()

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.graph(g, stream=side):
        _round(w, rin, inp, out, ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for rep in range(4):
        print(f"graph round cfg={cfg}: replay {rep}", flush=True)
        _round(w, rin, other, out, ws)       # eager round on other inputs, same buffers
        torch.cuda.synchronize()
        for v in list(out.values()):
            for t in (v.values() if isinstance(v, dict) else [v]):
                if t is not out["flags"]:
                    t.view(torch.uint8).fill_(0xA5)
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(out)
        for k in ref:
            if k == "flags":
                continue
            np.testing.assert_array_equal(got[k], ref[k], err_msg=f"replay {rep}: {k}")
