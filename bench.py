#!/usr/bin/env python3
"""Tree-verify rounds/s of the PRESTO draft-to-verify hot path on one MI355X.

One step = one whole round on one batch of synthetic inputs already resident
in HBM: presto_topk -> presto_build_tree -> presto_tree_attention (every
layer of the workload) -> presto_accept, enqueued on one stream with no host
synchronisation inside (--launch graph replays each round from a HIP graph
captured once per input replica instead).  Inputs are replicated in device memory and the steps
cycle through the replicas, so that every step reads data that has been
pushed out of the 256 MB last-level cache by the steps in between (the
numbers are DRAM numbers, not cache numbers).

Printed: one JSON line with rounds/s, per-stage times and achieved
bandwidth, the roofline of the dominant kernel and the CPU oracle timed on
the host's cores on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tree-verify rounds/sec at Qwen3-8B shapes; HBM GB/s of tree-attn + top-k"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_TFLOPS = 2500.0
MALL_BYTES = 256 << 20


def algorithmic_work(w, ctx, n_nodes, depth_of_nodes):
    """Bytes/flops the method must move or compute (padding and masks excluded)."""
    e = 2 if w.dtype == "bf16" else 4
    rows = w.batch * w.depth
    topk_bytes = rows * w.vocab * e + rows * (8 * w.k + 4)
    argmax_bytes = int(n_nodes.sum()) * w.vocab * e
    attn_bytes = sum(w.hkv * (int(c) + int(n)) * w.head_dim * 2 * e + int(n) * w.hq * w.head_dim * 2 * e
                     for c, n in zip(ctx, n_nodes))
    attn_flops = 0
    for s in range(w.batch):
        d = depth_of_nodes[s, : int(n_nodes[s])].astype(np.int64)
        attn_flops += int((w.hq * 4 * w.head_dim * (int(ctx[s]) + d + 1)).sum())
    return {"topk_bytes": topk_bytes, "argmax_bytes": argmax_bytes,
            "attn_bytes_per_layer": attn_bytes, "attn_flops_per_layer": attn_flops}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=2, help="synthetic workload 1..5")
    ap.add_argument("--replicas", type=int, default=0, help="input copies cycled (0 = auto)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-at-scale", action="store_true",
                    help="skip the kernels timed at the larger workloads' shapes")
    ap.add_argument("--launch", choices=["stream", "graph"], default="stream",
                    help="timed rounds: every kernel launched on the stream (default), or one "
                         "captured HIP graph per input replica, replayed (measured slower)")
    ap.add_argument("--at-scale-run", action="store_true",
                    help="only the at-scale kernels (printed as JSON), for rocprofv3 counter runs")
    ap.add_argument("--round-run", type=int, default=0,
                    help="only the whole rounds of workload 3, 4 or 5 (printed as JSON), for rocprofv3")
    ap.add_argument("--traffic-run", action="store_true",
                    help="only the workload's tree attention (5 calls) and a 256 MiB device copy "
                         "(3 calls), for rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the round is independent per sequence and this "
              "build measures one GPU's share; use --gpus 1", file=sys.stderr)
        return 2

    import torch

    import paper_2607_22634_amd as P
    import synthetic as sy

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.at_scale_run:
        print(json.dumps(measure_at_scale(P, sy, dev)), flush=True)
        return 0
    if args.round_run:
        print(json.dumps({sy.workload(args.round_run).name:
                          measure_round_at_scale(P, sy, args.round_run, dev)}), flush=True)
        return 0
    w = sy.workload(args.workload)
    t_gen = time.time()
    rin = sy.round_inputs(w)

    def dv(a, dtype=None):
        if dtype == "bf16" or a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    drafter = dv(rin["drafter_logits"], w.dtype)
    rho, lam, root = dv(rin["rho"]), dv(rin["lam"]), dv(rin["root_token"])
    ctx = rin["ctx"]
    max_ctx = int(ctx.max())
    layers = []
    for layer in range(w.layers):
        att = sy.attention_inputs(w, layer, ctx)
        layers.append({k: dv(v, w.dtype if v.dtype == np.uint16 else None) for k, v in att.items()})

    # the tree (deterministic) fixes the target rows the verifier produces
    ids, lp, _ = P.presto_topk(drafter, w.k)
    tree = P.presto_build_tree(ids, lp, rho, lam, root, w.depth, w.k, w.budget)
    torch.cuda.synchronize()
    th = {k: v.cpu().numpy() for k, v in tree.items()}
    target = dv(sy.target_logits(w, rin["field"], th["parent"], th["rank"], th["n_nodes"]), w.dtype)
    gen_s = time.time() - t_gen

    if args.traffic_run:
        return traffic_run(P, w, layers, tree, max_ctx, dev)

    work = algorithmic_work(w, ctx, th["n_nodes"], th["depth"])
    step_bytes = (work["topk_bytes"] + work["argmax_bytes"] + w.layers * work["attn_bytes_per_layer"])
    reps = args.replicas or max(1, min(16, -(-2 * MALL_BYTES // max(step_bytes, 1))))

    # replicas of every input the round reads; outputs and workspaces preallocated
    def clone(t):
        return t.clone()

    R = []
    for r in range(reps):
        R.append({
            "drafter": drafter if r == 0 else clone(drafter),
            "target": target if r == 0 else clone(target),
            "layers": layers if r == 0 else [{k: clone(v) for k, v in L.items()} for L in layers],
        })
    i32 = dict(dtype=torch.int32, device=dev)
    rows = w.batch * w.depth
    topk_out = (torch.empty(rows, w.k, **i32), torch.empty(rows, w.k, dtype=torch.float32, device=dev),
                torch.empty(rows, dtype=torch.float32, device=dev))
    topk_ws = torch.zeros(max(1, P.lib().presto_topk_workspace(rows, w.vocab, w.k)), dtype=torch.uint8,
                          device=dev)
    N = w.n_max
    tree_out = {k: torch.empty_like(v) for k, v in tree.items()}
    attn_out = [torch.empty_like(L["q"]) for L in layers]
    total_ctx = int(np.asarray(ctx).sum())
    desc = P.AttnDesc(w.batch, N, w.hq, w.hkv, w.head_dim, max_ctx, w.scale,
                      P.PRESTO_DT_BF16 if w.dtype == "bf16" else P.PRESTO_DT_F32,
                      P.PRESTO_CTX_PACKED, total_ctx)
    import ctypes
    attn_ws_n = P.lib().presto_tree_attention_workspace(ctypes.byref(desc))
    attn_ws = torch.zeros(max(1, attn_ws_n), dtype=torch.uint8, device=dev) if attn_ws_n else None
    acc_out = {"accept_len": torch.empty(w.batch, **i32), "path": torch.empty(w.batch, w.depth + 1, **i32),
               "bonus": torch.empty(w.batch, **i32), "target_argmax": torch.empty(w.batch, N, **i32)}
    acc_ws = torch.zeros(P.lib().presto_accept_workspace(w.batch, N, w.vocab), dtype=torch.uint8,
                         device=dev)
    flags = torch.zeros(1, **i32)

    stream = torch.cuda.current_stream()

    def st_topk(r):
        P.presto_topk(R[r]["drafter"], w.k, ids=topk_out[0], logprob=topk_out[1], lse=topk_out[2],
                      flags=flags, workspace=topk_ws)

    def st_tree(r):
        P.presto_build_tree(topk_out[0], topk_out[1], rho, lam, root, w.depth, w.k, w.budget,
                            out=tree_out)

    def st_attn(r):
        for li, L in enumerate(R[r]["layers"]):
            P.presto_tree_attention(L["q"], L["k_cache"], L["v_cache"], L["ctx_offsets"],
                                    L["k_tree"], L["v_tree"], tree_out["anc"], tree_out["n_nodes"],
                                    max_ctx, w.scale, out=attn_out[li], workspace=attn_ws,
                                    total_ctx=total_ctx)

    def st_accept(r):
        P.presto_accept(R[r]["target"], tree_out["parent"], tree_out["token"], tree_out["n_nodes"],
                        w.depth, out=acc_out, flags=flags, workspace=acc_ws)

    stage_fns = [st_topk, st_tree, st_attn, st_accept]

    def step(r):
        for f in stage_fns:
            f(r)

    def timed(fn, n, offset):
        """Average ms of `fn` over n back-to-back launches (replicas cycled)."""
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for i in range(n):
            fn((offset + i) % reps)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    for i in range(args.warmup):
        step(i % reps)
    torch.cuda.synchronize()
    # K whole rounds back to back, every kernel launched on the stream
    ms_stream = timed(step, args.steps, args.warmup)
    ms_per_step = ms_stream
    if args.launch == "graph":
        # The same rounds as HIP graphs: one capture per replica (the library
        # only launches kernels), checked bit for bit against the eager round
        # of replica 0 before timing.
        def outputs():
            t = [topk_out[0], topk_out[1], tree_out["parent"], tree_out["token"], tree_out["anc"],
                 tree_out["n_nodes"], acc_out["path"], acc_out["accept_len"], acc_out["bonus"]]
            return [x.detach().clone() for x in t + attn_out]

        step(0)
        torch.cuda.synchronize()
        ref = outputs()
        graphs = []
        side = torch.cuda.Stream()
        for r in range(reps):
            g = torch.cuda.CUDAGraph()
            side.wait_stream(stream)
            with torch.cuda.graph(g, stream=side):
                step(r)
            stream.wait_stream(side)
            graphs.append(g)
        torch.cuda.synchronize()
        step(1 % reps)
        graphs[0].replay()
        torch.cuda.synchronize()
        for a, b in zip(outputs(), ref):
            assert torch.equal(a, b), "graph replay differs from the eager round"
        ms_per_step = timed(lambda r: graphs[r].replay(), args.steps, args.warmup)
    # distribution of single rounds (each bracketed by its own event pair, still
    # back to back with no host synchronisation), and the warm-cache rate with
    # one replica repeated (labelled; every other figure is cold, DRAM)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i, (a0, a1) in enumerate(ev):
        a0.record(stream)
        if args.launch == "graph":
            graphs[(args.warmup + i) % reps].replay()
        else:
            step((args.warmup + i) % reps)
        a1.record(stream)
    torch.cuda.synchronize()
    per_round_us = np.array([a0.elapsed_time(a1) * 1e3 for a0, a1 in ev])
    warm_ms = timed(lambda r: step(0), args.steps, 0)
    # per-stage device time per launch: each stage alone, launched back to
    # back from a captured HIP graph (so the host's launch cost is not in the
    # figure), cycling the replicas as the rounds do
    stage_ms = np.array([graph_time_us(f, reps) * 1e-3 for f in stage_fns])
    assert int(flags.item()) == 0, "device flagged NaN inputs"

    names = ["topk", "build_tree", "tree_attention", "accept"]
    stages = {"timing": "device time per launch, from graph replays of back-to-back launches"}
    for j, nme in enumerate(names):
        us = float(stage_ms[j] * 1e3)
        entry = {"us": round(us, 2)}
        if nme == "topk":
            entry["GB/s"] = round(work["topk_bytes"] / (us * 1e3), 1)
        elif nme == "build_tree":
            # a sequential search per sequence: latency per committed node
            entry["ns_per_node"] = round(us * 1e3 / max(1, int(np.asarray(th["n_nodes"]).max()) - 1), 1)
        elif nme == "tree_attention":
            entry["GB/s"] = round(w.layers * work["attn_bytes_per_layer"] / (us * 1e3), 1)
            entry["TFLOP/s"] = round(w.layers * work["attn_flops_per_layer"] / (us * 1e6), 2)
        elif nme == "accept":
            entry["GB/s"] = round(work["argmax_bytes"] / (us * 1e3), 1)
        stages[nme] = entry

    # roofline of the dominant kernel among the bandwidth/compute-bound stages
    dom = max(["topk", "tree_attention", "accept"], key=lambda s_: stages[s_]["us"])
    us = stages[dom]["us"]
    if dom == "tree_attention":
        t_hbm = w.layers * work["attn_bytes_per_layer"] / (HBM_PEAK_GBS * 1e3)
        t_mfma = w.layers * work["attn_flops_per_layer"] / (MFMA_BF16_TFLOPS * 1e6)
        if t_mfma > t_hbm:
            roof = {"bound": "mfma", "achieved": stages[dom]["TFLOP/s"], "peak": MFMA_BF16_TFLOPS,
                    "unit": "TFLOP/s"}
        else:
            roof = {"bound": "hbm", "achieved": stages[dom]["GB/s"], "peak": HBM_PEAK_GBS,
                    "unit": "GB/s"}
    else:
        roof = {"bound": "hbm", "achieved": stages[dom]["GB/s"], "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["kernel"] = dom
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = measured_traffic(dom, w)

    extra = measure_next_rows(P, sy, w, R, reps, timed, topk_out, topk_ws, tree_out, rin, dev)
    rounds = None if args.no_at_scale else {
        sy.workload(c).name: measure_round_at_scale(P, sy, c, dev) for c in (3, 4, 5)}
    at_scale = None if args.no_at_scale else measure_at_scale(P, sy, dev)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, rin, layers, args.cpu_seconds)

    line = {
        "metric": METRIC, "value": round(1e3 / ms_per_step, 2), "unit": "rounds/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "launch": "hip-graph" if args.launch == "graph" else "stream",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: batch {w.batch}, block {w.depth}, vocab {w.vocab}, "
                               f"top-{w.k}, budget {w.budget}, GQA {w.hq}q/{w.hkv}kv d{w.head_dim}, "
                               f"ctx {w.ctx[0]}-{w.ctx[1]}, {w.layers} layer(s)",
                   "global_batch": w.batch, "replicas": reps},
        "sequence_rounds_per_s": round(w.batch * 1e3 / ms_per_step, 2),
        "round_us": {"p10": round(float(np.percentile(per_round_us, 10)), 2),
                     "p50": round(float(np.percentile(per_round_us, 50)), 2),
                     "p90": round(float(np.percentile(per_round_us, 90)), 2),
                     "rounds": int(per_round_us.size)},
        "warm_rounds_per_s": round(1e3 / warm_ms, 2),
        "stages": stages, "roofline": roof, "cpu_baseline": cpu, "next_rows": extra,
        "rounds_at_scale": rounds, "at_scale": at_scale,
        "accept_len": acc_out["accept_len"].cpu().tolist(),
        "gen_seconds": round(gen_s, 1),
    }
    if args.launch == "graph":
        line["ms_per_step_stream"] = round(ms_stream, 5)
    print(json.dumps(line), flush=True)
    return 0


TRAFFIC_PROFILE = {"tree_attention": ("profiles/traffic_tree_attention_qwen3-8b-single.md",
                                      "paper_2607_22634_amd/csrc/tree_attn.hip")}


def measured_traffic(kernel: str, w):
    """HBM bytes per launch of `kernel` from the committed FETCH_SIZE /
    WRITE_SIZE summary, when that summary is for this workload and for the
    kernel source as it is now (its sha256 is recorded there); else None."""
    import hashlib

    if kernel not in TRAFFIC_PROFILE or w.name != "qwen3-8b-single":
        return None
    summary, source = (os.path.join(ROOT, x) for x in TRAFFIC_PROFILE[kernel])
    if not os.path.exists(summary):
        return None
    fields = {}
    for line in open(summary):
        if line.startswith("- ") and ":" in line:
            key, val = line[2:].split(":", 1)
            fields[key.strip()] = val.strip().strip("`")
    digest = hashlib.sha256(open(source, "rb").read()).hexdigest()
    if fields.get("source sha256") != digest or "bytes per launch" not in fields:
        return None
    return int(fields["bytes per launch"])


def traffic_run(P, w, layers, tree, max_ctx, dev) -> int:
    """A short process for counter runs: 5 tree-attention calls of the
    workload, then 3 plain copies of 256 MiB (the calibration kernel)."""
    import torch

    L = layers[0]
    out = torch.empty_like(L["q"])
    for _ in range(5):
        P.presto_tree_attention(L["q"], L["k_cache"], L["v_cache"], L["ctx_offsets"], L["k_tree"],
                                L["v_tree"], tree["anc"], tree["n_nodes"], max_ctx, w.scale, out=out)
    src = torch.ones(64 << 20, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print("traffic run done: 5 tree-attention calls, 3 copies of 256 MiB", flush=True)
    return 0


def graph_time_us(fn, calls: int, reps: int = 5) -> float:
    """Device time per call of fn(i) (i = 0 .. calls-1, so the caller can
    cycle input replicas): `calls` launches captured into one HIP graph,
    the graph replayed `reps` times, the fastest replay divided by `calls`.
    The library only launches kernels, so its calls capture as they are."""
    import torch

    stream = torch.cuda.current_stream()
    for i in range(calls):
        fn(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.graph(g, stream=side):
        for i in range(calls):
            fn(i)
    stream.wait_stream(side)
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    best = float("inf")
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1) * 1e3 / calls)
    del g
    return best


def measure_round_at_scale(P, sy, cfg: int, dev, rounds: int = 10):
    """Whole rounds (top-k -> tree -> every layer's tree attention -> accept)
    at workload `cfg`, launched on one stream as the bench workload's rounds.
    Drafter logits, lattice, lambda, root tokens and context lengths follow
    the workload's recipe (host draws); the attention inputs of every layer
    are N(0, 1) device draws of the workload's shapes, and the target logits
    follow the recipe on the device (field row of the node's depth plus
    sigma_t N(0, 1) noise) for the tree the library builds: timing inputs
    only, parity at these shapes is in the tests.  One round touches far
    more than the 256 MB last-level cache, so every round is cold."""
    import ctypes

    import torch

    w = sy.workload(cfg)
    rin = sy.round_inputs(w)
    gen = torch.Generator(device=dev)
    gen.manual_seed(1000 + cfg)
    bf = torch.bfloat16

    def up(a, bf16=False):
        t = torch.from_numpy(np.ascontiguousarray(a))
        if bf16:
            t = t.view(torch.int16).view(bf)
        return t.to(dev)

    drafter = up(rin["drafter_logits"], w.dtype == "bf16")
    rho, lam, root = up(rin["rho"]), up(rin["lam"]), up(rin["root_token"])
    ctx = rin["ctx"].astype(np.int64)
    total = int(ctx.sum())
    offs = up(np.concatenate([[0], np.cumsum(ctx)]).astype(np.int32))
    N = w.n_max

    def randn(*shape):
        return torch.randn(*shape, device=dev, generator=gen).to(bf)

    layers = [{"q": randn(w.batch, N, w.hq, w.head_dim), "kc": randn(total, w.hkv, w.head_dim),
               "vc": randn(total, w.hkv, w.head_dim), "kt": randn(w.batch, N, w.hkv, w.head_dim),
               "vt": randn(w.batch, N, w.hkv, w.head_dim)} for _ in range(w.layers)]
    rows = w.batch * w.depth
    i32 = dict(dtype=torch.int32, device=dev)
    ids = torch.empty(rows, w.k, **i32)
    lp = torch.empty(rows, w.k, dtype=torch.float32, device=dev)
    lse = torch.empty(rows, dtype=torch.float32, device=dev)
    tws = torch.zeros(max(1, P.lib().presto_topk_workspace(rows, w.vocab, w.k)), dtype=torch.uint8,
                      device=dev)
    P.presto_topk(drafter, w.k, ids=ids, logprob=lp, lse=lse, workspace=tws)
    tree = P.presto_build_tree(ids, lp, rho, lam, root, w.depth, w.k, w.budget)
    torch.cuda.synchronize()
    # target logits of the tree's nodes: F[b, depth(n)] + sigma_t N(0, 1)
    field = up(rin["field"])
    dep = tree["depth"].clamp(min=0).long()
    target = torch.empty(w.batch, N, w.vocab, dtype=bf, device=dev)
    for b in range(w.batch):
        t = field[b].index_select(0, dep[b])
        t += float(w.sigma_t) * torch.randn(t.shape, device=dev, generator=gen)
        target[b] = t.to(bf)
    del field
    out = [torch.empty_like(L["q"]) for L in layers]
    desc = P.AttnDesc(w.batch, N, w.hq, w.hkv, w.head_dim, int(ctx.max()), w.scale, P.PRESTO_DT_BF16,
                      P.PRESTO_CTX_PACKED, total)
    nws = P.lib().presto_tree_attention_workspace(ctypes.byref(desc))
    aws = torch.zeros(max(1, nws), dtype=torch.uint8, device=dev)
    acc = {"accept_len": torch.empty(w.batch, **i32), "path": torch.empty(w.batch, w.depth + 1, **i32),
           "bonus": torch.empty(w.batch, **i32), "target_argmax": torch.empty(w.batch, N, **i32)}
    accws = torch.zeros(P.lib().presto_accept_workspace(w.batch, N, w.vocab), dtype=torch.uint8, device=dev)
    flags = torch.zeros(1, **i32)

    def st_topk(i=0):
        P.presto_topk(drafter, w.k, ids=ids, logprob=lp, lse=lse, flags=flags, workspace=tws)

    def st_tree(i=0):
        P.presto_build_tree(ids, lp, rho, lam, root, w.depth, w.k, w.budget, out=tree)

    def st_attn(i=0):
        for li, L in enumerate(layers):
            P.presto_tree_attention(L["q"], L["kc"], L["vc"], offs, L["kt"], L["vt"], tree["anc"],
                                    tree["n_nodes"], int(ctx.max()), w.scale, out=out[li], workspace=aws,
                                    total_ctx=total)

    def st_accept(i=0):
        P.presto_accept(target, tree["parent"], tree["token"], tree["n_nodes"], w.depth, out=acc,
                        flags=flags, workspace=accws)

    fns = [st_topk, st_tree, st_attn, st_accept]

    def step():
        for f in fns:
            f()

    stream = torch.cuda.current_stream()
    for _ in range(2):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(rounds):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    assert int(flags.item()) == 0, "device flagged NaN inputs"
    ms = e0.elapsed_time(e1) / rounds
    nn = tree["n_nodes"].cpu().numpy()
    work = algorithmic_work(w, ctx, nn, tree["depth"].cpu().numpy())
    stage_us = [graph_time_us(lambda i, f=f: f(), 4 if f is not st_attn else 1, 3) for f in fns]
    attn_bytes = w.layers * work["attn_bytes_per_layer"]
    attn_flops = w.layers * work["attn_flops_per_layer"]
    res = {
        "rounds_per_s": round(1e3 / ms, 2), "sequence_rounds_per_s": round(w.batch * 1e3 / ms, 2),
        "ms_per_round": round(ms, 4), "rounds": rounds, "layers": w.layers,
        "stages_us": {"topk": round(stage_us[0], 2), "build_tree": round(stage_us[1], 2),
                      "tree_attention": round(stage_us[2], 2), "accept": round(stage_us[3], 2)},
        "topk_GB/s": round(work["topk_bytes"] / (stage_us[0] * 1e3), 1),
        "attention_GB/s": round(attn_bytes / (stage_us[2] * 1e3), 1),
        "attention_TFLOP/s": round(attn_flops / (stage_us[2] * 1e6), 1),
        "accept_GB/s": round(work["argmax_bytes"] / (stage_us[3] * 1e3), 1),
        "accept_len_mean": round(float(acc["accept_len"].float().mean().item()), 3),
        "inputs": "drafter logits, lattice, lambda, roots and contexts by the workload recipe; "
                  "Q/K/V N(0,1) device draws; target logits by the recipe on the device",
    }
    del layers, out, target, drafter
    torch.cuda.empty_cache()
    return res


def measure_at_scale(P, sy, dev):
    """Single stages at the larger workloads' shapes, each against its
    roofline (device time per launch from graph replays after a warm-up):
    top-k over 1024 drafter rows at k = 4, 8 and 10 (with the count of
    chunks that took the exact tie path), the accept argmax over 4128 node
    rows, tree attention at workloads 3 and 4, and tree builds (best-first
    and beam search, W = 10) at workloads 3, 4 and 5 and at the paper's
    operating point (block 16, k = 10, budgets 128 / 256 / 512).  Logits are
    N(0, 4^2) device draws of those shapes; candidate tables come from
    presto_topk on them.  Timing only: parity at these shapes is covered by
    the tests."""
    import ctypes

    import torch

    def time_us(fn, calls=8):
        t0 = time.time()
        while time.time() - t0 < 0.05:  # clocks up before timing
            fn(0)
        torch.cuda.synchronize()
        return graph_time_us(fn, calls, 5)

    def roof(bytes_, flops, us):
        gbs = bytes_ / (us * 1e3)
        tfs = flops / (us * 1e6)
        t_hbm = bytes_ / (HBM_PEAK_GBS * 1e3)
        t_mfma = flops / (MFMA_BF16_TFLOPS * 1e6)
        if t_mfma > t_hbm:
            return {"us": round(us, 2), "bound": "mfma", "TFLOP/s": round(tfs, 1), "GB/s": round(gbs, 1),
                    "frac": round(tfs / MFMA_BF16_TFLOPS, 4)}
        return {"us": round(us, 2), "bound": "hbm", "GB/s": round(gbs, 1), "TFLOP/s": round(tfs, 1),
                "frac": round(gbs / HBM_PEAK_GBS, 4)}

    def tree_latency(us, tree):
        # one wave per sequence, all sequences at once: the launch takes as
        # long as the longest sequence's search
        nodes = int(tree["n_nodes"].max().item())
        return {"us": round(us, 2), "bound": "latency", "nodes_per_seq": nodes,
                "ns_per_node": round(us * 1e3 / nodes, 1)}

    gen = torch.Generator(device=dev)
    gen.manual_seed(1234)
    i32 = dict(dtype=torch.int32, device=dev)
    out = {}

    def candidates(batch, D, V, k):
        """A candidate table from presto_topk over N(0, 4^2) bf16 drafter rows."""
        rows = batch * D
        x = (torch.randn(rows, V, device=dev, generator=gen) * 4).to(torch.bfloat16)
        ids, lp, _ = P.presto_topk(x, k)
        del x
        return ids.contiguous(), lp.contiguous()

    # top-k over workload 5's 1024 drafter rows, at k = 4, 8 and 10
    w5 = sy.workload(5)
    rows = w5.batch * w5.depth
    logits = (torch.randn(rows, w5.vocab, device=dev, generator=gen) * 4).to(torch.bfloat16)
    for k in (4, 8, 10):
        ws = torch.zeros(P.lib().presto_topk_workspace(rows, w5.vocab, k), dtype=torch.uint8, device=dev)
        o = (torch.empty(rows, k, **i32), torch.empty(rows, k, dtype=torch.float32, device=dev),
             torch.empty(rows, dtype=torch.float32, device=dev))
        us = time_us(lambda i: P.presto_topk(logits, k, ids=o[0], logprob=o[1], lse=o[2], workspace=ws))
        P.presto_topk(logits, k, ids=o[0], logprob=o[1], lse=o[2], workspace=ws)
        torch.cuda.synchronize()
        r = roof(rows * w5.vocab * 2 + rows * (8 * k + 4), 0, us)
        r["fallback_chunks"] = P.topk_fallback_chunks(ws)
        out[f"topk_1024_rows_k{k}"] = r
    del logits
    # accept argmax over workload 5's 4128 node rows
    lam = torch.full((w5.depth,), 0.2, dtype=torch.float32, device=dev)
    root = torch.zeros(w5.batch, **i32)
    ids5, lp5 = candidates(w5.batch, w5.depth, w5.vocab, w5.k)
    tree = P.presto_build_tree(ids5, lp5, None, lam, root, w5.depth, w5.k, w5.budget)
    target = (torch.randn(w5.batch * w5.n_max, w5.vocab, device=dev, generator=gen) * 4).to(torch.bfloat16)
    aws = torch.zeros(P.lib().presto_accept_workspace(w5.batch, w5.n_max, w5.vocab), dtype=torch.uint8,
                      device=dev)
    accout = {"accept_len": torch.empty(w5.batch, **i32), "path": torch.empty(w5.batch, w5.depth + 1, **i32),
              "bonus": torch.empty(w5.batch, **i32), "target_argmax": torch.empty(w5.batch, w5.n_max, **i32)}
    us = time_us(lambda i: P.presto_accept(target, tree["parent"], tree["token"], tree["n_nodes"], w5.depth,
                                           out=accout, workspace=aws))
    live = int(tree["n_nodes"].sum().item())
    out["accept_4128_rows"] = roof(live * w5.vocab * 2, 0, us)
    del target

    # tree builds: workloads 3, 4, 5 and the paper's point (k = 10, block 16)
    def trees(name, batch, D, k, B, lam_v=0.2, lattice=True):
        ids, lp = candidates(batch, D, 151936, k)
        lamw = torch.full((D,), lam_v, dtype=torch.float32, device=dev)
        rootw = torch.zeros(batch, **i32)
        rho = None
        if lattice:
            g2 = torch.Generator(device=dev)
            g2.manual_seed(77)
            u = torch.rand(batch, D, k, k, k, device=dev, generator=g2)
            rho = torch.where(torch.rand(u.shape, device=dev, generator=g2) < 0.5,
                              torch.full_like(u, float(np.log(np.float32(1e-4)))),
                              torch.log(u * (1 - 1e-3) + 1e-3))
        tr = P.presto_build_tree(ids, lp, rho, lamw, rootw, D, k, B)
        us = time_us(lambda i: P.presto_build_tree(ids, lp, rho, lamw, rootw, D, k, B, out=tr))
        out[f"tree_build_{name}"] = tree_latency(us, tr)
        bm = {kk: torch.empty_like(v) for kk, v in tr.items()}
        us = time_us(lambda i: P.presto_build_tree(ids, lp, rho, lamw, rootw, D, k, B,
                                                   mode=P.PRESTO_TREE_BEAM, beam_width=10, out=bm))
        out[f"tree_build_beam10_{name}"] = tree_latency(us, bm)

    for cfg in (3, 4, 5):
        w = sy.workload(cfg)
        trees(w.name, w.batch, w.depth, w.k, w.budget, w.lam)
    for B in (128, 256, 512):
        trees(f"paper-k10-B{B}", 1, 16, 10, B)

    # tree attention at workloads 3 and 4
    for cfg in (3, 4):
        w = sy.workload(cfg)
        ctx = sy.ctx_lengths(w).astype(np.int64)
        offs = torch.from_numpy(np.concatenate([[0], np.cumsum(ctx)]).astype(np.int32)).to(dev)
        total = int(ctx.sum())
        ids, lp = candidates(w.batch, w.depth, w.vocab, w.k)
        lamw = torch.full((w.depth,), 0.2, dtype=torch.float32, device=dev)
        tr = P.presto_build_tree(ids, lp, None, lamw, torch.zeros(w.batch, **i32), w.depth, w.k, w.budget)
        q = torch.randn(w.batch, w.n_max, w.hq, w.head_dim, device=dev, generator=gen).to(torch.bfloat16)
        kc = torch.randn(total, w.hkv, w.head_dim, device=dev, generator=gen).to(torch.bfloat16)
        vc = torch.randn(total, w.hkv, w.head_dim, device=dev, generator=gen).to(torch.bfloat16)
        kt = torch.randn(w.batch, w.n_max, w.hkv, w.head_dim, device=dev, generator=gen).to(torch.bfloat16)
        vt = torch.randn(w.batch, w.n_max, w.hkv, w.head_dim, device=dev, generator=gen).to(torch.bfloat16)
        ao = torch.empty_like(q)
        desc = P.AttnDesc(w.batch, w.n_max, w.hq, w.hkv, w.head_dim, int(ctx.max()), w.scale,
                          P.PRESTO_DT_BF16, P.PRESTO_CTX_PACKED, total)
        nws = P.lib().presto_tree_attention_workspace(ctypes.byref(desc))
        aw = torch.zeros(max(1, nws), dtype=torch.uint8, device=dev)
        us = time_us(lambda i: P.presto_tree_attention(q, kc, vc, offs, kt, vt, tr["anc"], tr["n_nodes"],
                                                       int(ctx.max()), w.scale, out=ao, workspace=aw,
                                                       total_ctx=total), calls=4)
        nn = tr["n_nodes"].cpu().numpy()
        dep = tr["depth"].cpu().numpy()
        ww = algorithmic_work(w, ctx, nn, dep)
        out[f"tree_attention_{w.name}"] = roof(ww["attn_bytes_per_layer"], ww["attn_flops_per_layer"], us)
        del q, kc, vc, kt, vt, ao, aw
    torch.cuda.empty_cache()
    return out


def measure_next_rows(P, sy, w, R, reps, timed, topk_out, topk_ws, tree_out, rin, dev):
    """Per-launch times of the parts adjacent to the round (not in the step):
    top-k with the entropy output, the entropy-adaptive weight, the trigram
    lattice gather (and the one-time table build), beam-search trees and the
    bookkeeping calls.  Device time per call from graph replays (so the
    host's launch cost is not in the figures), except the table build."""
    import torch

    rows = w.batch * w.depth
    e = 2 if w.dtype == "bf16" else 4
    n = min(8, reps)  # calls per captured graph (input replicas cycled)
    ent = torch.empty(rows, dtype=torch.float32, device=dev)
    lam_t = torch.empty(rows, dtype=torch.float32, device=dev)
    out = {"timing": "device time per call, from graph replays of back-to-back calls "
                     "(table_build_ms: host-bracketed)"}

    def topk_ent(r):
        P.presto_topk(R[r]["drafter"], w.k, ids=topk_out[0], logprob=topk_out[1], lse=topk_out[2],
                      entropy=ent, workspace=topk_ws)

    us = graph_time_us(topk_ent, n)
    out["topk_entropy"] = {"us": round(us, 2),
                           "GB/s": round((rows * w.vocab * e + rows * (8 * w.k + 8)) / (us * 1e3), 1)}
    out["entropy_lambda"] = {"us": round(graph_time_us(
        lambda r: P.presto_entropy_lambda(ent, 0.6, 2.0, out=lam_t), n), 2)}

    # trigram table: walks through this round's candidates plus 1M background trigrams
    ids_h = topk_out[0].view(w.batch, w.depth, w.k).cpu().numpy()
    t2, t1, t, lr = sy.trigram_entries(w, ids_h, 64, 1_000_000)
    cap = 1 << max(6, int(np.ceil(np.log2(2 * len(t)))))
    table = torch.empty(P.presto_ngram_table_bytes(cap), dtype=torch.uint8, device=dev)
    cols = [torch.from_numpy(x).to(dev) for x in (t2, t1, t, lr)]
    flags = torch.zeros(1, dtype=torch.int32, device=dev)

    def build(r):
        P.presto_ngram_clear(table, cap)
        P.presto_ngram_insert(table, cap, *cols, flags=flags)

    build_ms = timed(build, 3, 0)
    assert int(flags.item()) == 0, "trigram table build flagged an entry"
    prev = torch.from_numpy(sy.prev_tokens(w)).to(dev)
    root = torch.from_numpy(rin["root_token"]).to(dev)
    lat = torch.empty(w.batch, w.depth, w.k, w.k, w.k, dtype=torch.float32, device=dev)
    us = graph_time_us(lambda r: P.presto_ngram_gather(table, cap, float(np.log(1e-4)), topk_out[0],
                                                       prev, root, w.depth, w.k, out=lat), n)
    out["ngram_gather"] = {"us": round(us, 2), "lattice_entries": int(lat.numel()),
                           "table_entries": int(len(t)), "table_slots": cap,
                           "table_build_ms": round(build_ms, 3)}

    lam = torch.from_numpy(rin["lam"]).to(dev)
    rho = torch.from_numpy(rin["rho"]).to(dev)
    beam_out = {k: torch.empty_like(v) for k, v in tree_out.items()}
    us = graph_time_us(lambda r: P.presto_build_tree(topk_out[0], topk_out[1], rho, lam, root,
                                                     w.depth, w.k, w.budget, mode=P.PRESTO_TREE_BEAM,
                                                     beam_width=10, out=beam_out), n)
    out["build_tree_beam10"] = {"us": round(us, 2)}
    us = graph_time_us(lambda r: P.presto_build_tree(topk_out[0], topk_out[1], rho, lam, root,
                                                     w.depth, w.k, w.budget,
                                                     mode=P.PRESTO_TREE_BEST_FIRST_ALG2,
                                                     out=beam_out), n)
    out["build_tree_alg2"] = {"us": round(us, 2)}

    # bookkeeping after accept: commit the accepted path into a slotted cache
    L0 = R[0]["layers"][0]
    ctx_h = rin["ctx"].astype(np.int64)
    room = 64 * (w.depth + 1)
    starts = np.concatenate([[0], np.cumsum(ctx_h + room)[:-1]])
    rows_total = int((ctx_h + room).sum())
    kc = torch.zeros((rows_total,) + tuple(L0["k_cache"].shape[1:]), dtype=L0["k_cache"].dtype,
                     device=dev)
    vc = torch.zeros_like(kc)
    ctx0 = torch.from_numpy(np.stack([starts, ctx_h], 1).astype(np.int32)).to(dev)
    ctx_t = ctx0.clone()
    cap = torch.from_numpy((ctx_h + room).astype(np.int32)).to(dev)
    acc = P.presto_accept(R[0]["target"], tree_out["parent"], tree_out["token"], tree_out["n_nodes"],
                          w.depth)
    flags = torch.zeros(1, dtype=torch.int32, device=dev)
    # every call appends up to depth + 1 rows per sequence: 8 calls per graph,
    # 40 calls in all, within the 64 (depth + 1) rows of room
    us = graph_time_us(lambda r: P.presto_commit_kv(L0["k_tree"], L0["v_tree"], acc["path"],
                                                    acc["accept_len"], kc, vc, ctx_t, cap,
                                                    flags=flags), 8, 3)
    assert int(flags.item()) == 0, "commit flagged a sequence"
    m = int(acc["accept_len"].sum().item()) + w.batch
    row_b = w.hkv * w.head_dim * e
    out["commit_kv"] = {"us": round(us, 2), "rows": m, "GB/s": round(4 * m * row_b / (us * 1e3), 1)}

    # quadratic self-speculation: slot selection + in-place top-k, flattening
    S = max(1, min(1024 // w.n_max - 1, w.depth, (2 << 30) // (w.batch * w.n_max * w.vocab * e)))
    slot_rows = w.batch * w.n_max * S
    slot_logits = torch.empty(slot_rows, w.vocab, dtype=R[0]["drafter"].dtype, device=dev)
    slot_logits.copy_(R[0]["drafter"][torch.arange(slot_rows, device=dev) % rows])
    sel = P.presto_select_slots(acc["path"], acc["accept_len"], w.n_max, S, 1)
    nrows = sel.numel()
    sws = torch.zeros(max(1, P.lib().presto_topk_workspace(nrows, w.vocab, w.k)), dtype=torch.uint8,
                      device=dev)
    sel_out = (torch.empty(nrows, w.k, dtype=torch.int32, device=dev),
               torch.empty(nrows, w.k, dtype=torch.float32, device=dev),
               torch.empty(nrows, dtype=torch.float32, device=dev))

    def select_topk(r):
        P.presto_select_slots(acc["path"], acc["accept_len"], w.n_max, S, 1, out=sel)
        P.presto_topk_rows(slot_logits, sel.view(-1), w.k, ids=sel_out[0], logprob=sel_out[1],
                           lse=sel_out[2], workspace=sws)

    us = graph_time_us(select_topk, n)
    out["select_slots_topk"] = {"us": round(us, 2), "slots": S, "rows": nrows,
                                "GB/s": round(nrows * w.vocab * e / (us * 1e3), 1)}
    root_pos = torch.from_numpy(rin["ctx"].astype(np.int32)).to(dev)
    us = graph_time_us(lambda r: P.presto_flatten_slots(tree_out["depth"], tree_out["anc"],
                                                        tree_out["n_nodes"], root_pos, S), n)
    out["flatten_slots"] = {"us": round(us, 2), "rows": w.n_max * (1 + S)}
    return out


def cpu_baseline(w, rin, layers, seconds):
    """The oracle, as it stands, on whole rounds of the same workload for ~`seconds`."""
    import oracle

    threads = len(os.sched_getaffinity(0))
    oracle.set_threads(threads)

    def host(t):
        import torch
        t = t.detach().cpu()
        return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()

    import synthetic as sy

    att = [{k: host(v) for k, v in L.items()} for L in layers]
    D, k = w.depth, w.k
    # the target rows follow the oracle's own tree (input synthesis, untimed)
    ids0, lp0, _, _ = oracle.topk(rin["drafter_logits"], k, w.dtype)
    tr0 = oracle.build_tree(ids0.reshape(w.batch, D, k), lp0.reshape(w.batch, D, k), rin["rho"],
                            rin["lam"], rin["root_token"], D, k, w.budget)
    T = sy.target_logits(w, rin["field"], tr0["parent"], tr0["rank"], tr0["n_nodes"])
    n = 0
    t0 = time.time()
    while True:
        ids, lp, _, _ = oracle.topk(rin["drafter_logits"], k, w.dtype)
        tr = oracle.build_tree(ids.reshape(w.batch, D, k), lp.reshape(w.batch, D, k), rin["rho"],
                               rin["lam"], rin["root_token"], D, k, w.budget)
        for L in att:
            oracle.tree_attention(w.dtype, L["q"], L["k_cache"], L["v_cache"], L["ctx_offsets"],
                                  L["k_tree"], L["v_tree"], tr["anc"], tr["n_nodes"], w.scale)
        oracle.accept(w.dtype, T, tr["parent"], tr["token"], tr["n_nodes"], D)
        n += 1
        if time.time() - t0 >= seconds:
            break
    el = time.time() - t0
    cores = oracle.get_threads()
    # the two sequential stages on one thread as well (one call each)
    oracle.set_threads(1)
    t1 = time.time()
    ids, lp, _, _ = oracle.topk(rin["drafter_logits"], k, w.dtype)
    t2 = time.time()
    oracle.build_tree(ids.reshape(w.batch, D, k), lp.reshape(w.batch, D, k), rin["rho"], rin["lam"],
                      rin["root_token"], D, k, w.budget)
    t3 = time.time()
    oracle.set_threads(threads)
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(n / el, 4), "unit": "rounds/s", "cores": cores,
            "kind": "oracle", "sample": f"{n} whole round(s) of the same workload ({el:.1f} s)",
            "cpu_model": model,
            "one_thread_ms": {"topk": round((t2 - t1) * 1e3, 2), "build_tree": round((t3 - t2) * 1e3, 2)}}


if __name__ == "__main__":
    sys.exit(main())
