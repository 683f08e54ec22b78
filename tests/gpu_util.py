"""Helpers shared by the GPU tests: device transfer of synthetic inputs and
cached per-workload data (inputs are drawn once per process)."""
from __future__ import annotations

import functools

import numpy as np
import torch

import synthetic as sy

DEV = "cuda"


def to_dev(a: np.ndarray, dtype: str | None = None) -> torch.Tensor:
    """Storage array -> device tensor (uint16 bit patterns become bfloat16)."""
    if dtype == "bf16" or a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)
    if a.dtype == np.uint64:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int64)).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def to_host(t: torch.Tensor) -> np.ndarray:
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def tree_to_host(tree: dict) -> dict:
    out = {k: to_host(v) for k, v in tree.items()}
    out["anc"] = out["anc"].view(np.uint64)
    return out


@functools.lru_cache(maxsize=2)
def round_data(cfg: int, **over) -> tuple:
    w = sy.workload(cfg, **over)
    return w, sy.round_inputs(w)


@functools.lru_cache(maxsize=2)
def oracle_candidates(cfg: int) -> tuple:
    """The oracle's top-k of a workload's drafter logits, [b, D, k] each.
    Stages after top-k are fed these on both sides, so no oracle input ever
    comes from the GPU."""
    import oracle

    w, rin = round_data(cfg)
    ids, lp, _, _ = oracle.topk(rin["drafter_logits"], w.k, w.dtype)
    return ids.reshape(w.batch, w.depth, w.k), lp.reshape(w.batch, w.depth, w.k)


@functools.lru_cache(maxsize=2)
def oracle_tree(cfg: int) -> dict:
    """The oracle's tree of a workload (from oracle_candidates)."""
    import oracle

    w, rin = round_data(cfg)
    ids, lp = oracle_candidates(cfg)
    return oracle.build_tree(ids, lp, rin["rho"], rin["lam"], rin["root_token"], w.depth, w.k,
                             w.budget)


def tree_to_dev(tree: dict) -> dict:
    return {k: to_dev(v) for k, v in tree.items()}


@functools.lru_cache(maxsize=2)
def attn_data(cfg: int, layer: int = 0) -> tuple:
    w = sy.workload(cfg)
    return w, sy.attention_inputs(w, layer)
