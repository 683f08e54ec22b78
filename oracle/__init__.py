"""CPU oracle for the PRESTO draft-to-verify round -- TEST INFRASTRUCTURE.

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It never serves the product path and
shares no code with the HIP library (``paper_2607_22634_amd``).

Each function wraps one entry point of ``liboracle.so`` (oracle.c), taking
and returning NumPy arrays.  Storage dtype "bf16" means uint16 bit patterns.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None

BEST_FIRST = 0
BEST_FIRST_ALG2 = 1
BEAM = 2


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _LIB = ctypes.CDLL(_build.LIB)
        _LIB.oracle_set_threads.argtypes = [ctypes.c_int]
        _LIB.oracle_get_threads.restype = ctypes.c_int
    return _LIB


def _p(a):
    return ctypes.c_void_p(0 if a is None else a.ctypes.data)


def _dt(dtype: str) -> int:
    return {"bf16": 0, "f32": 1}[dtype]


def _check(a: np.ndarray, dtype: str):
    want = np.uint16 if dtype == "bf16" else np.float32
    if a.dtype != want or not a.flags.c_contiguous:
        raise TypeError(f"expected contiguous {want.__name__} array for {dtype}")


def set_threads(n: int) -> None:
    lib().oracle_set_threads(int(n))


def get_threads() -> int:
    return int(lib().oracle_get_threads())


def topk(logits: np.ndarray, k: int, dtype: str):
    """Per row of logits [rows, V]: top-k ids, log q of those ids, log-sum-exp."""
    _check(logits, dtype)
    rows, V = logits.shape
    ids = np.empty((rows, k), np.int32)
    lp = np.empty((rows, k), np.float32)
    lse = np.empty(rows, np.float32)
    f = lib().oracle_topk
    f.restype = ctypes.c_int
    nan_rows = f(ctypes.c_int(_dt(dtype)), _p(logits), ctypes.c_int64(rows), ctypes.c_int32(V),
                 ctypes.c_int64(V), ctypes.c_int32(k), _p(ids), _p(lp), _p(lse))
    return ids, lp, lse, int(nan_rows)


def entropy(logits: np.ndarray, dtype: str) -> np.ndarray:
    """fp64 softmax entropy H of every row of logits [rows, V] (Appendix F)."""
    _check(logits, dtype)
    rows, V = logits.shape
    h = np.empty(rows, np.float64)
    lib().oracle_entropy(ctypes.c_int(_dt(dtype)), _p(logits), ctypes.c_int64(rows),
                         ctypes.c_int32(V), ctypes.c_int64(V), _p(h))
    return h


def entropy_lambda(h, beta: float, c: float) -> np.ndarray:
    """fp64 entropy-adaptive weight beta * H / (H + C) (Appendix F)."""
    h = np.ascontiguousarray(h, np.float64)
    out = np.empty_like(h)
    lib().oracle_entropy_lambda(ctypes.c_int64(h.size), _p(h), ctypes.c_double(beta),
                                ctypes.c_double(c), _p(out))
    return out


NGRAM_TOKEN_LIMIT = 1 << 21


def ngram_table(t2, t1, t, log_rho) -> dict:
    """Trigram model (Sec. 5.1: rho is an n-gram model with n = 3) as a
    dictionary (t2, t1, t) -> log rho(t | t2, t1).  Entries with a token
    outside [0, 2^21) or a log rho that is not finite and <= 0 are ignored;
    a key given more than once keeps its largest value; -0.0 reads as +0.0."""
    table = {}
    for a, b, c, v in zip(np.asarray(t2).tolist(), np.asarray(t1).tolist(),
                          np.asarray(t).tolist(), np.asarray(log_rho, np.float32).tolist()):
        if not all(0 <= x < NGRAM_TOKEN_LIMIT for x in (a, b, c)):
            continue
        if not (np.isfinite(v) and v <= 0.0):
            continue
        v = v + 0.0
        key = (a, b, c)
        if key not in table or v > table[key]:
            table[key] = v
    return table


def ngram_lattice(table: dict, floor: float, ids, prev_token, root_token) -> np.ndarray:
    """log_rho lattice [b, D, k, k, k] for the tree stage (Eq. 9): entry
    (b, d, r2, r1, r) is log rho(t | t2, t1) of candidate t = ids[b, d, r]
    after the two tokens before it on a path: the parent t1 = ids[b, d-1, r1]
    (the root token at d = 0) and the grandparent t2 = ids[b, d-2, r2] (the
    root token at d = 1, the token before the root at d = 0); `floor` when
    the table lacks the trigram."""
    ids = np.asarray(ids)
    B, D, k = ids.shape
    out = np.empty((B, D, k, k, k), np.float32)
    for b in range(B):
        root, prev = int(root_token[b]), int(prev_token[b])
        for d in range(D):
            for r2 in range(k):
                for r1 in range(k):
                    parent = int(ids[b, d - 1, r1]) if d >= 1 else root
                    if d >= 2:
                        grand = int(ids[b, d - 2, r2])
                    elif d == 1:
                        grand = root
                    else:
                        grand = prev
                    for r in range(k):
                        out[b, d, r2, r1, r] = table.get((grand, parent, int(ids[b, d, r])),
                                                         floor)
    return out


def build_tree(ids, logprob, rho, lam, root_token, depth: int, k: int, budget: int,
               branch: int | None = None, mode: int = BEST_FIRST, beam_width: int = 0) -> dict:
    """Tree per sequence (best-first, literal Alg. 2, or beam search with beam
    width `beam_width`); ids/logprob [b, D, k], rho [b, D, k, k, k] or None;
    lam [D], or [b, D] for a weight per sequence and position."""
    branch = k if branch is None else branch
    ids = np.ascontiguousarray(ids, np.int32)
    logprob = np.ascontiguousarray(logprob, np.float32)
    lam = np.ascontiguousarray(lam, np.float32)
    root_token = np.ascontiguousarray(root_token, np.int32)
    rho = None if rho is None else np.ascontiguousarray(rho, np.float32)
    b = root_token.shape[0]
    per_seq = lam.ndim == 2
    if per_seq and lam.shape != (b, depth):
        raise ValueError("a 2-D lambda must be [batch, depth]")
    N = budget + 1
    W = (N + 63) // 64
    out = {
        "n_nodes": np.empty(b, np.int32), "parent": np.empty((b, N), np.int32),
        "token": np.empty((b, N), np.int32), "depth": np.empty((b, N), np.int32),
        "rank": np.empty((b, N), np.int32), "score": np.empty((b, N), np.float32),
        "anc": np.empty((b, N, W), np.uint64),
    }
    f = lib().oracle_build_tree
    f.restype = ctypes.c_int
    rc = f(ctypes.c_int(mode), ctypes.c_int32(b), ctypes.c_int32(depth), ctypes.c_int32(k),
           ctypes.c_int32(branch), ctypes.c_int32(budget), ctypes.c_int32(beam_width), _p(ids),
           _p(logprob), _p(rho), _p(lam), ctypes.c_int32(int(per_seq)),
           _p(root_token), _p(out["n_nodes"]), _p(out["parent"]), _p(out["token"]),
           _p(out["depth"]), _p(out["rank"]), _p(out["score"]), _p(out["anc"]))
    if rc != 0:
        raise ValueError("oracle_build_tree rejected its arguments")
    return out


def _attn_args(dtype, q, k_cache, v_cache, ctx_offsets, k_tree, v_tree, anc, n_nodes, hkv):
    for a in (q, k_cache, v_cache, k_tree, v_tree):
        _check(a, dtype)
    b, N, hq, d = q.shape
    return b, N, hq, d, [np.ascontiguousarray(ctx_offsets, np.int32),
                         np.ascontiguousarray(anc, np.uint64),
                         np.ascontiguousarray(n_nodes, np.int32)]


def tree_attention(dtype, q, k_cache, v_cache, ctx_offsets, k_tree, v_tree, anc, n_nodes,
                   scale: float | None = None):
    """Tree-masked attention output [b, N, Hq, d] in the storage dtype."""
    hkv = k_cache.shape[1]
    b, N, hq, d, (offs, anc, nn) = _attn_args(dtype, q, k_cache, v_cache, ctx_offsets, k_tree,
                                              v_tree, anc, n_nodes, hkv)
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    out = np.empty_like(q)
    lib().oracle_tree_attention(
        ctypes.c_int(_dt(dtype)), ctypes.c_int32(b), ctypes.c_int32(N), ctypes.c_int32(hq),
        ctypes.c_int32(hkv), ctypes.c_int32(d), ctypes.c_double(scale), _p(q), _p(k_cache),
        _p(v_cache), _p(offs), _p(k_tree), _p(v_tree), _p(anc), _p(nn), _p(out))
    return out


def tree_attention_rows(dtype, q, k_cache, v_cache, ctx_offsets, k_tree, v_tree, anc, n_nodes,
                        rows, scale: float | None = None):
    """fp64 attention output for the listed (b, n, h) rows only: [len(rows), d]."""
    hkv = k_cache.shape[1]
    b, N, hq, d, (offs, anc, nn) = _attn_args(dtype, q, k_cache, v_cache, ctx_offsets, k_tree,
                                              v_tree, anc, n_nodes, hkv)
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    rows = np.ascontiguousarray(rows, np.int32).reshape(-1, 3)
    out = np.empty((rows.shape[0], d), np.float64)
    lib().oracle_tree_attention_rows(
        ctypes.c_int(_dt(dtype)), ctypes.c_int32(b), ctypes.c_int32(N), ctypes.c_int32(hq),
        ctypes.c_int32(hkv), ctypes.c_int32(d), ctypes.c_double(scale), _p(q), _p(k_cache),
        _p(v_cache), _p(offs), _p(k_tree), _p(v_tree), _p(anc), _p(nn),
        ctypes.c_int64(rows.shape[0]), _p(rows), _p(out))
    return out


def accept(dtype, target_logits, parent, token, n_nodes, depth: int) -> dict:
    """Greedy verification of the tree: accept_len [b], path [b, D+1], bonus [b], argmax [b, N]."""
    _check(target_logits, dtype)
    b, N, V = target_logits.shape
    parent = np.ascontiguousarray(parent, np.int32)
    token = np.ascontiguousarray(token, np.int32)
    n_nodes = np.ascontiguousarray(n_nodes, np.int32)
    out = {"accept_len": np.empty(b, np.int32), "path": np.empty((b, depth + 1), np.int32),
           "bonus": np.empty(b, np.int32), "target_argmax": np.empty((b, N), np.int32)}
    f = lib().oracle_accept
    f.restype = ctypes.c_int
    nan_rows = f(ctypes.c_int(_dt(dtype)), _p(target_logits), ctypes.c_int32(V), ctypes.c_int64(V),
                 ctypes.c_int32(b), ctypes.c_int32(N), ctypes.c_int32(depth), _p(parent), _p(token),
                 _p(n_nodes), _p(out["accept_len"]), _p(out["path"]), _p(out["bonus"]),
                 _p(out["target_argmax"]))
    out["nan_rows"] = int(nan_rows)
    return out


# ----------------------------------------------------------------------------
# Bookkeeping between rounds (Appendix C stages I, II and IV)

def commit_kv(k_tree, v_tree, path, accept_len, k_cache, v_cache, ctx, ctx_cap):
    """The root and the accepted draft tokens join the committed prefix
    (Appendix C stage I): for each sequence, the tree K/V rows of its path
    (root first, as the accept stage lists it) are appended after its cache
    rows, and its length grows by their count.  ctx [b, 2] = (start, len),
    ctx_cap [b] = rows the sequence owns.  A sequence that would overflow
    its rows, lies outside the cache, or has an invalid path is left as it
    is.  Returns (k_cache, v_cache, ctx, skipped) as new arrays."""
    kc, vc, cx = k_cache.copy(), v_cache.copy(), np.array(ctx, np.int32, copy=True)
    B, N = k_tree.shape[:2]
    depth = path.shape[1] - 1
    skipped = np.zeros(B, bool)
    for b in range(B):
        start, length, cap = int(cx[b, 0]), int(cx[b, 1]), int(ctx_cap[b])
        al = int(accept_len[b])
        nodes = [int(x) for x in path[b, :al + 1]] if 0 <= al <= depth else []
        ok = (0 <= al <= depth and start >= 0 and length >= 0 and cap >= 0
              and start + cap <= kc.shape[0] and length + al + 1 <= cap
              and nodes[0] == 0 and all(0 <= x < N for x in nodes))
        if not ok:
            skipped[b] = True
            continue
        for i, node in enumerate(nodes):
            kc[start + length + i] = k_tree[b, node]
            vc[start + length + i] = v_tree[b, node]
        cx[b, 1] = length + len(nodes)
    return kc, vc, cx, skipped


def select_slots(path, accept_len, n_max: int, slots: int, first_slot: int = 1) -> np.ndarray:
    """Rows of the next round's drafter positions in the slot-logit matrix
    [b * n_max * slots, V] (Appendix C stage II): only the mask slots after the
    last accepted node are used, from slot first_slot + 1 (1-based) on."""
    B = len(accept_len)
    out = np.empty((B, slots - first_slot), np.int64)
    for b in range(B):
        last = int(path[b, int(accept_len[b])])
        for d in range(slots - first_slot):
            out[b, d] = (b * n_max + last) * slots + first_slot + d
    return out


def flatten_slots(parent, depth, n_nodes, root_pos, slots: int) -> dict:
    """Composite input of the next forward (Appendix C stage IV): every tree node
    is followed by a block of `slots` mask slots; row n * (1 + slots) + j is
    node n (j = 0) or its slot j.  A node row attends to the node rows on its
    root path (itself included), a slot row to those same node rows and to
    its whole block; positions are root_pos + depth(n) + j.  Built from
    parent pointers."""
    B, N = parent.shape
    blk = 1 + slots
    R = N * blk
    WO = (R + 63) // 64
    pos = np.full((B, R), -1, np.int32)
    anc = np.zeros((B, R, WO), np.uint64)
    n_rows = np.zeros(B, np.int32)

    def setbit(b, r, c):
        anc[b, r, c // 64] |= np.uint64(1) << np.uint64(c % 64)

    for b in range(B):
        nn = int(n_nodes[b])
        n_rows[b] = nn * blk
        for n in range(nn):
            chain = [n]
            while chain[-1] != 0:
                chain.append(int(parent[b, chain[-1]]))
            for j in range(blk):
                r = n * blk + j
                pos[b, r] = int(root_pos[b]) + int(depth[b, n]) + j
                for m in chain:
                    setbit(b, r, m * blk)
                if j > 0:
                    for jj in range(1, blk):
                        setbit(b, r, n * blk + jj)
    return {"pos": pos, "anc": anc, "n_rows": n_rows}
