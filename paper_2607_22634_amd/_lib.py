"""ctypes binding of libpresto (include/presto.h).

Argument marshalling only: every step of a round runs in the HIP kernels of
libpresto.so.  Tensors are PyTorch device tensors (memory and streams only);
the binding checks their dtype/shape/contiguity, allocates outputs and the
workspace with torch when the caller does not pass them, and enqueues the
call on the current (or given) stream.  There is no fallback: a missing
library raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpresto.so")

PRESTO_OK = 0
PRESTO_ERR_INVALID_ARG = -1
PRESTO_ERR_UNSUPPORTED = -2
PRESTO_ERR_WORKSPACE = -3
PRESTO_ERR_HIP = -4

PRESTO_DT_BF16 = 0
PRESTO_DT_F32 = 1

PRESTO_TREE_BEST_FIRST = 0
PRESTO_TREE_BEST_FIRST_ALG2 = 1
PRESTO_TREE_BEAM = 2

PRESTO_FLAG_NAN_DRAFTER = 1
PRESTO_FLAG_NAN_TARGET = 2
PRESTO_FLAG_NGRAM_BAD = 4
PRESTO_FLAG_NGRAM_FULL = 8
PRESTO_FLAG_BAD_INDEX = 16
PRESTO_FLAG_KV_COMMIT = 32
PRESTO_CTX_PACKED = 0
PRESTO_CTX_SLOTS = 1

EXPORTS = (
    "presto_topk_workspace", "presto_topk", "presto_topk_noalloc", "presto_entropy_lambda",
    "presto_ngram_table_bytes",
    "presto_ngram_clear", "presto_ngram_insert", "presto_ngram_gather", "presto_build_tree_workspace",
    "presto_build_tree",
    "presto_tree_attention_workspace", "presto_tree_attention", "presto_accept_workspace",
    "presto_accept", "presto_topk_rows", "presto_commit_kv", "presto_select_slots",
    "presto_flatten_slots", "presto_status_string", "presto_last_error", "presto_version",
)


class PrestoError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status}: {detail}")
        self.status = status


class TreeDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("depth", ctypes.c_int32), ("k", ctypes.c_int32),
                ("branch", ctypes.c_int32), ("budget", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("beam_width", ctypes.c_int32), ("lambda_per_seq", ctypes.c_int32)]


class AttnDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_max", ctypes.c_int32), ("hq", ctypes.c_int32),
                ("hkv", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("max_ctx", ctypes.c_int32),
                ("scale", ctypes.c_float), ("dt", ctypes.c_int32), ("ctx_layout", ctypes.c_int32),
                ("total_ctx", ctypes.c_int64)]


class CommitDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_max", ctypes.c_int32), ("hkv", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("depth", ctypes.c_int32), ("dt", ctypes.c_int32)]


_VP, _I32, _I64, _SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
_LIB = None


def lib() -> ctypes.CDLL:
    """Load libpresto.so (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2607_22634_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        L.presto_topk_workspace.argtypes = [_I64, _I32, _I32]
        L.presto_topk_workspace.restype = _SZ
        L.presto_topk.argtypes = [_I32, _VP, _I64, _I32, _I64, _I32] + [_VP] * 6 + [_SZ, _VP]
        L.presto_topk.restype = _I32
        L.presto_topk_noalloc.argtypes = [_I32, _VP, _I64, _I32, _I64, _I32] + [_VP] * 6
        L.presto_topk_noalloc.restype = _I32
        L.presto_entropy_lambda.argtypes = [_I64, _VP, ctypes.c_float, ctypes.c_float, _VP, _VP]
        L.presto_entropy_lambda.restype = _I32
        L.presto_ngram_table_bytes.argtypes = [_I64]
        L.presto_ngram_table_bytes.restype = _SZ
        L.presto_ngram_clear.argtypes = [_VP, _I64, _VP]
        L.presto_ngram_clear.restype = _I32
        L.presto_ngram_insert.argtypes = [_VP, _I64, _I64, _VP, _VP, _VP, _VP, _VP, _VP]
        L.presto_ngram_insert.restype = _I32
        L.presto_ngram_gather.argtypes = [_VP, _I64, ctypes.c_float, _I32, _I32, _I32, _VP, _VP,
                                          _VP, _VP, _VP]
        L.presto_ngram_gather.restype = _I32
        L.presto_build_tree_workspace.argtypes = [ctypes.POINTER(TreeDesc)]
        L.presto_build_tree_workspace.restype = _SZ
        L.presto_build_tree.argtypes = [ctypes.POINTER(TreeDesc)] + [_VP] * 13 + [_SZ, _VP]
        L.presto_build_tree.restype = _I32
        L.presto_tree_attention_workspace.argtypes = [ctypes.POINTER(AttnDesc)]
        L.presto_tree_attention_workspace.restype = _SZ
        L.presto_tree_attention.argtypes = [ctypes.POINTER(AttnDesc)] + [_VP] * 10 + [_SZ, _VP]
        L.presto_tree_attention.restype = _I32
        L.presto_accept_workspace.argtypes = [_I32, _I32, _I32]
        L.presto_accept_workspace.restype = _SZ
        L.presto_accept.argtypes = [_I32, _VP, _I32, _I64, _I32, _I32, _I32] + [_VP] * 9 + [_SZ, _VP]
        L.presto_accept.restype = _I32
        L.presto_topk_rows.argtypes = [_I32, _VP, _I64, _VP, _I64, _I32, _I64, _I32] + [_VP] * 6 \
            + [_SZ, _VP]
        L.presto_topk_rows.restype = _I32
        L.presto_commit_kv.argtypes = [ctypes.POINTER(CommitDesc)] + [_VP] * 6 + [_I64] + \
            [_VP] * 4
        L.presto_commit_kv.restype = _I32
        L.presto_select_slots.argtypes = [_I32, _I32, _I32, _I32, _I32] + [_VP] * 5
        L.presto_select_slots.restype = _I32
        L.presto_flatten_slots.argtypes = [_I32, _I32, _I32] + [_VP] * 8
        L.presto_flatten_slots.restype = _I32
        L.presto_status_string.argtypes = [_I32]
        L.presto_status_string.restype = ctypes.c_char_p
        L.presto_last_error.restype = ctypes.c_char_p
        L.presto_version.restype = ctypes.c_char_p
        _LIB = L
    return _LIB


def _check(status: int, where: str) -> None:
    if status != PRESTO_OK:
        raise PrestoError(status, where, lib().presto_last_error().decode())


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int | None:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return PRESTO_DT_BF16
    if t.dtype == torch.float32:
        return PRESTO_DT_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _dev(*ts):
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError("tensors must be contiguous device tensors")


def _rows(t: torch.Tensor) -> None:
    """Row-strided matrices: any row stride, contiguous innermost dimension."""
    if not t.is_cuda or t.stride(-1) != 1 or (t.dim() == 3 and t.stride(0) != t.shape[1] * t.stride(1)):
        raise ValueError("logits must be a device tensor with a contiguous innermost dimension")


def _workspace(nbytes: int, device, ws):
    if nbytes == 0:
        return None, 0
    if ws is not None:
        return ws, ws.numel() * ws.element_size()
    t = torch.empty(nbytes, dtype=torch.uint8, device=device)  # contents on entry are ignored
    return t, nbytes


def version() -> str:
    return lib().presto_version().decode()


def presto_topk(logits: torch.Tensor, k: int, *, ids=None, logprob=None, lse=None, entropy=None,
                flags=None, workspace=None, stream=None):
    """Top-k ids, log q and LSE of every row of logits [rows, V] (bf16 or fp32).

    With ``entropy`` (a [rows] fp32 tensor, or True to allocate one) the
    softmax entropy of each row is written too and returned fourth."""
    _rows(logits)
    rows, V = logits.shape
    dev = logits.device
    ids = torch.empty(rows, k, dtype=torch.int32, device=dev) if ids is None else ids
    logprob = torch.empty(rows, k, dtype=torch.float32, device=dev) if logprob is None else logprob
    lse = torch.empty(rows, dtype=torch.float32, device=dev) if lse is None else lse
    want_h = entropy is not None and entropy is not False
    if entropy is True:
        entropy = torch.empty(rows, dtype=torch.float32, device=dev)
    h = entropy if want_h else None
    _dev(ids, logprob, lse, h, flags)
    need = lib().presto_topk_workspace(rows, V, k)
    ws, nb = _workspace(need, dev, workspace)
    _check(lib().presto_topk(_dt(logits), _ptr(logits), rows, V, logits.stride(0), k, _ptr(ids),
                             _ptr(logprob), _ptr(lse), _ptr(h), _ptr(flags), _ptr(ws), nb,
                             _stream(stream)),
           "presto_topk")
    return (ids, logprob, lse, h) if want_h else (ids, logprob, lse)


def presto_topk_noalloc(logits: torch.Tensor, k: int, *, ids=None, logprob=None, lse=None,
                        entropy=None, flags=None, stream=None):
    """presto_topk without a workspace (the library's static scratch; for
    callers that cannot allocate).  Returns (ids, logprob, lse[, entropy])."""
    _rows(logits)
    rows, V = logits.shape
    dev = logits.device
    ids = torch.empty(rows, k, dtype=torch.int32, device=dev) if ids is None else ids
    logprob = torch.empty(rows, k, dtype=torch.float32, device=dev) if logprob is None else logprob
    lse = torch.empty(rows, dtype=torch.float32, device=dev) if lse is None else lse
    want_h = entropy is not None and entropy is not False
    if entropy is True:
        entropy = torch.empty(rows, dtype=torch.float32, device=dev)
    h = entropy if want_h else None
    _dev(ids, logprob, lse, h, flags)
    _check(lib().presto_topk_noalloc(_dt(logits), _ptr(logits), rows, V, logits.stride(0), k,
                                     _ptr(ids), _ptr(logprob), _ptr(lse), _ptr(h), _ptr(flags),
                                     _stream(stream)),
           "presto_topk_noalloc")
    return (ids, logprob, lse, h) if want_h else (ids, logprob, lse)


def topk_workspace(rows: int, vocab: int, k: int, device) -> torch.Tensor:
    """A workspace for presto_topk / presto_topk_rows of this size."""
    return torch.empty(max(1, lib().presto_topk_workspace(rows, vocab, k)), dtype=torch.uint8,
                       device=device)


def topk_fallback_chunks(workspace: torch.Tensor) -> int:
    """The diagnostic count a completed top-k call leaves in the first four
    bytes of its workspace: chunks that took the exact tie pass."""
    return int(workspace[:4].cpu().view(torch.int32).item())


def presto_entropy_lambda(entropy: torch.Tensor, beta: float, c: float, *, out=None, stream=None):
    """Entropy-adaptive weight beta * H / (H + C) of every entry of entropy."""
    out = torch.empty_like(entropy) if out is None else out
    _dev(entropy, out)
    if entropy.dtype != torch.float32 or out.dtype != torch.float32 or out.shape != entropy.shape:
        raise ValueError("entropy and out must be fp32 tensors of one shape")
    _check(lib().presto_entropy_lambda(entropy.numel(), _ptr(entropy), float(beta), float(c),
                                       _ptr(out), _stream(stream)),
           "presto_entropy_lambda")
    return out


def presto_ngram_table_bytes(capacity: int) -> int:
    """Bytes of device memory a trigram table of `capacity` slots needs."""
    return int(lib().presto_ngram_table_bytes(capacity))


def presto_ngram_clear(table: torch.Tensor, capacity: int, *, stream=None) -> None:
    """Empty the trigram table held in `table` (a device byte tensor)."""
    _dev(table)
    _check(lib().presto_ngram_clear(_ptr(table), capacity, _stream(stream)), "presto_ngram_clear")


def presto_ngram_insert(table: torch.Tensor, capacity: int, t2: torch.Tensor, t1: torch.Tensor,
                        t: torch.Tensor, log_rho: torch.Tensor, *, flags=None, stream=None) -> None:
    """Add entries log rho(t | t2, t1) (int32 / fp32 device vectors of one length)."""
    _dev(table, t2, t1, t, log_rho, flags)
    n = t.numel()
    if not (t2.numel() == t1.numel() == log_rho.numel() == n):
        raise ValueError("t2, t1, t and log_rho must have one length")
    _check(lib().presto_ngram_insert(_ptr(table), capacity, n, _ptr(t2), _ptr(t1), _ptr(t),
                                     _ptr(log_rho), _ptr(flags), _stream(stream)),
           "presto_ngram_insert")


def presto_ngram_gather(table: torch.Tensor, capacity: int, floor_log_rho: float,
                        ids: torch.Tensor, prev_token: torch.Tensor, root_token: torch.Tensor,
                        depth: int, k: int, *, out=None, stream=None) -> torch.Tensor:
    """log_rho lattice [b, depth, k, k, k] for the candidates ids [b*depth, k]
    or [b, depth, k]."""
    b = root_token.shape[0]
    out = torch.empty(b, depth, k, k, k, dtype=torch.float32, device=ids.device) if out is None \
        else out
    _dev(table, ids, prev_token, root_token, out)
    _check(lib().presto_ngram_gather(_ptr(table), capacity, float(floor_log_rho), b, depth, k,
                                     _ptr(ids), _ptr(prev_token), _ptr(root_token), _ptr(out),
                                     _stream(stream)),
           "presto_ngram_gather")
    return out


def presto_build_tree(ids: torch.Tensor, logprob: torch.Tensor, log_rho, lam: torch.Tensor,
                      root_token: torch.Tensor, depth: int, k: int, budget: int,
                      branch: int | None = None, mode: int = PRESTO_TREE_BEST_FIRST, *, out=None,
                      workspace=None, stream=None, beam_width: int = 0) -> dict:
    """Draft tree per sequence (best-first, or beam search of width
    `beam_width`): ids/logprob [b*D, k] or [b, D, k]; lam [D], or [b, D]
    for a weight per sequence and position."""
    branch = k if branch is None else branch
    b = root_token.shape[0]
    N = budget + 1
    W = (N + 63) // 64
    dev = root_token.device
    _dev(ids, logprob, log_rho, lam, root_token)
    if out is None:
        i32 = dict(dtype=torch.int32, device=dev)
        out = {
            "n_nodes": torch.empty(b, **i32), "parent": torch.empty(b, N, **i32),
            "token": torch.empty(b, N, **i32), "depth": torch.empty(b, N, **i32),
            "rank": torch.empty(b, N, **i32),
            "score": torch.empty(b, N, dtype=torch.float32, device=dev),
            "anc": torch.empty(b, N, W, dtype=torch.int64, device=dev),
        }
    per_seq = lam.dim() == 2
    if per_seq and tuple(lam.shape) != (b, depth):
        raise ValueError("a 2-D lambda must be [batch, depth]")
    desc = TreeDesc(b, depth, k, branch, budget, mode, beam_width, int(per_seq))
    need = lib().presto_build_tree_workspace(ctypes.byref(desc))
    ws, nb = _workspace(need, dev, workspace)
    _check(lib().presto_build_tree(
        ctypes.byref(desc), _ptr(ids), _ptr(logprob), _ptr(log_rho), _ptr(lam), _ptr(root_token),
        _ptr(out["n_nodes"]), _ptr(out["parent"]), _ptr(out["token"]), _ptr(out["depth"]),
        _ptr(out["rank"]), _ptr(out["score"]), _ptr(out["anc"]), _ptr(ws), nb, _stream(stream)),
        "presto_build_tree")
    return out


def presto_tree_attention(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                          ctx_offsets: torch.Tensor, k_tree: torch.Tensor, v_tree: torch.Tensor,
                          anc: torch.Tensor, n_nodes: torch.Tensor, max_ctx: int,
                          scale: float | None = None, *, out=None, workspace=None, stream=None,
                          ctx_layout: int = PRESTO_CTX_PACKED, total_ctx: int = 0):
    """Tree-masked attention of q [b, N, Hq, d] over [cache ; ancestors].
    ctx_offsets: [b + 1] packed offsets, or [b, 2] (start, len) pairs with
    ctx_layout=PRESTO_CTX_SLOTS.  total_ctx: the sum of the context lengths
    when the caller knows it (a scheduling hint for ragged batches; 0 =
    unknown); a workspace passed in must be sized for the same hint."""
    b, N, hq, d = q.shape
    hkv = k_tree.shape[2]
    scale = d ** -0.5 if scale is None else scale
    _dev(q, k_cache, v_cache, ctx_offsets, k_tree, v_tree, anc, n_nodes)
    out = torch.empty_like(q) if out is None else out
    _dev(out)
    desc = AttnDesc(b, N, hq, hkv, d, int(max_ctx), float(scale), _dt(q), int(ctx_layout),
                    int(total_ctx))
    need = lib().presto_tree_attention_workspace(ctypes.byref(desc))
    ws, nb = _workspace(need, q.device, workspace)
    _check(lib().presto_tree_attention(
        ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(ctx_offsets), _ptr(k_tree),
        _ptr(v_tree), _ptr(anc), _ptr(n_nodes), _ptr(out), _ptr(ws), nb, _stream(stream)),
        "presto_tree_attention")
    return out


def presto_accept(target_logits: torch.Tensor, parent: torch.Tensor, token: torch.Tensor,
                  n_nodes: torch.Tensor, depth: int, *, out=None, flags=None, workspace=None,
                  stream=None) -> dict:
    """Greedy acceptance: target_logits [b, N, V] (or [b*N, V]) against the tree."""
    b, N = parent.shape
    V = target_logits.shape[-1]
    dev = parent.device
    _rows(target_logits)
    _dev(parent, token, n_nodes, flags)
    if out is None:
        i32 = dict(dtype=torch.int32, device=dev)
        out = {"accept_len": torch.empty(b, **i32), "path": torch.empty(b, depth + 1, **i32),
               "bonus": torch.empty(b, **i32), "target_argmax": torch.empty(b, N, **i32)}
    need = lib().presto_accept_workspace(b, N, V)
    ws, nb = _workspace(need, dev, workspace)
    _check(lib().presto_accept(
        _dt(target_logits), _ptr(target_logits), V, target_logits.stride(-2), b, N, depth,
        _ptr(parent), _ptr(token), _ptr(n_nodes), _ptr(out["accept_len"]), _ptr(out["path"]),
        _ptr(out["bonus"]), _ptr(out.get("target_argmax")), _ptr(flags), _ptr(ws), nb,
        _stream(stream)), "presto_accept")
    return out


def presto_topk_rows(logits: torch.Tensor, row_index: torch.Tensor, k: int, *, ids=None,
                     logprob=None, lse=None, entropy=None, flags=None, workspace=None, stream=None):
    """presto_topk on the rows logits[row_index] (int64 device indices), read in place."""
    _rows(logits)
    _dev(row_index)
    if row_index.dtype != torch.int64:
        raise TypeError("row_index must be int64")
    rows = row_index.numel()
    L, V = logits.shape
    dev = logits.device
    ids = torch.empty(rows, k, dtype=torch.int32, device=dev) if ids is None else ids
    logprob = torch.empty(rows, k, dtype=torch.float32, device=dev) if logprob is None else logprob
    lse = torch.empty(rows, dtype=torch.float32, device=dev) if lse is None else lse
    want_h = entropy is not None and entropy is not False
    if entropy is True:
        entropy = torch.empty(rows, dtype=torch.float32, device=dev)
    h = entropy if want_h else None
    _dev(ids, logprob, lse, h, flags)
    need = lib().presto_topk_workspace(rows, V, k)
    ws, nb = _workspace(need, dev, workspace)
    _check(lib().presto_topk_rows(_dt(logits), _ptr(logits), L, _ptr(row_index), rows, V,
                                  logits.stride(0), k, _ptr(ids), _ptr(logprob), _ptr(lse), _ptr(h),
                                  _ptr(flags), _ptr(ws), nb, _stream(stream)),
           "presto_topk_rows")
    return (ids, logprob, lse, h) if want_h else (ids, logprob, lse)


def presto_commit_kv(k_tree: torch.Tensor, v_tree: torch.Tensor, path: torch.Tensor,
                     accept_len: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                     ctx: torch.Tensor, ctx_cap: torch.Tensor, *, flags=None, stream=None) -> None:
    """Append each sequence's root and accepted tree K/V rows to its cache
    slot; ctx [b, 2] (start, len) is advanced in place."""
    b, N, hkv, d = k_tree.shape
    depth = path.shape[1] - 1
    _dev(k_tree, v_tree, path, accept_len, k_cache, v_cache, ctx, ctx_cap, flags)
    desc = CommitDesc(b, N, hkv, d, depth, _dt(k_tree))
    _check(lib().presto_commit_kv(ctypes.byref(desc), _ptr(k_tree), _ptr(v_tree), _ptr(path),
                                  _ptr(accept_len), _ptr(k_cache), _ptr(v_cache),
                                  k_cache.shape[0], _ptr(ctx), _ptr(ctx_cap), _ptr(flags),
                                  _stream(stream)),
           "presto_commit_kv")


def presto_select_slots(path: torch.Tensor, accept_len: torch.Tensor, n_max: int, slots: int,
                        first_slot: int = 1, *, out=None, flags=None, stream=None) -> torch.Tensor:
    """Row indices [b, slots - first_slot] of the next drafter rows in the
    slot-logit matrix [b * n_max * slots, V]."""
    b = accept_len.shape[0]
    depth = path.shape[1] - 1
    out = torch.empty(b, slots - first_slot, dtype=torch.int64, device=path.device) \
        if out is None else out
    _dev(path, accept_len, out, flags)
    _check(lib().presto_select_slots(b, n_max, depth, slots, first_slot, _ptr(path),
                                     _ptr(accept_len), _ptr(out), _ptr(flags), _stream(stream)),
           "presto_select_slots")
    return out


def presto_flatten_slots(depth: torch.Tensor, anc: torch.Tensor, n_nodes: torch.Tensor,
                         root_pos: torch.Tensor, slots: int, *, stream=None) -> dict:
    """Composite layout of a tree with `slots` mask slots after every node:
    pos [b, R], anc [b, R, ceil(R/64)], n_rows [b] with R = N * (1 + slots)."""
    b, N = depth.shape
    R = N * (1 + slots)
    dev = depth.device
    out = {"pos": torch.empty(b, R, dtype=torch.int32, device=dev),
           "anc": torch.empty(b, R, (R + 63) // 64, dtype=torch.int64, device=dev),
           "n_rows": torch.empty(b, dtype=torch.int32, device=dev)}
    _dev(depth, anc, n_nodes, root_pos)
    _check(lib().presto_flatten_slots(b, N, slots, _ptr(depth), _ptr(anc), _ptr(n_nodes),
                                      _ptr(root_pos), _ptr(out["pos"]), _ptr(out["anc"]),
                                      _ptr(out["n_rows"]), _stream(stream)),
           "presto_flatten_slots")
    return out
