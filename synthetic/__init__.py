"""Seeded synthetic inputs for the PRESTO draft-to-verify round.

This module only draws and casts random inputs. It holds none of the
method's arithmetic (no softmax, no scoring, no tree search, no attention,
no acceptance), so the CPU oracle and the HIP path can both consume its
bytes without sharing any computation.

The paper (Sec. 5.1, Appendix D) evaluates on trained Qwen3 targets with
dFlash drafters over public benchmark suites; neither the weights nor the
suites are available here, so these generators stand in for them with
the shapes of those runs: Qwen3 vocabulary (151936) and GQA geometry
(32 query heads, 8 KV heads, head_dim 128), a drafter block of 16
positions, tree budgets of 32 to 256 draft nodes, 1 to 32 sequences.

Recipe (every tensor is generated in fp32, then cast by round-to-nearest-
even on the bit pattern when the workload is bf16):

* RNG: ``numpy.random.default_rng([seed, seq, layer, stream, *extra])``
  (PCG64 seeded through SeedSequence).  ``stream`` names the tensor.
  SeedSequence ignores trailing zero words, so every variable-length
  suffix is written with non-zero digits.
* Field ``F[b, D+1, V]``: i.i.d. N(0, sigma_f^2) plus planted peaks.  A
  planted peak sets one token to (that row's Gaussian maximum) + h.
  Drafter logits are ``F[:, :D]``.
* Target logits for a tree node of depth delta: ``F[:, delta] +
  sigma_t * E`` with ``E ~ N(0, 1)`` seeded by the node's rank path, so
  the simulated target world does not depend on node numbering.
* Prefix-signal lattice ``R[b, D, k, k, k]`` (log rho of a trigram over
  candidate ranks): each entry is, with probability 1/2, the unseen-trigram
  floor ``ln(1e-4)``, otherwise ``ln(u)`` with ``u ~ U(1e-3, 1)``.
* Q, K, V ~ N(0, 1), independent per layer; the KV cache is packed
  varlen ``[sum ctx, Hkv, d]`` with ``ctx_offsets[b+1]``.
* Trigram table entries (the n-gram rho of Sec. 5.1, whose training corpus
  is not available): the trigrams of random walks that start from the
  two committed tokens (the token before the root, the root) and pick one
  of the k candidate tokens at each drafter position, plus uniformly random
  background trigrams; each distinct trigram gets ln(u), u ~ U(1e-3, 1).
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field as dc_field

import numpy as np

# Stream identifiers: one per tensor kind.
S_FIELD, S_PEAKS, S_TNOISE, S_RHO, S_Q, S_K, S_V, S_KT, S_VT, S_CTX, S_TOKENS, S_NGRAM = range(1, 13)

# Positions of the KV cache drawn from one generator call.
_KV_CHUNK = 1024


@dataclass(frozen=True)
class Workload:
    """One synthetic draft-to-verify round."""

    name: str
    dtype: str            # "f32" or "bf16": logits, Q/K/V and attention output
    batch: int
    depth: int            # drafter block D (tree depth cap)
    vocab: int
    k: int                # candidates per position (= children per expansion)
    budget: int           # draft nodes B, root excluded
    hq: int
    hkv: int
    head_dim: int
    ctx: tuple            # (lo, hi) inclusive; lo == hi for a fixed length
    layers: int
    lam: float            # lambda_d, constant over depth
    sigma_f: float        # field standard deviation
    peaks: tuple          # (min peaks, max peaks, min height, max height) per row
    sigma_t: float        # target-side noise standard deviation
    seed: int
    extra: dict = dc_field(default_factory=dict)

    @property
    def n_max(self) -> int:
        return self.budget + 1

    @property
    def words(self) -> int:
        return (self.n_max + 63) // 64

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def with_(self, **kw) -> "Workload":
        d = self.__dict__.copy()
        d.update(kw)
        return Workload(**d)


WORKLOADS = {
    1: Workload("tiny-fp32", "f32", 1, 4, 1024, 2, 8, 2, 1, 64, (128, 128), 1, 0.2,
                3.0, (0, 0, 0.0, 0.0), 1.0, 0),
    2: Workload("qwen3-8b-single", "bf16", 1, 16, 151936, 4, 64, 32, 8, 128, (4096, 4096), 1, 0.2,
                4.0, (1, 1, 8.0, 8.0), 2.0, 2),
    3: Workload("batched-serving", "bf16", 16, 16, 151936, 4, 32, 32, 8, 128, (1024, 8192), 1, 0.2,
                4.0, (1, 1, 8.0, 8.0), 2.0, 3),
    4: Workload("large-tree", "bf16", 4, 16, 151936, 8, 256, 32, 8, 128, (32768, 32768), 1, 0.2,
                4.0, (1, 3, 4.0, 10.0), 2.0, 4),
    5: Workload("self-spec-36l", "bf16", 32, 32, 151936, 4, 128, 32, 8, 128, (2048, 2048), 36, 0.0,
                4.0, (0, 0, 0.0, 0.0), 1.0, 5),
}


def workload(i: int, **overrides) -> Workload:
    w = WORKLOADS[i]
    return w.with_(**overrides) if overrides else w


# ----------------------------------------------------------------------------
# casting helpers (input preparation only)

def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + r) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def cast(x: np.ndarray, dtype: str) -> np.ndarray:
    """Cast fp32 data to the workload dtype's storage (float32 or bf16 bits)."""
    return to_bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def as_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_bits_to_f32(x) if dtype == "bf16" else np.asarray(x, dtype=np.float32)


def _rng(w: Workload, seq: int, layer: int, stream: int, *extra: int) -> np.random.Generator:
    return np.random.default_rng([w.seed, seq, layer, stream, *extra])


def _pool() -> int:
    return max(1, min(16, len(os.sched_getaffinity(0))))


def _parallel(fn, items):
    items = list(items)
    if len(items) <= 1:
        for it in items:
            fn(it)
        return
    with ThreadPoolExecutor(_pool()) as ex:
        list(ex.map(fn, items))


# ----------------------------------------------------------------------------
# drafter / target field

def field(w: Workload) -> np.ndarray:
    """F[b, D+1, V] fp32 with planted peaks."""
    b, rows, V = w.batch, w.depth + 1, w.vocab
    F = np.empty((b, rows, V), np.float32)

    def fill(it):
        s, r = it
        _rng(w, s, 0, S_FIELD, r + 1).standard_normal(V, dtype=np.float32, out=F[s, r])
        F[s, r] *= np.float32(w.sigma_f)

    _parallel(fill, [(s, r) for s in range(b) for r in range(rows)])
    lo, hi, hlo, hhi = w.peaks
    if hi > 0:
        for s in range(b):
            g = _rng(w, s, 0, S_PEAKS)
            for r in range(rows):
                m = int(g.integers(lo, hi + 1))
                toks = g.choice(V, size=m, replace=False)
                hs = g.uniform(hlo, hhi, size=m) if hhi > hlo else np.full(m, hlo)
                top = F[s, r].max()
                for t, h in zip(toks, hs):
                    F[s, r, t] = np.float32(top + np.float32(h))
    return F


def drafter_logits(w: Workload, F: np.ndarray | None = None) -> np.ndarray:
    """Drafter logits [b*D, V] in the workload's storage dtype."""
    if F is None:
        F = field(w)
    return cast(F[:, : w.depth].reshape(w.batch * w.depth, w.vocab), w.dtype)


def rho_lattice(w: Workload) -> np.ndarray:
    """log rho lattice R[b, D, k, k, k] fp32 (all entries <= 0, finite)."""
    D, k = w.depth, w.k
    R = np.empty((w.batch, D, k, k, k), np.float32)
    floor = np.float32(np.log(np.float32(1e-4)))
    for s in range(w.batch):
        g = _rng(w, s, 0, S_RHO)
        coin = g.random(size=(D, k, k, k)) < 0.5
        u = g.uniform(1e-3, 1.0, size=(D, k, k, k))
        R[s] = np.where(coin, floor, np.log(u).astype(np.float32))
    return R


def lambdas(w: Workload) -> np.ndarray:
    return np.full(w.depth, w.lam, np.float32)


def root_tokens(w: Workload) -> np.ndarray:
    return np.array([int(_rng(w, s, 0, S_TOKENS).integers(0, w.vocab)) for s in range(w.batch)],
                    np.int32)


def prev_tokens(w: Workload) -> np.ndarray:
    """The committed token before the root, per sequence."""
    return np.array([int(_rng(w, s, 0, S_TOKENS, 2).integers(0, w.vocab)) for s in range(w.batch)],
                    np.int32)


def trigram_entries(w: Workload, ids: np.ndarray, n_walks: int, n_background: int) -> tuple:
    """Trigram table entries (t2, t1, t, log rho) as four arrays: the
    trigrams along n_walks random walks per sequence through its candidate
    rows ids [b, D, k] after (prev token, root token), and n_background
    random trigrams over the vocabulary."""
    rng = np.random.default_rng([w.seed, 7, S_NGRAM])
    prev, root = prev_tokens(w), root_tokens(w)
    B, D, k = ids.shape
    walks = []
    for b in range(B):
        pick = rng.integers(0, k, (n_walks, D))
        toks = np.take_along_axis(np.broadcast_to(ids[b], (n_walks, D, k)), pick[:, :, None],
                                  axis=2)[:, :, 0]
        seq = np.concatenate([np.full((n_walks, 1), prev[b]), np.full((n_walks, 1), root[b]), toks],
                             axis=1)
        walks.append(np.stack([seq[:, :-2], seq[:, 1:-1], seq[:, 2:]], axis=2).reshape(-1, 3))
    bg = rng.integers(0, w.vocab, (n_background, 3))
    tri = np.unique(np.concatenate(walks + [bg]).astype(np.int64), axis=0)
    tri = tri[rng.permutation(len(tri))]
    logp = np.log(rng.uniform(1e-3, 1.0, len(tri))).astype(np.float32)
    return (tri[:, 0].astype(np.int32), tri[:, 1].astype(np.int32), tri[:, 2].astype(np.int32),
            logp)


def ctx_lengths(w: Workload) -> np.ndarray:
    lo, hi = w.ctx
    if lo == hi:
        return np.full(w.batch, lo, np.int32)
    return _rng(w, 0, 0, S_CTX).integers(lo, hi + 1, size=w.batch).astype(np.int32)


# ----------------------------------------------------------------------------
# target logits, keyed by the node's rank path

def rank_paths(parent: np.ndarray, rank: np.ndarray, n_nodes: np.ndarray) -> list:
    """Per sequence, per node: tuple of (rank + 1) digits from depth 1 down."""
    out = []
    for s in range(parent.shape[0]):
        paths = []
        for n in range(int(n_nodes[s])):
            digits = []
            c = n
            while c > 0:
                digits.append(int(rank[s, c]) + 1)
                c = int(parent[s, c])
            paths.append(tuple(reversed(digits)))
        out.append(paths)
    return out


def target_logits(w: Workload, F: np.ndarray, parent: np.ndarray, rank: np.ndarray,
                  n_nodes: np.ndarray) -> np.ndarray:
    """Target logits [b, N, V]: node of depth delta sees F[:, delta] + sigma_t * E(path).

    Rows of padding nodes (n >= n_nodes) are zero.
    """
    b, N, V = w.batch, w.n_max, w.vocab
    T = np.zeros((b, N, V), np.float32)
    paths = rank_paths(parent, rank, n_nodes)

    def fill(it):
        s, n = it
        p = paths[s][n]
        e = _rng(w, s, 0, S_TNOISE, len(p) + 1, *p).standard_normal(V, dtype=np.float32)
        T[s, n] = F[s, len(p)] + np.float32(w.sigma_t) * e

    _parallel(fill, [(s, n) for s in range(b) for n in range(int(n_nodes[s]))])
    return cast(T, w.dtype)


# ----------------------------------------------------------------------------
# attention inputs

def _normal_rows(w: Workload, shape, seq: int, layer: int, stream: int) -> np.ndarray:
    """N(0,1) tensor whose leading axis is drawn in fixed chunks (thread-count independent)."""
    out = np.empty(shape, np.float32)
    n0 = shape[0]
    chunks = [(c, min(n0, c + _KV_CHUNK)) for c in range(0, n0, _KV_CHUNK)]

    def fill(ci):
        i, (a, e) = ci
        _rng(w, seq, layer, stream, i + 1).standard_normal(out[a:e].shape, dtype=np.float32,
                                                           out=out[a:e])

    _parallel(fill, list(enumerate(chunks)))
    return out


def attention_inputs(w: Workload, layer: int = 0, ctx: np.ndarray | None = None) -> dict:
    """Q [b,N,Hq,d], packed KV cache [sum ctx,Hkv,d], ctx_offsets [b+1], tree K/V [b,N,Hkv,d]."""
    if ctx is None:
        ctx = ctx_lengths(w)
    b, N, hq, hkv, d = w.batch, w.n_max, w.hq, w.hkv, w.head_dim
    offs = np.zeros(b + 1, np.int64)
    offs[1:] = np.cumsum(ctx)
    total = int(offs[-1])
    kc = np.empty((total, hkv, d), np.float32)
    vc = np.empty((total, hkv, d), np.float32)
    q = np.empty((b, N, hq, d), np.float32)
    kt = np.empty((b, N, hkv, d), np.float32)
    vt = np.empty((b, N, hkv, d), np.float32)
    for s in range(b):
        a, e = int(offs[s]), int(offs[s + 1])
        kc[a:e] = _normal_rows(w, (e - a, hkv, d), s, layer + 1, S_K)
        vc[a:e] = _normal_rows(w, (e - a, hkv, d), s, layer + 1, S_V)
        q[s] = _normal_rows(w, (N, hq, d), s, layer + 1, S_Q)
        kt[s] = _normal_rows(w, (N, hkv, d), s, layer + 1, S_KT)
        vt[s] = _normal_rows(w, (N, hkv, d), s, layer + 1, S_VT)
    return {
        "q": cast(q, w.dtype), "k_cache": cast(kc, w.dtype), "v_cache": cast(vc, w.dtype),
        "ctx_offsets": offs.astype(np.int32), "k_tree": cast(kt, w.dtype),
        "v_tree": cast(vt, w.dtype),
    }


def round_inputs(w: Workload) -> dict:
    """Everything a round needs before the tree exists (target logits come after the build)."""
    F = field(w)
    return {
        "field": F,
        "drafter_logits": drafter_logits(w, F),
        "rho": rho_lattice(w),
        "lam": lambdas(w),
        "root_token": root_tokens(w),
        "ctx": ctx_lengths(w),
    }
