"""Brute-force checkers used to pin the oracle on tiny inputs.

Each checker restates what the paper fixes in a different form from the
oracle's algorithm:

* ``full_tree`` / ``top_b``: enumerate every node of the candidate tree and
  keep the B best prefixes (Sec. 4.2: the optimal tree is the B prefixes
  with the largest S; Eq. 3 and Appendix A).
* ``max_prefix_mass``: exhaustive search over prefix-closed node sets of size
  B for the largest surrogate mass sum exp(S) (Eq. 3), with no ranking rule.
* ``path_attention``: each node's output recomputed as ordinary attention
  over the explicit sequence [cached prefix ; root .. node] (Appendix C
  stage I), from parent pointers rather than the ancestor mask.
* ``brute_accept``: every root-to-node path tested for acceptance token by
  token (Eq. 1 at temperature 0), keeping the longest.
"""
from __future__ import annotations

import itertools

import numpy as np
from scipy.special import softmax


def token_score(lp, lam, R, row, a, b, r):
    """s = log q + lambda * log rho, each operation rounded to fp32."""
    if R is None:
        return np.float32(lp[row, r])
    return np.float32(np.float32(lp[row, r]) + np.float32(np.float32(lam[row]) * np.float32(R[row, a, b, r])))


def full_tree(lp, lam, R, D, k, branch=None):
    """All nodes of the candidate tree: dict path(tuple of ranks) -> S (fp32)."""
    branch = k if branch is None else branch
    nodes = {(): np.float32(0.0)}
    frontier = [()]
    while frontier:
        nxt = []
        for u in frontier:
            d = len(u)
            if d >= D:
                continue
            a = u[-2] if d >= 2 else 0
            b = u[-1] if d >= 1 else 0
            s = [token_score(lp, lam, R, d, a, b, r) for r in range(k)]
            order = sorted(range(k), key=lambda r: (-float(s[r]), r))[:branch]
            for r in order:
                c = u + (r,)
                nodes[c] = np.float32(nodes[u] + s[r])
                nxt.append(c)
        frontier = nxt
    return nodes


def top_b(nodes, B):
    """The B best non-root prefixes: larger S first, then lexicographic rank path."""
    cands = [u for u in nodes if u]
    cands.sort(key=lambda u: (-float(nodes[u]), u))
    return cands[:B]


def paths_of(tree, s=0):
    """Rank path of every live node of one sequence of a tree dict (oracle layout)."""
    out = []
    for n in range(int(tree["n_nodes"][s])):
        p = []
        c = n
        while c > 0:
            p.append(int(tree["rank"][s, c]))
            c = int(tree["parent"][s, c])
        out.append(tuple(reversed(p)))
    return out


def prefix_closed_subsets(nodes, B):
    """All prefix-closed sets of B non-root nodes (tiny trees only)."""
    cands = [u for u in nodes if u]
    for combo in itertools.combinations(cands, B):
        s = set(combo)
        if all(len(u) == 1 or u[:-1] in s for u in combo):
            yield combo


def max_prefix_mass(nodes, B):
    best = -np.inf
    for combo in prefix_closed_subsets(nodes, B):
        best = max(best, sum(np.exp(np.float64(nodes[u])) for u in combo))
    return best


def anc_from_parent(parent, n_nodes, N):
    """Ancestor-or-self bit rows built from parent pointers."""
    W = (N + 63) // 64
    anc = np.zeros((parent.shape[0], N, W), np.uint64)
    for s in range(parent.shape[0]):
        for n in range(int(n_nodes[s])):
            c = n
            while c >= 0:
                anc[s, n, c // 64] |= np.uint64(1) << np.uint64(c % 64)
                c = int(parent[s, c]) if c > 0 else -1
    return anc


def path_attention(q, kc, vc, offs, kt, vt, parent, b, n, h, scale):
    """fp64 attention of query (b, n, h) over [cache ; root .. n] built from parent pointers."""
    hq, hkv = q.shape[2], kc.shape[1]
    g = h // (hq // hkv)
    chain = []
    c = n
    while True:
        chain.append(c)
        if c == 0:
            break
        c = int(parent[b, c])
    chain = chain[::-1]
    K = np.concatenate([kc[offs[b]:offs[b + 1], g], kt[b, chain, g]], 0).astype(np.float64)
    V = np.concatenate([vc[offs[b]:offs[b + 1], g], vt[b, chain, g]], 0).astype(np.float64)
    p = softmax(K @ q[b, n, h].astype(np.float64) * scale)
    return p @ V


def brute_accept(T, parent, token, n_nodes, b):
    """Longest accepted root-to-node path, checking each token against np.argmax."""
    a = [int(np.argmax(T[b, n])) for n in range(int(n_nodes[b]))]
    best = [0]
    for n in range(1, int(n_nodes[b])):
        chain = []
        c = n
        while c > 0:
            chain.append(c)
            c = int(parent[b, c])
        chain = [0] + chain[::-1]
        if all(int(token[b, chain[i + 1]]) == a[chain[i]] for i in range(len(chain) - 1)):
            if len(chain) > len(best):
                best = chain
    return len(best) - 1, best, a[best[-1]], a
