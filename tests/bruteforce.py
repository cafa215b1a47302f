"""Pure-Python brute force for tiny draft blocks: an independent check of the oracle.

It enumerates every node of the candidate lattice (all prefixes y_{1:d}, d <= gamma, of
the K^gamma candidate paths), scores each from scratch as a path sum (Appendix A, Eq.
ubtree-path and ubtree-depth-bonus), and ranks nodes by the total order the build uses
for ties: within a depth, score desc, then the parent's own order, then the candidate
rank; across depths, score desc, then depth asc.  Unlike the oracle it keeps no
incremental state: no frontier arrays, no parent positions, no stable sorts.
"""
from __future__ import annotations

import itertools

import numpy as np


def path_score(logq: np.ndarray, path: tuple, zeta: float) -> float:
    """l_zeta(y_{1:d}) = sum_i log q_i^bi(y_i | y_{i-1}) + zeta * d, with y_0 the anchor (row 0)."""
    s = 0.0
    prev = 0
    for i, c in enumerate(path):
        s += float(logq[i, prev, c])
        prev = c
    return s + zeta * len(path)


def depth_key(scores: dict, path: tuple) -> tuple:
    """Sort key of the within-depth order: (-l(y_{1:d}), -l(y_{1:d-1}), ..., -l(y_1), c_1, ..., c_d).

    Comparing two nodes of one depth walks their scores from the node towards the root and
    then their candidate ranks from the root down; the first candidate rank that differs
    sits where the two paths split, i.e. where they have a common parent."""
    return tuple(-scores[path[:k]] for k in range(len(path), 0, -1)) + tuple(path)


def global_key(scores: dict, path: tuple) -> tuple:
    return (-scores[path], len(path)) + depth_key(scores, path)


def lattice(logq: np.ndarray, zeta: float) -> dict:
    """Every non-root node of the lattice -> its score."""
    gamma, K = logq.shape[0], logq.shape[2]
    out = {}
    for d in range(1, gamma + 1):
        for path in itertools.product(range(K), repeat=d):
            out[path] = path_score(logq, path, zeta)
    return out


def best_first(logq: np.ndarray, budget: int, zeta: float = 0.0) -> list:
    """The global top-`budget` nodes of the whole lattice, in order (no width limit)."""
    sc = lattice(logq, zeta)
    return sorted(sc, key=lambda p: global_key(sc, p))[:budget]


def beam(logq: np.ndarray, W: int, budget: int, zeta: float = 0.0) -> tuple[list, list]:
    """Depth-wise expansion with width W, then global pruning; returns (frontiers, tree).

    F_d is taken from the full lattice as the W best depth-d nodes whose parent is in
    F_{d-1}; the tree is the `budget` best nodes of the union of the F_d."""
    gamma = logq.shape[0]
    sc = lattice(logq, zeta)
    frontiers = []
    keep = {()}
    for d in range(1, gamma + 1):
        ext = [p for p in sc if len(p) == d and p[:-1] in keep]
        ext.sort(key=lambda p: depth_key(sc, p))
        fd = ext[:W]
        frontiers.append(fd)
        keep = set(fd)
    sup = [p for fd in frontiers for p in fd]
    tree = sorted(sup, key=lambda p: global_key(sc, p))[:budget]
    return frontiers, tree


def tree_as_paths(out: dict, b: int) -> list:
    """The oracle's (or the GPU's) emitted tree of sequence b as candidate-rank paths, in slot order."""
    n = int(out["n_nodes"][b])
    par, cr = out["parent"][b], out["cand_rank"][b]
    paths = [()]
    for i in range(1, n):
        paths.append(paths[int(par[i])] + (int(cr[i]),))
    return paths[1:]


def frontier_as_paths(out: dict, b: int) -> list:
    """The supertree dump F_1..F_gamma of sequence b as candidate-rank paths."""
    gamma = out["f_count"].shape[1]
    prev = [()]
    res = []
    for d in range(gamma):
        cnt = int(out["f_count"][b, d])
        cur = [prev[int(out["f_parent"][b, d, j])] + (int(out["f_cand"][b, d, j]),) for j in range(cnt)]
        res.append(cur)
        prev = cur
    return res


def closure_best_first(edge: np.ndarray, budget: int, zeta: float = 0.0) -> list:
    """Best-first growth under arbitrary (not necessarily monotone) edge scores, by brute
    force: every lattice node is scored from scratch as a path sum; then, `budget` times,
    the best node not yet taken whose parent is taken is added, under (score desc, depth
    asc, parent's position in the taken list asc, candidate rank asc).  Returns the taken
    nodes in order.  No frontier is kept: each round rescans the whole lattice."""
    sc = lattice(edge, zeta)
    taken = [()]
    pos = {(): 0}
    while len(taken) - 1 < budget:
        best, best_key = None, None
        for p in sc:
            if p in pos or p[:-1] not in pos:
                continue
            key = (-sc[p], len(p), pos[p[:-1]], p[-1])
            if best_key is None or key < best_key:
                best, best_key = p, key
        if best is None:
            break
        pos[best] = len(taken)
        taken.append(best)
    return taken[1:]
