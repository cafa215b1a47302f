"""TEST INFRASTRUCTURE: the fp64 CPU oracle of the UBTree draft-tree construction step.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (``paper_2609_39972_amd``)
never does, and the two share no code.

This module only marshals numpy arrays into the plain C++ oracle
(``ubt_oracle.cpp``), which holds the arithmetic.  bf16 arrays travel as their
``uint16`` bit patterns and are decoded exactly inside the oracle.
"""
from __future__ import annotations

import contextlib
import ctypes
import os

import numpy as np

from . import _build

_lib = None
DTYPE_CODE = {"f32": 0, "bf16": 1}

_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int
_f64 = ctypes.c_double


def _load(path: str) -> ctypes.CDLL:
    L = ctypes.CDLL(path)
    L.ubt_oracle_topk.argtypes = [_p, _i32, _i64, _i64, _i32, _p, _p, _p, _p, _i32]
    L.ubt_oracle_bigram.argtypes = [_p, _p, _p, _i32, _i64, _i32, _p, _p, _p, _p, _p,
                                    _i32, _i32, _i32, _p, _p, _i32]
    L.ubt_oracle_build_tree.argtypes = [_p, _p, _p, _i32, _i32, _i32, _i32, _i32, _f64,
                                        _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _i32]
    L.ubt_oracle_tree_mask.argtypes = [_p, _p, _i32, _i32, _p]
    L.ubt_oracle_edge_scores.argtypes = [_p, _p, _p, _p, _i32, _i32, _i32, _p]
    L.ubt_oracle_best_first.argtypes = [_p, _p, _p, _i32, _i32, _i32, _i32, _f64, _p, _p, _p, _p, _p, _p, _p, _i32]
    for f in (L.ubt_oracle_topk, L.ubt_oracle_bigram, L.ubt_oracle_build_tree, L.ubt_oracle_tree_mask,
              L.ubt_oracle_edge_scores, L.ubt_oracle_best_first):
        f.restype = _i32
    return L


def lib() -> ctypes.CDLL:
    """The oracle library; compiled on first use if no build is present."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _lib = _load(_build.LIB)
    return _lib


@contextlib.contextmanager
def using_library(path: str):
    """Routes every call to the oracle library at ``path`` for the duration (mutation tests)."""
    global _lib
    saved = _lib
    _lib = _load(path)
    try:
        yield
    finally:
        _lib = saved


def default_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(_p)


def _dtype_of(a: np.ndarray) -> int:
    if a.dtype == np.uint16:
        return DTYPE_CODE["bf16"]
    if a.dtype == np.float32:
        return DTYPE_CODE["f32"]
    raise TypeError(f"stored values must be float32 or bf16 bits (uint16), got {a.dtype}")


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with status {rc}")


def topk(logits: np.ndarray, K: int, threads: int | None = None) -> dict:
    """Candidate sets of every row of ``logits [..., V]``: ids, logits, log q_i and LSE."""
    x = np.ascontiguousarray(logits)
    lead, V = x.shape[:-1], x.shape[-1]
    rows = int(np.prod(lead)) if lead else 1
    ids = np.empty(lead + (K,), np.int32)
    val = np.empty(lead + (K,), np.float64)
    lp = np.empty(lead + (K,), np.float64)
    lse = np.empty(lead, np.float64)
    _check(lib().ubt_oracle_topk(_ptr(x), _dtype_of(x), rows, V, K, _ptr(ids), _ptr(val), _ptr(lp), _ptr(lse),
                                 threads or default_threads()), "topk")
    return dict(cand_ids=ids, cand_logit=val, cand_logprob=lp, lse=lse)


def bigram(phi: np.ndarray, psi: np.ndarray, gate: np.ndarray, anchor: np.ndarray, cand_ids: np.ndarray,
           cand_logit: np.ndarray, alpha: np.ndarray, lam: np.ndarray, threads: int | None = None) -> dict:
    """Selector scores delta and normalised log q^bi for all adjacent candidate pairs."""
    phi, psi, gate = (np.ascontiguousarray(a) for a in (phi, psi, gate))
    if not (phi.dtype == psi.dtype == gate.dtype):
        raise TypeError("phi, psi and gate must share one storage dtype")
    V, r = phi.shape
    B, gamma, K = cand_ids.shape
    ids = np.ascontiguousarray(cand_ids, np.int32)
    anc = np.ascontiguousarray(anchor, np.int32)
    cl = np.ascontiguousarray(cand_logit, np.float64)
    al = np.ascontiguousarray(alpha, np.float64)
    la = np.ascontiguousarray(lam, np.float64)
    delta = np.empty((B, gamma, K, K), np.float64)
    logq = np.empty((B, gamma, K, K), np.float64)
    _check(lib().ubt_oracle_bigram(_ptr(phi), _ptr(psi), _ptr(gate), _dtype_of(phi), V, r, _ptr(anc), _ptr(ids),
                                   _ptr(cl), _ptr(al), _ptr(la), B, gamma, K, _ptr(delta), _ptr(logq),
                                   threads or default_threads()), "bigram")
    return dict(delta=delta, logq=logq)


def build_tree(anchor: np.ndarray, cand_ids: np.ndarray, logq: np.ndarray, W: int, budget: int,
               zeta: float = 0.0, threads: int | None = None) -> dict:
    """Algorithm 1 on every sequence; returns the tree, its mask and the supertree F_d."""
    B, gamma, K = cand_ids.shape
    N = budget + 1
    words = (N + 31) // 32
    anc = np.ascontiguousarray(anchor, np.int32)
    ids = np.ascontiguousarray(cand_ids, np.int32)
    q = np.ascontiguousarray(logq, np.float64)
    out = dict(n_nodes=np.empty(B, np.int32), token=np.empty((B, N), np.int32), parent=np.empty((B, N), np.int32),
               depth=np.empty((B, N), np.int32), cand_rank=np.empty((B, N), np.int32),
               score=np.empty((B, N), np.float64), mask=np.empty((B, N, words), np.uint32),
               f_count=np.empty((B, gamma), np.int32), f_parent=np.empty((B, gamma, W), np.int32),
               f_cand=np.empty((B, gamma, W), np.int32), f_score=np.empty((B, gamma, W), np.float64))
    o = out
    _check(lib().ubt_oracle_build_tree(_ptr(anc), _ptr(ids), _ptr(q), B, gamma, K, W, budget, float(zeta),
                                       _ptr(o["n_nodes"]), _ptr(o["token"]), _ptr(o["parent"]), _ptr(o["depth"]),
                                       _ptr(o["cand_rank"]), _ptr(o["score"]), _ptr(o["mask"]), _ptr(o["f_count"]),
                                       _ptr(o["f_parent"]), _ptr(o["f_cand"]), _ptr(o["f_score"]),
                                       threads or default_threads()), "build_tree")
    return out


def tree_mask(parent: np.ndarray, n_nodes: np.ndarray) -> np.ndarray:
    """Ancestor mask rows ``[B, N, ceil(N/32)]`` from parent pointers ``[B, N]``."""
    par = np.ascontiguousarray(parent, np.int32)
    nn = np.ascontiguousarray(n_nodes, np.int32)
    B, N = par.shape
    mask = np.empty((B, N, (N + 31) // 32), np.uint32)
    _check(lib().ubt_oracle_tree_mask(_ptr(par), _ptr(nn), B, N, _ptr(mask)), "tree_mask")
    return mask


def pipeline(logits: np.ndarray, phi: np.ndarray, psi: np.ndarray, gate: np.ndarray, anchor: np.ndarray,
             alpha: np.ndarray, lam: np.ndarray, K: int, W: int, budget: int, zeta: float = 0.0,
             threads: int | None = None) -> dict:
    """The whole step on ``logits [B, gamma, V]``: candidates, selector scores, tree."""
    t = topk(logits, K, threads)
    g = bigram(phi, psi, gate, anchor, t["cand_ids"], t["cand_logit"], alpha, lam, threads)
    tr = build_tree(anchor, t["cand_ids"], g["logq"], W, budget, zeta, threads)
    return {**t, **g, **tr}


def edge_scores(cand_logprob: np.ndarray, delta: np.ndarray, alpha: np.ndarray, lam: np.ndarray) -> np.ndarray:
    """Unigram-plus-bigram edge scores ``[B, gamma, K, K]``: alpha_i log q_i(c) + lambda_i
    delta_i(a, c), not normalised over the successors."""
    B, gamma, K = cand_logprob.shape
    lp = np.ascontiguousarray(cand_logprob, np.float64)
    dl = np.ascontiguousarray(delta, np.float64)
    al = np.ascontiguousarray(alpha, np.float64)
    la = np.ascontiguousarray(lam, np.float64)
    edge = np.empty((B, gamma, K, K), np.float64)
    _check(lib().ubt_oracle_edge_scores(_ptr(lp), _ptr(dl), _ptr(al), _ptr(la), B, gamma, K, _ptr(edge)),
           "edge_scores")
    return edge


def best_first(anchor: np.ndarray, cand_ids: np.ndarray, edge: np.ndarray, budget: int, zeta: float = 0.0,
               threads: int | None = None) -> dict:
    """Best-first tree over the candidate lattice under cumulative edge scores, grown
    from the root one node at a time (a node is eligible once its parent is in)."""
    B, gamma, K = cand_ids.shape
    N = budget + 1
    words = (N + 31) // 32
    anc = np.ascontiguousarray(anchor, np.int32)
    ids = np.ascontiguousarray(cand_ids, np.int32)
    e = np.ascontiguousarray(edge, np.float64)
    o = dict(n_nodes=np.empty(B, np.int32), token=np.empty((B, N), np.int32), parent=np.empty((B, N), np.int32),
             depth=np.empty((B, N), np.int32), cand_rank=np.empty((B, N), np.int32),
             score=np.empty((B, N), np.float64), mask=np.empty((B, N, words), np.uint32))
    _check(lib().ubt_oracle_best_first(_ptr(anc), _ptr(ids), _ptr(e), B, gamma, K, budget, float(zeta),
                                       _ptr(o["n_nodes"]), _ptr(o["token"]), _ptr(o["parent"]), _ptr(o["depth"]),
                                       _ptr(o["cand_rank"]), _ptr(o["score"]), _ptr(o["mask"]),
                                       threads or default_threads()), "best_first")
    return o


def pipeline_unigram_bigram(logits: np.ndarray, phi: np.ndarray, psi: np.ndarray, gate: np.ndarray,
                            anchor: np.ndarray, alpha: np.ndarray, lam: np.ndarray, K: int, budget: int,
                            zeta: float = 0.0, threads: int | None = None) -> dict:
    """The step under the unigram-plus-bigram scoring: candidates, selector scores, edge
    scores and the best-first tree."""
    t = topk(logits, K, threads)
    g = bigram(phi, psi, gate, anchor, t["cand_ids"], t["cand_logit"], alpha, lam, threads)
    e = edge_scores(t["cand_logprob"], g["delta"], alpha, lam)
    tr = best_first(anchor, t["cand_ids"], e, budget, zeta, threads)
    return {**t, **g, "edge": e, **tr}
