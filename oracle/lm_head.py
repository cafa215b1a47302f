"""TEST INFRASTRUCTURE: fp64 oracle of the LM-head projection followed by the softmax
statistics and candidate sets.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module; the product path never does, and the two share no
code.

Background, "DFlash & DFlash 2": the proposer's hidden state h_i is mapped to its logits
u_i by the frozen target LM head, u_i = W_lm h_i.  Method / Unigram Proposer, Eq.
(ubtree-unigram) and "Candidate Sets": q_i = softmax(u_i) and C_i = the K tokens of
largest q_i (ties to the lower token id; softmax is increasing, so C_i ranks u_i).

Plain numpy in fp64: the bf16 inputs are widened exactly, the products h_k W_vk are exact
in fp64 and each logit is a fp64 sum of d of them.  W is taken in blocks of vocabulary
rows only to bound memory; every logit is the same fp64 matmul of one row of h with one
row of W.
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to fp64."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def logits(h_bits: np.ndarray, w_bits: np.ndarray, block: int = 8192) -> np.ndarray:
    """u[m, v] = sum_k h[m, k] W[v, k] in fp64, shape [M, V]."""
    h = bf16_to_f64(h_bits)
    V = w_bits.shape[0]
    out = np.empty((h.shape[0], V), np.float64)
    for v0 in range(0, V, block):
        out[:, v0:v0 + block] = h @ bf16_to_f64(w_bits[v0:v0 + block]).T
    return out


def abs_logits(h_bits: np.ndarray, w_bits: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """sum_k |h[m, k] W[v, k]| for v = ids[m, :] (the scale of a logit's rounding error)."""
    h = np.abs(bf16_to_f64(h_bits))
    return np.stack([np.abs(bf16_to_f64(w_bits[ids[m]])) @ h[m] for m in range(h.shape[0])])


def topk_of_logits(u: np.ndarray, K: int) -> dict:
    """Candidate sets and softmax statistics of fp64 logit rows: ids ordered by (logit
    desc, id asc), their logits and log-probabilities, and LSE (max-shifted)."""
    M, V = u.shape
    ids = np.empty((M, K), np.int32)
    for m in range(M):
        ids[m] = np.lexsort((np.arange(V), -u[m]))[:K]
    mx = u.max(axis=1, keepdims=True)
    lse = (mx + np.log(np.exp(u - mx).sum(axis=1, keepdims=True)))[:, 0]
    val = np.take_along_axis(u, ids.astype(np.int64), 1)
    return dict(cand_ids=ids, cand_logit=val, cand_logprob=val - lse[:, None], lse=lse)


def lm_head_topk(h_bits: np.ndarray, w_bits: np.ndarray, K: int) -> dict:
    """The LM head then the candidate sets of every row of h ([M, d] bf16 bits) under the
    head W ([V, d] bf16 bits); also returns the fp64 logits."""
    u = logits(h_bits, w_bits)
    return {**topk_of_logits(u, K), "logits": u}
