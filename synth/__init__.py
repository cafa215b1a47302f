"""Seeded synthetic workloads for the UBTree draft-tree construction step.

This module only draws random numbers and rounds them to the storage dtype.  It
holds none of the method's arithmetic, so both the fp64 oracle (``oracle/``) and the
HIP path (``paper_2609_39972_amd``) can be fed from it without sharing code.

The five workloads stand in for the DFlash proposer outputs of the paper's
Qwen3-scale experiments (vocabulary 151936), which are not available: proposer
logits, the selector gate ``P(h_i)``, the vocabulary-wide codebook tables
``phi``/``psi`` (Method, "Deep Codebooks") and the anchor token.

Every array is drawn from ``numpy.random.default_rng(SeedSequence([cfg, buf, field,
...]))`` with field ids 0 logits, 1 permutation, 2 noise, 3 phi table, 4 psi table,
5 gate, 6 anchor.  Logit rows are drawn one row at a time (the row index is part of
the seed), so any subset of rows can be regenerated on its own.  Values are drawn in
fp64, rounded to fp32 (round-to-nearest-even) and, for bf16 storage, rounded once
more to bf16 (round-to-nearest-even).  bf16 arrays are returned as ``uint16`` bit
patterns; fp32 arrays as ``float32``.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import math
import os

import numpy as np

F_LOGIT, F_PERM, F_NOISE, F_PHI, F_PSI, F_GATE, F_ANCHOR = range(7)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload.  ``L`` is the drafting block including the anchor, so a
    sequence carries ``gamma = L - 1`` logit rows; ``budget`` counts non-root nodes."""

    cfg: int
    name: str
    B: int
    L: int
    V: int
    K: int
    r: int
    budget: int
    W: int
    dtype: str  # logits storage: "f32" | "bf16"
    feat_dtype: str  # phi/psi/gate storage
    logits: str  # "normal" | "zipf"
    logit_std: float = 0.0  # for "normal"
    zipf_s: float = 1.1
    noise_var: float = 0.5
    temperature: float = 1.0
    steps: int = 1
    zeta: float = 0.0

    @property
    def gamma(self) -> int:
        return self.L - 1

    @property
    def rows(self) -> int:
        return self.B * self.gamma

    @property
    def N(self) -> int:
        return self.budget + 1

    @property
    def logit_bytes(self) -> int:
        return self.rows * self.V * (2 if self.dtype == "bf16" else 4)

    def describe(self) -> str:
        return (f"B={self.B} L={self.L} (gamma={self.gamma}) V={self.V} {self.dtype} {self.logits} logits, "
                f"K={self.K} r={self.r} {self.feat_dtype} features, budget={self.budget} W={self.W}")


WORKLOADS = {
    1: Workload(1, "normal3-v32000-b1", B=1, L=8, V=32000, K=4, r=32, budget=16, W=3,
                dtype="f32", feat_dtype="f32", logits="normal", logit_std=3.0, steps=1),
    2: Workload(2, "zipf-v151936-b8", B=8, L=16, V=151936, K=8, r=64, budget=32, W=8,
                dtype="bf16", feat_dtype="bf16", logits="zipf", steps=100),
    3: Workload(3, "zipf-v151936-b32", B=32, L=16, V=151936, K=8, r=128, budget=64, W=12,
                dtype="bf16", feat_dtype="bf16", logits="zipf", steps=1000),
    4: Workload(4, "highentropy-v151936-b32", B=32, L=16, V=151936, K=16, r=128, budget=128, W=24,
                dtype="bf16", feat_dtype="bf16", logits="normal", logit_std=0.7, steps=1000),
    5: Workload(5, "zipf-v151936-b256", B=256, L=32, V=151936, K=16, r=256, budget=128, W=24,
                dtype="bf16", feat_dtype="bf16", logits="zipf", steps=200),
    # The paper's own configuration (Appendix, Table "UBTree configuration": 15 future
    # positions plus the anchor, K = 64, W = 12, budget 64, selector rank 256, zeta = 0)
    # on the headline batch of 32 sequences.
    6: Workload(6, "paper-k64-v151936-b32", B=32, L=16, V=151936, K=64, r=256, budget=64, W=12,
                dtype="bf16", feat_dtype="bf16", logits="zipf", steps=1000),
}


def custom(cfg: int = 100, **kw) -> Workload:
    """A workload of arbitrary shape (tests).  Unspecified fields take small defaults."""
    base = dict(name=f"custom{cfg}", B=2, L=5, V=1000, K=4, r=16, budget=8, W=3, dtype="f32",
                feat_dtype="f32", logits="normal", logit_std=2.0)
    base.update(kw)
    return Workload(cfg, **base)


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(k) for k in key]))


def round_f32(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def round_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp64 -> fp32 (RNE) -> bf16 (RNE); returns the bf16 bit patterns as uint16."""
    bits = round_f32(x).view(np.uint32)
    bias = ((bits >> 16) & 1) + np.uint32(0x7FFF)
    return ((bits + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32 values (for inspection / plots)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    return round_bf16_bits(x) if dtype == "bf16" else round_f32(x)


def _zipf_base(V: int, s: float) -> np.ndarray:
    k = np.arange(1, V + 1, dtype=np.float64)
    logk = -s * np.log(k)
    return logk - np.log(np.exp(logk).sum())


def logit_row(w: Workload, buf: int, row: int, _base_cache: dict = {}) -> np.ndarray:
    """fp64 logits of one (sequence, position) row, before rounding to storage."""
    if w.logits == "normal":
        return _rng(w.cfg, buf, F_LOGIT, row).normal(0.0, w.logit_std, w.V)
    if w.logits == "zipf":
        key = (w.V, w.zipf_s)
        if key not in _base_cache:
            _base_cache[key] = _zipf_base(w.V, w.zipf_s)
        base = _base_cache[key]
        perm = _rng(w.cfg, buf, F_PERM, row).permutation(w.V)
        noise = _rng(w.cfg, buf, F_NOISE, row).normal(0.0, math.sqrt(w.noise_var), w.V)
        u = np.empty(w.V, dtype=np.float64)
        u[perm] = (base + noise) / w.temperature
        return u
    raise ValueError(w.logits)


def logits(w: Workload, buf: int = 0, rows: np.ndarray | None = None, workers: int | None = None) -> np.ndarray:
    """Stored logits ``[B, gamma, V]`` (or ``[len(rows), V]`` for a row subset)."""
    idx = np.arange(w.rows) if rows is None else np.asarray(rows)
    out = np.empty((len(idx), w.V), dtype=np.uint16 if w.dtype == "bf16" else np.float32)

    def fill(j: int) -> None:
        out[j] = store(logit_row(w, buf, int(idx[j])), w.dtype)

    workers = workers or min(16, os.cpu_count() or 1)
    if len(idx) > 8 and workers > 1:
        with _cf.ThreadPoolExecutor(workers) as ex:
            list(ex.map(fill, range(len(idx))))
    else:
        for j in range(len(idx)):
            fill(j)
    return out.reshape(w.B, w.gamma, w.V) if rows is None else out


def tables(w: Workload) -> tuple[np.ndarray, np.ndarray]:
    """Vocabulary-wide codebook tables ``phi, psi`` of shape ``[V, r]``, entries N(0, 1/r).
    They are model constants, so they do not depend on the buffer index."""
    sd = 1.0 / math.sqrt(w.r)
    phi = store(_rng(w.cfg, 0, F_PHI).normal(0.0, sd, (w.V, w.r)), w.feat_dtype)
    psi = store(_rng(w.cfg, 0, F_PSI).normal(0.0, sd, (w.V, w.r)), w.feat_dtype)
    return phi, psi


def gate(w: Workload, buf: int = 0) -> np.ndarray:
    """Selector gate ``P(h_i)`` per (sequence, position): ``[B, gamma, r]``, entries N(0, 1)."""
    return store(_rng(w.cfg, buf, F_GATE).normal(0.0, 1.0, (w.B, w.gamma, w.r)), w.feat_dtype)


def anchor(w: Workload, buf: int = 0) -> np.ndarray:
    """Anchor token per sequence, uniform over the vocabulary: ``int32[B]``."""
    return _rng(w.cfg, buf, F_ANCHOR).integers(0, w.V, w.B).astype(np.int32)


def calibration(w: Workload) -> tuple[np.ndarray, np.ndarray]:
    """Depth scales alpha, lambda (``float32[gamma]``): unit weights, as initialised in the paper."""
    return np.ones(w.gamma, np.float32), np.ones(w.gamma, np.float32)


def inputs(w: Workload, buf: int = 0, with_tables: bool = True) -> dict:
    d = dict(logits=logits(w, buf), gate=gate(w, buf), anchor=anchor(w, buf))
    d["alpha"], d["lam"] = calibration(w)
    if with_tables:
        d["phi"], d["psi"] = tables(w)
    return d


def dyadic_logq(B: int, gamma: int, K: int, seed: int = 0, step: float = 2.0 ** -6,
                levels: int = 64, tie_frac: float = 0.0) -> np.ndarray:
    """Synthetic normalised-score slabs ``[B, gamma, K, K]`` whose entries are exact
    multiples of ``step`` in ``(-levels*step, 0]``.  Sums along any path are then exact in
    fp32 and fp64 alike, so tree construction can be compared bit for bit, exact ties
    included.  With ``tie_frac`` > 0 that share of entries is copied from another entry of
    the same slab to force ties.  The rows are not normalised: the tree search only
    needs them to be <= 0."""
    rng = _rng(900, seed, B, gamma, K)
    q = -rng.integers(0, levels, size=(B, gamma, K, K)).astype(np.float64) * step
    if tie_frac > 0:
        m = rng.random((B, gamma, K, K)) < tie_frac
        src = rng.integers(0, K * K, size=(B, gamma, K, K))
        flat = q.reshape(B, gamma, K * K)
        q = np.where(m, np.take_along_axis(flat, src.reshape(B, gamma, K * K), 2).reshape(B, gamma, K, K), q)
    return q.astype(np.float32)


def candidate_ids(B: int, gamma: int, K: int, V: int, seed: int = 0) -> np.ndarray:
    """Arbitrary candidate token ids ``int32[B, gamma, K]`` (tree tests that start from logq)."""
    return _rng(901, seed, B, gamma, K).integers(0, V, size=(B, gamma, K)).astype(np.int32)


# ---- verification inputs ----------------------------------------------------------------
F_VQ, F_VKC, F_VVC, F_VKT, F_VVT, F_VTARGET = range(20, 26)


def verify_inputs(seed: int, B: int, N: int, H: int, Hkv: int, D: int, Pmax: int) -> dict:
    """Synthetic operands of tree verification as bf16 bit patterns (uint16): queries of
    the tree nodes ``q [B, N, H, D]``, cached keys/values ``[B, Pmax, Hkv, D]`` and the
    tree nodes' keys/values ``[B, N, Hkv, D]``, all i.i.d. N(0, 1) (so that q.k / sqrt(D)
    is of unit scale, as after the target's normalisation layers)."""
    def draw(field, shape):
        return round_bf16_bits(_rng(seed, field).normal(0.0, 1.0, size=shape))

    return dict(q=draw(F_VQ, (B, N, H, D)), k_cache=draw(F_VKC, (B, Pmax, Hkv, D)),
                v_cache=draw(F_VVC, (B, Pmax, Hkv, D)), k_tree=draw(F_VKT, (B, N, Hkv, D)),
                v_tree=draw(F_VVT, (B, N, Hkv, D)))


def verify_targets(seed: int, token: np.ndarray, parent: np.ndarray, n_nodes: np.ndarray, V: int,
                   follow: float = 0.7) -> np.ndarray:
    """Target samples ``[B, N]`` for the acceptance walk: from the root, with probability
    ``follow`` per step the sample equals the token of a uniformly drawn child (so the walk
    goes on), otherwise a uniform token; nodes off that walk get uniform tokens."""
    rng = _rng(seed, F_VTARGET)
    B, N = token.shape
    tgt = rng.integers(0, V, size=(B, N)).astype(np.int32)
    for b in range(B):
        cur = 0
        while True:
            kids = [c for c in range(cur + 1, int(n_nodes[b])) if parent[b, c] == cur]
            if not kids or rng.random() >= follow:
                break
            c = kids[int(rng.integers(0, len(kids)))]
            tgt[b, cur] = token[b, c]
            cur = c
    return tgt


# ---- training-objective inputs ------------------------------------------------------------
F_TNOISE, F_YSTAR = 30, 31


def loss_inputs(w: Workload, buf: int = 0, invalid_frac: float = 0.05) -> dict:
    """Synthetic operands of the training objective for workload ``w``:

    * ``target_logits [B, gamma, V]`` (stored like the logits): each proposer row plus
      N(0, 1) noise, so the target agrees with the proposer only roughly;
    * ``y_star int32[B, gamma]``: the ground-truth tokens.  For Zipf rows the token of
      rank k (in the row's permutation) with probability proportional to k^-s over the
      first 64 ranks, so it usually lies in the candidate set; for normal rows a uniform
      token.  A share ``invalid_frac`` of the positions is -1 (not valid)."""
    rng = _rng(w.cfg, buf, F_YSTAR)
    z = np.empty((w.rows, w.V), dtype=np.uint16 if w.dtype == "bf16" else np.float32)
    y = np.empty(w.rows, np.int32)
    ranks = np.arange(1, 65, dtype=np.float64)
    pr = ranks ** -w.zipf_s
    pr /= pr.sum()
    for row in range(w.rows):
        u = logit_row(w, buf, row)
        z[row] = store(u + _rng(w.cfg, buf, F_TNOISE, row).normal(0.0, 1.0, w.V), w.dtype)
        if w.logits == "zipf":
            perm = _rng(w.cfg, buf, F_PERM, row).permutation(w.V)
            y[row] = perm[int(rng.choice(64, p=pr))]
        else:
            y[row] = int(rng.integers(0, w.V))
    y[rng.random(w.rows) < invalid_frac] = -1
    return dict(target_logits=z.reshape(w.B, w.gamma, w.V), y_star=y.reshape(w.B, w.gamma))


# ---- LM-head inputs ---------------------------------------------------------------------
F_LMH, F_LMW = 40, 41


def lm_head_inputs(seed: int, M: int, d: int, V: int, logit_std: float = 3.0) -> dict:
    """Synthetic operands of the LM-head projection as bf16 bit patterns (uint16): hidden
    states ``h [M, d]`` i.i.d. N(0, 1) (unit scale, as after the proposer's final
    normalisation) and a head ``W [V, d]`` i.i.d. N(0, logit_std^2 / d), so each logit is
    roughly N(0, logit_std^2).  W is drawn in blocks of rows to bound memory."""
    h = round_bf16_bits(_rng(seed, F_LMH).normal(0.0, 1.0, size=(M, d)))
    w = np.empty((V, d), np.uint16)
    sd = logit_std / math.sqrt(d)
    block = 8192
    for i, v0 in enumerate(range(0, V, block)):
        n = min(block, V - v0)
        w[v0:v0 + n] = round_bf16_bits(_rng(seed, F_LMW, i).normal(0.0, sd, size=(n, d)))
    return dict(h=h, w=w)
