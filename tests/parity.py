"""Comparison of GPU outputs with the fp64 oracle.

Candidate ids, tree topology, tokens and masks are compared bit for bit.  Floating-point
outputs are compared within ``EPS * max(1, |ref|)`` (EPS = 1e-5).

Tree construction takes discrete decisions on floating-point scores.  The GPU scores in
fp32, the oracle in fp64, so two candidates whose scores differ by less than the
rounding can be ordered differently; both trees are then correct.  When the GPU tree is
not identical to the oracle's, :func:`check_tree` validates the GPU's own selections
against the oracle's fp64 scores step by step ("guided"): at every Top_W and at the
final Top_budget, every node the GPU kept or dropped must be on the right side of the
oracle's selection boundary, unless its fp64 score lies within ``EPS * max(1, |score|)``
of that boundary (the tie gap).  Structure (parents, depths, tokens, mask) must still
be exact for the GPU's tree.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np

EPS = 1e-5

# Largest share of a call's trees that may need the tie excusal.  A selection differs
# from the oracle's only when two fp64 scores lie within fp32 rounding (about 1e-6) of
# each other at a selection boundary, which at these score spreads happens for well
# under one tree in a thousand.
MAX_EXCUSED_SHARE = 0.05


def tol(ref: np.ndarray) -> np.ndarray:
    return EPS * np.maximum(1.0, np.abs(ref))


def close(gpu: np.ndarray, ref: np.ndarray, what: str) -> None:
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    same_inf = np.isinf(gpu) & np.isinf(ref) & (np.sign(gpu) == np.sign(ref))
    with np.errstate(invalid="ignore"):
        err = np.where(same_inf, 0.0, np.abs(gpu - ref))
    bad = ~(err <= tol(np.where(np.isinf(ref), 0.0, ref)))
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {int(bad.sum())} entries out of tolerance; first at {tuple(i)}: "
                             f"gpu={gpu[tuple(i)]!r} ref={ref[tuple(i)]!r}")


def check_topk(g: dict, ref: dict, rows: np.ndarray | None = None) -> None:
    """g: GPU outputs (numpy) for all rows; ref: oracle outputs for `rows` (flattened row
    indices) or for all rows."""
    K = g["cand_ids"].shape[-1]
    gid = g["cand_ids"].reshape(-1, K)
    glog = g["cand_logit"].reshape(-1, K)
    glp = g["cand_logprob"].reshape(-1, K) if g.get("cand_logprob") is not None else None
    glse = g["lse"].reshape(-1)
    if rows is not None:
        gid, glog, glse = gid[rows], glog[rows], glse[rows]
        glp = glp[rows] if glp is not None else None
    rid = ref["cand_ids"].reshape(-1, K)
    if not np.array_equal(gid, rid):
        r = int(np.argwhere((gid != rid).any(-1))[0][0])
        raise AssertionError(f"candidate ids differ in row {r}: gpu={gid[r].tolist()} ref={rid[r].tolist()}")
    np.testing.assert_array_equal(glog.astype(np.float64), ref["cand_logit"].reshape(-1, K), "candidate logits")
    close(glse, ref["lse"].reshape(-1), "lse")
    if glp is not None:
        close(glp, ref["cand_logprob"].reshape(-1, K), "cand_logprob")


def check_selector(g: dict, ref: dict, seqs: np.ndarray | None = None) -> None:
    for k in ("delta", "logq"):
        if g.get(k) is None:
            continue
        gv = g[k] if seqs is None else g[k][seqs]
        close(gv, ref[k], k)


def _paths_from_dump(g: dict, b: int) -> list:
    gamma = g["f_count"].shape[1]
    prev, out = [()], []
    for d in range(gamma):
        n = int(g["f_count"][b, d])
        cur = [prev[int(g["f_parent"][b, d, j])] + (int(g["f_cand"][b, d, j]),) for j in range(n)]
        out.append(cur)
        prev = cur
    return out


def _mask_bits(mask_row: np.ndarray, N: int) -> set:
    words = mask_row.view(np.uint32)
    return {m for m in range(N) if (int(words[m // 32]) >> (m % 32)) & 1}


def check_structure(g: dict, b: int, cand_ids: np.ndarray, anchor: int, budget: int, with_mask: bool = True) -> list:
    """Exact structural checks of the GPU tree of sequence b; returns its node paths."""
    N = budget + 1
    n = int(g["n_nodes"][b])
    par, dep, cr, tok = g["parent"][b], g["depth"][b], g["cand_rank"][b], g["token"][b]
    assert 1 <= n <= N
    assert par[0] == -1 and dep[0] == 0 and tok[0] == anchor and cr[0] == -1 and g["score"][b, 0] == 0
    paths = [()]
    for i in range(1, n):
        p = int(par[i])
        assert 0 <= p < i, f"slot {i}: parent {p} does not precede it"
        assert dep[i] == dep[p] + 1, f"slot {i}: depth {dep[i]} vs parent depth {dep[p]}"
        assert 0 <= cr[i] < cand_ids.shape[-1]
        assert tok[i] == cand_ids[dep[i] - 1, cr[i]], f"slot {i}: token is not C_d[c]"
        assert g["score"][b, i] <= g["score"][b, p], f"slot {i}: score above its parent's"
        paths.append(paths[p] + (int(cr[i]),))
    assert len(set(paths)) == len(paths), "a prefix appears twice"
    assert (par[n:] == -1).all() and (dep[n:] == -1).all() and (tok[n:] == -1).all() and (cr[n:] == -1).all()
    assert np.isneginf(g["score"][b, n:]).all()
    if with_mask and g.get("mask") is not None:
        for i in range(N):
            bits = _mask_bits(g["mask"][b, i], N)
            if i >= n:
                assert not bits, f"mask row {i} beyond n_nodes is not zero"
                continue
            anc, m = set(), i
            while m >= 0:
                anc.add(m)
                m = int(par[m])
            assert bits == anc, f"mask row {i} is not the ancestor set"
    return paths[1:]


def check_tree(g: dict, ref: dict, logq: np.ndarray, cand_ids: np.ndarray, anchor: np.ndarray, W: int,
               budget: int, zeta: float = 0.0, seqs=None, allow_ties: bool = True) -> dict:
    """Compares GPU trees (all sequences in `g`, or `seqs` of them) with the oracle's
    (`ref`, `logq` and `cand_ids` indexed like `seqs`).  Returns counts of exact and
    excused sequences; raises on a failure."""
    seqs = list(range(g["n_nodes"].shape[0])) if seqs is None else list(seqs)
    counts = dict(exact=0, excused=0)
    for j, b in enumerate(seqs):
        paths = check_structure(g, b, cand_ids[j], int(anchor[j]), budget)
        n = int(g["n_nodes"][b])
        same = (n == int(ref["n_nodes"][j])
                and np.array_equal(g["parent"][b], ref["parent"][j])
                and np.array_equal(g["cand_rank"][b], ref["cand_rank"][j])
                and np.array_equal(g["token"][b], ref["token"][j]))
        if same and g.get("mask") is not None:
            same = np.array_equal(g["mask"][b].view(np.uint32), ref["mask"][j])
        if same:
            close(g["score"][b, :n], ref["score"][j, :n], f"seq {b} scores")
            counts["exact"] += 1
            continue
        if not allow_ties:
            raise AssertionError(f"seq {b}: tree differs from the oracle and ties are not allowed here")
        _guided(g, b, paths, logq[j], W, budget, zeta)
        counts["excused"] += 1
    return counts


def _guided(g: dict, b: int, tree_paths: list, q: np.ndarray, W: int, budget: int, zeta: float) -> None:
    if "f_count" not in g:
        raise AssertionError(f"seq {b}: tree differs and no supertree dump is available to validate it")
    gamma, K = q.shape[0], q.shape[2]
    fr = _paths_from_dump(g, b)
    score = {(): 0.0}
    prev = [()]
    for d in range(1, gamma + 1):
        ext = []
        for p, pp in enumerate(prev):
            row = 0 if d == 1 else pp[-1]
            for c in range(K):
                path = pp + (c,)
                score[path] = score[pp] + float(q[d - 1, row, c]) + zeta
                ext.append(path)
        keep = fr[d - 1]
        assert len(keep) == min(W, len(ext)), f"seq {b} depth {d}: |F_d| = {len(keep)}"
        assert set(keep) <= set(ext), f"seq {b} depth {d}: F_d holds a node outside E_d"
        _validate_cut(ext, set(keep), score, len(keep), f"seq {b} depth {d}")
        for x, y in zip(keep, keep[1:]):
            assert score[x] >= score[y] - EPS * max(1.0, abs(score[y])), f"seq {b} depth {d}: F_d out of order"
        for jj, x in enumerate(keep):
            gs = float(g["f_score"][b, d - 1, jj])
            assert abs(gs - score[x]) <= EPS * max(1.0, abs(score[x])), f"seq {b} depth {d}: F_d score {gs}"
        prev = keep
    sup = [p for f in fr for p in f]
    n_sel = min(budget, len(sup))
    assert len(tree_paths) == n_sel, f"seq {b}: {len(tree_paths)} nodes, expected {n_sel}"
    assert set(tree_paths) <= set(sup)
    _validate_cut(sup, set(tree_paths), score, n_sel, f"seq {b} pruning")
    for x, y in zip(tree_paths, tree_paths[1:]):
        assert score[x] >= score[y] - EPS * max(1.0, abs(score[y])), f"seq {b}: emission out of order"


def _validate_cut(items: list, chosen: set, score: dict, n: int, where: str) -> None:
    """`chosen` (n items) must be a top-n of `items` by fp64 score up to the tie gap."""
    if n >= len(items):
        assert len(chosen) == len(items)
        return
    vals = sorted((score[x] for x in items), reverse=True)
    boundary = vals[n - 1]
    for x in items:
        s = score[x]
        gap = EPS * max(1.0, abs(s), abs(boundary))
        if s > boundary + gap:
            assert x in chosen, f"{where}: dropped {x} with score {s} above the boundary {boundary}"
        if s < boundary - gap:
            assert x not in chosen, f"{where}: kept {x} with score {s} below the boundary {boundary}"


def record(label: str, counts: dict) -> None:
    """Bounds the excused share of one comparison and, when the environment variable
    UBT_PARITY_RECORD names a file, appends the counts to it as a JSON line."""
    trees = counts["exact"] + counts["excused"]
    assert counts["excused"] <= max(1, math.ceil(MAX_EXCUSED_SHARE * trees)), \
        f"{label}: {counts['excused']} of {trees} trees needed the tie excusal"
    path = os.environ.get("UBT_PARITY_RECORD")
    if path:
        with open(path, "a") as fh:
            fh.write(json.dumps({"case": label, **counts, "failed": 0}) + "\n")


def check_best_first(g: dict, ref: dict, edge: np.ndarray, cand_ids: np.ndarray, anchor: np.ndarray, budget: int,
                     zeta: float = 0.0, seqs=None, allow_ties: bool = True) -> dict:
    """Compares GPU trees grown best-first (all sequences in `g`, or `seqs` of them) with
    the oracle's (`ref`, `edge` and `cand_ids` indexed like `seqs`).  Structure is exact:
    parents precede children, depths, tokens and the mask match the parents.  A tree that
    differs from the oracle's is validated step by step: each node the GPU added must be
    a child of the nodes added before it and score within the tie gap of the best such
    child (fp64 path sums).  Returns counts of exact and excused sequences."""
    seqs = list(range(g["n_nodes"].shape[0])) if seqs is None else list(seqs)
    counts = dict(exact=0, excused=0)
    N = budget + 1
    for j, b in enumerate(seqs):
        n = int(g["n_nodes"][b])
        assert n == int(ref["n_nodes"][j]), f"seq {b}: {n} nodes, oracle {int(ref['n_nodes'][j])}"
        par, dep, cr, tok = g["parent"][b], g["depth"][b], g["cand_rank"][b], g["token"][b]
        assert par[0] == -1 and dep[0] == 0 and tok[0] == anchor[j] and cr[0] == -1 and g["score"][b, 0] == 0
        paths = [()]
        for i in range(1, n):
            p = int(par[i])
            assert 0 <= p < i and dep[i] == dep[p] + 1 and 0 <= cr[i] < cand_ids.shape[-1]
            assert tok[i] == cand_ids[j, dep[i] - 1, cr[i]], f"seq {b} slot {i}: token is not C_d[c]"
            paths.append(paths[p] + (int(cr[i]),))
        assert len(set(paths)) == n, f"seq {b}: a prefix appears twice"
        assert (par[n:] == -1).all() and (tok[n:] == -1).all() and np.isneginf(g["score"][b, n:]).all()
        if g.get("mask") is not None:
            for i in range(N):
                bits = _mask_bits(g["mask"][b, i], N)
                anc, m = set(), i
                while i < n and m >= 0:
                    anc.add(m)
                    m = int(par[m])
                assert bits == anc, f"seq {b}: mask row {i} is not the ancestor set"
        same = (np.array_equal(par, ref["parent"][j]) and np.array_equal(cr, ref["cand_rank"][j])
                and np.array_equal(tok, ref["token"][j]))
        if same:
            for i in range(1, n):
                sx, ax = _path_sum(edge[j], paths[i], zeta)
                gs = float(g["score"][b, i])
                assert abs(gs - float(ref["score"][j, i])) <= EPS * max(1.0, ax), \
                    f"seq {b} slot {i}: GPU score {gs} vs {float(ref['score'][j, i])}"
            counts["exact"] += 1
            continue
        if not allow_ties:
            raise AssertionError(f"seq {b}: tree differs from the oracle and ties are not allowed here")
        _guided_best_first(g, b, paths, edge[j], zeta)
        counts["excused"] += 1
    return counts


def _path_sum(e: np.ndarray, path: tuple, zeta: float) -> tuple[float, float]:
    """fp64 path score and the sum of its terms' magnitudes.  Edge scores can have either
    sign, so a path sum may cancel; its fp32 rounding error is bounded relative to the sum
    of magnitudes, which is what the best-first tolerance scales with (for edges <= 0 the
    two coincide, as in the normalised scoring)."""
    s, a, prev = 0.0, 0.0, 0
    for i, c in enumerate(path):
        t = float(e[i, prev, c])
        s += t + zeta
        a += abs(t) + abs(zeta)
        prev = c
    return s, a


def _guided_best_first(g: dict, b: int, paths: list, e: np.ndarray, zeta: float) -> None:
    gamma, K = e.shape[0], e.shape[2]
    taken = {()}
    for t, x in enumerate(paths[1:], start=1):
        front = [p + (c,) for p in taken if len(p) < gamma for c in range(K) if p + (c,) not in taken]
        scored = [_path_sum(e, f, zeta) for f in front]
        bi = max(range(len(front)), key=lambda i: scored[i][0])
        best, best_abs = scored[bi]
        assert x in front, f"seq {b} slot {t}: {x} is not a child of the tree so far"
        sx, ax = _path_sum(e, x, zeta)
        assert sx >= best - EPS * max(1.0, best_abs, ax), f"seq {b} slot {t}: score {sx} below the best child {best}"
        gs = float(g["score"][b, t])
        assert abs(gs - sx) <= EPS * max(1.0, ax), f"seq {b} slot {t}: GPU score {gs} vs {sx}"
        taken.add(x)


def lm_head_tol(abs_sum: np.ndarray, d: int) -> np.ndarray:
    """Bound on the fp32 rounding of a logit formed from exact bf16 products: at most
    d/32 accumulating matrix-core steps, each of which may round up to 32 times, so
    (d/32 + 32) unit roundoffs (2^-24) of the sum of the terms' magnitudes."""
    return (d / 32 + 32) * 2.0 ** -24 * abs_sum


def check_lm_head(g: dict, h_bits: np.ndarray, w_bits: np.ndarray, K: int, exact: bool = False) -> dict:
    """GPU candidates of the LM head (numpy outputs, rows flattened) against the fp64
    oracle.  exact: logits exact in fp32 (integer-valued inputs), so ids and logits must
    match bit for bit, ties included.  Otherwise every reported logit must be its id's
    fp64 logit within lm_head_tol, the order (logit desc, id asc) must hold on the
    reported values, and no excluded id may beat an included one by more than both
    tolerances; rows whose ids differ from the oracle's only that way are 'excused'."""
    from oracle import lm_head as LH

    M, d = h_bits.shape
    u = LH.logits(h_bits, w_bits)
    ref = LH.topk_of_logits(u, K)
    gid = np.asarray(g["cand_ids"]).reshape(M, K).astype(np.int64)
    gval = np.asarray(g["cand_logit"]).reshape(M, K).astype(np.float64)
    glse = np.asarray(g["lse"]).reshape(M).astype(np.float64)
    glp = None if g.get("cand_logprob") is None else np.asarray(g["cand_logprob"]).reshape(M, K).astype(np.float64)
    if exact:
        if not np.array_equal(gid, ref["cand_ids"]):
            r = int(np.argwhere((gid != ref["cand_ids"]).any(-1))[0][0])
            raise AssertionError(f"ids differ in row {r}: gpu={gid[r].tolist()} ref={ref['cand_ids'][r].tolist()}")
        np.testing.assert_array_equal(gval, ref["cand_logit"], "candidate logits")
        close(glse, ref["lse"], "lse")
        if glp is not None:
            close(glp, ref["cand_logprob"], "cand_logprob")
        return {"exact": M, "excused": 0}
    # Sum of |h_k W_vk| for every (row, id): the oracle's logits of the magnitudes.
    tolu = lm_head_tol(LH.logits(h_bits & np.uint16(0x7FFF), w_bits & np.uint16(0x7FFF)), d)
    V = u.shape[1]
    counts = {"exact": 0, "excused": 0}
    for m in range(M):
        ids = gid[m]
        assert ((ids >= 0) & (ids < V)).all() and len(set(ids.tolist())) == K, f"row {m}: invalid ids {ids.tolist()}"
        uv, tv = u[m, ids], tolu[m, ids]
        err = np.abs(gval[m] - uv)
        assert (err <= tv).all(), f"row {m}: logit of id {ids[np.argmax(err - tv)]} off by {err.max()} (tol {tv.max()})"
        dv = np.diff(gval[m])
        assert (dv <= 0).all(), f"row {m}: reported logits not descending"
        assert ((dv < 0) | (np.diff(ids) > 0)).all(), f"row {m}: equal logits not in id order"
        out = np.ones(V, bool)
        out[ids] = False
        if out.any():
            worst_out = np.max(u[m, out] - tolu[m, out])
            assert worst_out <= np.min(uv + tv), f"row {m}: an excluded id beats the selection beyond the tolerance"
        lse_tol = tolu[m].max() + EPS * max(1.0, abs(ref["lse"][m]))
        assert abs(glse[m] - ref["lse"][m]) <= lse_tol, f"row {m}: lse {glse[m]} vs {ref['lse'][m]}"
        if glp is not None:
            lp_err = np.abs(glp[m] - (uv - ref["lse"][m]))
            assert (lp_err <= tv + lse_tol).all(), f"row {m}: cand_logprob off by {lp_err.max()}"
        counts["exact" if np.array_equal(ids, ref["cand_ids"][m]) else "excused"] += 1
    return counts
