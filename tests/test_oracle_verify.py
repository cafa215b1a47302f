"""Pins of the verification oracle (``oracle/verify.py``) against what the definition
fixes independently of it: brute-force attention over each node's explicit root path
(walked from parent pointers, not read from the mask), causal attention for a chain
tree (a library routine), invariances, and brute-force enumeration of every root path
for the acceptance walk.  Planted mistakes in copies of the oracle must fail a pin."""
from __future__ import annotations

import math
import os

import numpy as np
import pytest

import oracle
from oracle import verify as V


def _random_tree(rng, N: int, branch: int = 3):
    """Topological tree (parent[n] < n) whose children of one parent carry distinct tokens."""
    parent = np.full(N, -1, np.int32)
    token = np.zeros(N, np.int32)
    token[0] = rng.integers(0, 50)
    for n in range(1, N):
        lo = max(0, n - branch * 2)
        parent[n] = rng.integers(lo, n)
        used = {int(token[c]) for c in range(1, n) if parent[c] == parent[n]}
        t = int(rng.integers(0, 50))
        while t in used:
            t = int(rng.integers(0, 50))
        token[n] = t
    return parent, token


def _mask_by_walking(parent: np.ndarray, nn: int, N: int) -> np.ndarray:
    words = (N + 31) // 32
    m = np.zeros((N, words), np.uint32)
    for n in range(nn):
        a = n
        while a >= 0:
            m[n, a // 32] |= np.uint32(1 << (a % 32))
            a = int(parent[a])
    return m


def _inputs(seed: int, B=2, N=9, H=4, Hkv=2, D=8, Pmax=6, plen=(5, 0), nn=(9, 6)):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=(B, N, H, D))
    kc = rng.normal(size=(B, Pmax, Hkv, D))
    vc = rng.normal(size=(B, Pmax, Hkv, D))
    kt = rng.normal(size=(B, N, Hkv, D))
    vt = rng.normal(size=(B, N, Hkv, D))
    parents = np.full((B, N), -1, np.int32)
    mask = np.zeros((B, N, (N + 31) // 32), np.uint32)
    for b in range(B):
        parents[b], _ = _random_tree(rng, N)
        mask[b] = _mask_by_walking(parents[b], nn[b], N)
    return dict(q=q, k_cache=kc, v_cache=vc, prefix_len=np.array(plen, np.int32), k_tree=kt, v_tree=vt,
                mask=mask, n_nodes=np.array(nn, np.int32)), parents


def _brute_attention(d: dict, parents: np.ndarray, scale: float):
    """Per node: the explicit sequence prefix + (root .. node) from parent pointers, then
    a single-query softmax attention with scalar loops."""
    q, kc, vc, kt, vt = d["q"], d["k_cache"], d["v_cache"], d["k_tree"], d["v_tree"]
    B, N, H, D = q.shape
    g = H // kc.shape[2]
    out = np.zeros((B, N, H, D))
    lse = np.full((B, N, H), -np.inf)
    for b in range(B):
        for n in range(int(d["n_nodes"][b])):
            path, a = [], n
            while a >= 0:
                path.append(a)
                a = int(parents[b, a])
            path.reverse()
            for h in range(H):
                kv = h // g
                seq = [(kc[b, p, kv], vc[b, p, kv]) for p in range(int(d["prefix_len"][b]))]
                seq += [(kt[b, m, kv], vt[b, m, kv]) for m in path]
                scores = [scale * sum(float(q[b, n, h, i]) * float(k[i]) for i in range(D)) for k, _ in seq]
                top = max(scores)
                w = [math.exp(s - top) for s in scores]
                tot = sum(w)
                for i in range(D):
                    out[b, n, h, i] = sum(wj * float(v[i]) for wj, (_, v) in zip(w, seq)) / tot
                lse[b, n, h] = top + math.log(tot)
    return out, lse


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_attention_matches_explicit_paths(seed):
    d, parents = _inputs(seed)
    out, lse = V.tree_attention(**d, scale=0.3)
    ref, ref_lse = _brute_attention(d, parents, 0.3)
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-12)
    assert np.array_equal(np.isinf(lse), np.isinf(ref_lse))
    fin = np.isfinite(ref_lse)
    assert np.allclose(lse[fin], ref_lse[fin], rtol=1e-12, atol=1e-12)
    # rows past n_nodes are zero
    assert not out[1, 6:].any()


@pytest.mark.parametrize("seed", [3, 4])
def test_fast_form_equals_plain_form(seed):
    d, _ = _inputs(seed, B=3, N=40, H=6, Hkv=3, D=16, Pmax=20, plen=(20, 0, 7), nn=(40, 33, 1))
    a, la = V.tree_attention(**d, scale=0.25)
    b, lb = V.tree_attention_fast(**d, scale=0.25)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)
    assert np.array_equal(np.isinf(la), np.isinf(lb))
    fin = np.isfinite(la)
    assert np.allclose(la[fin], lb[fin], rtol=1e-12, atol=1e-12)


def test_chain_tree_is_causal_attention():
    """A chain (parent[n] = n - 1) is an ordinary sequence: node n's output is row P + n of
    causal attention over prefix + chain (torch's scaled_dot_product_attention)."""
    import torch

    rng = np.random.default_rng(5)
    B, N, H, Hkv, D, P = 1, 12, 4, 4, 16, 7
    d, _ = _inputs(5, B=B, N=N, H=H, Hkv=Hkv, D=D, Pmax=P, plen=(P,), nn=(N,))
    parent = np.arange(-1, N - 1, dtype=np.int32)
    d["mask"] = _mask_by_walking(parent, N, N)[None]
    out, _ = V.tree_attention(**d, scale=1 / math.sqrt(D))
    k = np.concatenate([d["k_cache"][0], d["k_tree"][0]], axis=0)  # [P + N, Hkv, D]
    v = np.concatenate([d["v_cache"][0], d["v_tree"][0]], axis=0)
    qf = np.concatenate([rng.normal(size=(P, H, D)), d["q"][0]], axis=0)  # queries for every position
    T = torch.from_numpy
    ref = torch.nn.functional.scaled_dot_product_attention(T(qf).transpose(0, 1), T(k).transpose(0, 1),
                                                           T(v).transpose(0, 1), is_causal=True)
    ref = ref.transpose(0, 1).numpy()[P:]
    assert np.allclose(out[0], ref, rtol=1e-10, atol=1e-10)


def test_non_ancestors_do_not_matter():
    d, parents = _inputs(6, B=1, N=20, plen=(4,), nn=(20,), Pmax=4)
    out, _ = V.tree_attention(**d, scale=0.5)
    n = 19
    anc, a = set(), n
    while a >= 0:
        anc.add(a)
        a = int(parents[0, a])
    d2 = {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in d.items()}
    others = [m for m in range(20) if m not in anc]
    d2["k_tree"][0, others] += 5.0
    d2["v_tree"][0, others] -= 3.0
    out2, _ = V.tree_attention(**d2, scale=0.5)
    assert np.array_equal(out[0, n], out2[0, n])
    d2["v_cache"][0, 0] += 1.0
    out3, _ = V.tree_attention(**d2, scale=0.5)
    assert not np.allclose(out3[0, n], out[0, n])


def test_zero_query_averages_visible_values():
    d, parents = _inputs(7, B=1, N=10, plen=(3,), nn=(10,), Pmax=3)
    d["q"][:] = 0.0
    out, lse = V.tree_attention(**d, scale=1.0)
    for n in range(10):
        path, a = [], n
        while a >= 0:
            path.append(a)
            a = int(parents[0, a])
        for h in range(d["q"].shape[2]):
            kv = h // 2
            vals = np.concatenate([d["v_cache"][0, :3, kv], d["v_tree"][0, path, kv]])
            assert np.allclose(out[0, n, h], vals.mean(axis=0), rtol=1e-13, atol=1e-13)
            assert math.isclose(lse[0, n, h], math.log(len(vals)), rel_tol=1e-13)


def test_bf16_inputs_are_decoded_exactly():
    d, _ = _inputs(8, B=1, N=5, plen=(2,), nn=(5,), Pmax=2)
    bits = {k: (np.asarray(d[k], np.float32).view(np.uint32) >> 16).astype(np.uint16)
            for k in ("q", "k_cache", "v_cache", "k_tree", "v_tree")}
    vals = {k: (bits[k].astype(np.uint32) << 16).view(np.float32).astype(np.float64) for k in bits}
    a, _ = V.tree_attention(**{**d, **bits}, scale=0.5)
    b, _ = V.tree_attention(**{**d, **vals}, scale=0.5)
    assert np.array_equal(a, b)


def test_mask_from_the_tree_oracle_is_the_walked_mask():
    """The packed masks the draft-tree oracle emits are the ancestor sets used above."""
    rng = np.random.default_rng(9)
    B, N = 3, 40
    parent = np.full((B, N), -1, np.int32)
    for b in range(B):
        parent[b], _ = _random_tree(rng, N)
    nn = np.array([40, 17, 1], np.int32)
    m = oracle.tree_mask(parent, nn)
    for b in range(B):
        assert np.array_equal(m[b], _mask_by_walking(parent[b], int(nn[b]), N))


# ---- acceptance walk --------------------------------------------------------------------
def _brute_accept(token, parent, nn, target):
    """Every root path, checked edge by edge; the deepest valid one is accepted (unique:
    siblings carry distinct tokens), its last node's sample is the bonus."""
    best = [0]
    for n in range(1, nn):
        path, a = [], n
        while a >= 0:
            path.append(a)
            a = int(parent[a])
        path.reverse()
        if all(token[c] == target[p] for p, c in zip(path, path[1:])) and len(path) > len(best):
            best = path
    return len(best) - 1, best, int(target[best[-1]])


@pytest.mark.parametrize("seed", range(6))
def test_accept_matches_path_enumeration(seed):
    rng = np.random.default_rng(100 + seed)
    B, N = 4, 33
    token = np.zeros((B, N), np.int32)
    parent = np.full((B, N), -1, np.int32)
    target = rng.integers(0, 50, size=(B, N)).astype(np.int32)
    nn = np.array([33, 20, 1, 33], np.int32)
    for b in range(B):
        parent[b], token[b] = _random_tree(rng, N)
        # steer the target along a random root path for part of its length
        a = int(rng.integers(0, nn[b]))
        path = []
        while a >= 0:
            path.append(a)
            a = int(parent[b, a])
        path.reverse()
        stop = int(rng.integers(0, len(path)))
        for p, c in zip(path[:stop], path[1:stop + 1]):
            target[b, p] = token[b, c]
    alen, nodes, bonus = V.verify_accept(token, parent, nn, target)
    for b in range(B):
        L, path, y = _brute_accept(token[b], parent[b], int(nn[b]), target[b])
        assert alen[b] == L and bonus[b] == y
        assert list(nodes[b, :L + 1]) == path and (nodes[b, L + 1:] == -1).all()


def test_accept_edge_cases():
    # chain that matches to the end: every node accepted, bonus = the leaf's sample
    N = 6
    parent = np.arange(-1, N - 1, dtype=np.int32)[None]
    token = np.arange(10, 10 + N, dtype=np.int32)[None]
    target = np.concatenate([token[0, 1:], [99]]).astype(np.int32)[None]
    alen, nodes, bonus = V.verify_accept(token, parent, np.array([N]), target)
    assert alen[0] == N - 1 and bonus[0] == 99 and list(nodes[0]) == list(range(N))
    # mismatch at the root
    target2 = target.copy()
    target2[0, 0] = 7
    alen, nodes, bonus = V.verify_accept(token, parent, np.array([N]), target2)
    assert alen[0] == 0 and bonus[0] == 7 and nodes[0, 0] == 0 and (nodes[0, 1:] == -1).all()


def test_commit_kv():
    rng = np.random.default_rng(11)
    B, N, Hkv, D, Pmax = 2, 8, 2, 4, 10
    kt, vt = rng.normal(size=(B, N, Hkv, D)), rng.normal(size=(B, N, Hkv, D))
    kc, vc = np.zeros((B, Pmax, Hkv, D)), np.zeros((B, Pmax, Hkv, D))
    nodes = np.array([[0, 2, 5, -1, -1, -1, -1, -1], [0, 1, 3, 4, 6, 7, -1, -1]], np.int32)
    alen = np.array([2, 5], np.int32)
    plen = np.array([3, 7], np.int32)
    k2, v2, p2 = V.commit_kv(kt, vt, nodes, alen, plen, kc, vc)
    assert list(p2) == [6, 10]
    assert np.array_equal(k2[0, 3:6], kt[0, [0, 2, 5]]) and np.array_equal(v2[0, 3:6], vt[0, [0, 2, 5]])
    assert np.array_equal(k2[1, 7:10], kt[1, [0, 1, 3]])  # the rest fell past the cache
    assert not k2[0, 6:].any() and not k2[0, :3].any()


# ---- planted mistakes ------------------------------------------------------------------
MUTANTS = {
    "gqa head mapping": ("kv = h // g\n                keys", "kv = h % Hkv\n                keys"),
    "self not attended": ("if mask_bit(mask, b, n, m)]", "if mask_bit(mask, b, n, m) and m != n]"),
    "lse without its shift": ("lse[b, n, h] = mx + np.log(tot)", "lse[b, n, h] = np.log(tot)"),
    "prefix one short": ("P = int(prefix_len[b])\n        nn = int(n_nodes[b])\n        for n in range(nn):",
                         "P = max(int(prefix_len[b]) - 1, 0)\n        nn = int(n_nodes[b])\n        for n in range(nn):"),
    "sample read at the child": ("token[b, c] == y), None)", "token[b, c] == int(target[b, c])), None)"),
    "bonus from the parent": ("bonus[b] = y\n", "bonus[b] = int(target[b, max(int(parent[b, cur]), 0)])\n"),
    "commit one row short": ("cnt = int(accept_len[b]) + 1", "cnt = int(accept_len[b])"),
}


def _mutant(name: str):
    src = open(os.path.join(os.path.dirname(V.__file__), "verify.py")).read()
    a, b = MUTANTS[name]
    assert src.count(a) == 1, name
    ns: dict = {}
    exec(compile(src.replace(a, b), f"mutant:{name}", "exec"), ns)
    return ns


def _pins_pass(ns) -> bool:
    saved = {k: getattr(V, k) for k in ("tree_attention", "verify_accept", "commit_kv")}
    try:
        for k in saved:
            setattr(V, k, ns[k])
        tests = [lambda: test_attention_matches_explicit_paths(0), lambda: test_accept_matches_path_enumeration(0),
                 test_accept_edge_cases, test_commit_kv, test_zero_query_averages_visible_values]
        for t in tests:
            t()
        return True
    except AssertionError:
        return False
    finally:
        for k, f in saved.items():
            setattr(V, k, f)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    assert not _pins_pass(_mutant(name)), f"planted mistake '{name}' passed every pin"
