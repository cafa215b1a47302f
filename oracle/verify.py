"""TEST INFRASTRUCTURE: fp64 CPU oracle of the verification step that consumes a draft
tree (Appendix A / Verification via Tree-attention; Background, "Tree Drafting").

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may
import this module; the product path never does, and the two share no code.

Three functions, each the plain definition written out in numpy float64:

* ``tree_attention`` -- every tree node attends to the committed prefix and to the tree
  nodes its ancestor-mask row allows (its ancestors and itself), i.e. it is evaluated
  under its own autoregressive prefix.  Scaled dot-product softmax attention, grouped
  query heads (head h reads key/value head h // (H / H_kv)).
* ``verify_accept`` -- from the root, follow the child whose token equals the target
  model's sample at the current node, until no child matches; that sample is the bonus
  token.
* ``commit_kv`` -- the key/value rows of the root and of the accepted nodes are appended
  to the cache, in path order; those of every other branch are dropped.

bf16 arrays are given as their uint16 bit patterns and decoded exactly here.
"""
from __future__ import annotations

import numpy as np


def _widen(a: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) or float arrays -> float64, exactly."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def mask_bit(mask: np.ndarray, b: int, n: int, m: int) -> bool:
    """Bit m of row n of sequence b of a packed mask [B, N, words] (LSB-first words)."""
    return bool((int(mask[b, n, m // 32]) >> (m % 32)) & 1)


def tree_attention(q, k_cache, v_cache, prefix_len, k_tree, v_tree, mask, n_nodes, scale: float):
    """out [B, N, H, D] float64 and lse [B, N, H] (natural log).

    q [B, N, H, D]; k_cache, v_cache [B, P_max, H_kv, D]; prefix_len [B]; k_tree, v_tree
    [B, N, H_kv, D]; mask [B, N, ceil(N/32)] uint32; n_nodes [B].  Node n < n_nodes[b]
    attends to cache positions 0..prefix_len[b]-1 and to tree nodes m < n_nodes[b] whose
    bit m is set in its mask row.  Rows n >= n_nodes[b] are 0 with lse = -inf."""
    q, kc, vc, kt, vt = (_widen(x) for x in (q, k_cache, v_cache, k_tree, v_tree))
    B, N, H, D = q.shape
    Hkv = kc.shape[2]
    g = H // Hkv
    out = np.zeros((B, N, H, D))
    lse = np.full((B, N, H), -np.inf)
    for b in range(B):
        P = int(prefix_len[b])
        nn = int(n_nodes[b])
        for n in range(nn):
            allowed = [m for m in range(nn) if mask_bit(mask, b, n, m)]
            for h in range(H):
                kv = h // g
                keys = np.concatenate([kc[b, :P, kv], kt[b, allowed, kv]], axis=0)
                vals = np.concatenate([vc[b, :P, kv], vt[b, allowed, kv]], axis=0)
                if keys.shape[0] == 0:
                    continue
                s = scale * (keys @ q[b, n, h])
                mx = s.max()
                e = np.exp(s - mx)
                tot = e.sum()
                out[b, n, h] = (e @ vals) / tot
                lse[b, n, h] = mx + np.log(tot)
    return out, lse


def tree_attention_fast(q, k_cache, v_cache, prefix_len, k_tree, v_tree, mask, n_nodes, scale: float,
                        seqs=None):
    """The same definition evaluated per (sequence, key/value head) with dense matrix
    products and a boolean visibility matrix, for sizes where the per-node loops of
    ``tree_attention`` are too slow.  ``seqs`` restricts the work to some sequences
    (the other rows are left at 0 / -inf)."""
    q, kc, vc, kt, vt = (_widen(x) for x in (q, k_cache, v_cache, k_tree, v_tree))
    B, N, H, D = q.shape
    Hkv = kc.shape[2]
    g = H // Hkv
    out = np.zeros((B, N, H, D))
    lse = np.full((B, N, H), -np.inf)
    bits = np.unpackbits(np.ascontiguousarray(mask).view(np.uint8), axis=-1, bitorder="little")[..., :N]
    for b in (range(B) if seqs is None else seqs):
        P = int(prefix_len[b])
        nn = int(n_nodes[b])
        if nn == 0:
            continue
        vis = np.concatenate([np.ones((nn, P), bool), bits[b, :nn, :nn].astype(bool)], axis=1)  # [nn, P + nn]
        for kv in range(Hkv):
            keys = np.concatenate([kc[b, :P, kv], kt[b, :nn, kv]], axis=0)
            vals = np.concatenate([vc[b, :P, kv], vt[b, :nn, kv]], axis=0)
            qs = q[b, :nn, kv * g:(kv + 1) * g]  # [nn, g, D]
            s = scale * np.einsum("ngd,kd->ngk", qs, keys)
            s = np.where(vis[:, None, :], s, -np.inf)
            mx = s.max(axis=-1, keepdims=True)
            e = np.exp(s - mx)
            tot = e.sum(axis=-1, keepdims=True)
            out[b, :nn, kv * g:(kv + 1) * g] = np.einsum("ngk,kd->ngd", e, vals) / tot
            lse[b, :nn, kv * g:(kv + 1) * g] = (mx + np.log(tot))[..., 0]
    return out, lse


def verify_accept(token, parent, n_nodes, target):
    """accept_len [B], accept_nodes [B, N] (root first, then the accepted nodes, -1
    after), bonus [B].  target[b, n] is the target model's sample at node n (the token
    it predicts after node n's prefix).  Among several matching children the lowest
    node index is taken."""
    B, N = token.shape
    alen = np.zeros(B, np.int32)
    nodes = np.full((B, N), -1, np.int32)
    bonus = np.zeros(B, np.int32)
    for b in range(B):
        nn = max(1, min(int(n_nodes[b]), N))
        cur, path = 0, [0]
        while True:
            y = int(target[b, cur])
            nxt = next((c for c in range(cur + 1, nn) if parent[b, c] == cur and token[b, c] == y), None)
            if nxt is None:
                bonus[b] = y
                break
            path.append(nxt)
            cur = nxt
        alen[b] = len(path) - 1
        nodes[b, :len(path)] = path
    return alen, nodes, bonus


def commit_kv(k_tree, v_tree, accept_nodes, accept_len, prefix_len, k_cache, v_cache):
    """New (k_cache, v_cache, prefix_len): rows of nodes accept_nodes[b, 0..accept_len[b]]
    copied to positions prefix_len[b], prefix_len[b] + 1, ...; positions at or past the
    cache length are dropped and prefix_len stops there."""
    kc, vc = k_cache.copy(), v_cache.copy()
    plen = np.asarray(prefix_len, np.int32).copy()
    Pmax = kc.shape[1]
    for b in range(kc.shape[0]):
        P = int(plen[b])
        cnt = int(accept_len[b]) + 1
        for i in range(cnt):
            if P + i < Pmax:
                kc[b, P + i] = k_tree[b, accept_nodes[b, i]]
                vc[b, P + i] = v_tree[b, accept_nodes[b, i]]
        plen[b] = min(Pmax, P + cnt)
    return kc, vc, plen
