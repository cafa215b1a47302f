"""TEST INFRASTRUCTURE: fp64 CPU oracle of UBTree's renormalised-KL training objective
(Method / Tree-native Training, Eqs. (ubtree-training-distributions) and
(ubtree-training-loss)), its value and its gradients.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may
import this module; the product path never does, and the two share no code.

For sequence b and draft position i (row i = 0..gamma-1, depth i + 1) with ground-truth
token y = y_star[b, i] (negative: the position is not valid, loss and gradients 0) and
predecessor a = the anchor (i = 0) or y_star[b, i - 1]:

* C_i = cand_ids[b, i] (the proposer's top-K support); y outside [0, V) marks the
  position invalid, and a predecessor outside [0, V) gives delta = 0;
* selector logits s(b') = alpha_i u_i(b') + lambda_i delta_i(a, b') for b' in C_i, with
  delta_i(a, b') = (P(h_i) * phi(a)) . psi(b')  (Eqs. (dflash2-selector), (ubtree-depth));
* p~(b') = softmax over C_i of z_i(b') / T (T = 0: uniform over the maximisers of z_i
  on C_i, the limit T -> 0+), q~(b') = softmax over C_i of s(b');
* KL = sum_b' p~ (log p~ - log q~) (0 log 0 = 0); CE = -log q_i(y) = LSE_V(u_i) - u_i(y);
  loss = KL + beta * CE.
* d loss / d s(b') = q~(b') - p~(b');
  d loss / d u_i(v) = beta (softmax(u_i)(v) - [v = y]) + alpha_i [v in C_i] (q~ - p~)(v).

bf16 arrays are uint16 bit patterns, decoded exactly here.
"""
from __future__ import annotations

import numpy as np


def _widen(a: np.ndarray) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def _logsumexp(x: np.ndarray) -> float:
    m = x.max()
    return float(m + np.log(np.exp(x - m).sum()))


def target_probs(zc: np.ndarray, T: float) -> np.ndarray:
    """p~ on the K candidates from their target logits."""
    if T == 0.0:
        hit = zc == zc.max()
        return hit / hit.sum()
    x = zc / T
    return np.exp(x - _logsumexp(x))


def tree_kl_loss(logits, cand_ids, target_logits, y_star, anchor, phi, psi, gate, alpha, lam, T: float,
                 beta: float, rows=None, with_grad: bool = True):
    """Returns dict(loss, kl, ce [B, gamma], grad_s [B, gamma, K], grad_logits [B, gamma, V]
    (None unless with_grad)).  ``rows`` = list of (b, i) to evaluate (others stay 0)."""
    u = _widen(logits)
    z = _widen(target_logits)
    ph, ps, gt = _widen(phi), _widen(psi), _widen(gate)
    B, G, V = u.shape
    K = cand_ids.shape[2]
    out = dict(loss=np.zeros((B, G)), kl=np.zeros((B, G)), ce=np.zeros((B, G)), grad_s=np.zeros((B, G, K)),
               grad_logits=np.zeros((B, G, V)) if with_grad else None)
    todo = [(b, i) for b in range(B) for i in range(G)] if rows is None else rows
    for b, i in todo:
        y = int(y_star[b, i])
        if not 0 <= y < V:
            continue
        a = int(anchor[b]) if i == 0 else int(y_star[b, i - 1])
        C = cand_ids[b, i].astype(np.int64)
        feat = gt[b, i] * ph[a] if 0 <= a < V else np.zeros_like(gt[b, i])
        delta = ps[C] @ feat
        s = alpha[i] * u[b, i, C] + lam[i] * delta
        logq = s - _logsumexp(s)
        qt = np.exp(logq)
        pt = target_probs(z[b, i, C], T)
        nz = pt > 0
        kl = float((pt[nz] * (np.log(pt[nz]) - logq[nz])).sum())
        lse = _logsumexp(u[b, i])
        ce = lse - u[b, i, y]
        out["kl"][b, i] = kl
        out["ce"][b, i] = ce
        out["loss"][b, i] = kl + beta * ce
        out["grad_s"][b, i] = qt - pt
        if with_grad:
            g = beta * np.exp(u[b, i] - lse)
            g[y] -= beta
            np.add.at(g, C, alpha[i] * (qt - pt))
            out["grad_logits"][b, i] = g
    return out
