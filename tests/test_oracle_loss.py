"""Pins of the renormalised-KL oracle (``oracle/loss.py``): finite differences of the loss
against its gradients, scipy's relative entropy and log-softmax, the T -> 0 limit,
invariances, and planted mistakes in copies of the oracle."""
from __future__ import annotations

import os

import numpy as np
import pytest
import scipy.special as sp

from oracle import loss as Lo


def _case(seed: int, B=2, G=4, V=50, K=6, r=8, T=0.7, beta=0.1):
    rng = np.random.default_rng(seed)
    u = rng.normal(0, 2.0, size=(B, G, V))
    z = u + rng.normal(0, 1.0, size=(B, G, V))
    cand = np.stack([np.stack([rng.choice(V, K, replace=False) for _ in range(G)]) for _ in range(B)]).astype(np.int32)
    y = rng.integers(0, V, size=(B, G)).astype(np.int32)
    y[0, 1] = cand[0, 1, 2]  # a ground truth inside the support
    anchor = rng.integers(0, V, size=B).astype(np.int32)
    phi, psi = rng.normal(0, 0.5, size=(V, r)), rng.normal(0, 0.5, size=(V, r))
    gate = rng.normal(0, 1.0, size=(B, G, r))
    alpha, lam = rng.uniform(0.5, 2.0, G), rng.uniform(0.5, 2.0, G)
    return dict(logits=u, cand_ids=cand, target_logits=z, y_star=y, anchor=anchor, phi=phi, psi=psi, gate=gate,
                alpha=alpha, lam=lam, T=T, beta=beta)


@pytest.mark.parametrize("seed", [0, 1])
def test_gradient_of_logits_by_finite_differences(seed):
    c = _case(seed)
    g = Lo.tree_kl_loss(**c)["grad_logits"]
    h = 1e-6
    for b, i in [(0, 0), (0, 1), (1, 3)]:
        vs = sorted(set(c["cand_ids"][b, i][:3].tolist()) | {int(c["y_star"][b, i]), 7, 31})
        for v in vs:
            up, dn = {k: (x.copy() if isinstance(x, np.ndarray) else x) for k, x in c.items()}, None
            dn = {k: (x.copy() if isinstance(x, np.ndarray) else x) for k, x in c.items()}
            up["logits"][b, i, v] += h
            dn["logits"][b, i, v] -= h
            fd = (Lo.tree_kl_loss(**up, rows=[(b, i)], with_grad=False)["loss"][b, i] -
                  Lo.tree_kl_loss(**dn, rows=[(b, i)], with_grad=False)["loss"][b, i]) / (2 * h)
            assert abs(fd - g[b, i, v]) <= 1e-7, (b, i, v, fd, g[b, i, v])


@pytest.mark.parametrize("which", ["alpha", "lam"])
def test_gradient_of_scores_through_the_calibration(which):
    """d loss / d alpha_i = sum grad_s * u(C_i);  d loss / d lambda_i = sum grad_s * delta."""
    c = _case(2)
    r = Lo.tree_kl_loss(**c)
    h = 1e-6
    for b, i in [(0, 0), (1, 2)]:
        up = dict(c, **{which: c[which].copy()})
        dn = dict(c, **{which: c[which].copy()})
        up[which][i] += h
        dn[which][i] -= h
        fd = (Lo.tree_kl_loss(**up, rows=[(b, i)], with_grad=False)["loss"][b, i] -
              Lo.tree_kl_loss(**dn, rows=[(b, i)], with_grad=False)["loss"][b, i]) / (2 * h)
        C = c["cand_ids"][b, i]
        if which == "alpha":
            inner = c["logits"][b, i, C]
        else:
            a = c["anchor"][b] if i == 0 else c["y_star"][b, i - 1]
            inner = c["psi"][C] @ (c["gate"][b, i] * c["phi"][a])
        assert abs(fd - float(r["grad_s"][b, i] @ inner)) <= 1e-7


def test_terms_match_scipy():
    c = _case(3)
    r = Lo.tree_kl_loss(**c)
    for b in range(2):
        for i in range(4):
            C = c["cand_ids"][b, i]
            a = c["anchor"][b] if i == 0 else c["y_star"][b, i - 1]
            s = c["alpha"][i] * c["logits"][b, i, C] + c["lam"][i] * (c["psi"][C] @ (c["gate"][b, i] * c["phi"][a]))
            p = sp.softmax(c["target_logits"][b, i, C] / c["T"])
            q = sp.softmax(s)
            assert np.isclose(r["kl"][b, i], sp.rel_entr(p, q).sum(), rtol=1e-12, atol=1e-14)
            ce = -sp.log_softmax(c["logits"][b, i])[c["y_star"][b, i]]
            assert np.isclose(r["ce"][b, i], ce, rtol=1e-12)
            assert np.isclose(r["loss"][b, i], r["kl"][b, i] + c["beta"] * ce, rtol=1e-12)
            assert np.allclose(r["grad_s"][b, i], q - p, atol=1e-14)
    assert np.allclose(r["grad_logits"].sum(axis=-1), 0.0, atol=1e-12)  # softmax - onehot and q~ - p~ sum to 0


def test_zero_temperature_limit():
    c = _case(4, T=0.0)
    r0 = Lo.tree_kl_loss(**c)
    c2 = dict(c, T=1e-4)
    r1 = Lo.tree_kl_loss(**c2)
    assert np.allclose(r0["grad_s"], r1["grad_s"], atol=1e-9)
    assert np.allclose(r0["kl"], r1["kl"], atol=1e-6)
    # ties at the maximum: the limit is uniform over the tied candidates
    p = Lo.target_probs(np.array([1.0, 3.0, 3.0, -2.0]), 0.0)
    assert np.array_equal(p, [0.0, 0.5, 0.5, 0.0])
    assert np.allclose(Lo.target_probs(np.array([1.0, 3.0, 3.0, -2.0]), 1e-3), p)


def test_invariances_and_invalid_positions():
    c = _case(5)
    r = Lo.tree_kl_loss(**c)
    shifted = dict(c, target_logits=c["target_logits"] + 3.0, logits=c["logits"])
    r2 = Lo.tree_kl_loss(**shifted)
    assert np.allclose(r["kl"], r2["kl"], atol=1e-12)
    c3 = dict(c, y_star=c["y_star"].copy())
    c3["y_star"][1, 2] = -1
    r3 = Lo.tree_kl_loss(**c3)
    assert r3["loss"][1, 2] == 0 and not r3["grad_logits"][1, 2].any() and not r3["grad_s"][1, 2].any()
    # the next position's predecessor is now invalid: its selector drops delta
    C = c["cand_ids"][1, 3]
    q = sp.softmax(c["alpha"][3] * c["logits"][1, 3, C])
    assert np.allclose(r3["grad_s"][1, 3], q - sp.softmax(c["target_logits"][1, 3, C] / c["T"]), atol=1e-14)


MUTANTS = {
    "predecessor = own token": ("else int(y_star[b, i - 1])", "else int(y_star[b, i])"),
    "temperature ignored": ("    x = zc / T\n", "    x = zc\n"),
    "reverse KL": ("kl = float((pt[nz] * (np.log(pt[nz]) - logq[nz])).sum())",
                   "kl = float((qt * (logq - np.log(np.maximum(pt, 1e-300)))).sum())"),
    "gate dropped": ("feat = gt[b, i] * ph[a]", "feat = ph[a]"),
    "gradient sign": ("out[\"grad_s\"][b, i] = qt - pt", "out[\"grad_s\"][b, i] = pt - qt"),
    "alpha missing in the logit gradient": ("np.add.at(g, C, alpha[i] * (qt - pt))", "np.add.at(g, C, qt - pt)"),
    "CE on the wrong token": ("ce = lse - u[b, i, y]", "ce = lse - u[b, i, C[0]]"),
}


def _mutant(name):
    src = open(os.path.join(os.path.dirname(Lo.__file__), "loss.py")).read()
    a, b = MUTANTS[name]
    assert src.count(a) == 1, name
    ns: dict = {}
    exec(compile(src.replace(a, b), f"mutant:{name}", "exec"), ns)
    return ns


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    ns = _mutant(name)
    saved = (Lo.tree_kl_loss, Lo.target_probs)
    Lo.tree_kl_loss, Lo.target_probs = ns["tree_kl_loss"], ns["target_probs"]
    try:
        tests = [lambda: test_gradient_of_logits_by_finite_differences(0),
                 lambda: test_gradient_of_scores_through_the_calibration("lam"), test_terms_match_scipy,
                 test_zero_temperature_limit, test_invariances_and_invalid_positions]
        failed = False
        for t in tests:
            try:
                t()
            except (AssertionError, ValueError, FloatingPointError):
                failed = True
                break
        assert failed, f"planted mistake '{name}' passed every pin"
    finally:
        Lo.tree_kl_loss, Lo.target_probs = saved
