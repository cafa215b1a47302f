"""GPU parity of ubt_tree_kl_loss (the renormalised-KL objective and its gradients)
against the fp64 oracle in ``oracle/loss.py``, through the C ABI.

The GPU takes its candidates and LSE from ubt_topk; the oracle takes its own (the two
candidate sets are first checked to be identical, so the oracle never reads a GPU
output).  Tolerances, from the arithmetic: the loss terms are fp32 sums of at most K
exponentials and one LSE of the vocabulary (relative error ~1e-6), so loss, KL and CE
must agree within 1e-5 * max(1, |ref|); d loss / d s within 1e-5; the logit gradient
within 1e-5 |ref| + 1e-6 (its dense part is one fp32 exp per element)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import synth
from oracle import loss as Lo

pytestmark = pytest.mark.gpu


def _run(w: synth.Workload, d: dict, li: dict, T: float, beta: float, with_grad: bool = True):
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, dev_values

    logits = dev_values(d["logits"])
    cand = ubt.topk(logits, w.K)
    out = ubt.tree_kl_loss(logits, cand, dev_values(li["target_logits"]), dev_i32(li["y_star"]), dev_i32(d["anchor"]),
                           dev_values(d["phi"]), dev_values(d["psi"]), dev_values(d["gate"]), d["alpha"], d["lam"],
                           T_train=T, beta=beta, with_grad=with_grad)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy().astype(np.float64) for k, v in out.items() if v is not None}
    res["cand_ids"] = cand["cand_ids"].cpu().numpy()
    return res


def _check(w: synth.Workload, d: dict, li: dict, T: float, beta: float, grad_rows=None):
    from gpu_util import say

    say(f"tree_kl_loss workload {w.cfg} ({w.describe()}) T={T} beta={beta}")
    g = _run(w, d, li, T, beta)
    ref_c = oracle.topk(d["logits"], w.K)
    assert np.array_equal(g["cand_ids"], ref_c["cand_ids"]), "candidate sets differ"
    rows = None if grad_rows is None else [(r // w.gamma, r % w.gamma) for r in grad_rows]
    ref = Lo.tree_kl_loss(d["logits"], ref_c["cand_ids"], li["target_logits"], li["y_star"], d["anchor"], d["phi"],
                          d["psi"], d["gate"], d["alpha"], d["lam"], T, beta, with_grad=grad_rows is None)
    for k in ("loss", "kl", "ce"):
        err = np.abs(g[k] - ref[k])
        assert np.all(err <= 1e-5 * np.maximum(1.0, np.abs(ref[k]))), f"{k}: max error {err.max():.3g}"
    assert np.all(np.abs(g["grad_s"] - ref["grad_s"]) <= 1e-5), "grad_s differs"
    if grad_rows is None:
        gl, rl = g["grad_logits"], ref["grad_logits"]
    else:
        sub = Lo.tree_kl_loss(d["logits"], ref_c["cand_ids"], li["target_logits"], li["y_star"], d["anchor"],
                              d["phi"], d["psi"], d["gate"], d["alpha"], d["lam"], T, beta, rows=rows)
        gl = np.stack([g["grad_logits"][b, i] for b, i in rows])
        rl = np.stack([sub["grad_logits"][b, i] for b, i in rows])
    err = np.abs(gl - rl)
    assert np.all(err <= 1e-5 * np.abs(rl) + 1e-6), f"grad_logits: max error {err.max():.3g}"
    invalid = li["y_star"] < 0
    assert (~invalid).any(), "the case has no valid position: it would only compare zeros"
    assert not g["loss"][invalid].any() and not g["grad_s"][invalid].any()
    say(f"  valid positions {int((~invalid).sum())}, mean loss {g['loss'][~invalid].mean():.4f}")


@pytest.mark.parametrize("kw,T", [
    (dict(B=3, L=6, V=3001, dtype="f32", feat_dtype="f32", K=8, r=32), 0.7),   # ragged V: per-element pass
    (dict(B=3, L=6, V=3001, dtype="f32", feat_dtype="f32", K=8, r=32), 0.0),   # T -> 0
    (dict(B=2, L=9, V=4096, dtype="bf16", feat_dtype="bf16", K=16, r=64), 1.0),  # vector pass
    (dict(B=2, L=4, V=2048, dtype="bf16", feat_dtype="f32", K=64, r=16), 0.0),   # K = 64, ties likely
    (dict(B=2, L=4, V=512, dtype="f32", feat_dtype="bf16", K=1, r=512), 1.0),   # K = 1: KL = 0; r = 512
])
def test_loss_small(kw, T):
    base = dict(logits="normal", logit_std=2.0, budget=8, W=3)
    w = synth.custom(400 + kw["K"], **{**base, **kw})
    d = synth.inputs(w, 0)
    rng = np.random.default_rng(kw["V"])
    d["alpha"] = rng.uniform(0.5, 2.0, w.gamma).astype(np.float32)
    d["lam"] = rng.uniform(0.5, 2.0, w.gamma).astype(np.float32)
    li = synth.loss_inputs(w, 0, invalid_frac=0.2)
    # Keep the first position of every sequence valid (its predecessor is the anchor), so
    # each case compares real losses, also the smallest ones.
    y = li["y_star"]
    y[:, 0] = np.where(y[:, 0] < 0, 0, y[:, 0])
    _check(w, d, li, T, 0.1)


def test_loss_ties_at_zero_temperature():
    """Target logits equal on several candidates: the T -> 0 target is uniform over them."""
    w = synth.custom(450, B=2, L=5, V=2000, dtype="f32", feat_dtype="f32", K=8, r=32, logits="normal",
                     logit_std=2.0, budget=8, W=3)
    d = synth.inputs(w, 0)
    li = synth.loss_inputs(w, 0, invalid_frac=0.0)
    c = oracle.topk(d["logits"], w.K)["cand_ids"]
    z = li["target_logits"].copy()
    for b in range(w.B):
        for i in range(w.gamma):
            z[b, i, c[b, i, :3]] = 50.0  # three tied maxima
    li["target_logits"] = z
    _check(w, d, li, 0.0, 0.1)


@pytest.mark.parametrize("T", [1.0, 0.0])
def test_loss_headline_workload(T):
    w = synth.WORKLOADS[3]
    d = synth.inputs(w, 0)
    li = synth.loss_inputs(w, 0)
    _check(w, d, li, T, 0.1, grad_rows=[0, 17, 233, 479])
