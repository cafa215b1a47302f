"""End-to-end GPU parity of one draft step (top-K -> selector -> tree + mask) against
the oracle, on the six workloads at full size and at the exact best-first width."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import parity
import synth

pytestmark = pytest.mark.gpu


def _check_workload(w: synth.Workload, W: int, buf: int = 0, allow_ties: bool = True) -> dict:
    from gpu_util import run_pipeline, say

    say(f"pipeline workload {w.cfg} buf={buf} W={W}: {w.describe()}")
    d = synth.inputs(w, buf)
    g = run_pipeline(w, d, W=W)
    ref_t = oracle.topk(d["logits"], w.K)
    parity.check_topk(g, ref_t)
    ref_s = oracle.bigram(d["phi"], d["psi"], d["gate"], d["anchor"], ref_t["cand_ids"], ref_t["cand_logit"],
                          d["alpha"], d["lam"])
    parity.check_selector(g, ref_s)
    ref = oracle.build_tree(d["anchor"], ref_t["cand_ids"], ref_s["logq"], W, w.budget, w.zeta)
    counts = parity.check_tree(g, ref, ref_s["logq"], ref_t["cand_ids"], d["anchor"], W, w.budget, w.zeta,
                               allow_ties=allow_ties)
    assert (g["n_nodes"] == w.N).all(), "every tree should use the whole budget"
    parity.record(f"pipeline wl{w.cfg} buf={buf} W={W}", counts)
    say(f"  trees: {counts}")
    return counts


def test_workload1_exact():
    """Workload 1 (fp32 logits and features): every tree identical to the oracle's, with
    no tie excused."""
    counts = _check_workload(synth.WORKLOADS[1], synth.WORKLOADS[1].W, allow_ties=False)
    assert counts["excused"] == 0


@pytest.mark.parametrize("cfg", [2, 3, 4, 5, 6])
def test_workload_full_size(cfg):
    w = synth.WORKLOADS[cfg]
    _check_workload(w, w.W)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6])
def test_workload_best_first_width(cfg):
    w = synth.WORKLOADS[cfg]
    _check_workload(w, w.budget)


def test_pool_buffers_and_repeatability():
    """Each distinct pool buffer of the headline workload, and bitwise-identical reruns."""
    from gpu_util import run_pipeline

    w = synth.WORKLOADS[3]
    for buf in (1, 2, 3):
        _check_workload(w, w.W, buf=buf)
    d = synth.inputs(w, 0)
    a = run_pipeline(w, d)
    b = run_pipeline(w, d)
    for k in a:
        assert np.array_equal(a[k], b[k]), f"{k} differs between identical runs"
