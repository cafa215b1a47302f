"""GPU parity of the unigram-plus-bigram scoring with best-first growth
(ubt_edge_scores, ubt_build_tree_best_first) against the fp64 oracle, through the C ABI.

* Dyadic edge slabs (multiples of 2^-5, positive and negative, with planted ties): every
  path sum is exact in fp32 and fp64, so trees, slots and scores must match bit for bit,
  the tie order included.  Shapes cover K = 1..64, budgets beyond the lattice, the depth
  bonus, edges far above zero (children outscoring their parents), and slabs staged in
  LDS or read from memory.
* The whole step on the workloads: ubt_topk's log-probabilities, ubt_edge_scores (within
  1e-5 * max(1, |ref|) of the oracle's fp64 edges) and the tree, exact or within the 1e-5
  tie gap of the oracle's path sums, validated growth step by growth step."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import parity
import synth

pytestmark = pytest.mark.gpu


def _dyadic(B, gamma, K, seed, lift=0.0, tie_frac=0.3):
    """Multiples of 2^-5 plus `lift` (itself a multiple of 2^-5, so every path sum stays
    exact in fp32), with a share of entries copied within the slab to plant ties."""
    assert lift * 32 == int(lift * 32)
    rng = np.random.default_rng(seed)
    e = rng.integers(-64, 24, size=(B, gamma, K, K)).astype(np.float64) * 2.0 ** -5 + lift
    m = rng.random(e.shape) < tie_frac
    src = rng.integers(0, K * K, size=(B, gamma, K, K))
    flat = e.reshape(B, gamma, K * K)
    e = np.where(m, np.take_along_axis(flat, src.reshape(B, gamma, K * K), 2).reshape(B, gamma, K, K), e)
    e[:, 0, 1:, :] = 0.0
    return e.astype(np.float32)


def _run_tree(anchor, ids, edge, budget, zeta):
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, to_np

    out = ubt.build_tree_best_first(dev_i32(anchor), dev_i32(ids), torch.from_numpy(edge).cuda(), budget, zeta)
    torch.cuda.synchronize()
    return to_np(out)


@pytest.mark.parametrize("B,gamma,K,budget,zeta,lift", [
    (3, 4, 4, 20, 0.0, 0.0),
    (2, 3, 2, 14, 0.0, 0.0),        # budget = the whole lattice (2 + 4 + 8)
    (2, 3, 2, 40, 0.0, 0.0),        # budget beyond the lattice
    (4, 15, 8, 64, 0.0, 0.0),       # the headline shape
    (4, 15, 8, 64, -0.25, 0.0),     # depth bonus
    (4, 15, 8, 64, 0.0, 0.5),       # edges mostly above zero: sums rise along paths
    (2, 15, 16, 128, 0.0, 0.0),
    (2, 31, 16, 128, 0.0, 0.0),     # slab 31.7 KB: still in LDS
    (2, 40, 16, 200, 0.0, 0.25),    # slab 40 KB: read from memory
    (2, 15, 64, 64, 0.0, 0.0),      # K = 64: read from memory
    (2, 64, 4, 255, -0.0625, 0.0),  # the longest block and the largest budget
    (2, 6, 1, 10, 0.0, 0.0),        # K = 1: a chain, shorter than the budget
    (2, 5, 5, 30, 0.0, 0.0),        # K outside the powers of two
])
def test_dyadic_trees_are_exact(B, gamma, K, budget, zeta, lift):
    from gpu_util import say

    say(f"best-first dyadic B={B} gamma={gamma} K={K} budget={budget} zeta={zeta} lift={lift}")
    edge = _dyadic(B, gamma, K, seed=gamma * 100 + K, lift=lift)
    rng = np.random.default_rng(K)
    anchor = rng.integers(0, 5000, B).astype(np.int32)
    ids = rng.integers(0, 5000, size=(B, gamma, K)).astype(np.int32)
    g = _run_tree(anchor, ids, edge, budget, zeta)
    ref = oracle.best_first(anchor, ids, edge.astype(np.float64), budget, zeta)
    for k in ("n_nodes", "token", "parent", "depth", "cand_rank"):
        np.testing.assert_array_equal(g[k], ref[k], err_msg=k)
    np.testing.assert_array_equal(g["score"].astype(np.float64), ref["score"])
    np.testing.assert_array_equal(g["mask"], ref["mask"])
    parity.check_best_first(g, ref, edge.astype(np.float64), ids, anchor, budget, zeta, allow_ties=False)
    if lift > 0:
        rises = sum(int(g["score"][b, i] > g["score"][b, g["parent"][b, i]]) for b in range(B)
                    for i in range(1, int(g["n_nodes"][b])))
        assert rises > 0


def _step(w: synth.Workload, buf: int = 0, lam_scale: float = 1.0):
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, dev_values, say, to_np

    say(f"best-first step workload {w.cfg}: {w.describe()} lambda x{lam_scale}")
    d = synth.inputs(w, buf)
    lam = d["lam"] * lam_scale
    logits = dev_values(d["logits"])
    anchor = dev_i32(d["anchor"])
    cand = ubt.topk(logits, w.K)
    sel = ubt.edge_scores(dev_values(d["phi"]), dev_values(d["psi"]), dev_values(d["gate"]), anchor,
                          cand["cand_ids"], cand["cand_logprob"], d["alpha"], lam, with_delta=True)
    tree = ubt.build_tree_best_first(anchor, cand["cand_ids"], sel["edge"], w.budget, w.zeta)
    torch.cuda.synchronize()
    g = {**to_np(cand), **to_np(sel), **to_np(tree)}
    ref = oracle.pipeline_unigram_bigram(d["logits"], d["phi"], d["psi"], d["gate"], d["anchor"], d["alpha"], lam,
                                         w.K, w.budget, w.zeta)
    parity.check_topk(g, ref)
    parity.close(g["delta"], ref["delta"], "delta")
    parity.close(g["edge"], ref["edge"], "edge")
    counts = parity.check_best_first(g, ref, ref["edge"], ref["cand_ids"], d["anchor"], w.budget, w.zeta)
    parity.record(f"best-first wl{w.cfg} lambda x{lam_scale}", counts)
    say(f"  trees vs oracle: {counts}")
    return g


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6])
def test_workload_step(cfg):
    _step(synth.WORKLOADS[cfg])


def test_strong_selector_makes_sums_rise():
    """lambda = 40 on the headline workload: selector scores outweigh the log-probabilities,
    so many nodes outscore their parents; the trees must still match the oracle's."""
    g = _step(synth.WORKLOADS[3], lam_scale=40.0)
    rises = sum(int(g["score"][b, i] > g["score"][b, g["parent"][b, i]]) for b in range(g["n_nodes"].shape[0])
                for i in range(1, int(g["n_nodes"][b])))
    assert rises > 0
