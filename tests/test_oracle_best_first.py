"""Pins of the oracle's unigram-plus-bigram scoring with best-first prefix closure (CPU).

Edge scores e_i(a, c) = alpha_i log q_i(c) + lambda_i delta_i(a, c): the unigram
log-probability of Eq. (ubtree-unigram) plus the raw selector score of Eq.
(dflash2-selector), weighted as in Eq. (ubtree-depth), not normalised over the
successors.  Paths are ranked by their cumulative edge score and grown best-first
(Background, "Tree Drafting"): a node becomes eligible once its parent is in the tree, so
the tree stays prefix-closed although the sums are not monotone along a path.

Each test pins the oracle to something other than itself: the brute-force closure in
``bruteforce.py`` (path sums from scratch, a full rescan per step), scipy's log-softmax,
the already-pinned beam oracle in the monotone case, and closed forms.  Planted mistakes
at the end must each fail one of them.
"""
from __future__ import annotations

import numpy as np
import pytest
import scipy.special

import bruteforce as bf
import oracle
import synth


def _tree(B, gamma, K, V=1000, seed=0):
    anchor = synth._rng(950, seed).integers(0, V, B).astype(np.int32)
    return anchor, synth.candidate_ids(B, gamma, K, V, seed)


def _edges(B, gamma, K, seed, spread=3.0, dyadic=False, tie_frac=0.0):
    """Edge slabs with positive and negative entries (so sums are not monotone)."""
    rng = np.random.default_rng(seed)
    if dyadic:
        e = rng.integers(-96, 32, size=(B, gamma, K, K)).astype(np.float64) * 2.0 ** -5
        if tie_frac:
            m = rng.random(e.shape) < tie_frac
            e = np.where(m, e.reshape(B, gamma, -1)[..., :1].reshape(B, gamma, 1, 1), e)
    else:
        e = rng.normal(-1.0, spread, size=(B, gamma, K, K))
    e[:, 0, 1:, :] = 0.0
    return e


def _paths(o, b):
    return bf.tree_as_paths(o, b)


@pytest.mark.parametrize("K,gamma,budget,seed", [(2, 3, 7, 0), (3, 3, 20, 1), (4, 3, 30, 2), (3, 4, 25, 3),
                                                 (2, 5, 40, 4), (5, 2, 12, 5)])
def test_matches_brute_force_closure(K, gamma, budget, seed):
    B = 3
    e = _edges(B, gamma, K, seed)
    anchor, ids = _tree(B, gamma, K, seed=seed)
    o = oracle.best_first(anchor, ids, e, budget, 0.0)
    for b in range(B):
        want = bf.closure_best_first(e[b], budget)
        assert _paths(o, b) == want
        assert o["n_nodes"][b] == 1 + len(want)
        np.testing.assert_allclose(o["score"][b, 1:1 + len(want)], [bf.path_score(e[b], p, 0.0) for p in want])


@pytest.mark.parametrize("seed,zeta", [(10, 0.0), (11, -0.25), (12, -1.0)])
def test_dyadic_ties_match_brute_force(seed, zeta):
    """Exact ties everywhere (dyadic values, many copies): the tie order decides."""
    B, gamma, K, budget = 4, 3, 3, 22
    e = _edges(B, gamma, K, seed, dyadic=True, tie_frac=0.4)
    anchor, ids = _tree(B, gamma, K, seed=seed)
    o = oracle.best_first(anchor, ids, e, budget, zeta)
    for b in range(B):
        assert _paths(o, b) == bf.closure_best_first(e[b], budget, zeta)


def test_sums_are_not_monotone_but_the_tree_is_closed():
    """Edges far above zero: children outscore their parents, and still every node's
    parent precedes it; the mask is each node's ancestor set."""
    B, gamma, K, budget = 4, 4, 3, 30
    e = _edges(B, gamma, K, 20, spread=4.0) + 2.0
    anchor, ids = _tree(B, gamma, K, seed=20)
    o = oracle.best_first(anchor, ids, e, budget)
    rises = 0
    for b in range(B):
        n = o["n_nodes"][b]
        for i in range(1, n):
            p = o["parent"][b, i]
            assert 0 <= p < i and o["depth"][b, i] == o["depth"][b, p] + 1
            assert o["token"][b, i] == ids[b, o["depth"][b, i] - 1, o["cand_rank"][b, i]]
            rises += o["score"][b, i] > o["score"][b, p]
        np.testing.assert_array_equal(oracle.tree_mask(o["parent"], o["n_nodes"])[b], o["mask"][b])
    assert rises > 0


@pytest.mark.parametrize("K,gamma,budget", [(3, 3, 12), (4, 3, 20), (2, 5, 25)])
def test_monotone_edges_give_the_global_best_first_of_the_beam_oracle(K, gamma, budget):
    """With every edge <= 0 the sums fall along each path, so best-first growth takes the
    global top-`budget` nodes: the beam oracle at W = budget (pinned separately) and the
    brute-force global ranking agree on the node set."""
    B = 3
    e = -np.abs(_edges(B, gamma, K, 40 + K))
    anchor, ids = _tree(B, gamma, K, seed=K)
    o = oracle.best_first(anchor, ids, e, budget)
    beam = oracle.build_tree(anchor, ids, e, budget, budget)
    for b in range(B):
        assert set(_paths(o, b)) == set(bf.tree_as_paths(beam, b)) == set(bf.best_first(e[b], budget))


def test_gamma1_is_the_sorted_first_row_and_k1_is_a_chain():
    anchor, ids = _tree(2, 1, 6, seed=3)
    e = _edges(2, 1, 6, 3)
    o = oracle.best_first(anchor, ids, e, 4)
    for b in range(2):
        order = np.lexsort((np.arange(6), -e[b, 0, 0]))[:4]
        assert [p[0] for p in _paths(o, b)] == order.tolist()
    anchor, ids = _tree(2, 5, 1, seed=4)
    e = _edges(2, 5, 1, 4)
    o = oracle.best_first(anchor, ids, e, 3)
    for b in range(2):
        assert _paths(o, b) == [(0,), (0, 0), (0, 0, 0)]


def test_very_negative_zeta_is_breadth_first_and_budget_caps_at_the_lattice():
    """zeta = -1e9 makes every deeper node worse than every shallower one: the tree is all
    of depth 1, then the best depth-2 nodes by score.  A budget beyond the lattice takes
    every node."""
    B, gamma, K = 2, 3, 3
    e = _edges(B, gamma, K, 50)
    anchor, ids = _tree(B, gamma, K, seed=50)
    o = oracle.best_first(anchor, ids, e, K + 4, -1e9)
    for b in range(B):
        paths = _paths(o, b)
        assert sorted(paths[:K]) == [(c,) for c in range(K)]
        d2 = sorted((p for p in bf.lattice(e[b], 0.0) if len(p) == 2), key=lambda p: -bf.path_score(e[b], p, 0.0))
        assert set(paths[K:]) == set(d2[:4])
    full = K + K * K + K ** 3
    o = oracle.best_first(anchor, ids, e, 255)
    assert (o["n_nodes"] == 1 + full).all()


def test_edges_normalised_are_the_selector_log_probabilities():
    """log-softmax over the successors of an edge row gives the normalised log q^bi of
    Appendix A (Eq. ubtree-path): the two differ by alpha_i LSE_i, constant per row."""
    w = synth.custom(60, B=2, L=5, V=700, K=6, r=16, dtype="f32", feat_dtype="f32")
    d = synth.inputs(w, 0)
    rng = np.random.default_rng(1)
    d["alpha"] = rng.uniform(0.5, 2, w.gamma)
    d["lam"] = rng.uniform(0.5, 2, w.gamma)
    t = oracle.topk(d["logits"], w.K)
    g = oracle.bigram(d["phi"], d["psi"], d["gate"], d["anchor"], t["cand_ids"], t["cand_logit"], d["alpha"], d["lam"])
    e = oracle.edge_scores(t["cand_logprob"], g["delta"], d["alpha"], d["lam"])
    for i in range(w.gamma):
        rows = 1 if i == 0 else w.K
        np.testing.assert_allclose(scipy.special.log_softmax(e[:, i, :rows], axis=-1), g["logq"][:, i, :rows],
                                   atol=1e-12)
        assert not e[:, 0, 1:].any()


def test_edges_without_the_selector_are_unigram_log_probabilities():
    """lambda = 0: every row of an edge slab is alpha_i times the candidates' log q_i, which
    scipy's log-softmax over the whole vocabulary gives."""
    w = synth.custom(61, B=2, L=4, V=900, K=5, r=16, dtype="f32", feat_dtype="f32")
    d = synth.inputs(w, 0)
    alpha = np.array([0.5, 1.0, 2.0])
    t = oracle.topk(d["logits"], w.K)
    g = oracle.bigram(d["phi"], d["psi"], d["gate"], d["anchor"], t["cand_ids"], t["cand_logit"], alpha,
                      np.ones(w.gamma))
    e = oracle.edge_scores(t["cand_logprob"], g["delta"], alpha, np.zeros(w.gamma))
    lq = scipy.special.log_softmax(d["logits"].astype(np.float64), axis=-1)
    for b in range(w.B):
        for i in range(w.gamma):
            want = alpha[i] * lq[b, i, t["cand_ids"][b, i]]
            for a in range(1 if i == 0 else w.K):
                np.testing.assert_allclose(e[b, i, a], want, rtol=1e-13, atol=1e-13)


# ----------------------------------------------------------------------------------
# Planted mistakes: each mutant of the oracle source must fail a pin above.
# ----------------------------------------------------------------------------------

MUTANTS = {
    "no_closure": ("if (d >= gamma) return;\n      const int row",
                   "if (d >= gamma) return;\n      slot = 0;\n      const int row"),
    "deeper_first_on_ties": ("if (x.depth != y.depth) return x.depth < y.depth;",
                             "if (x.depth != y.depth) return x.depth > y.depth;"),
    "later_parent_first": ("if (x.pslot != y.pslot) return x.pslot < y.pslot;",
                           "if (x.pslot != y.pslot) return x.pslot > y.pslot;"),
    "row_always_anchor": ("const int row = (d == 0) ? 0 : c;", "const int row = 0;"),
    "zeta_dropped": ("frontier.push_back({s + e[k] + zeta,", "frontier.push_back({s + e[k],"),
    "edge_raw_logit": ("alpha[i] * cand_logprob[bi * K + c] + lambda[i] * delta[o]",
                       "alpha[i] * (cand_logprob[bi * K + c] + 1.0) + lambda[i] * delta[o]"),
    "edge_lambda_on_unigram": ("alpha[i] * cand_logprob[bi * K + c] + lambda[i] * delta[o]",
                               "lambda[i] * cand_logprob[bi * K + c] + alpha[i] * delta[o]"),
    "budget_counts_root": ("while (n <= budget && !frontier.empty())", "while (n < budget && !frontier.empty())"),
}


def _run_pins_against(lib_path: str) -> list:
    tests = [
        lambda: test_matches_brute_force_closure(3, 3, 20, 1),
        lambda: test_matches_brute_force_closure(2, 5, 40, 4),
        lambda: test_dyadic_ties_match_brute_force(10, 0.0),
        lambda: test_dyadic_ties_match_brute_force(11, -0.25),
        test_sums_are_not_monotone_but_the_tree_is_closed,
        lambda: test_monotone_edges_give_the_global_best_first_of_the_beam_oracle(4, 3, 20),
        test_gamma1_is_the_sorted_first_row_and_k1_is_a_chain,
        test_very_negative_zeta_is_breadth_first_and_budget_caps_at_the_lattice,
        test_edges_normalised_are_the_selector_log_probabilities,
        test_edges_without_the_selector_are_unigram_log_probabilities,
    ]
    failures = []
    with oracle.using_library(lib_path):
        for t in tests:
            try:
                t()
            except Exception as e:  # noqa: BLE001 - any failure counts
                failures.append(repr(e)[:80])
    return failures


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, tmp_path):
    import subprocess
    src = open(oracle._build.SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(old, new, 1)
    cpp = tmp_path / "mut.cpp"
    cpp.write_text(mutated)
    so = tmp_path / f"libmut_{name}.so"
    subprocess.run(["g++", "-O1", "-std=c++17", "-shared", "-fPIC", "-pthread", str(cpp), "-o", str(so)], check=True)
    assert _run_pins_against(str(so)), f"mutant {name} passed every pin"


def test_unmutated_oracle_passes_compact_pins():
    assert _run_pins_against(oracle._build.LIB) == []
