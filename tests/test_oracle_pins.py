"""Pins of the fp64 oracle against what the paper and the mathematics fix (CPU only).

Each test pins one oracle function to something other than itself: a library routine
it does not use, a closed form, an invariant, or the brute-force lattice enumerator in
``bruteforce.py``.  The mutation tests at the end show that plausible mistakes in the
oracle's source fail at least one of these pins.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import scipy.special

import bruteforce as bf
import oracle
import synth

# ----------------------------------------------------------------------------------
# Candidate sets and softmax statistics (Method, Unigram Proposer / Candidate Sets)
# ----------------------------------------------------------------------------------


def _np_topk(u: np.ndarray, K: int) -> np.ndarray:
    """Library pin: lexsort by (value desc, id asc); -0.0 and 0.0 compare equal in numpy."""
    return np.stack([np.lexsort((np.arange(u.shape[-1]), -row))[:K] for row in u.reshape(-1, u.shape[-1])])


@pytest.mark.parametrize("V,K", [(1, 1), (7, 3), (33, 8), (1000, 64), (4099, 16)])
def test_topk_matches_lexsort_f32(V, K):
    rng = np.random.default_rng(V * 31 + K)
    u = rng.normal(0, 3, (5, V)).astype(np.float32)
    o = oracle.topk(u, K)
    np.testing.assert_array_equal(o["cand_ids"].reshape(-1, K), _np_topk(u.astype(np.float64), K))
    np.testing.assert_array_equal(o["cand_logit"], np.take_along_axis(u, o["cand_ids"], -1).astype(np.float64))


def test_topk_bf16_duplicates_lower_id_first():
    # bf16 has few distinct values near the top of a row: many exact ties.
    rng = np.random.default_rng(5)
    u = synth.round_bf16_bits(np.round(rng.normal(0, 1, (6, 3000)) * 4) / 4)
    o = oracle.topk(u, 32)
    vals = synth.bf16_bits_to_f32(u).astype(np.float64)
    np.testing.assert_array_equal(o["cand_ids"], _np_topk(vals, 32))
    # within equal values the ids ascend
    for row_ids, row_vals in zip(o["cand_ids"], o["cand_logit"]):
        for j in range(31):
            assert row_vals[j] > row_vals[j + 1] or (row_vals[j] == row_vals[j + 1] and row_ids[j] < row_ids[j + 1])


def test_topk_all_equal_row_gives_first_ids():
    u = np.full((3, 500), 1.25, np.float32)
    o = oracle.topk(u, 10)
    np.testing.assert_array_equal(o["cand_ids"], np.tile(np.arange(10), (3, 1)))


def test_topk_signed_zero_and_neg_inf():
    u = np.full((1, 12), -np.inf, np.float32)
    u[0, 3] = -0.0
    u[0, 7] = 0.0
    u[0, 9] = -1.0
    o = oracle.topk(u, 5)
    # -0 == +0: ties by id; then -1; then the -inf entries by id.
    np.testing.assert_array_equal(o["cand_ids"][0], [3, 7, 9, 0, 1])
    assert o["cand_logit"][0, 3] == -np.inf
    np.testing.assert_allclose(o["lse"][0], math.log(2 + math.exp(-1)), rtol=1e-15)


def test_topk_brute_force_all_orders():
    # Every ordering of a tiny row with ties, checked against an explicit pairwise count.
    rng = np.random.default_rng(9)
    for _ in range(200):
        V = int(rng.integers(1, 9))
        u = rng.integers(-2, 3, V).astype(np.float32)
        K = int(rng.integers(1, V + 1))
        ids = oracle.topk(u[None], K)["cand_ids"][0]
        rank = [sum(1 for j in range(V) if u[j] > u[i] or (u[j] == u[i] and j < i)) for i in range(V)]
        expect = [i for r in range(K) for i in range(V) if rank[i] == r]
        assert list(ids) == expect


def test_lse_matches_scipy_and_logprob():
    rng = np.random.default_rng(11)
    u = rng.normal(0, 3, (4, 32000)).astype(np.float32)
    o = oracle.topk(u, 4)
    ref = scipy.special.logsumexp(u.astype(np.float64), axis=-1)
    np.testing.assert_allclose(o["lse"], ref, rtol=1e-13, atol=1e-12)
    np.testing.assert_allclose(o["cand_logprob"], o["cand_logit"] - ref[:, None], rtol=1e-13, atol=1e-12)


@pytest.mark.parametrize("c", [-7.5, 0.0, 3.0, 120.0])
def test_lse_constant_row_closed_form(c):
    V = 151936
    o = oracle.topk(np.full((1, V), c, np.float32), 8)
    np.testing.assert_allclose(o["lse"][0], c + math.log(V), rtol=1e-14)
    np.testing.assert_array_equal(o["cand_ids"][0], np.arange(8))


def test_lse_shift_equivariance():
    rng = np.random.default_rng(2)
    u = (np.round(rng.normal(0, 2, (3, 5000)) * 64) / 64).astype(np.float32)
    a, b = oracle.topk(u, 8), oracle.topk(u + np.float32(16.0), 8)
    np.testing.assert_array_equal(a["cand_ids"], b["cand_ids"])
    np.testing.assert_allclose(b["lse"], a["lse"] + 16.0, rtol=1e-14)
    np.testing.assert_allclose(b["cand_logprob"], a["cand_logprob"], atol=1e-12)


# ----------------------------------------------------------------------------------
# Selector scores and normalisation (Eq. dflash2-selector, ubtree-depth, ubtree-edge-matrix,
# ubtree-path)
# ----------------------------------------------------------------------------------


def _small_selector(dtype="f32", K=4, gamma=5, V=50, r=16, B=3, seed=0, lam_scale=1.0):
    rng = np.random.default_rng(seed)
    phi = synth.store(rng.normal(0, r ** -0.5, (V, r)), dtype)
    psi = synth.store(rng.normal(0, r ** -0.5, (V, r)), dtype)
    gate = synth.store(rng.normal(0, 1, (B, gamma, r)), dtype)
    ids = np.stack([np.stack([rng.permutation(V)[:K] for _ in range(gamma)]) for _ in range(B)]).astype(np.int32)
    logit = rng.normal(0, 2, (B, gamma, K))
    anchor = rng.integers(0, V, B).astype(np.int32)
    alpha = rng.uniform(0.5, 2, gamma)
    lam = rng.uniform(0.5, 2, gamma) * lam_scale
    return phi, psi, gate, ids, logit, anchor, alpha, lam


def _decode(a):
    return synth.bf16_bits_to_f32(a).astype(np.float64) if a.dtype == np.uint16 else a.astype(np.float64)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_delta_matches_einsum(dtype):
    phi, psi, gate, ids, logit, anchor, alpha, lam = _small_selector(dtype)
    o = oracle.bigram(phi, psi, gate, anchor, ids, logit, alpha, lam)
    P, S, G = _decode(phi), _decode(psi), _decode(gate)
    B, gamma, K = ids.shape
    for b in range(B):
        for i in range(gamma):
            pred = [anchor[b]] if i == 0 else ids[b, i - 1]
            ref = np.einsum("k,ak,ck->ac", G[b, i], P[pred], S[ids[b, i]])
            np.testing.assert_allclose(o["delta"][b, i, : len(pred)], ref, rtol=1e-12, atol=1e-14)
            if i == 0:
                assert not o["delta"][b, 0, 1:].any() and not o["logq"][b, 0, 1:].any()


def test_pair_count():
    # K + (gamma-1) K^2 predecessor-successor pairs per sequence (Method, Parallel Computation):
    # one normalised row (the anchor) at depth 1, K rows at every later depth.
    phi, psi, gate, ids, logit, anchor, alpha, lam = _small_selector(K=3, gamma=6)
    o = oracle.bigram(phi, psi, gate, anchor, ids, logit, alpha, lam)
    B, gamma, K = ids.shape
    rows = np.isclose(np.exp(o["logq"]).sum(-1), 1.0, rtol=0, atol=1e-12)
    assert int(rows[0].sum()) * K == K + (gamma - 1) * K * K
    assert not o["delta"][0, 0, 1:].any()


def test_logq_rows_normalised_and_nonpositive():
    phi, psi, gate, ids, logit, anchor, alpha, lam = _small_selector("bf16", K=8)
    o = oracle.bigram(phi, psi, gate, anchor, ids, logit, alpha, lam)
    lq = o["logq"]
    sums = np.exp(lq).sum(-1)
    np.testing.assert_allclose(sums[:, 1:], 1.0, rtol=1e-13)
    np.testing.assert_allclose(sums[:, 0, 0], 1.0, rtol=1e-13)
    assert (lq <= 0).all()


def test_logq_definition_by_softmax():
    # log q^bi(b|a) = log softmax_b(alpha u(b) + lambda delta(a,b)), via scipy.
    phi, psi, gate, ids, logit, anchor, alpha, lam = _small_selector(K=5, seed=3)
    o = oracle.bigram(phi, psi, gate, anchor, ids, logit, alpha, lam)
    s = alpha[None, :, None, None] * logit[:, :, None, :] + lam[None, :, None, None] * o["delta"]
    ref = scipy.special.log_softmax(s, axis=-1)
    np.testing.assert_allclose(o["logq"][:, 1:], ref[:, 1:], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(o["logq"][:, 0, 0], ref[:, 0, 0], rtol=1e-12, atol=1e-13)


def test_lambda_zero_is_separable():
    phi, psi, gate, ids, logit, anchor, alpha, lam = _small_selector(K=4, seed=4, lam_scale=0.0)
    lq = oracle.bigram(phi, psi, gate, anchor, ids, logit, alpha, lam)["logq"]
    np.testing.assert_allclose(lq[:, 1:], np.broadcast_to(lq[:, 1:, :1, :], lq[:, 1:].shape), atol=1e-14)
    ref = scipy.special.log_softmax(alpha[None, :, None] * logit, axis=-1)
    np.testing.assert_allclose(lq[:, :, 0, :], ref, atol=1e-13)


def test_logq_invariant_to_unigram_shift():
    # Replacing u_i by log q_i = u_i - LSE_i shifts every row of s_i by a constant.
    phi, psi, gate, ids, logit, anchor, alpha, lam = _small_selector(K=6, seed=5)
    a = oracle.bigram(phi, psi, gate, anchor, ids, logit, alpha, lam)["logq"]
    b = oracle.bigram(phi, psi, gate, anchor, ids, logit - 11.5, alpha, lam)["logq"]
    np.testing.assert_allclose(a, b, atol=1e-12)


# ----------------------------------------------------------------------------------
# Tree construction (Appendix A, Algorithm 1)
# ----------------------------------------------------------------------------------

TINY = [  # (gamma, K, budget, W)
    (1, 1, 1, 1), (1, 4, 3, 2), (2, 2, 3, 1), (3, 2, 6, 2), (3, 3, 8, 2), (4, 2, 10, 3),
    (4, 3, 12, 4), (5, 2, 20, 3), (5, 3, 24, 5), (6, 2, 30, 4), (3, 4, 9, 9), (4, 4, 24, 6),
]


def _tree_pair(gamma, K, budget, W, seed, zeta=0.0, tie_frac=0.0, levels=16):
    q = synth.dyadic_logq(2, gamma, K, seed=seed, levels=levels, tie_frac=tie_frac).astype(np.float64)
    ids = synth.candidate_ids(2, gamma, K, 1000, seed)
    anchor = np.array([5, 7], np.int32)
    o = oracle.build_tree(anchor, ids, q, W, budget, zeta)
    return q, o


@pytest.mark.parametrize("gamma,K,budget,W", TINY)
@pytest.mark.parametrize("tie_frac", [0.0, 0.5])
def test_tree_matches_brute_force_beam(gamma, K, budget, W, tie_frac):
    for seed in range(3):
        q, o = _tree_pair(gamma, K, budget, W, seed, zeta=-0.125 * (seed % 2), tie_frac=tie_frac, levels=6)
        zeta = -0.125 * (seed % 2)
        for b in range(2):
            fr, tree = bf.beam(q[b], W, budget, zeta)
            assert bf.frontier_as_paths(o, b) == fr
            assert bf.tree_as_paths(o, b) == tree


@pytest.mark.parametrize("gamma,K,budget", [(3, 3, 8), (4, 2, 10), (4, 3, 20), (5, 2, 12), (3, 4, 15)])
def test_wide_beam_is_global_best_first(gamma, K, budget):
    # With W >= budget the beam loses nothing: T is the global top-budget of the lattice.
    for seed in range(4):
        for W in (budget, budget + 3):
            q, o = _tree_pair(gamma, K, budget, W, seed, tie_frac=0.3, levels=8)
            for b in range(2):
                assert bf.tree_as_paths(o, b) == bf.best_first(q[b], budget)


def test_tree_scores_are_path_sums_and_tokens_follow_ranks():
    q, o = _tree_pair(5, 3, 20, 4, seed=1, zeta=-0.25)
    ids = synth.candidate_ids(2, 5, 3, 1000, 1)
    for b in range(2):
        paths = bf.tree_as_paths(o, b)
        for n, p in enumerate(paths, start=1):
            assert o["score"][b, n] == bf.path_score(q[b], p, -0.25)
            assert o["depth"][b, n] == len(p)
            assert o["token"][b, n] == ids[b, len(p) - 1, p[-1]]
        assert o["token"][b, 0] == [5, 7][b] and o["parent"][b, 0] == -1 and o["score"][b, 0] == 0


def test_k1_is_argmax_chain():
    q, o = _tree_pair(6, 1, 4, 2, seed=0)
    for b in range(2):
        assert o["n_nodes"][b] == 5
        np.testing.assert_array_equal(o["parent"][b], [-1, 0, 1, 2, 3])
        np.testing.assert_array_equal(o["depth"][b], [0, 1, 2, 3, 4])


def test_gamma1_is_sorted_first_row():
    q, o = _tree_pair(1, 8, 5, 3, seed=2, tie_frac=0.4, levels=4)
    for b in range(2):
        row = q[b, 0, 0]
        expect = np.lexsort((np.arange(8), -row))[:3]
        np.testing.assert_array_equal(o["cand_rank"][b, 1:4], expect)
        assert o["n_nodes"][b] == 4 and (o["cand_rank"][b, 4:] == -1).all()


def test_frontier_sizes_and_node_count():
    for gamma, K, budget, W in [(6, 3, 12, 2), (5, 4, 30, 7), (8, 2, 15, 16)]:
        q, o = _tree_pair(gamma, K, budget, W, seed=3)
        prev = 1
        for d in range(gamma):
            assert o["f_count"][0, d] == min(W, K * prev)
            prev = o["f_count"][0, d]
        assert o["n_nodes"][0] == 1 + min(budget, int(o["f_count"][0].sum()))


def test_zeta_keeps_supertree_and_very_negative_zeta_is_breadth_first():
    q, o0 = _tree_pair(5, 3, 14, 3, seed=4)
    _, o1 = _tree_pair(5, 3, 14, 3, seed=4, zeta=-0.5)
    _, o2 = _tree_pair(5, 3, 14, 3, seed=4, zeta=-1e6)
    for b in range(2):
        assert bf.frontier_as_paths(o0, b) == bf.frontier_as_paths(o1, b) == bf.frontier_as_paths(o2, b)
        # zeta -> -inf: whole frontiers in depth order
        fr = bf.frontier_as_paths(o2, b)
        expect = [p for fd in fr for p in fd][:14]
        assert bf.tree_as_paths(o2, b) == expect
        assert (np.diff(o2["depth"][b, 1:15]) >= 0).all()


def test_prefix_closed_and_mask_is_ancestor_set():
    w = synth.custom(7, B=3, L=9, V=600, K=5, budget=40, W=6)
    d = synth.inputs(w)
    o = oracle.pipeline(d["logits"], d["phi"], d["psi"], d["gate"], d["anchor"], d["alpha"], d["lam"],
                        w.K, w.W, w.budget)
    N = w.N
    for b in range(w.B):
        n = o["n_nodes"][b]
        assert n == N
        for i in range(1, n):
            p = o["parent"][b, i]
            assert 0 <= p < i and o["depth"][b, i] == o["depth"][b, p] + 1
            assert o["score"][b, i] <= o["score"][b, p]
        for i in range(n):
            anc, m = set(), i
            while m >= 0:
                anc.add(m)
                m = o["parent"][b, m]
            bits = {m for m in range(N) if (o["mask"][b, i, m // 32] >> (m % 32)) & 1}
            assert bits == anc
            assert len(bits) == o["depth"][b, i] + 1
        np.testing.assert_array_equal(oracle.tree_mask(o["parent"], o["n_nodes"])[b], o["mask"][b])


# ----------------------------------------------------------------------------------
# Planted mistakes: each mutant of the oracle source must fail a pin above.
# ----------------------------------------------------------------------------------

MUTANTS = {
    "tie_to_higher_id": ("(u[a] == u[b] && a < b)", "(u[a] == u[b] && a > b)"),
    "lse_drops_shift": ("return m + std::log(s);", "return std::log(s);"),
    "gate_dropped": ("d += load_value(gate, feat_dtype, bi * r + k) *", "d += 1.0 *"),
    "phi_psi_swapped": ("load_value(phi_tab, feat_dtype, pred * r + k)", "load_value(psi_tab, feat_dtype, pred * r + k)"),
    "predecessor_same_depth": ("cand_ids[(bi - 1) * K + a]", "cand_ids[bi * K + a]"),
    "alpha_on_delta": ("alpha[i] * cand_logit[bi * K + c] + lambda[i] * d", "lambda[i] * cand_logit[bi * K + c] + alpha[i] * d"),
    "zeta_sign": ("F[d - 1][p].score + q[c] + zeta", "F[d - 1][p].score + q[c] - zeta"),
    "row_from_rank_zero": ("const int row = (d == 1) ? 0 : F[d - 1][p].c;", "const int row = 0;"),
    "width_per_parent": ("E.resize(std::min<size_t>(E.size(), static_cast<size_t>(W)));",
                         "E.resize(std::min<size_t>(E.size(), static_cast<size_t>(W) * F[d - 1].size()));"),
    "unstable_global_sort": ("std::stable_sort(S.begin(), S.end()", "std::sort(S.rbegin(), S.rend()"),
    "budget_counts_root": ("std::min<int>(static_cast<int>(S.size()), budget)", "std::min<int>(static_cast<int>(S.size()), budget - 1)"),
}


def _run_pins_against(lib_path: str) -> list:
    """Runs a compact set of the pins above with the oracle at `lib_path`; returns failures."""
    tests = [
        test_topk_bf16_duplicates_lower_id_first, test_lse_matches_scipy_and_logprob,
        lambda: test_lse_constant_row_closed_form(3.0),
        lambda: test_delta_matches_einsum("f32"), test_logq_definition_by_softmax,
        lambda: test_tree_matches_brute_force_beam(4, 3, 12, 4, 0.5),
        lambda: test_wide_beam_is_global_best_first(4, 3, 20), test_frontier_sizes_and_node_count,
        test_zeta_keeps_supertree_and_very_negative_zeta_is_breadth_first, test_gamma1_is_sorted_first_row,
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
