"""GPU parity of ubt_bigram_scores (selector scores, depth calibration, successor
normalisation) against the oracle, on identical inputs."""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
import parity
import synth

pytestmark = pytest.mark.gpu


def _inputs(B, gamma, K, V, r, dt, seed, alpha_lam="unit"):
    rng = np.random.default_rng(seed)
    phi = synth.store(rng.normal(0, r ** -0.5, (V, r)), dt)
    psi = synth.store(rng.normal(0, r ** -0.5, (V, r)), dt)
    gate = synth.store(rng.normal(0, 1, (B, gamma, r)), dt)
    ids = np.stack([np.stack([rng.permutation(V)[:K] for _ in range(gamma)]) for _ in range(B)]).astype(np.int32)
    logit = synth.round_f32(rng.normal(0, 3, (B, gamma, K)))
    anchor = rng.integers(0, V, B).astype(np.int32)
    if alpha_lam == "unit":
        alpha = lam = np.ones(gamma, np.float32)
    elif alpha_lam == "random":
        alpha = synth.round_f32(rng.uniform(0.5, 2, gamma))
        lam = synth.round_f32(rng.uniform(0.5, 2, gamma))
    else:  # lambda = sqrt(r)
        alpha = np.ones(gamma, np.float32)
        lam = np.full(gamma, math.sqrt(r), np.float32)
    return phi, psi, gate, ids, logit, anchor, alpha, lam


def _run(phi, psi, gate, ids, logit, anchor, alpha, lam):
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, dev_values, to_np

    out = ubt.bigram_scores(dev_values(phi), dev_values(psi), dev_values(gate), dev_i32(anchor), dev_i32(ids),
                            dev_values(logit), alpha, lam)
    torch.cuda.synchronize()
    return to_np(out)


CASES = [  # B, gamma, K, V, r
    (2, 3, 1, 50, 16), (3, 5, 4, 300, 32), (2, 4, 8, 1000, 64), (2, 15, 8, 5000, 128), (2, 6, 16, 3000, 128),
    (1, 4, 17, 500, 48), (1, 3, 32, 800, 256), (1, 3, 33, 800, 80), (1, 2, 64, 2000, 512), (4, 31, 16, 2000, 256),
    # K > 16 splits each position's contraction over K/16 waves: the paper's shape (K = 64, r = 256),
    # fewer k-steps than waves (r = 48), a half last step (r = 208), and rows past K in the last tile row
    (2, 15, 64, 5000, 256), (2, 5, 40, 3000, 48), (1, 3, 24, 700, 208), (2, 4, 49, 1500, 144),
]


@pytest.mark.parametrize("B,gamma,K,V,r", CASES)
@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_selector_matches_oracle(B, gamma, K, V, r, dt):
    from gpu_util import say

    say(f"bigram B={B} gamma={gamma} K={K} V={V} r={r} {dt}")
    args = _inputs(B, gamma, K, V, r, dt, seed=B * 1000 + K * 10 + r)
    g = _run(*args)
    ref = oracle.bigram(args[0], args[1], args[2], args[5], args[3], args[4], args[6], args[7])
    parity.check_selector(g, ref)
    assert (g["logq"] <= 0).all()
    assert not g["delta"][:, 0, 1:].any() and not g["logq"][:, 0, 1:].any()


@pytest.mark.parametrize("mode", ["random", "sqrt_r"])
def test_depth_calibration(mode):
    args = _inputs(3, 7, 8, 2000, 128, "bf16", seed=77, alpha_lam=mode)
    g = _run(*args)
    ref = oracle.bigram(args[0], args[1], args[2], args[5], args[3], args[4], args[6], args[7])
    parity.check_selector(g, ref)


def test_rows_normalised():
    args = _inputs(2, 9, 16, 4000, 128, "bf16", seed=5)
    g = _run(*args)
    s = np.exp(g["logq"].astype(np.float64)).sum(-1)
    np.testing.assert_allclose(s[:, 1:], 1.0, atol=2e-6)
    np.testing.assert_allclose(s[:, 0, 0], 1.0, atol=2e-6)
