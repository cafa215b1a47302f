"""Pins of the LM-head oracle (``oracle/lm_head.py``) against what the mathematics fixes
(CPU only): exact integer arithmetic, a plain-Python brute force, the already-pinned C
oracle on logits that fp32 represents exactly, scipy's logsumexp, and closed forms.
Planted mistakes in a copy of the module must each fail one of them."""
from __future__ import annotations

import math
import types

import numpy as np
import pytest
import scipy.special

import oracle
import synth
from oracle import lm_head as LH


def _bits(x: np.ndarray) -> np.ndarray:
    return synth.round_bf16_bits(np.asarray(x, np.float64))


def _int_inputs(M, d, V, seed, lo=-8, hi=8, scale=0.25):
    """bf16 inputs that are small integers times `scale` (exact in bf16)."""
    rng = np.random.default_rng(seed)
    h = rng.integers(lo, hi + 1, size=(M, d)) * scale
    w = rng.integers(lo, hi + 1, size=(V, d)) * scale
    return h, w


def test_logits_are_exact_integer_arithmetic(lib=None):
    """Integer-valued inputs: every logit is an exact integer sum, computed here with
    Python integers."""
    L = lib or LH
    h, w = _int_inputs(3, 40, 57, 1, scale=1.0)
    u = L.logits(_bits(h), _bits(w), block=16)  # several blocks, a ragged last one
    hi, wi = h.astype(np.int64), w.astype(np.int64)
    for m in range(3):
        for v in range(57):
            assert u[m, v] == sum(int(hi[m, k]) * int(wi[v, k]) for k in range(40))


def test_logits_brute_force_random(lib=None):
    """General bf16 values: a plain-Python dot product of the widened values."""
    L = lib or LH
    rng = np.random.default_rng(2)
    hb, wb = _bits(rng.normal(0, 1, (2, 24))), _bits(rng.normal(0, 0.3, (11, 24)))
    u = L.logits(hb, wb, block=4)
    hv = [[float(x) for x in row] for row in synth.bf16_bits_to_f32(hb)]
    wv = [[float(x) for x in row] for row in synth.bf16_bits_to_f32(wb)]
    for m in range(2):
        for v in range(11):
            ref = math.fsum(hv[m][k] * wv[v][k] for k in range(24))
            assert abs(u[m, v] - ref) <= 1e-12 * max(1.0, abs(ref))


def test_candidates_match_the_c_oracle_on_exact_logits(lib=None):
    """Logits that are integers (exact in fp32): the candidates and LSE equal those of
    the C oracle's top-K run on the same values (pinned separately)."""
    L = lib or LH
    h, w = _int_inputs(4, 16, 3000, 3)
    out = L.lm_head_topk(_bits(h), _bits(w), 8)
    ref = oracle.topk(out["logits"].astype(np.float32), 8)
    np.testing.assert_array_equal(out["cand_ids"], ref["cand_ids"])
    np.testing.assert_array_equal(out["cand_logit"], ref["cand_logit"])
    np.testing.assert_allclose(out["lse"], ref["lse"], rtol=1e-13)
    np.testing.assert_allclose(out["cand_logprob"], ref["cand_logprob"], rtol=1e-12, atol=1e-12)


def test_lse_matches_scipy_and_handles_large_logits(lib=None):
    L = lib or LH
    rng = np.random.default_rng(4)
    hb = _bits(rng.normal(0, 1, (3, 64)))
    wb = _bits(rng.normal(0, 40, (500, 64)))  # logits near a thousand: exp overflows unshifted
    out = L.lm_head_topk(hb, wb, 4)
    np.testing.assert_allclose(out["lse"], scipy.special.logsumexp(out["logits"], axis=1), rtol=1e-13)
    assert np.isfinite(out["lse"]).all()


def test_zero_hidden_state_and_permuted_head(lib=None):
    """h = 0: every logit is 0, the candidates are ids 0..K-1 and LSE = ln V.  Permuting
    the head's rows permutes the candidate ids (distinct logits)."""
    L = lib or LH
    V = 777
    rng = np.random.default_rng(5)
    wb = _bits(rng.normal(0, 1, (V, 32)))
    out = L.lm_head_topk(_bits(np.zeros((2, 32))), wb, 5)
    np.testing.assert_array_equal(out["cand_ids"], np.tile(np.arange(5), (2, 1)))
    np.testing.assert_allclose(out["lse"], math.log(V), rtol=1e-14)
    hb = _bits(rng.normal(0, 1, (2, 32)))
    base = L.lm_head_topk(hb, wb, 6)
    perm = rng.permutation(V)
    permuted = L.lm_head_topk(hb, wb[perm], 6)
    np.testing.assert_array_equal(perm[permuted["cand_ids"]], base["cand_ids"])


def test_ties_go_to_the_lower_id(lib=None):
    L = lib or LH
    wb = _bits(np.repeat(np.array([[1.0, 2.0], [3.0, -1.0]]), 5, axis=0))  # rows 0-4 equal, 5-9 equal
    out = L.lm_head_topk(_bits(np.array([[1.0, 1.0]])), wb, 7)
    assert out["cand_ids"][0].tolist() == [0, 1, 2, 3, 4, 5, 6]


# ----------------------------------------------------------------------------------
# Planted mistakes: each mutant of the module must fail a pin above.
# ----------------------------------------------------------------------------------

MUTANTS = {
    "ties_to_higher_id": ("np.lexsort((np.arange(V), -u[m]))", "np.lexsort((-np.arange(V), -u[m]))"),
    "lse_without_shift": ("lse = (mx + np.log(np.exp(u - mx).sum(axis=1, keepdims=True)))[:, 0]",
                          "lse = np.log(np.exp(u).sum(axis=1, keepdims=True))[:, 0]"),
    "last_block_dropped": ("for v0 in range(0, V, block):", "for v0 in range(0, V - block + 1, block):"),
    "logprob_sign": ("cand_logprob=val - lse[:, None]", "cand_logprob=val + lse[:, None]"),
    "bf16_truncated_to_8_bits": ("astype(np.uint32) << 16)", "astype(np.uint32) << 16) & np.uint32(0xFFFF0000) & np.uint32(0xFFF0FFFF)"),
    "head_row_offset": ("out[:, v0:v0 + block] = h @ bf16_to_f64(w_bits[v0:v0 + block]).T",
                        "out[:, v0:v0 + block] = h @ bf16_to_f64(w_bits[max(v0 - 1, 0):max(v0 - 1, 0) + min(block, V - v0)]).T"),
}


def _mutant(name: str) -> types.ModuleType:
    src = open(LH.__file__).read()
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mod = types.ModuleType(f"lm_head_{name}")
    exec(compile(src.replace(old, new, 1), mod.__name__, "exec"), mod.__dict__)
    return mod


PINS = [test_logits_are_exact_integer_arithmetic, test_logits_brute_force_random,
        test_candidates_match_the_c_oracle_on_exact_logits, test_lse_matches_scipy_and_handles_large_logits,
        test_zero_hidden_state_and_permuted_head, test_ties_go_to_the_lower_id]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    mod = _mutant(name)
    failures = 0
    for pin in PINS:
        try:
            with np.errstate(over="ignore", invalid="ignore"):
                pin(lib=mod)
        except Exception:  # noqa: BLE001 - any failure counts
            failures += 1
    assert failures > 0, f"mutant {name} passed every pin"
