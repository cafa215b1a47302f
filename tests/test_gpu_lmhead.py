"""GPU parity of the LM-head projection fused with the candidate sets (ubt_lm_head_topk)
against the fp64 oracle, through the C ABI.

* Integer-valued hidden states and head rows: every logit is an exact integer in fp32,
  whatever the accumulation order, so ids and logits must match bit for bit, and the many
  equal logits test the tie order (id asc) across tiles, waves and workgroups.  Hidden
  sizes cover both kernels: the one that splits d over a workgroup's waves (d a multiple
  of 512, every slice width) and the one that does not.
* Gaussian operands at the drafting block of the paper's latency breakdown (16 rows of a
  2560-wide hidden state against a 151,936-token head), at d = 4096, and at small and
  ragged shapes (M not a multiple of 16, V not a multiple of 16, d/32 odd): logits within
  the derived fp32 accumulation bound, the candidate order valid under it.
* Degenerate cases: h = 0 (every logit 0), K = V, K = 1, one row; reuse of a workspace
  across calls of different shapes and kernels."""
from __future__ import annotations

import math

import numpy as np
import pytest

import parity
import synth

pytestmark = pytest.mark.gpu


def _run(h_bits, w_bits, K, workspace=None):
    import torch

    import paper_2609_39972_amd as ubt

    h = ubt.bf16_tensor_from_bits(h_bits)
    w = ubt.bf16_tensor_from_bits(w_bits)
    out = ubt.lm_head_topk(h, w, K, workspace=workspace)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items() if v is not None}


def _int_bits(M, d, V, seed, lo=-8, hi=8):
    rng = np.random.default_rng(seed)
    h = rng.integers(lo, hi + 1, size=(M, d)).astype(np.float64)
    w = rng.integers(lo, hi + 1, size=(V, d)).astype(np.float64)
    return synth.round_bf16_bits(h), synth.round_bf16_bits(w)


@pytest.mark.parametrize("M,d,V,K", [
    # d not a multiple of 512: one wave per tile over the whole of d
    (1, 32, 64, 1), (5, 96, 1000, 8), (16, 256, 4099, 64), (17, 64, 2500, 16), (33, 128, 777, 64),
    # d a multiple of 512: the eight waves of a workgroup split d (every slice width built)
    (3, 2560, 3000, 64), (2, 1024, 3001, 64), (16, 1536, 4099, 64), (17, 2048, 1500, 16), (5, 3072, 999, 8),
    (5, 3584, 2000, 8), (1, 4096, 130, 64), (1, 5120, 777, 64), (20, 2560, 70001, 64),
])
def test_lm_head_integer_inputs_exact(M, d, V, K):
    print(f"lm_head exact M={M} d={d} V={V} K={K}", flush=True)
    hb, wb = _int_bits(M, d, V, seed=M * 1000 + d + V)
    g = _run(hb, wb, K)
    parity.check_lm_head(g, hb, wb, K, exact=True)


def test_lm_head_ties_in_many_workgroups():
    """Heads with only a few distinct rows: most logits tie, across every workgroup."""
    print("lm_head ties", flush=True)
    rng = np.random.default_rng(7)
    base = rng.integers(-4, 5, size=(3, 64)).astype(np.float64)
    wb = synth.round_bf16_bits(base[rng.integers(0, 3, size=20011)])
    hb = synth.round_bf16_bits(rng.integers(-4, 5, size=(9, 64)).astype(np.float64))
    parity.check_lm_head(_run(hb, wb, 64), hb, wb, 64, exact=True)


@pytest.mark.parametrize("M,d,V,K,seed", [
    (15, 2560, 151936, 64, 1),   # the drafting block of the paper's latency breakdown
    (16, 4096, 151936, 64, 2),
    (1, 64, 1000, 8, 3),
    (17, 96, 5003, 16, 4),
    (40, 256, 20000, 64, 5),
    (3, 2560, 32000, 1, 6),
])
def test_lm_head_gaussian(M, d, V, K, seed):
    print(f"lm_head gaussian M={M} d={d} V={V} K={K} seed={seed}", flush=True)
    x = synth.lm_head_inputs(seed, M, d, V)
    counts = parity.check_lm_head(_run(x["h"], x["w"], K), x["h"], x["w"], K)
    parity.record(f"lm_head M={M} d={d} V={V} K={K}", {"exact": counts["exact"], "excused": counts["excused"]})


def test_lm_head_zero_hidden_state():
    """h = 0: every logit is 0, so C = ids 0..K-1 and LSE = ln V."""
    print("lm_head zero h", flush=True)
    V, d = 70001, 128
    x = synth.lm_head_inputs(8, 1, d, V)
    hb = np.zeros((4, d), np.uint16)
    g = _run(hb, x["w"], 64)
    np.testing.assert_array_equal(g["cand_ids"], np.tile(np.arange(64), (4, 1)))
    np.testing.assert_array_equal(g["cand_logit"], 0.0)
    np.testing.assert_allclose(g["lse"], math.log(V), rtol=1e-6)
    np.testing.assert_allclose(g["cand_logprob"], -math.log(V), rtol=1e-6)


def test_lm_head_k_equals_v():
    print("lm_head K = V", flush=True)
    x = synth.lm_head_inputs(9, 6, 64, 64)
    g = _run(x["h"], x["w"], 64)
    parity.check_lm_head(g, x["h"], x["w"], 64)
    assert all(sorted(r.tolist()) == list(range(64)) for r in g["cand_ids"])


def test_lm_head_workspace_reuse():
    """One workspace (sized for the larger call) serves calls of different shapes in a
    row; nothing carries over between them."""
    import paper_2609_39972_amd as ubt

    print("lm_head workspace reuse", flush=True)
    ws = ubt.lm_head_workspace(40, 128, 50000, 64)
    a = synth.lm_head_inputs(10, 40, 128, 50000)
    b = synth.lm_head_inputs(11, 7, 128, 3001)
    for x, K in ((a, 64), (b, 8), (a, 64)):
        parity.check_lm_head(_run(x["h"], x["w"], K, workspace=ws), x["h"], x["w"], K)


def test_lm_head_workspace_reuse_across_shapes():
    """One workspace serves calls with different numbers of row groups, hidden sizes and
    kernels in any order: nothing in it is read before the call writes it."""
    import paper_2609_39972_amd as ubt

    print("lm_head workspace reuse across shapes", flush=True)
    cases = [(40, 2560, 30011, 64), (5, 2560, 9000, 8), (17, 1024, 20000, 16), (3, 96, 3000, 4), (40, 2560, 30011, 64)]
    n = max(ubt.lib().ubt_lm_head_topk_workspace_bytes(M, d, V, K) for M, d, V, K in cases)
    import torch
    ws = torch.full((n,), 0xA5, dtype=torch.uint8, device="cuda")  # stale bytes must not matter
    for i, (M, d, V, K) in enumerate(cases):
        x = synth.lm_head_inputs(20 + i, M, d, V)
        parity.check_lm_head(_run(x["h"], x["w"], K, workspace=ws), x["h"], x["w"], K)
