"""GPU tests of ubt_draft_tree: the selector and the tree search in one call must give
bit-identical logq and trees to ubt_bigram_scores followed by ubt_build_tree (whose
parity with the oracle the pipeline and tree tests establish), on the five workloads,
at their width and at the exact best-first width, and on shapes that exercise the
one-launch kernel's edges (fewer positions than waves, several positions per wave,
every K it handles, a depth bonus, and the two-launch fallback)."""
from __future__ import annotations

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu

TREE_KEYS = ("n_nodes", "token", "parent", "depth", "cand_rank", "score", "mask")


def _both(w: synth.Workload, W: int, buf: int = 0) -> tuple[dict, dict]:
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, dev_values, say, to_np

    say(f"fused vs separate: workload {w.cfg} W={W}: {w.describe()}")
    d = synth.inputs(w, buf)
    args = (w.B, w.gamma, w.V, w.K, W, w.budget, dev_values(d["phi"]), dev_values(d["psi"]), dev_values(d["gate"]),
            dev_i32(d["anchor"]), d["alpha"], d["lam"], w.zeta)
    logits = dev_values(d["logits"])
    sep = ubt.DraftStep(*args, fused=False)
    fus = ubt.DraftStep(*args, fused=True, one_call=False)
    assert fus.fused and not sep.fused
    a = to_np(sep.run(logits))
    torch.cuda.synchronize()
    b = to_np(fus.run(logits))
    torch.cuda.synchronize()
    return a, b


def _same(a: dict, b: dict) -> None:
    for k in ("cand_ids", "logq") + TREE_KEYS:
        assert a[k].dtype == b[k].dtype
        if a[k].dtype == np.float32:
            assert np.array_equal(a[k].view(np.uint32), b[k].view(np.uint32)), f"{k} differs"
        else:
            assert np.array_equal(a[k], b[k]), f"{k} differs"


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6])
def test_fused_workload(cfg):
    w = synth.WORKLOADS[cfg]
    _same(*_both(w, w.W))


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6])
def test_fused_best_first_width(cfg):
    w = synth.WORKLOADS[cfg]
    _same(*_both(w, w.budget))


@pytest.mark.parametrize("kw", [
    dict(B=3, L=3, K=4, r=16, budget=5, W=3),                 # 2 positions: 2 waves
    dict(B=2, L=9, K=8, r=32, budget=20, W=4),                # 8 positions: one per wave
    dict(B=3, L=10, K=16, r=32, budget=40, W=6),              # 9 positions: wave 0 takes two
    dict(B=2, L=33, K=8, r=64, budget=100, W=10),             # 32 positions: four per wave
    dict(B=2, L=65, K=4, r=16, budget=255, W=16),             # 64 positions, gamma * W = 1024
    dict(B=2, L=6, K=16, r=48, budget=60, W=32),              # W * K = 512
    dict(B=2, L=7, K=8, r=32, budget=30, W=5, zeta=-0.75),    # depth bonus
    dict(B=2, L=6, K=5, r=32, budget=20, W=4),                # K outside {4, 8, 16}: two launches
    dict(B=2, L=6, K=8, r=32, budget=40, W=65),               # W > 64: two launches
])
def test_fused_edges(kw):
    w = synth.custom(200, V=3000, dtype="bf16", feat_dtype="bf16", logits="normal", logit_std=2.0, **kw)
    _same(*_both(w, w.W))
