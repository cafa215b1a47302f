"""GPU test of ubt_draft_step_noalloc, the draft step for callers that cannot allocate:
its outputs must be bit-identical to ubt_draft_step's (the same kernels, with the
library's static per-device workspace instead of the caller's), on two calls in a row,
the second on a smaller input, so the shared array is reused with less of it in play.
Called through the C ABI."""
from __future__ import annotations

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu

KEYS = ("cand_ids", "cand_logit", "cand_logprob", "lse", "logq", "n_nodes", "token", "parent", "depth", "cand_rank",
        "score", "mask")


def _both(w: synth.Workload, buf: int = 0):
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, dev_values, say, to_np

    say(f"draft_step_noalloc vs draft_step: {w.describe()}")
    d = synth.inputs(w, buf)
    logits = dev_values(d["logits"])
    args = (dev_values(d["phi"]), dev_values(d["psi"]), dev_values(d["gate"]), dev_i32(d["anchor"]), d["alpha"],
            d["lam"], w.K, w.W, w.budget, w.zeta)
    ws = ubt.draft_step_workspace(w.B, w.gamma, w.V, w.K, logits.dtype)
    ref = to_np(ubt.draft_step(logits, *args, workspace=ws))
    torch.cuda.synchronize()
    assert ubt.draft_step_error(ws) == 0
    got = to_np(ubt.draft_step_noalloc(logits, *args))
    torch.cuda.synchronize()
    for k in KEYS:
        a, b = ref[k], got[k]
        if a.dtype == np.float32:
            a, b = a.view(np.uint32), b.view(np.uint32)
        assert np.array_equal(a, b), f"{k} differs between ubt_draft_step_noalloc and ubt_draft_step"
    assert (got["n_nodes"] >= 1).all()
    return got


def test_noalloc_matches_draft_step_twice():
    """The headline workload, then a smaller one (fewer sequences, rows and candidates)."""
    big = synth.WORKLOADS[3]
    small = synth.custom(500, B=5, L=7, V=20000, K=4, r=32, budget=20, W=4, dtype="bf16", feat_dtype="bf16",
                         logits="zipf")
    a = _both(big)
    b = _both(small)
    assert a["n_nodes"].shape[0] == 32 and b["n_nodes"].shape[0] == 5


def test_noalloc_separate_kernel_shape():
    """A shape the one launch does not take (K = 5): the separate kernels, no scratch."""
    w = synth.custom(501, B=2, L=6, V=10000, K=5, r=32, budget=20, W=4, dtype="bf16", feat_dtype="bf16",
                     logits="normal", logit_std=2.0)
    _both(w)


def test_noalloc_k64_twice():
    """K = 64 (the selector and the search in one launch, ready words in the static array):
    the paper's shape at B = 32, then a smaller one."""
    big = synth.WORKLOADS[6]
    small = synth.custom(502, B=3, L=5, V=8000, K=64, r=64, budget=30, W=8, dtype="bf16", feat_dtype="bf16",
                         logits="zipf")
    a = _both(big)
    b = _both(small)
    assert a["n_nodes"].shape[0] == 32 and b["n_nodes"].shape[0] == 3
