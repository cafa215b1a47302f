"""GPU tests of ubt_draft_step, the whole step in one launch (rows swept depth by depth in
chunks beside per-sequence searchers that merge the chunks and search as the rows come
out).

Every case is checked against the fp64 oracle: candidate ids bit-exact, LSE, log-probs
and logq within the fp32 score tolerance, and the trees exact or within the 1e-5 tie
gap.  The guided tie check needs the supertree F_d, which only ubt_build_tree can dump:
the one-launch outputs are first shown bit-identical to ubt_topk + ubt_bigram_scores +
ubt_build_tree (candidates, logq, tree and mask), then validated with that path's dump.

Also: the workspace error word is clear and every row counter reset after every call,
repeated calls on one workspace give identical bits, graph replays match eager calls,
and the shapes that stress the split (ties across many tiles, rows whose top elements sit
late in the row, few tiles per row, a last chunk shorter than K, fp32 logits, one
position, 64 sequences) and the fallback to the separate calls."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import parity
import synth

pytestmark = pytest.mark.gpu

EXACT_KEYS = ("cand_ids", "cand_logit", "logq", "n_nodes", "token", "parent", "depth", "cand_rank", "score", "mask")


def _args(w: synth.Workload, d: dict, W: int):
    from gpu_util import dev_i32, dev_values

    return (w.B, w.gamma, w.V, w.K, W, w.budget, dev_values(d["phi"]), dev_values(d["psi"]), dev_values(d["gate"]),
            dev_i32(d["anchor"]), d["alpha"], d["lam"], w.zeta)


def _logits_tensor(w: synth.Workload, d: dict):
    from gpu_util import dev_values

    return dev_values(d["logits"])


def _run_both(w: synth.Workload, d: dict, W: int) -> tuple[dict, dict, object]:
    """The separate calls (with the supertree dump) and the one-launch call on the same
    inputs."""
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import to_np

    args = _args(w, d, W)
    logits = _logits_tensor(w, d)
    dtype = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    sep = ubt.DraftStep(*args, fused=False, debug=True)
    one = ubt.DraftStep(*args, one_call=True, logit_dtype=dtype)
    a = to_np(sep.run(logits))
    torch.cuda.synchronize()
    b = to_np(one.run(logits))
    one.check()
    return a, b, one


def _check_workspace(step) -> None:
    """The error word is clear and every row's chunk counter is back to zero."""
    B, gamma = step.shape[:2]
    ws = step.workspace.cpu().numpy()
    assert ws.size >= 256 + B * gamma * 4
    assert int(ws[:4].view(np.uint32)[0]) == 0, "a wait inside the launch timed out"
    assert not ws[256:256 + B * gamma * 4].any(), "row counters were not reset"


def _same(a: dict, b: dict, logit_dtype: str) -> None:
    for k in EXACT_KEYS:
        assert a[k].dtype == b[k].dtype
        if a[k].dtype == np.float32:
            assert np.array_equal(a[k].view(np.uint32), b[k].view(np.uint32)), f"{k} differs"
        else:
            assert np.array_equal(a[k], b[k]), f"{k} differs"
    # LSE and log-probs: fp32 sums in another order.
    for k in ("lse", "cand_logprob"):
        ref = a[k].astype(np.float64)
        assert np.all(np.abs(b[k] - ref) <= 1e-5 * np.maximum(1.0, np.abs(ref))), f"{k} differs beyond 1e-5"


def check_vs_oracle(w: synth.Workload, W: int, d: dict, sep: dict, one: dict) -> dict:
    """The one-launch outputs against the oracle pipeline; `sep` (bit-identical to `one`
    on the tree) supplies the supertree dump for the guided tie check.  Returns the tree
    counts (exact / excused)."""
    ref = oracle.pipeline(d["logits"], d["phi"], d["psi"], d["gate"], d["anchor"], d["alpha"], d["lam"], w.K, W,
                          w.budget, w.zeta)
    parity.check_topk(one, ref)
    parity.check_selector({"logq": one["logq"]}, ref)
    g = dict(one)
    for k in ("f_count", "f_parent", "f_cand", "f_score"):
        g[k] = sep[k]
    return parity.check_tree(g, ref, ref["logq"], ref["cand_ids"], d["anchor"], W, w.budget, w.zeta)


def _check(w: synth.Workload, W: int, d: dict | None = None, buf: int = 0) -> dict:
    from gpu_util import say

    say(f"draft_step workload {w.cfg} buf={buf} W={W}: {w.describe()}")
    if d is None:
        d = synth.inputs(w, buf)
    a, b, one = _run_both(w, d, W)
    _same(a, b, w.dtype)
    if one.workspace is not None:
        _check_workspace(one)
    counts = check_vs_oracle(w, W, d, a, b)
    parity.record(f"draft_step wl{w.cfg} W={W}", counts)
    say(f"  trees vs oracle: {counts}")
    return counts


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6])
def test_step_workload(cfg):
    w = synth.WORKLOADS[cfg]
    _check(w, w.W)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_step_best_first_width(cfg):
    w = synth.WORKLOADS[cfg]
    _check(w, w.budget)


def test_step_repeat_and_pool():
    """One workspace, consecutive calls over different logit buffers and back: bitwise
    identical results for the same input, and the workspace clean after each."""
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import say, to_np

    w = synth.WORKLOADS[3]
    say("draft_step repeat: workload 3, buffers 0, 1, 0")
    d0, d1 = synth.inputs(w, 0), synth.inputs(w, 1)
    one = ubt.DraftStep(*_args(w, d0, w.W), one_call=True)
    r0 = to_np(one.run(_logits_tensor(w, d0)))
    torch.cuda.synchronize()
    _check_workspace(one)
    r1 = to_np(one.run(_logits_tensor(w, d1)))
    torch.cuda.synchronize()
    _check_workspace(one)
    r2 = to_np(one.run(_logits_tensor(w, d0)))
    torch.cuda.synchronize()
    _check_workspace(one)
    for k in r0:
        assert np.array_equal(r0[k], r2[k]), f"{k} differs between identical calls"
    assert not np.array_equal(r0["cand_ids"], r1["cand_ids"])
    # The step holds buffer 0's gate and anchor; only the logits come from buffer 1.
    ref1 = oracle.pipeline(d1["logits"], d0["phi"], d0["psi"], d0["gate"], d0["anchor"], d0["alpha"], d0["lam"], w.K,
                           w.W, w.budget, w.zeta)
    parity.check_topk(r1, ref1)
    parity.check_selector({"logq": r1["logq"]}, ref1)


def test_step_graph_replay():
    """The step captured in a HIP graph: every replay, with eager work in between,
    matches the eager call."""
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import say, to_np

    w = synth.WORKLOADS[3]
    say("draft_step graph replay: workload 3")
    d = synth.inputs(w, 0)
    logits = _logits_tensor(w, d)
    one = ubt.DraftStep(*_args(w, d, w.W), one_call=True)
    ref = to_np(one.run(logits))
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        one.run(logits)  # warm-up on the capture stream
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=s):
            out = one.run(logits)
    torch.cuda.synchronize()
    for _ in range(3):
        for v in out.values():
            if v is not None:
                v.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        got = to_np(out)
        for k in ref:
            assert np.array_equal(ref[k], got[k]), f"{k} differs after a graph replay"
        _check_workspace(one)
        one.run(logits)  # eager call between replays
        torch.cuda.synchronize()


def _custom(cfg: int, **kw) -> synth.Workload:
    base = dict(V=20000, dtype="bf16", feat_dtype="bf16", logits="normal", logit_std=2.0, K=8, r=32, budget=24, W=6)
    base.update(kw)
    return synth.custom(cfg, **base)


@pytest.mark.parametrize("kw", [
    dict(B=3, L=4),                                   # few rows
    dict(B=1, L=2, K=16, W=8, budget=40),             # one position
    dict(B=2, L=9, V=5000, K=4, W=3, budget=12),      # 3 tiles per row
    dict(B=2, L=9, V=16384 + 8, K=8),                 # a ragged last tile of 8 elements
    dict(B=2, L=5, V=8192 + 8, K=16, W=8, budget=40), # a last chunk of 8 elements, fewer than K
    dict(B=64, L=3, V=3000, K=4, W=4, budget=16),     # 64 searchers
    dict(B=8, L=33, V=6000, K=8, W=8, budget=64),     # 32 positions over 7 helper waves
    dict(B=2, L=65, V=4000, K=4, W=8, budget=100),    # the longest block (gamma = 64)
    dict(B=2, L=6, V=30000, dtype="f32", feat_dtype="bf16", K=8),  # fp32 logits
    dict(B=2, L=6, V=10000, K=16, W=32, budget=60),   # W * K = 512
    dict(B=2, L=6, V=10000, K=5, W=4, budget=20),     # K outside {4, 8, 16}: the separate calls
    dict(B=2, L=6, V=10001, K=8, W=4, budget=20),     # V * 2 bytes not a multiple of 16
    # K = 64: the sweep, then the selector and the four-wave search in one launch
    dict(B=2, L=7, V=6000, K=64, W=12, r=256, budget=64),   # the paper's search shape, fewer positions
    dict(B=3, L=2, V=3000, K=64, W=4, r=64, budget=20),     # one position (no slab two depths ahead)
    dict(B=2, L=17, V=5000, K=64, W=16, r=48, budget=120),  # W = 16, 16 positions, fewer k-steps than waves
    dict(B=2, L=9, V=6000, K=64, W=16, r=32, budget=16),    # W = budget
])
def test_step_shapes(kw):
    w = _custom(300, **kw)
    _check(w, w.W)


def test_step_ties_everywhere():
    """Constant rows and rows with long runs of equal top values: waves hold more
    groups at the threshold than their buffers keep and scan again; ids must come out
    lowest first."""
    w = _custom(301, B=2, L=5, V=40000)
    d = synth.inputs(w, 0)
    lg = d["logits"].copy()
    lg[0, 0, :] = lg[0, 0, 0]                      # constant row
    lg[0, 1, :] = lg[0, 1, :].min()                # floor everywhere ...
    lg[0, 1, 25000:25000 + 3000] = lg[0, 1, 5]     # ... and a run of 3000 equal values late in the row
    lg[1, 2, ::7] = lg[1, 2, 3]                    # every 7th element equal
    d["logits"] = lg
    _check(w, w.W, d=d)


def test_step_top_outside_samples():
    """Rows whose largest values all sit far from the first tiles."""
    w = _custom(302, B=2, L=5, V=60000, K=16, W=8, budget=40)
    d = synth.inputs(w, 0)
    lg = d["logits"].copy()
    rng = np.random.default_rng(7)
    for b in range(w.B):
        for i in range(w.gamma):
            idx = rng.choice(np.arange(40000, 60000), size=40, replace=False)
            lg[b, i, idx] = synth.store(np.full(40, 12.0) + rng.normal(0, 0.5, 40), w.dtype)
    d["logits"] = lg
    _check(w, w.W, d=d)


def test_step_neg_inf():
    """Rows that are mostly -inf (bf16 0xFF80), with a few finite values in late tiles."""
    w = _custom(303, B=2, L=4, V=30000, K=8)
    d = synth.inputs(w, 0)
    lg = d["logits"].copy()
    lg[0, 0, :] = 0xFF80
    lg[0, 0, 29990:] = synth.store(np.linspace(-1, 1, 10), "bf16")
    lg[1, 1, 100:] = 0xFF80
    d["logits"] = lg
    _check(w, w.W, d=d)
