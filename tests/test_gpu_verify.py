"""GPU parity of tree verification (ubt_tree_attention, ubt_verify_accept, ubt_commit_kv)
against the fp64 oracle in ``oracle/verify.py``, called through the C ABI.

Tolerance of the attention output, from the arithmetic: q.k runs on bf16 MFMA with fp32
accumulation (the products are exact, the sums round at 2^-24 relative); the softmax
weights are rounded to bf16 before the value product, a relative error of at most 2^-9
per weight, so |out - ref| <= 2^-9 * max|v| plus fp32 rounding.  The test allows
2^-8 * max|v| + 1e-5 (and one more bf16 rounding of the output, 2^-8 |ref|, for bf16
outputs).  lse uses the unrounded weights: 1e-4 absolute.  The acceptance walk and the
KV commit are integer / copy work and must be bit-exact."""
from __future__ import annotations

import math

import numpy as np
import pytest

import synth
from oracle import verify as V

pytestmark = pytest.mark.gpu


def _tree(rng, B: int, N: int, nn):
    """Random topological trees with distinct sibling tokens, their ancestor masks."""
    parent = np.full((B, N), -1, np.int32)
    token = np.full((B, N), -1, np.int32)
    words = (N + 31) // 32
    mask = np.zeros((B, N, words), np.uint32)
    for b in range(B):
        token[b, 0] = rng.integers(0, 1000)
        for n in range(1, int(nn[b])):
            parent[b, n] = rng.integers(max(0, n - 8), n)
            used = {int(token[b, c]) for c in range(1, n) if parent[b, c] == parent[b, n]}
            t = int(rng.integers(0, 1000))
            while t in used:
                t = int(rng.integers(0, 1000))
            token[b, n] = t
        for n in range(int(nn[b])):
            a = n
            while a >= 0:
                mask[b, n, a // 32] |= np.uint32(1 << (a % 32))
                a = int(parent[b, a])
    return parent, token, mask


def _run_attention(d, plen, mask, nn, scale, out_dtype, D):
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, dev_values

    kc = dev_values(d["k_cache"]) if d["k_cache"].shape[1] > 0 else None
    vc = dev_values(d["v_cache"]) if d["v_cache"].shape[1] > 0 else None
    out, lse = ubt.tree_attention(dev_values(d["q"]), kc, vc, dev_i32(plen), dev_values(d["k_tree"]),
                                  dev_values(d["v_tree"]), dev_i32(mask.view(np.int32)), dev_i32(nn), scale=scale,
                                  out_dtype=out_dtype)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64), lse.cpu().numpy().astype(np.float64)


def _check_attention(out, lse, ref, ref_lse, d, bf16_out: bool, seqs=None):
    seqs = range(out.shape[0]) if seqs is None else seqs
    vmax = max(np.abs(synth.bf16_bits_to_f32(d["v_tree"])).max(),
               np.abs(synth.bf16_bits_to_f32(d["v_cache"])).max() if d["v_cache"].size else 0.0)
    for b in seqs:
        tol = 2.0 ** -8 * vmax + 1e-5 + (2.0 ** -8 * np.abs(ref[b]) if bf16_out else 0.0)
        err = np.abs(out[b] - ref[b])
        assert np.all(err <= tol), f"sequence {b}: max error {err.max():.3g} (tolerance {np.max(tol):.3g})"
        fin = np.isfinite(ref_lse[b])
        assert np.array_equal(fin, np.isfinite(lse[b])), f"sequence {b}: lse -inf pattern differs"
        assert np.all(np.abs(lse[b][fin] - ref_lse[b][fin]) <= 1e-4), f"sequence {b}: lse differs"


@pytest.mark.parametrize("B,N,H,Hkv,D,Pmax,plen,nn", [
    (2, 17, 4, 2, 64, 40, (37, 0), (17, 9)),          # ragged prefix, empty prefix, partial tree
    (2, 65, 32, 8, 128, 100, (100, 33), (65, 64)),    # Qwen3-8B heads, budget 64
    (1, 129, 8, 8, 128, 64, (64,), (129,)),           # no grouping, budget 128 (5 mask words)
    (3, 33, 16, 2, 64, 70, (70, 1, 32), (33, 1, 20)),  # group of 8, a root-only tree
    (1, 1, 4, 4, 128, 0, (0,), (1,)),                 # root only, no context at all
    (2, 256, 4, 1, 128, 31, (31, 5), (256, 200)),      # largest tree: 8 mask words
    (1, 129, 8, 2, 128, 64, (64,), (129,)),           # 516 query rows per head: two row groups
    (2, 256, 16, 4, 64, 40, (40, 7), (256, 100)),      # 1024 rows per head: four groups, partial tree
])
@pytest.mark.parametrize("out_dtype", ["f32", "bf16"])
def test_tree_attention_small(B, N, H, Hkv, D, Pmax, plen, nn, out_dtype):
    import torch

    from gpu_util import say

    say(f"tree_attention B={B} N={N} H={H} Hkv={Hkv} D={D} P={plen} nn={nn} out={out_dtype}")
    rng = np.random.default_rng(1000 + N + D)
    plen, nn = np.array(plen, np.int32), np.array(nn, np.int32)
    _, _, mask = _tree(rng, B, N, nn)
    d = synth.verify_inputs(N * 7 + D, B, N, H, Hkv, D, Pmax)
    scale = 1.0 / math.sqrt(D)
    out, lse = _run_attention(d, plen, mask, nn, scale, torch.float32 if out_dtype == "f32" else torch.bfloat16, D)
    ref, ref_lse = V.tree_attention_fast(d["q"], d["k_cache"], d["v_cache"], plen, d["k_tree"], d["v_tree"], mask, nn,
                                         scale)
    _check_attention(out, lse, ref, ref_lse, d, out_dtype == "bf16")
    for b in range(B):
        assert not out[b, int(nn[b]):].any(), "rows past n_nodes must be zero"


def test_tree_attention_on_draft_trees():
    """Trees, masks and node counts from the draft step of the headline workload,
    attended over a 1000-token context with Qwen3-8B's head layout."""
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, dev_values, say, to_np

    w = synth.WORKLOADS[3]
    say("tree_attention on draft trees of workload 3, context 1000")
    di = synth.inputs(w, 0)
    step = ubt.DraftStep(w.B, w.gamma, w.V, w.K, w.W, w.budget, dev_values(di["phi"]), dev_values(di["psi"]),
                         dev_values(di["gate"]), dev_i32(di["anchor"]), di["alpha"], di["lam"], w.zeta)
    tree = to_np(step.run(dev_values(di["logits"])))
    torch.cuda.synchronize()
    H, Hkv, D, P = 32, 8, 128, 1000
    d = synth.verify_inputs(3, w.B, w.N, H, Hkv, D, P)
    plen = np.full(w.B, P, np.int32)
    out, lse = _run_attention(d, plen, tree["mask"], tree["n_nodes"], D ** -0.5, torch.float32, D)
    seqs = [0, 13, 31]
    ref, ref_lse = V.tree_attention_fast(d["q"], d["k_cache"], d["v_cache"], plen, d["k_tree"], d["v_tree"],
                                         tree["mask"], tree["n_nodes"], D ** -0.5, seqs=seqs)
    _check_attention(out, lse, ref, ref_lse, d, False, seqs=seqs)


def test_tree_attention_full_size_sampled():
    """The measured shape (B=32, budget 64, Qwen3-8B heads, 4096-token context), sampled
    sequences against the oracle."""
    import torch

    from gpu_util import say

    B, N, H, Hkv, D, P = 32, 65, 32, 8, 128, 4096
    say(f"tree_attention full size B={B} N={N} H={H} Hkv={Hkv} D={D} P={P}")
    rng = np.random.default_rng(77)
    nn = np.full(B, N, np.int32)
    _, _, mask = _tree(rng, B, N, nn)
    d = synth.verify_inputs(4096, B, N, H, Hkv, D, P)
    plen = np.array([P - (b % 3) * 17 for b in range(B)], np.int32)
    out, lse = _run_attention(d, plen, mask, nn, D ** -0.5, torch.bfloat16, D)
    seqs = [0, 1, 17, 31]
    ref, ref_lse = V.tree_attention_fast(d["q"], d["k_cache"], d["v_cache"], plen, d["k_tree"], d["v_tree"], mask,
                                         nn, D ** -0.5, seqs=seqs)
    _check_attention(out, lse, ref, ref_lse, d, True, seqs=seqs)


@pytest.mark.parametrize("B,N,follow", [(8, 65, 0.7), (16, 129, 0.9), (4, 256, 1.0), (3, 1, 1.0), (5, 33, 0.0)])
def test_verify_accept(B, N, follow):
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, say

    say(f"verify_accept B={B} N={N} follow={follow}")
    rng = np.random.default_rng(N + B)
    nn = np.array([N if b % 2 == 0 else max(1, N // 2) for b in range(B)], np.int32)
    parent, token, _ = _tree(rng, B, N, nn)
    target = synth.verify_targets(N, token, parent, nn, 1000, follow)
    g = ubt.verify_accept(dev_i32(token), dev_i32(parent), dev_i32(nn), dev_i32(target))
    torch.cuda.synchronize()
    alen, nodes, bonus = V.verify_accept(token, parent, nn, target)
    assert np.array_equal(g["accept_len"].cpu().numpy(), alen)
    assert np.array_equal(g["accept_nodes"].cpu().numpy(), nodes)
    assert np.array_equal(g["bonus"].cpu().numpy(), bonus)


def test_verify_accept_on_draft_trees():
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, dev_values, say, to_np

    w = synth.WORKLOADS[4]
    say("verify_accept on draft trees of workload 4")
    di = synth.inputs(w, 0)
    step = ubt.DraftStep(w.B, w.gamma, w.V, w.K, w.W, w.budget, dev_values(di["phi"]), dev_values(di["psi"]),
                         dev_values(di["gate"]), dev_i32(di["anchor"]), di["alpha"], di["lam"], w.zeta)
    tree = to_np(step.run(dev_values(di["logits"])))
    target = synth.verify_targets(44, tree["token"], tree["parent"], tree["n_nodes"], w.V, 0.8)
    g = ubt.verify_accept(dev_i32(tree["token"]), dev_i32(tree["parent"]), dev_i32(tree["n_nodes"]), dev_i32(target))
    torch.cuda.synchronize()
    alen, nodes, bonus = V.verify_accept(tree["token"], tree["parent"], tree["n_nodes"], target)
    assert np.array_equal(g["accept_len"].cpu().numpy(), alen)
    assert np.array_equal(g["accept_nodes"].cpu().numpy(), nodes)
    assert np.array_equal(g["bonus"].cpu().numpy(), bonus)
    assert alen.max() > 1, "the steered targets should accept some paths"


@pytest.mark.parametrize("D", [64, 128])
def test_commit_kv(D):
    import torch

    import paper_2609_39972_amd as ubt
    from gpu_util import dev_i32, dev_values, say

    B, N, Hkv, Pmax = 6, 65, 8, 300
    say(f"commit_kv B={B} N={N} Hkv={Hkv} D={D} Pmax={Pmax}")
    rng = np.random.default_rng(D)
    nn = np.full(B, N, np.int32)
    parent, token, _ = _tree(rng, B, N, nn)
    target = synth.verify_targets(D, token, parent, nn, 1000, 0.9)
    alen, nodes, _ = V.verify_accept(token, parent, nn, target)
    d = synth.verify_inputs(D + 1, B, N, 1, Hkv, D, Pmax)
    plen = np.array([0, 10, 299, 290, 150, 300], np.int32)  # one exactly full, two that overflow
    kc, vc = dev_values(d["k_cache"]), dev_values(d["v_cache"])
    pl = dev_i32(plen)
    ubt.commit_kv(dev_values(d["k_tree"]), dev_values(d["v_tree"]), dev_i32(nodes), dev_i32(alen), pl, kc, vc)
    torch.cuda.synchronize()
    rk, rv, rp = V.commit_kv(d["k_tree"], d["v_tree"], nodes, alen, plen, d["k_cache"], d["v_cache"])
    assert np.array_equal(pl.cpu().numpy(), rp)
    assert np.array_equal(kc.view(torch.int16).cpu().numpy().view(np.uint16), rk)
    assert np.array_equal(vc.view(torch.int16).cpu().numpy().view(np.uint16), rv)
