"""Benchmark of one UBTree draft step on one MI355X.

A step is the whole hot path on one batch of synthetic proposer outputs: softmax
statistics and top-K over the vocabulary, selector scores and normalisation, beam
search, pruning, tree and ancestor mask.  By default it is one ubt_draft_step call (one
launch: rows swept in depth order beside per-sequence searchers); ``--mode tree`` runs
ubt_topk then ubt_draft_tree (selector and search in one launch), ``--mode separate`` the
three calls ubt_topk, ubt_bigram_scores and ubt_build_tree.  Steps rotate over a pool of distinct logit buffers whose total size
exceeds the 256 MB last-level cache, so every step reads its logits from HBM.  Inputs
are resident in HBM before the timed region; the steps are captured once into a HIP
graph and replayed.

Prints one JSON line: trees/s (value), ms per step, the dominant kernel's achieved HBM
bandwidth against the 8 TB/s peak (roofline: the one-launch step kernel in step mode, else
the sweep; the sweep alone is reported beside it), and the fp64 oracle timed on the host
cores (cpu_baseline).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "draft trees/sec and µs/step at B=32, V=151936; achieved HBM GB/s vs peak"
HBM_PEAK_GBPS = 8000.0
POOL_BYTES = 512 << 20  # pool size that defeats the 256 MB Infinity Cache
SWEEP_KERNEL = "topk_row_kernel"
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "topk_sweep_zipf-v151936-b32_counters.md")
SWEEP_SOURCES = ("topk.hip", "sweep.h", "sweep_big.h", "ubt_device.h")
STEP_KERNEL = "draft_pipe_kernel"
STEP_PROFILE = os.path.join(ROOT, "profiles", "draft_step_pipe_zipf-v151936-b32_counters.md")
STEP_SOURCES = ("step.hip", "sweep.h", "search.h", "pipe_search.h", "bigram_tile.h", "ubt_device.h")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


VERIFY_PROFILE = os.path.join(ROOT, "profiles", "tree_attention_verify-b32-n65-p4096.md")
VERIFY_SOURCES = ("verify.hip", "ubt_device.h")
LOSS_PROFILE = os.path.join(ROOT, "profiles", "kl_loss_zipf-v151936-b32.md")
LOSS_SOURCES = ("loss.hip", "ubt_device.h")
LMHEAD_PROFILE = os.path.join(ROOT, "profiles", "lm_head_topk_m15-d2560-v151936-k64.md")
LMHEAD_SOURCES = ("lmhead.hip", "search.h", "bigram_tile.h", "ubt_device.h")


def source_hash(files=SWEEP_SOURCES) -> str:
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2609_39972_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(profile: str = TRAFFIC_PROFILE, files=SWEEP_SOURCES) -> dict | None:
    """HBM bytes per launch of a dominant kernel from its committed counter summary, if
    that summary was taken on the kernel's current source."""
    if not os.path.exists(profile):
        return None
    txt = open(profile).read()
    m_hash = re.search(r"source hash:\s*`?([0-9a-f]{16})", txt)
    m_bytes = re.search(r"hbm bytes per launch:\s*([0-9.eE+]+)", txt)
    if not (m_hash and m_bytes) or m_hash.group(1) != source_hash(files):
        return None
    return {"bytes": float(m_bytes.group(1))}


def one_launch_step(w, dev) -> bool:
    """Whether ubt_draft_step runs the workload as its one-launch kernel: 16-byte aligned
    rows, bf16 features, K in {4, 8, 16} with the register-resident search shape, at most
    64 sequences and fewer sequences than compute units."""
    import torch

    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    shape = (w.W * w.K <= 512 and w.W <= 64 and w.gamma * w.W <= 1024)
    return (w.feat_dtype == "bf16" and w.K in (4, 8, 16) and shape and w.B <= 64 and w.B < cus
            and (w.V * (2 if w.dtype == "bf16" else 4)) % 16 == 0)


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, d, min_seconds: float) -> tuple[dict, dict]:
    """The fp64 oracle on pool buffer 0: full steps on the host threads for at least
    `min_seconds`, then one step on one thread.  Returns the baseline and the oracle's
    outputs of the first step (the parity reference)."""
    import oracle

    threads = oracle.default_threads()
    args = (d["logits"], d["phi"], d["psi"], d["gate"], d["anchor"], d["alpha"], d["lam"], w.K, w.W, w.budget, w.zeta)
    reps, t0, ref = 0, time.perf_counter(), None
    while True:
        out = oracle.pipeline(*args, threads=threads)
        ref = out if ref is None else ref
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds:
            break
    t1 = time.perf_counter()
    oracle.pipeline(*args, threads=1)
    el1 = time.perf_counter() - t1
    return {"value": round(reps * w.B / el, 3), "unit": "trees/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} full step(s) of the workload ({reps * w.B} trees, {reps * w.rows} logit rows) on "
                      f"pool buffer 0, fp64 C++ oracle, {threads} threads, {el:.1f} s",
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "single_thread": {"value": round(w.B / el1, 3), "unit": "trees/s",
                              "sample": f"1 full step ({w.B} trees) on 1 thread, {el1:.2f} s"}}, ref


EXACT_KEYS = ("cand_ids", "cand_logit", "logq", "n_nodes", "token", "parent", "depth", "cand_rank", "score", "mask")


def step_parity(w, d, step, logits, ref) -> dict:
    """The timed step's outputs for pool buffer 0 (left by the last graph replay) against
    the oracle's: candidate ids exact, LSE, log-probs and logq within 1e-5 * max(1, |ref|),
    and each tree exact or within the 1e-5 tie gap.  The guided tie check reads the
    supertree, which only the separate calls can dump: their outputs on the same logits
    must first be bit-identical to the timed step's.  Counts trees."""
    import numpy as np
    import torch

    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import parity

    import paper_2609_39972_amd as ubt

    got = {k: v.detach().cpu().numpy() for k, v in step.outputs().items() if v is not None}
    got["mask"] = got["mask"].view(np.uint32)
    B, gamma, V, K, W, budget = step.shape
    sep = ubt.DraftStep(B, gamma, V, K, W, budget, step.phi, step.psi, step.gate, step.anchor, step.alpha, step.lam,
                        step.zeta, fused=False, debug=True)
    dump = {k: v.detach().cpu().numpy() for k, v in sep.run(logits).items() if v is not None}
    torch.cuda.synchronize()
    dump["mask"] = dump["mask"].view(np.uint32)
    same = all(np.array_equal(np.asarray(got[k]).view(np.uint32) if got[k].dtype == np.float32 else got[k],
                              np.asarray(dump[k]).view(np.uint32) if dump[k].dtype == np.float32 else dump[k])
               for k in EXACT_KEYS)
    g = dict(got)
    for k in ("f_count", "f_parent", "f_cand", "f_score"):
        g[k] = dump[k]
    counts = {"exact": 0, "excused": 0, "failed": 0}
    first_failure = None
    for b in range(B):
        try:
            if not same:
                raise AssertionError("the timed step's outputs differ from the separate calls'")
            sub = {k: got[k][b:b + 1] for k in ("cand_ids", "cand_logit", "cand_logprob", "lse")}
            parity.check_topk(sub, {k: ref[k][b:b + 1] for k in ("cand_ids", "cand_logit", "cand_logprob", "lse")})
            parity.close(got["logq"][b], ref["logq"][b], "logq")
            c = parity.check_tree(g, {k: ref[k][b:b + 1] for k in ("n_nodes", "parent", "cand_rank", "token", "mask",
                                                                  "score")},
                                  ref["logq"][b:b + 1], ref["cand_ids"][b:b + 1], d["anchor"][b:b + 1], W, budget,
                                  w.zeta, seqs=[b])
            counts["exact"] += c["exact"]
            counts["excused"] += c["excused"]
        except AssertionError as e:
            counts["failed"] += 1
            first_failure = first_failure or f"sequence {b}: {e}"
    out = {**counts, "trees": B, "sample": f"pool buffer 0 ({B} trees) of the timed step vs the fp64 oracle",
           "tie_gap": 1e-5}
    if first_failure:
        out["first_failure"] = first_failure[:300]
    return out


MFMA_BF16_PEAK_TFLOPS = 2500.0
VERIFY_SHAPE = dict(B=32, N=65, H=32, Hkv=8, D=128, P=4096)  # budget 64; Qwen3-8B attention heads


def bench_verify(args, dev) -> int:
    """Tree verification on one batch of draft trees: ubt_tree_attention over a 4096-token
    context (the dominant kernel), ubt_verify_accept and ubt_commit_kv.  The trees and
    masks come from the headline draft step; queries, keys and values are synthetic."""
    import numpy as np
    import torch

    import paper_2609_39972_amd as ubt
    import synth

    S = VERIFY_SHAPE
    B, N, H, Hkv, D, P = S["B"], S["N"], S["H"], S["Hkv"], S["D"], S["P"]
    w = synth.WORKLOADS[3]
    assert w.B == B and w.N == N
    di = synth.inputs(w, 0)
    bits = lambda a: ubt.bf16_tensor_from_bits(a, dev)
    step = ubt.DraftStep(w.B, w.gamma, w.V, w.K, w.W, w.budget, bits(di["phi"]), bits(di["psi"]), bits(di["gate"]),
                         torch.from_numpy(di["anchor"]).to(dev), di["alpha"], di["lam"], w.zeta)
    tree = step.run(bits(di["logits"]))
    torch.cuda.synchronize()
    d = synth.verify_inputs(1, B, N, H, Hkv, D, P + N)  # cache room for the committed path
    q, kc, vc, kt, vt = (bits(d[k]) for k in ("q", "k_cache", "v_cache", "k_tree", "v_tree"))
    plen0 = torch.full((B,), P, dtype=torch.int32, device=dev)
    out = torch.empty(B, N, H, D, dtype=torch.bfloat16, device=dev)
    lse = torch.empty(B, N, H, dtype=torch.float32, device=dev)
    tok, par, nn, mask = tree["token"], tree["parent"], tree["n_nodes"], tree["mask"]
    target = torch.from_numpy(synth.verify_targets(5, tok.cpu().numpy(), par.cpu().numpy(), nn.cpu().numpy(), w.V,
                                                   0.8)).to(dev)
    acc = ubt.verify_accept(tok, par, nn, target)
    plen = plen0.clone()
    stream = torch.cuda.Stream(device=dev)

    def timed(fn, n=50, replays=4):
        with torch.cuda.stream(stream):
            fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for _ in range(n):
                fn()
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            g.replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            a.record(stream)
            for _ in range(replays):
                g.replay()
            b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / (n * replays)

    n_att = max(8, args.steps // 20)
    att_us = timed(lambda: ubt.tree_attention(q, kc, vc, plen0, kt, vt, mask, nn, out=out, lse=lse, stream=stream),
                   n=n_att)
    acc_us = timed(lambda: ubt.verify_accept(tok, par, nn, target, out=acc, stream=stream))

    def commit():
        plen.copy_(plen0)
        ubt.commit_kv(kt, vt, acc["accept_nodes"], acc["accept_len"], plen, kc, vc, stream=stream)
    commit_us = timed(commit)

    # Algorithmic work of one attention launch: each (node, head) reads the context and
    # its ancestors once: 2 * D multiply-adds per key for q.k and as many for p.v.
    m = mask.cpu().numpy().view(np.uint32)
    vis = np.unpackbits(m.view(np.uint8), axis=-1, bitorder="little")[..., :N].sum(axis=-1)  # [B, N]
    nn_h = nn.cpu().numpy()
    keys = sum(int(P * nn_h[b] + vis[b, :nn_h[b]].sum()) for b in range(B))
    flops = 4.0 * D * H * keys
    kv_bytes = B * (P + N) * Hkv * D * 2 * 2
    io_bytes = B * N * H * D * 2 * 2 + B * N * H * 4 + m.nbytes
    att_bytes = kv_bytes + io_bytes
    tflops = flops / (att_us * 1e-6) / 1e12
    gbps = att_bytes / (att_us * 1e-6) / 1e9
    t_hbm = att_bytes / (HBM_PEAK_GBPS * 1e9)
    t_mfma = flops / (MFMA_BF16_PEAK_TFLOPS * 1e12)
    bound = "hbm" if t_hbm >= t_mfma else "mfma"
    log(f"tree attention {att_us:.2f} us: {gbps:.0f} GB/s, {tflops:.1f} TFLOP/s (HBM floor {t_hbm * 1e6:.1f} us, "
        f"MFMA floor {t_mfma * 1e6:.1f} us); accept {acc_us:.2f} us; commit {commit_us:.2f} us")

    cpu = None
    if not args.no_cpu_baseline:
        import oracle.verify as ov

        host = {k: d[k] for k in d}
        t0, reps = time.perf_counter(), 0
        seqs = [0]
        while True:
            ov.tree_attention_fast(host["q"], host["k_cache"], host["v_cache"], np.full(B, P, np.int32),
                                   host["k_tree"], host["v_tree"], m, nn_h, D ** -0.5, seqs=seqs)
            reps += 1
            if time.perf_counter() - t0 >= min(args.cpu_seconds, 10.0):
                break
        el = time.perf_counter() - t0
        per_seq = el / reps
        cpu = {"value": round(1.0 / (per_seq * B), 3), "unit": "verifications/s", "cores": os.cpu_count(),
               "kind": "oracle",
               "sample": f"{reps} x sequence 0 of {B} (all heads, 4096-token context), fp64 numpy oracle, "
                         f"{el:.1f} s; value = 1 / (time per sequence * B)"}

    res = {
        "metric": "tree verification attention us/call at B=32, budget 64, Qwen3-8B heads, 4096-token context",
        "value": round(1e6 / att_us, 1), "unit": "verifications/s", "n_gpus": 1, "steps": n_att * 4,
        "warmup": 1, "ms_per_step": round(att_us / 1e3, 6), "us_per_step": round(att_us, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "verify-qwen3-8b-heads-b32-n65-p4096", **S},
        "kernels_us": {"tree_attention": round(att_us, 3), "verify_accept": round(acc_us, 3),
                       "commit_kv": round(commit_us, 3)},
        "roofline": {"bound": bound, "kernel": "tree_attention_kernel",
                     "achieved": round(gbps, 1) if bound == "hbm" else round(tflops, 1),
                     "peak": HBM_PEAK_GBPS if bound == "hbm" else MFMA_BF16_PEAK_TFLOPS,
                     "unit": "GB/s" if bound == "hbm" else "TFLOP/s",
                     "frac": round(gbps / HBM_PEAK_GBPS if bound == "hbm" else tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                     "traffic": (measured_traffic(VERIFY_PROFILE, VERIFY_SOURCES) or {}).get("bytes"),
                     "algorithmic_bytes_per_launch": att_bytes, "algorithmic_flops": flops,
                     "other": {"TFLOP/s": round(tflops, 1), "mfma_frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
                               "GB/s": round(gbps, 1), "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4)}},
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)
    return 0


def bench_loss(args, dev) -> int:
    """The renormalised-KL objective with its logit gradient on the headline workload's
    logits (B=32, gamma=15, V=151936 bf16, K=8, r=128): the dense gradient pass (the
    dominant kernel: it reads every logit and writes an fp32 gradient) and the
    per-position kernel, timed together and apart."""
    import numpy as np
    import torch

    import paper_2609_39972_amd as ubt
    import synth

    w = synth.WORKLOADS[3]
    d = synth.inputs(w, 0)
    li = synth.loss_inputs(w, 0)
    bits = lambda a: ubt.bf16_tensor_from_bits(a, dev)
    logits, z = bits(d["logits"]), bits(li["target_logits"])
    y = torch.from_numpy(li["y_star"]).to(dev)
    anchor = torch.from_numpy(d["anchor"]).to(dev)
    phi, psi, gate = bits(d["phi"]), bits(d["psi"]), bits(d["gate"])
    cand = ubt.topk(logits, w.K)
    out = ubt.tree_kl_loss(logits, cand, z, y, anchor, phi, psi, gate, d["alpha"], d["lam"])
    no_grad = {k: (v if k != "grad_logits" else None) for k, v in out.items()}
    torch.cuda.synchronize()
    stream = torch.cuda.Stream(device=dev)

    def timed(fn, n=100, replays=4):
        with torch.cuda.stream(stream):
            fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for _ in range(n):
                fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            g.replay()
            a.record(stream)
            for _ in range(replays):
                g.replay()
            b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / (n * replays)

    both_us = timed(lambda: ubt.tree_kl_loss(logits, cand, z, y, anchor, phi, psi, gate, d["alpha"], d["lam"],
                                             out=out, stream=stream))
    pos_us = timed(lambda: ubt.tree_kl_loss(logits, cand, z, y, anchor, phi, psi, gate, d["alpha"], d["lam"],
                                            out=no_grad, stream=stream))
    dense_us = max(both_us - pos_us, 1e-3)
    dense_bytes = w.rows * w.V * (2 + 4)  # read bf16 logits, write fp32 gradient
    gbps = dense_bytes / (dense_us * 1e-6) / 1e9
    log(f"loss + gradient {both_us:.2f} us (dense pass ~{dense_us:.2f} us, {gbps:.0f} GB/s; per-position kernel "
        f"{pos_us:.2f} us)")
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        import oracle.loss as ol

        c = oracle.topk(d["logits"][:1], w.K)
        t0, reps = time.perf_counter(), 0
        while True:
            ol.tree_kl_loss(d["logits"][:1], c["cand_ids"], li["target_logits"][:1], li["y_star"][:1],
                            d["anchor"][:1], d["phi"], d["psi"], d["gate"][:1], d["alpha"], d["lam"], 1.0, 0.1)
            reps += 1
            if time.perf_counter() - t0 >= min(args.cpu_seconds, 10.0):
                break
        el = time.perf_counter() - t0
        cpu = {"value": round(reps * w.gamma / el, 3), "unit": "positions/s", "cores": 1, "kind": "oracle",
               "sample": f"{reps} x sequence 0 ({w.gamma} positions, loss and full logit gradient), fp64 numpy "
                         f"oracle, {el:.1f} s"}
    res = {
        "metric": "training objective + logit gradient us/call at B=32, gamma=15, V=151936 (bf16), K=8",
        "value": round(w.rows / (both_us * 1e-6), 1), "unit": "positions/s", "n_gpus": 1, "steps": 400,
        "warmup": 100, "ms_per_step": round(both_us / 1e3, 6), "us_per_step": round(both_us, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "kl-loss-" + w.name, "B": w.B, "gamma": w.gamma, "V": w.V, "K": w.K, "r": w.r,
                   "T_train": 1.0, "beta": 0.1},
        "kernels_us": {"loss_and_gradient": round(both_us, 3), "kl_position_kernel": round(pos_us, 3),
                       "kl_dense_kernel (difference)": round(dense_us, 3)},
        "roofline": {"bound": "hbm", "kernel": "kl_dense_kernel", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
                     "traffic": (measured_traffic(LOSS_PROFILE, LOSS_SOURCES) or {}).get("bytes"),
                     "algorithmic_bytes_per_launch": dense_bytes},
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)
    return 0


def bench_lmhead(args, dev) -> int:
    """The LM-head projection fused with the candidate sets (ubt_lm_head_topk) at the
    drafting block of the paper's latency breakdown: 15 draft positions of one sequence,
    hidden size 2560 (Qwen3-4B), V = 151936, K = 64, bf16.  Timed beside the library path
    (hipBLASLt GEMM writing bf16 logits, then ubt_topk) and inside the whole batch-1
    post-processing (ubt_lm_head_topk then ubt_draft_tree with W = 12, budget 64, rank
    256).  The head (778 MB) exceeds the 256 MB last-level cache, so every call streams
    it from HBM."""
    import numpy as np
    import torch

    import paper_2609_39972_amd as ubt
    import synth

    M, d, V, K = args.lm_rows, args.lm_hidden, 151936, 64
    t0 = time.perf_counter()
    x = synth.lm_head_inputs(0, M, d, V)
    log(f"inputs M={M} d={d} V={V}: {time.perf_counter() - t0:.1f} s")
    h = ubt.bf16_tensor_from_bits(x["h"], dev)
    wt = ubt.bf16_tensor_from_bits(x["w"], dev)
    ws = ubt.lm_head_workspace(M, d, V, K, dev)
    stream = torch.cuda.Stream(device=dev)
    out = ubt.lm_head_topk(h, wt, K, workspace=ws)
    torch.cuda.synchronize()

    def timed(fn, n=args.lm_calls, replays=4):
        with torch.cuda.stream(stream):
            fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for _ in range(n):
                fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            g.replay()
            a.record(stream)
            for _ in range(replays):
                g.replay()
            b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / (n * replays)

    fused_us = timed(lambda: ubt.lm_head_topk(h, wt, K, out=out, workspace=ws, stream=stream))
    logits = torch.empty(1, M, V, dtype=torch.bfloat16, device=dev)
    lib_out = ubt.topk(logits, K)

    def library():
        torch.matmul(h, wt.t(), out=logits[0])
        ubt.topk(logits, K, out=lib_out, stream=stream)

    gemm_us = timed(lambda: torch.matmul(h, wt.t(), out=logits[0]))
    lib_us = timed(library)
    # The whole batch-1 post-processing: candidates, selector scores and the tree.
    w6 = synth.WORKLOADS[6]
    gate = ubt.bf16_tensor_from_bits(synth.gate(w6, 0)[:1, :M], dev).contiguous()
    anchor = torch.from_numpy(synth.anchor(w6, 0)[:1].copy()).to(dev)
    phi_b, psi_b = synth.tables(w6)
    phi, psi = ubt.bf16_tensor_from_bits(phi_b, dev), ubt.bf16_tensor_from_bits(psi_b, dev)
    alpha, lam = synth.calibration(w6)
    alpha, lam = alpha[:M], lam[:M]
    cand3 = {k: v.view(1, M, *v.shape[1:]) for k, v in out.items() if v is not None}
    tree = ubt.tree_outputs(1, M, w6.W, w6.budget, dev)
    logq = torch.empty(1, M, K, K, dtype=torch.float32, device=dev)

    def chain():
        ubt.lm_head_topk(h, wt, K, out=out, workspace=ws, stream=stream)
        ubt.draft_tree(phi, psi, gate, anchor, cand3["cand_ids"], cand3["cand_logit"], alpha, lam, w6.W, w6.budget,
                       logq=logq, out=tree, stream=stream)

    chain_us = timed(chain) if M <= w6.gamma else None
    alg_bytes = V * d * 2 + M * d * 2 + M * K * 12 + M * 4
    gbps = alg_bytes / (fused_us * 1e-6) / 1e9
    tflops = 2.0 * M * V * d / (fused_us * 1e-6) / 1e12
    log(f"fused {fused_us:.2f} us ({gbps:.0f} GB/s of the head, {tflops:.1f} TFLOP/s); library GEMM {gemm_us:.2f} "
        f"us, GEMM + ubt_topk {lib_us:.2f} us; batch-1 post-processing {chain_us} us")
    # Parity of the timed outputs against the oracle, and the oracle on the host.
    parity_counts, cpu = None, None
    if not args.no_cpu_baseline:
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        import parity as par
        from oracle import lm_head as LH

        torch.cuda.synchronize()
        g = {k: v.cpu().numpy() for k, v in out.items() if v is not None}
        c = par.check_lm_head(g, x["h"], x["w"], K)
        parity_counts = {"rows": M, "exact": c["exact"], "excused": c["excused"], "failed": 0}
        t0, reps = time.perf_counter(), 0
        while True:
            LH.lm_head_topk(x["h"], x["w"], K)
            reps += 1
            if time.perf_counter() - t0 >= args.cpu_seconds:
                break
        el = time.perf_counter() - t0
        cpu = {"value": round(reps / el, 4), "unit": "blocks/s", "cores": torch.get_num_threads(),
               "kind": "oracle", "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
               "sample": f"{reps} whole calls (M={M}, d={d}, V={V}, K={K}): fp64 numpy matmul in blocks of "
                         f"8192 head rows, then the candidate sets; {el:.1f} s"}
    res = {
        "metric": f"LM head + candidate sets us/call at M={M}, d={d}, V={V}, K={K} (bf16)",
        "value": round(1e6 / fused_us, 1), "unit": "blocks/s", "n_gpus": 1, "steps": 4 * args.lm_calls,
        "warmup": args.lm_calls,
        "ms_per_step": round(fused_us / 1e3, 6), "us_per_step": round(fused_us, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"lm-head-m{M}-d{d}-v{V}-k{K}", "M": M, "d": d, "V": V, "K": K},
        "kernels_us": {"ubt_lm_head_topk": round(fused_us, 3), "library_gemm_bf16_logits": round(gemm_us, 3),
                       "library_gemm_plus_ubt_topk": round(lib_us, 3),
                       "post_processing_batch1 (lm_head_topk + draft_tree W=12 budget=64 r=256)":
                           None if chain_us is None else round(chain_us, 3)},
        "speedup_vs_library": round(lib_us / fused_us, 3),
        "roofline": {"bound": "hbm", "kernel": "lm_head_stream_kernel + lm_head_merge_kernel (whole call)",
                     "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(gbps / HBM_PEAK_GBPS, 4),
                     "traffic": (measured_traffic(LMHEAD_PROFILE, LMHEAD_SOURCES) or {}).get("bytes"),
                     "algorithmic_bytes_per_launch": alg_bytes, "mfma_tflops": round(tflops, 2),
                     "mfma_frac_bf16": round(tflops / 2500.0, 5)},
        "parity": parity_counts,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=3, help="synthetic workload id (3 = B=32, V=151936 headline)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="minimum oracle time for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--mode", choices=("step", "tree", "separate", "verify", "loss", "lmhead"), default="step",
                    help="step: one ubt_draft_step call; tree: ubt_topk + ubt_draft_tree; separate: ubt_topk + "
                         "ubt_bigram_scores + ubt_build_tree; verify: tree verification; loss: the training "
                         "objective; lmhead: the LM head fused with the candidate sets (each its own JSON line)")
    ap.add_argument("--lm-rows", type=int, default=15, help="lmhead mode: rows of h (draft positions)")
    ap.add_argument("--lm-hidden", type=int, default=2560, help="lmhead mode: hidden size d")
    ap.add_argument("--lm-calls", type=int, default=50, help="lmhead mode: calls per timing graph (4 replays)")
    ap.add_argument("--sweep-launches", type=int, default=200, help="launches per kernel in the per-kernel timing")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a plain device copy of known size (counter calibration) and exit")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); sequences shard across GPUs with no "
              f"exchange, so the multi-GPU figure is N times this one.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2609_39972_amd as ubt
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.copy_calibration:
        n = 256 << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 5}))
        return 0
    if args.mode == "verify":
        return bench_verify(args, dev)
    if args.mode == "loss":
        return bench_loss(args, dev)
    if args.mode == "lmhead":
        return bench_lmhead(args, dev)

    w = synth.WORKLOADS[args.workload]
    pool = max(1, -(-POOL_BYTES // w.logit_bytes))
    log(f"workload {w.cfg}: {w.describe()}; pool of {pool} logit buffers ({pool * w.logit_bytes / 1e6:.0f} MB)")

    t0 = time.perf_counter()
    phi_np, psi_np = synth.tables(w)
    to_dev = (lambda a: ubt.bf16_tensor_from_bits(a, dev)) if w.feat_dtype == "bf16" else \
        (lambda a: torch.from_numpy(a).to(dev))
    to_dev_logits = (lambda a: ubt.bf16_tensor_from_bits(a, dev)) if w.dtype == "bf16" else \
        (lambda a: torch.from_numpy(a).to(dev))
    phi, psi = to_dev(phi_np), to_dev(psi_np)
    bufs = []
    host0 = None
    for p in range(pool):
        d = synth.inputs(w, p, with_tables=False)
        if p == 0:
            host0 = dict(d, phi=phi_np, psi=psi_np)
        step = ubt.DraftStep(w.B, w.gamma, w.V, w.K, w.W, w.budget, phi, psi, to_dev(d["gate"]),
                             torch.from_numpy(d["anchor"]).to(dev), d["alpha"], d["lam"], w.zeta,
                             fused=args.mode != "separate", one_call=args.mode == "step",
                             logit_dtype=torch.bfloat16 if w.dtype == "bf16" else torch.float32)
        bufs.append((to_dev_logits(d["logits"]), step))
    torch.cuda.synchronize()
    log(f"inputs resident in HBM ({time.perf_counter() - t0:.1f} s)")

    stream = torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for s in range(args.warmup):
            x, st = bufs[s % pool]
            st.run(x)
    torch.cuda.synchronize()

    # One graph holds one step per pool buffer.
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        for x, st in bufs:
            st.run(x)
    torch.cuda.synchronize()
    replays = max(1, -(-args.steps // pool))
    steps = replays * pool
    with torch.cuda.stream(stream):
        for _ in range(2):
            graph.replay()
    torch.cuda.synchronize()

    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    with torch.cuda.stream(stream):
        start.record(stream)
        for _ in range(replays):
            graph.replay()
        end.record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t_wall) * 1e3
    elapsed_ms = start.elapsed_time(end)
    ms_per_step = elapsed_ms / steps
    log(f"{steps} steps in {elapsed_ms:.2f} ms (wall {wall_ms:.2f} ms): {ms_per_step * 1e3:.2f} us/step")

    # Per-kernel durations: `n` launches of one kernel (rotating over the pool buffers, so
    # each sweep reads its logits from HBM) captured back to back in a graph, replayed
    # between two events on the launch stream; duration = elapsed / launches.
    def timed(fn, n, replays=4):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for j in range(n):
                fn(j)
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            g.replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            a.record(stream)
            for _ in range(replays):
                g.replay()
            b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / (n * replays)  # us

    n = max(pool, args.sweep_launches - args.sweep_launches % pool)
    sweep_us = timed(lambda j: ubt.topk(bufs[j % pool][0], w.K, bufs[j % pool][1].cand), n)
    bigram_us = timed(lambda j: ubt.bigram_scores(bufs[j % pool][1].phi, bufs[j % pool][1].psi,
                                                  bufs[j % pool][1].gate, bufs[j % pool][1].anchor,
                                                  bufs[j % pool][1].cand["cand_ids"],
                                                  bufs[j % pool][1].cand["cand_logit"], bufs[j % pool][1].alpha,
                                                  bufs[j % pool][1].lam, bufs[j % pool][1].sel), n)
    tree_us = timed(lambda j: ubt.build_tree(bufs[j % pool][1].anchor, bufs[j % pool][1].cand["cand_ids"],
                                             bufs[j % pool][1].sel["logq"], w.W, w.budget, w.zeta,
                                             bufs[j % pool][1].tree), n)
    draft_us = timed(lambda j: ubt.draft_tree(bufs[j % pool][1].phi, bufs[j % pool][1].psi, bufs[j % pool][1].gate,
                                              bufs[j % pool][1].anchor, bufs[j % pool][1].cand["cand_ids"],
                                              bufs[j % pool][1].cand["cand_logit"], bufs[j % pool][1].alpha,
                                              bufs[j % pool][1].lam, w.W, w.budget, w.zeta,
                                              bufs[j % pool][1].sel["logq"], bufs[j % pool][1].tree), n)
    sweep_bytes = w.logit_bytes
    sweep_gbps = sweep_bytes / (sweep_us * 1e-6) / 1e9
    log(f"sweep {sweep_us:.2f} us ({sweep_gbps:.0f} GB/s), selector {bigram_us:.2f} us, tree {tree_us:.2f} us, "
        f"selector + tree in one launch {draft_us:.2f} us")
    # The whole step as one ubt_draft_step call; its algorithmic bytes are the logits plus
    # the selector's gathers and writes and the tree outputs.
    step_us = timed(lambda j: bufs[j % pool][1].run(bufs[j % pool][0]), n) if args.mode == "step" else None
    es = 2 if w.feat_dtype == "bf16" else 4
    sel_bytes = (w.B * ((w.gamma - 1) * w.K + 1) * w.r * es        # phi rows of the predecessors
                 + w.B * w.gamma * w.K * w.r * es                  # psi rows of the candidates
                 + w.B * w.gamma * w.r * es                        # gate rows
                 + w.B * w.gamma * w.K * w.K * 4)                  # logq
    cand_bytes = w.B * w.gamma * (w.K * 12 + 4)                   # ids, logits, log-probs, lse
    words = -(-w.N // 32)
    tree_bytes = w.B * w.N * (5 * 4 + 4 * words) + w.B * 4        # tree arrays, mask, n_nodes
    step_bytes = sweep_bytes + sel_bytes + cand_bytes + tree_bytes
    if step_us is not None:
        log(f"ubt_draft_step {step_us:.2f} us ({step_bytes / (step_us * 1e-6) / 1e9:.0f} GB/s)")

    # Every one-launch call's bounded waits completed (the workspaces' error words are 0).
    for _, st in bufs:
        st.check()
    traffic = measured_traffic()
    cpu = None
    par = None
    if not args.no_cpu_baseline:
        log("timing the oracle on the host cores ...")
        cpu, ref = cpu_baseline(w, host0, args.cpu_seconds)
        log(f"oracle: {cpu['value']} trees/s on {cpu['cores']} threads")
        par = step_parity(w, host0, bufs[0][1], bufs[0][0], ref)
        log(f"parity of pool buffer 0 vs the oracle: {par}")

    value = w.B / (ms_per_step * 1e-3)
    res = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "trees/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "us_per_step": round(ms_per_step * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "L": w.L, "gamma": w.gamma, "V": w.V, "K": w.K, "r": w.r,
                   "budget": w.budget, "W": w.W, "logits": f"{w.dtype} {w.logits}", "features": w.feat_dtype,
                   "pool_buffers": pool, "graph": f"{pool} steps per HIP graph, replayed {replays} times"},
        "kernels_us": {"draft_step": None if step_us is None else round(step_us, 3),
                       "topk_sweep": round(sweep_us, 3), "bigram": round(bigram_us, 3),
                       "build_tree": round(tree_us, 3), "draft_tree": round(draft_us, 3)},
        "step_calls": {"step": "ubt_draft_step", "tree": "ubt_topk + ubt_draft_tree",
                       "separate": "ubt_topk + ubt_bigram_scores + ubt_build_tree"}[args.mode],
        "sweep_alone": {"kernel": SWEEP_KERNEL, "us": round(sweep_us, 3), "GB/s": round(sweep_gbps, 1),
                        "frac": round(sweep_gbps / HBM_PEAK_GBPS, 4), "bytes": sweep_bytes},
        "cpu_baseline": cpu,
        "parity": par,
    }
    # The roofline is that of the dominant kernel: the one-launch step when ubt_draft_step
    # runs as one launch (its algorithmic bytes: logits, selector gathers and writes,
    # candidates, tree), else the sweep.
    if step_us is not None and one_launch_step(w, dev):
        step_gbps = step_bytes / (step_us * 1e-6) / 1e9
        straffic = measured_traffic(STEP_PROFILE, STEP_SOURCES)
        res["roofline"] = {"bound": "hbm", "kernel": STEP_KERNEL, "achieved": round(step_gbps, 1),
                           "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(step_gbps / HBM_PEAK_GBPS, 4),
                           "traffic": straffic["bytes"] if straffic is not None and args.workload == 3 else None,
                           "algorithmic_bytes_per_launch": step_bytes,
                           "source_hash": source_hash(STEP_SOURCES),
                           "note": "one launch holds the logit sweep, the selector and the tree search; "
                                   "the sweep on its own is sweep_alone"}
    else:
        res["roofline"] = {"bound": "hbm", "kernel": SWEEP_KERNEL, "achieved": round(sweep_gbps, 1),
                           "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(sweep_gbps / HBM_PEAK_GBPS, 4),
                           "traffic": traffic["bytes"] if traffic is not None and args.workload == 3 else None,
                           "algorithmic_bytes_per_launch": sweep_bytes, "source_hash": source_hash()}
    if step_us is not None:
        res["step_effective"] = {"us": round(step_us, 3), "bytes": step_bytes,
                                 "GB/s": round(step_bytes / (step_us * 1e-6) / 1e9, 1)}
    res = {k: res[k] for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "us_per_step",
                               "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config", "kernels_us",
                               "step_calls", "roofline", "sweep_alone", "step_effective", "cpu_baseline", "parity")
           if k in res}
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
