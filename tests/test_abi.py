"""The C ABI of libubt.so on the host: exported symbols, status strings and
argument validation, which returns an error before any device work (so
these run without a GPU; the pointers passed are never dereferenced)."""
from __future__ import annotations

import ctypes
import re
import subprocess

import pytest

import paper_2609_39972_amd as ubt

FAKE = ctypes.c_void_p(0x10000)  # never dereferenced: every call below fails validation first


def _declared() -> set:
    hdr = open(f"{ubt.PKG}/../include/ubt.h").read()
    return set(re.findall(r"\b(ubt_[a-z_]+)\s*\(", hdr))


def test_library_exports_every_declared_symbol():
    L = ubt.lib()
    declared = _declared()
    assert declared == set(ubt.EXPORTS)
    nm = subprocess.run(["nm", "-D", "--defined-only", ubt.LIB_PATH], capture_output=True, text=True, check=True)
    exported = set(re.findall(r" T (ubt_\w+)", nm.stdout))
    assert declared <= exported
    for name in declared:
        assert hasattr(L, name)


def test_version_and_status_strings():
    L = ubt.lib()
    assert L.ubt_abi_version() == 1
    for code, name in ubt.STATUS.items():
        assert L.ubt_status_str(code).decode() == name
    assert L.ubt_status_str(99).decode() == "UBT_ERR_UNKNOWN"


def _topk(**kw):
    a = dict(logits=FAKE, dt=1, B=2, gamma=3, V=1000, sb=3000, si=1000, K=8, ids=FAKE, val=FAKE, lp=None, lse=None)
    a.update(kw)
    return ubt.lib().ubt_topk(a["logits"], a["dt"], a["B"], a["gamma"], a["V"], a["sb"], a["si"], a["K"], a["ids"],
                              a["val"], a["lp"], a["lse"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(logits=None), 1), (dict(ids=None), 1), (dict(val=None), 1),
    (dict(dt=5), 3),
    (dict(B=0), 2), (dict(gamma=0), 2), (dict(gamma=65), 2), (dict(K=0), 2), (dict(K=65), 2), (dict(V=7), 2),
    (dict(si=999), 2), (dict(sb=2999), 2), (dict(V=2 ** 31, si=2 ** 31, sb=3 * 2 ** 31), 2),
])
def test_topk_validation(kw, code):
    assert _topk(**kw) == code


def _bigram(alpha=None, lam=None, **kw):
    g = kw.pop("gamma", 3)
    a = (ctypes.c_float * 64)(*([1.0] * 64)) if alpha is None else alpha
    l_ = (ctypes.c_float * 64)(*([1.0] * 64)) if lam is None else lam
    args = dict(phi=FAKE, psi=FAKE, gate=FAKE, dt=1, V=1000, r=64, anchor=FAKE, ids=FAKE, logit=FAKE, B=2, K=8,
                delta=None, logq=FAKE)
    args.update(kw)
    return ubt.lib().ubt_bigram_scores(args["phi"], args["psi"], args["gate"], args["dt"], args["V"], args["r"],
                                       args["anchor"], args["ids"], args["logit"], a, l_, args["B"], g, args["K"],
                                       args["delta"], args["logq"], None)


def _arr(vals):
    return (ctypes.c_float * len(vals))(*vals)


@pytest.mark.parametrize("kw,code", [
    (dict(phi=None), 1), (dict(gate=None), 1), (dict(anchor=None), 1), (dict(logq=None), 1),
    (dict(dt=9), 3), (dict(r=8), 2), (dict(r=72), 2), (dict(r=528), 2), (dict(K=65), 2), (dict(gamma=65), 2),
    (dict(V=5), 2), (dict(B=0), 2),
    (dict(alpha=_arr([1.0, 0.0, 1.0])), 3), (dict(lam=_arr([1.0, 1.0, -2.0])), 3),
    (dict(alpha=_arr([1.0, float("inf"), 1.0])), 3), (dict(lam=_arr([float("nan"), 1.0, 1.0])), 3),
    (dict(phi=ctypes.c_void_p(0x10002)), 4),
])
def test_bigram_validation(kw, code):
    assert _bigram(**kw) == code


def _tree(dbg=None, **kw):
    a = dict(anchor=FAKE, ids=FAKE, logq=FAKE, B=2, gamma=15, K=8, W=12, budget=64, zeta=0.0, nn=FAKE, tok=FAKE,
             par=FAKE, dep=FAKE, cr=FAKE, sc=FAKE, mask=None)
    a.update(kw)
    return ubt.lib().ubt_build_tree(a["anchor"], a["ids"], a["logq"], a["B"], a["gamma"], a["K"], a["W"],
                                    a["budget"], a["zeta"], a["nn"], a["tok"], a["par"], a["dep"], a["cr"], a["sc"],
                                    a["mask"], dbg, None)


@pytest.mark.parametrize("kw,code", [
    (dict(anchor=None), 1), (dict(logq=None), 1), (dict(nn=None), 1), (dict(sc=None), 1),
    (dict(B=0), 2), (dict(gamma=0), 2), (dict(gamma=65), 2), (dict(K=65), 2), (dict(W=0), 2), (dict(W=256), 2),
    (dict(budget=0), 2), (dict(budget=256), 2),
    (dict(W=65, K=64), 4), (dict(gamma=64, W=65, K=4), 4),
    (dict(zeta=0.5), 3), (dict(zeta=float("-inf")), 3), (dict(zeta=float("nan")), 3),
])
def test_build_tree_validation(kw, code):
    assert _tree(**kw) == code


def test_build_tree_incomplete_debug_struct():
    s = ubt._Supertree(FAKE, None, FAKE, FAKE)
    assert _tree(dbg=ctypes.byref(s)) == 1


def _draft(alpha=None, lam=None, **kw):
    a_ = (ctypes.c_float * 64)(*([1.0] * 64)) if alpha is None else alpha
    l_ = (ctypes.c_float * 64)(*([1.0] * 64)) if lam is None else lam
    a = dict(phi=FAKE, psi=FAKE, gate=FAKE, dt=1, V=1000, r=64, anchor=FAKE, ids=FAKE, logit=FAKE, B=2, gamma=3,
             K=8, W=4, budget=10, zeta=0.0, logq=FAKE, nn=FAKE, tok=FAKE, par=FAKE, dep=FAKE, cr=FAKE, sc=FAKE,
             mask=None)
    a.update(kw)
    return ubt.lib().ubt_draft_tree(a["phi"], a["psi"], a["gate"], a["dt"], a["V"], a["r"], a["anchor"], a["ids"],
                                    a["logit"], a_, l_, a["B"], a["gamma"], a["K"], a["W"], a["budget"], a["zeta"],
                                    a["logq"], a["nn"], a["tok"], a["par"], a["dep"], a["cr"], a["sc"], a["mask"],
                                    None)


@pytest.mark.parametrize("kw,code", [
    (dict(phi=None), 1), (dict(logit=None), 1), (dict(logq=None), 1), (dict(nn=None), 1), (dict(sc=None), 1),
    (dict(dt=9), 3), (dict(r=8), 2), (dict(K=65), 2), (dict(gamma=65), 2), (dict(V=5), 2), (dict(B=0), 2),
    (dict(W=0), 2), (dict(budget=256), 2), (dict(W=65, K=64), 4), (dict(gamma=64, W=65, K=4), 4),
    (dict(alpha=_arr([1.0, 0.0, 1.0])), 3), (dict(lam=_arr([1.0, 1.0, float("nan")])), 3),
    (dict(zeta=0.5), 3), (dict(zeta=float("nan")), 3), (dict(gate=ctypes.c_void_p(0x10008)), 4),
])
def test_draft_tree_validation(kw, code):
    """The one-call selector + search checks the union of the two calls' arguments."""
    assert _draft(**kw) == code


@pytest.mark.parametrize("args,code", [
    ((None, FAKE, 2, 65, FAKE), 1), ((FAKE, None, 2, 65, FAKE), 1), ((FAKE, FAKE, 2, 65, None), 1),
    ((FAKE, FAKE, 0, 65, FAKE), 2), ((FAKE, FAKE, 2, 0, FAKE), 2), ((FAKE, FAKE, 2, 257, FAKE), 2),
])
def test_tree_mask_validation(args, code):
    assert ubt.lib().ubt_tree_mask(*args, None) == code


def test_binding_refuses_host_tensors():
    import torch

    with pytest.raises(ValueError):
        ubt.topk(torch.zeros(1, 1, 16, dtype=torch.bfloat16), 4)


def _attn(**kw):
    a = dict(q=FAKE, kc=FAKE, vc=FAKE, plen=FAKE, Pmax=128, kt=FAKE, vt=FAKE, mask=FAKE, nn=FAKE, B=2, N=65, H=32,
             Hkv=8, D=128, scale=0.088, out=FAKE, odt=1, lse=None)
    a.update(kw)
    return ubt.lib().ubt_tree_attention(a["q"], a["kc"], a["vc"], a["plen"], a["Pmax"], a["kt"], a["vt"], a["mask"],
                                        a["nn"], a["B"], a["N"], a["H"], a["Hkv"], a["D"], a["scale"], a["out"],
                                        a["odt"], a["lse"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), 1), (dict(kt=None), 1), (dict(vt=None), 1), (dict(mask=None), 1), (dict(nn=None), 1),
    (dict(out=None), 1), (dict(plen=None), 1), (dict(kc=None), 1), (dict(vc=None), 1),
    (dict(B=0), 2), (dict(N=0), 2), (dict(N=257), 2), (dict(H=0), 2), (dict(Hkv=0), 2), (dict(H=30), 2),
    (dict(Pmax=-1), 2), (dict(Pmax=2 ** 31), 2),
    (dict(D=96), 4), (dict(D=256), 4), (dict(q=ctypes.c_void_p(0x10008)), 4), (dict(kc=ctypes.c_void_p(0x10004)), 4),
    (dict(odt=7), 3), (dict(scale=0.0), 3), (dict(scale=float("inf")), 3), (dict(scale=-1.0), 3),
])
def test_tree_attention_validation(kw, code):
    assert _attn(**kw) == code


def test_tree_attention_without_context_needs_no_cache():
    """P_max = 0 takes NULL caches; the call then fails only on what is still wrong."""
    assert _attn(Pmax=0, kc=None, vc=None, N=0) == 2


@pytest.mark.parametrize("args,code", [
    ((None, FAKE, FAKE, FAKE, 2, 65, FAKE, FAKE, FAKE), 1), ((FAKE, FAKE, FAKE, None, 2, 65, FAKE, FAKE, FAKE), 1),
    ((FAKE, FAKE, FAKE, FAKE, 2, 65, FAKE, FAKE, None), 1),
    ((FAKE, FAKE, FAKE, FAKE, 0, 65, FAKE, FAKE, FAKE), 2), ((FAKE, FAKE, FAKE, FAKE, 2, 257, FAKE, FAKE, FAKE), 2),
])
def test_verify_accept_validation(args, code):
    assert ubt.lib().ubt_verify_accept(*args, None) == code


@pytest.mark.parametrize("kw,code", [
    (dict(kt=None), 1), (dict(kc=None), 1), (dict(plen=None), 1), (dict(nodes=None), 1),
    (dict(B=0), 2), (dict(N=300), 2), (dict(Hkv=0), 2), (dict(Pmax=0), 2), (dict(D=32), 4),
    (dict(kc=ctypes.c_void_p(0x10002)), 4),
])
def test_commit_kv_validation(kw, code):
    a = dict(kt=FAKE, vt=FAKE, nodes=FAKE, alen=FAKE, plen=FAKE, kc=FAKE, vc=FAKE, B=2, N=65, Hkv=8, D=128, Pmax=64)
    a.update(kw)
    assert ubt.lib().ubt_commit_kv(a["kt"], a["vt"], a["nodes"], a["alen"], a["plen"], a["kc"], a["vc"], a["B"],
                                   a["N"], a["Hkv"], a["D"], a["Pmax"], None) == code


def _kl(**kw):
    g = kw.pop("gamma", 3)
    a = (ctypes.c_float * 64)(*([1.0] * 64))
    args = dict(logits=FAKE, dt=1, B=2, gamma=g, V=1000, sb=3000, si=1000, lse=FAKE, ids=FAKE, cl=FAKE, K=8, z=FAKE,
                tsb=3000, tsi=1000, y=FAKE, anchor=FAKE, phi=FAKE, psi=FAKE, gate=FAKE, fdt=1, r=64, alpha=a, lam=a,
                T=1.0, beta=0.1, loss=FAKE, kl=None, ce=None, gs=None, grad=None)
    args.update(kw)
    v = list(args.values())
    return ubt.lib().ubt_tree_kl_loss(*v, None)


@pytest.mark.parametrize("kw,code", [
    (dict(logits=None), 1), (dict(lse=None), 1), (dict(z=None), 1), (dict(y=None), 1), (dict(loss=None), 1),
    (dict(ids=None), 1), (dict(phi=None), 1), (dict(anchor=None), 1),
    (dict(dt=4), 3), (dict(fdt=4), 3), (dict(T=-0.5), 3), (dict(T=float("nan")), 3), (dict(beta=-1.0), 3),
    (dict(B=0), 2), (dict(K=65), 2), (dict(r=24), 2), (dict(si=999), 2), (dict(tsi=999), 2), (dict(tsb=2999), 2),
    (dict(grad=ctypes.c_void_p(0x10004)), 4), (dict(gate=ctypes.c_void_p(0x10008)), 4),
])
def test_tree_kl_loss_validation(kw, code):
    assert _kl(**kw) == code


def _step_ws_expected(B, gamma, V, K, es):
    """Workspace of the one-launch step: an error word, then 256-byte aligned regions
    for the row counters, the chunk ids and logits (C K each per row) and the chunk LSEs,
    with C = min(2, 64 // K, tiles per row) chunks of whole tiles (64 lanes x 64 bytes)."""
    al = lambda n: (n + 255) // 256 * 256
    tile = 64 * 64 // es
    tiles = -(-V // tile)
    c = min(2, max(1, 64 // K), tiles)
    length = -(-tiles // c) * tile
    C = -(-V // length)
    rows = B * gamma
    return 256 + al(rows * 4) + 2 * al(rows * C * K * 4) + al(rows * C * 4)


@pytest.mark.parametrize("B,gamma,V,K,dt", [
    (32, 15, 151936, 8, 1), (32, 15, 151936, 16, 1), (1, 7, 32000, 4, 0), (2, 4, 2048, 8, 1), (3, 2, 100, 16, 0),
    (64, 2, 3000, 4, 1), (2, 4, 8200, 16, 1),
])
def test_draft_step_workspace_bytes(B, gamma, V, K, dt):
    L = ubt.lib()
    got = L.ubt_draft_step_workspace_bytes(B, gamma, V, K, dt)
    assert got == _step_ws_expected(B, gamma, V, K, 2 if dt == 1 else 4)
    assert got >= 256 + 4 * B * gamma
    assert L.ubt_draft_step_workspace_bytes(0, gamma, V, K, dt) == 0
    assert L.ubt_draft_step_workspace_bytes(B, gamma, K - 1, K, dt) == 0


def _lmh(**kw):
    a = dict(h=FAKE, w=FAKE, M=15, d=2560, V=151936, K=64, ids=FAKE, val=FAKE, lp=None, lse=None, ws=FAKE,
             wsb=1 << 30)
    a.update(kw)
    return ubt.lib().ubt_lm_head_topk(a["h"], a["w"], a["M"], a["d"], a["V"], a["K"], a["ids"], a["val"], a["lp"],
                                      a["lse"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(h=None), 1), (dict(w=None), 1), (dict(ids=None), 1), (dict(val=None), 1),
    (dict(M=0), 2), (dict(d=48), 2), (dict(d=0), 2), (dict(d=65568), 2), (dict(K=0), 2), (dict(K=65), 2),
    (dict(V=63), 2), (dict(V=2 ** 31), 2),
    (dict(h=ctypes.c_void_p(0x10008)), 4), (dict(w=ctypes.c_void_p(0x10002)), 4),
    (dict(ws=None), 5), (dict(wsb=1000), 5), (dict(ws=ctypes.c_void_p(0x10010)), 5),
])
def test_lm_head_validation(kw, code):
    assert _lmh(**kw) == code


def test_lm_head_workspace_bytes():
    """One (max, sum) and K sorted (key, id) pairs per (row slot, workgroup),
    for 16 row slots per group of rows.  Workgroups: one per compute unit (256 on this GPU
    and when none is visible), at most one per 16-row tile when d is a multiple of 512
    (the k-split kernel), else at most one per 8 tiles."""
    L = ubt.lib()
    al = lambda n: (n + 255) // 256 * 256
    for M, d, V, K in ((15, 2560, 151936, 64), (17, 4096, 151936, 8), (1, 2560, 1000, 1), (3, 96, 1000, 4),
                       (2, 2560, 600, 8)):
        tiles = (V + 15) // 16
        G = min(256, tiles) if d % 512 == 0 else min(256, (tiles + 7) // 8)
        parts = (M + 15) // 16 * G * 16
        assert L.ubt_lm_head_topk_workspace_bytes(M, d, V, K) == al(parts * 8) + al(parts * K * 8)
    assert L.ubt_lm_head_topk_workspace_bytes(0, 2560, 1000, 8) == 0
    assert L.ubt_lm_head_topk_workspace_bytes(4, 2560, 7, 8) == 0
    assert L.ubt_lm_head_topk_workspace_bytes(4, 48, 1000, 8) == 0
    assert L.ubt_lm_head_topk_workspace_bytes(4, 2560, 2 ** 31 - 1, 64) == 0  # the merge's candidates would not fit
