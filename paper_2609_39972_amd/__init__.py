"""UBTree draft-tree construction on AMD Instinct MI355X (gfx950).

A thin binding over the C ABI of ``libubt.so`` (``include/ubt.h``).  Every step of the
path runs in the library's HIP kernels; this module only allocates outputs with torch,
passes raw device pointers and the current HIP stream, and turns status codes into
exceptions.  It fails loudly when the library is missing: there is no fallback.

Calls, in pipeline order (the paper's section and equation names in brackets):

* :func:`topk` -- softmax statistics and top-K candidates per row [Method / Unigram
  Proposer, Eq. ubtree-unigram; Candidate Sets];
* :func:`bigram_scores` -- selector scores and normalised transition log-probs
  [Eq. dflash2-selector, ubtree-depth, ubtree-edge-matrix, ubtree-path];
* :func:`build_tree` -- beam search with global pruning and the ancestor mask
  [Appendix A, Algorithm 1];
* :func:`tree_mask` -- the ancestor mask of any parent-pointer tree;
* :func:`draft_step` -- the whole step in one call (one kernel launch for the common
  shapes: rows swept in depth order while the searchers run; it needs a zero-filled
  workspace from :func:`draft_step_workspace`, whose error word
  :func:`draft_step_error` reads).

:class:`DraftStep` preallocates everything for one workload shape and runs the step on
one stream (graph-capturable).
"""
from __future__ import annotations

import ctypes
import os

import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libubt.so")

UBT_F32, UBT_BF16 = 0, 1
STATUS = {0: "UBT_OK", 1: "UBT_ERR_NULL", 2: "UBT_ERR_SHAPE", 3: "UBT_ERR_VALUE", 4: "UBT_ERR_UNSUPPORTED",
          5: "UBT_ERR_WORKSPACE", 6: "UBT_ERR_HIP"}

# Every symbol include/ubt.h declares.
EXPORTS = ("ubt_status_str", "ubt_abi_version", "ubt_last_hip_error", "ubt_topk",
           "ubt_lm_head_topk_workspace_bytes", "ubt_lm_head_topk", "ubt_bigram_scores", "ubt_build_tree", "ubt_draft_tree", "ubt_draft_step_workspace_bytes",
           "ubt_draft_step", "ubt_draft_step_noalloc", "ubt_edge_scores", "ubt_build_tree_best_first", "ubt_tree_mask", "ubt_tree_attention", "ubt_verify_accept", "ubt_commit_kv",
           "ubt_tree_kl_loss")

_p = ctypes.c_void_p
_i32 = ctypes.c_int
_i64 = ctypes.c_int64
_f32 = ctypes.c_float
_lib = None


class UbtError(RuntimeError):
    def __init__(self, call: str, status: int):
        self.status = status
        super().__init__(f"{call} failed: {STATUS.get(status, status)}")


class _Supertree(ctypes.Structure):
    _fields_ = [("f_count", _p), ("f_parent_slot", _p), ("f_cand", _p), ("f_score", _p)]


def lib() -> ctypes.CDLL:
    """The loaded ``libubt.so``.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        L.ubt_status_str.argtypes = [_i32]
        L.ubt_status_str.restype = ctypes.c_char_p
        L.ubt_abi_version.restype = _i32
        L.ubt_last_hip_error.restype = _i32
        L.ubt_topk.argtypes = [_p, _i32, _i32, _i32, _i64, _i64, _i64, _i32, _p, _p, _p, _p, _p]
        L.ubt_lm_head_topk_workspace_bytes.argtypes = [_i32, _i32, _i64, _i32]
        L.ubt_lm_head_topk_workspace_bytes.restype = ctypes.c_size_t
        L.ubt_lm_head_topk.argtypes = [_p, _p, _i32, _i32, _i64, _i32, _p, _p, _p, _p, _p, ctypes.c_size_t, _p]
        L.ubt_bigram_scores.argtypes = [_p, _p, _p, _i32, _i64, _i32, _p, _p, _p, _p, _p, _i32, _i32, _i32, _p, _p,
                                        _p]
        L.ubt_build_tree.argtypes = [_p, _p, _p, _i32, _i32, _i32, _i32, _i32, _f32, _p, _p, _p, _p, _p, _p, _p,
                                     ctypes.POINTER(_Supertree), _p]
        L.ubt_draft_tree.argtypes = [_p, _p, _p, _i32, _i64, _i32, _p, _p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32,
                                     _f32, _p, _p, _p, _p, _p, _p, _p, _p, _p]
        L.ubt_tree_mask.argtypes = [_p, _p, _i32, _i32, _p, _p]
        L.ubt_draft_step_workspace_bytes.argtypes = [_i32, _i32, _i64, _i32, _i32]
        L.ubt_draft_step_workspace_bytes.restype = ctypes.c_size_t
        L.ubt_draft_step.argtypes = [_p, _i32, _i32, _i32, _i64, _i64, _i64, _i32, _p, _p, _p, _i32, _i32, _p, _p,
                                     _p, _i32, _i32, _f32, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p,
                                     ctypes.c_size_t, _p]
        L.ubt_draft_step_noalloc.argtypes = [_p, _i32, _i32, _i32, _i64, _i64, _i64, _i32, _p, _p, _p, _i32, _i32,
                                             _p, _p, _p, _i32, _i32, _f32, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p,
                                             _p, _p, _p]
        L.ubt_edge_scores.argtypes = [_p, _p, _p, _i32, _i64, _i32, _p, _p, _p, _p, _p, _i32, _i32, _i32, _p, _p, _p]
        L.ubt_build_tree_best_first.argtypes = [_p, _p, _p, _i32, _i32, _i32, _i32, _f32, _p, _p, _p, _p, _p, _p, _p,
                                                _p]
        L.ubt_tree_attention.argtypes = [_p, _p, _p, _p, _i64, _p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32, _f32,
                                         _p, _i32, _p, _p]
        L.ubt_verify_accept.argtypes = [_p, _p, _p, _p, _i32, _i32, _p, _p, _p, _p]
        L.ubt_commit_kv.argtypes = [_p, _p, _p, _p, _p, _p, _p, _i32, _i32, _i32, _i32, _i64, _p]
        L.ubt_tree_kl_loss.argtypes = [_p, _i32, _i32, _i32, _i64, _i64, _i64, _p, _p, _p, _i32, _p, _i64, _i64, _p,
                                       _p, _p, _p, _p, _i32, _i32, _p, _p, _f32, _f32, _p, _p, _p, _p, _p, _p]
        for f in (L.ubt_topk, L.ubt_lm_head_topk, L.ubt_bigram_scores, L.ubt_build_tree, L.ubt_draft_tree, L.ubt_tree_mask,
                  L.ubt_draft_step, L.ubt_draft_step_noalloc, L.ubt_edge_scores, L.ubt_build_tree_best_first, L.ubt_tree_attention, L.ubt_verify_accept, L.ubt_commit_kv, L.ubt_tree_kl_loss):
            f.restype = _i32
        _lib = L
    return _lib


def _check(call: str, status: int) -> None:
    if status != 0:
        raise UbtError(call, status)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return UBT_BF16
    if t.dtype == torch.float32:
        return UBT_F32
    raise TypeError(f"unsupported dtype {t.dtype}: use torch.bfloat16 or torch.float32")


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _need_gpu(*ts: torch.Tensor) -> None:
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("all tensors must live on the GPU")


def _contig(t: torch.Tensor, name: str) -> torch.Tensor:
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def topk(logits: torch.Tensor, K: int, out: dict | None = None, with_logprob: bool = True, stream=None) -> dict:
    """Top-K candidates and softmax statistics of ``logits [B, gamma, V]`` (any strides with
    unit stride along V; e.g. ``u[:, 1:, :]`` of a ``[B, L, V]`` block)."""
    _need_gpu(logits)
    if logits.dim() != 3 or logits.stride(2) != 1:
        raise ValueError("logits must be [B, gamma, V] with unit stride along V")
    B, gamma, V = logits.shape
    code = _dtype_code(logits)
    dev = logits.device
    if out is None:
        out = dict(cand_ids=torch.empty(B, gamma, K, dtype=torch.int32, device=dev),
                   cand_logit=torch.empty(B, gamma, K, dtype=torch.float32, device=dev),
                   cand_logprob=torch.empty(B, gamma, K, dtype=torch.float32, device=dev) if with_logprob else None,
                   lse=torch.empty(B, gamma, dtype=torch.float32, device=dev))
    st = lib().ubt_topk(_ptr(logits), code, B, gamma, V, logits.stride(0), logits.stride(1), K,
                        _ptr(out["cand_ids"]), _ptr(out["cand_logit"]), _ptr(out.get("cand_logprob")),
                        _ptr(out.get("lse")), _stream(stream))
    _check("ubt_topk", st)
    return out


def lm_head_workspace(M: int, d: int, V: int, K: int, device="cuda") -> torch.Tensor:
    """A workspace for :func:`lm_head_topk` (uint8, 256-byte aligned; its contents are
    never read before they are written, so it serves calls of any shape in turn)."""
    n = lib().ubt_lm_head_topk_workspace_bytes(M, d, V, K)
    if n == 0:
        raise ValueError("invalid shape for ubt_lm_head_topk")
    ws = torch.empty(n, dtype=torch.uint8, device=device)
    if ws.data_ptr() % 256:
        raise RuntimeError("workspace is not 256-byte aligned")
    return ws


def lm_head_topk(h: torch.Tensor, w_lm: torch.Tensor, K: int, out: dict | None = None,
                 workspace: torch.Tensor | None = None, with_logprob: bool = True, stream=None) -> dict:
    """Candidates and softmax statistics of the logits ``h @ w_lm.T`` without forming them:
    ``h [..., d]`` and ``w_lm [V, d]``, both contiguous bf16.  Outputs have h's leading
    shape: ``cand_ids``/``cand_logit``/``cand_logprob`` [..., K] and ``lse`` [...]."""
    _need_gpu(h, w_lm)
    _contig(h, "h")
    _contig(w_lm, "w_lm")
    if h.dtype != torch.bfloat16 or w_lm.dtype != torch.bfloat16:
        raise TypeError("h and w_lm must be bfloat16")
    if w_lm.dim() != 2 or h.shape[-1] != w_lm.shape[1]:
        raise ValueError("h must be [..., d] and w_lm [V, d]")
    lead = tuple(h.shape[:-1])
    M = 1
    for n in lead:
        M *= n
    V, d = w_lm.shape
    dev = h.device
    if out is None:
        out = dict(cand_ids=torch.empty(*lead, K, dtype=torch.int32, device=dev),
                   cand_logit=torch.empty(*lead, K, dtype=torch.float32, device=dev),
                   cand_logprob=torch.empty(*lead, K, dtype=torch.float32, device=dev) if with_logprob else None,
                   lse=torch.empty(*lead, dtype=torch.float32, device=dev))
    if workspace is None:
        workspace = lm_head_workspace(M, d, V, K, dev)
    st = lib().ubt_lm_head_topk(_ptr(h), _ptr(w_lm), M, d, V, K, _ptr(out["cand_ids"]), _ptr(out["cand_logit"]),
                                _ptr(out.get("cand_logprob")), _ptr(out.get("lse")), _ptr(workspace),
                                workspace.numel(), _stream(stream))
    _check("ubt_lm_head_topk", st)
    return out


def _host_f32(x, n: int) -> ctypes.Array:
    vals = [float(v) for v in (x.tolist() if hasattr(x, "tolist") else x)]
    if len(vals) != n:
        raise ValueError(f"expected {n} values, got {len(vals)}")
    return (ctypes.c_float * n)(*vals)


def bigram_scores(phi: torch.Tensor, psi: torch.Tensor, gate: torch.Tensor, anchor: torch.Tensor,
                  cand_ids: torch.Tensor, cand_logit: torch.Tensor, alpha, lam, out: dict | None = None,
                  with_delta: bool = True, stream=None) -> dict:
    """Selector scores ``delta`` and ``logq`` ``[B, gamma, K, K]``; ``alpha``/``lam`` are
    per-depth host values (sequences or CPU tensors)."""
    _need_gpu(phi, psi, gate, anchor, cand_ids, cand_logit)
    for n, t in (("phi", phi), ("psi", psi), ("gate", gate), ("anchor", anchor), ("cand_ids", cand_ids),
                 ("cand_logit", cand_logit)):
        _contig(t, n)
    if not (phi.dtype == psi.dtype == gate.dtype):
        raise TypeError("phi, psi and gate must share one dtype")
    V, r = phi.shape
    B, gamma, K = cand_ids.shape
    dev = cand_ids.device
    if out is None:
        out = dict(delta=torch.empty(B, gamma, K, K, dtype=torch.float32, device=dev) if with_delta else None,
                   logq=torch.empty(B, gamma, K, K, dtype=torch.float32, device=dev))
    a, l = _host_f32(alpha, gamma), _host_f32(lam, gamma)
    st = lib().ubt_bigram_scores(_ptr(phi), _ptr(psi), _ptr(gate), _dtype_code(phi), V, r, _ptr(anchor),
                                 _ptr(cand_ids), _ptr(cand_logit), a, l, B, gamma, K, _ptr(out.get("delta")),
                                 _ptr(out["logq"]), _stream(stream))
    _check("ubt_bigram_scores", st)
    return out


def tree_outputs(B: int, gamma: int, W: int, budget: int, device="cuda", with_mask: bool = True,
                 debug: bool = False) -> dict:
    N = budget + 1
    words = (N + 31) // 32
    i32 = dict(dtype=torch.int32, device=device)
    out = dict(n_nodes=torch.empty(B, **i32), token=torch.empty(B, N, **i32), parent=torch.empty(B, N, **i32),
               depth=torch.empty(B, N, **i32), cand_rank=torch.empty(B, N, **i32),
               score=torch.empty(B, N, dtype=torch.float32, device=device),
               mask=torch.empty(B, N, words, **i32) if with_mask else None)
    if debug:
        out.update(f_count=torch.empty(B, gamma, **i32), f_parent=torch.empty(B, gamma, W, **i32),
                   f_cand=torch.empty(B, gamma, W, **i32),
                   f_score=torch.empty(B, gamma, W, dtype=torch.float32, device=device))
    return out


def build_tree(anchor: torch.Tensor, cand_ids: torch.Tensor, logq: torch.Tensor, W: int, budget: int,
               zeta: float = 0.0, out: dict | None = None, with_mask: bool = True, debug: bool = False,
               stream=None) -> dict:
    """Algorithm 1 per sequence: tree slots ``[B, budget+1]``, the packed ancestor mask
    (``int32`` view of the uint32 words) and, with ``debug``, the supertree F_d."""
    _need_gpu(anchor, cand_ids, logq)
    for n, t in (("anchor", anchor), ("cand_ids", cand_ids), ("logq", logq)):
        _contig(t, n)
    B, gamma, K = cand_ids.shape
    if out is None:
        out = tree_outputs(B, gamma, W, budget, cand_ids.device, with_mask, debug)
    dbg = None
    if "f_count" in out:
        dbg = ctypes.byref(_Supertree(_ptr(out["f_count"]), _ptr(out["f_parent"]), _ptr(out["f_cand"]),
                                      _ptr(out["f_score"])))
    st = lib().ubt_build_tree(_ptr(anchor), _ptr(cand_ids), _ptr(logq), B, gamma, K, W, budget, float(zeta),
                              _ptr(out["n_nodes"]), _ptr(out["token"]), _ptr(out["parent"]), _ptr(out["depth"]),
                              _ptr(out["cand_rank"]), _ptr(out["score"]), _ptr(out.get("mask")), dbg,
                              _stream(stream))
    _check("ubt_build_tree", st)
    return out


def draft_tree(phi: torch.Tensor, psi: torch.Tensor, gate: torch.Tensor, anchor: torch.Tensor,
               cand_ids: torch.Tensor, cand_logit: torch.Tensor, alpha, lam, W: int, budget: int,
               zeta: float = 0.0, logq: torch.Tensor | None = None, out: dict | None = None,
               with_mask: bool = True, stream=None) -> dict:
    """``bigram_scores`` (no delta) + ``build_tree`` in one library call; returns the tree
    outputs and ``logq``."""
    _need_gpu(phi, psi, gate, anchor, cand_ids, cand_logit)
    for n, t in (("phi", phi), ("psi", psi), ("gate", gate), ("anchor", anchor), ("cand_ids", cand_ids),
                 ("cand_logit", cand_logit)):
        _contig(t, n)
    if not (phi.dtype == psi.dtype == gate.dtype):
        raise TypeError("phi, psi and gate must share one dtype")
    V, r = phi.shape
    B, gamma, K = cand_ids.shape
    if logq is None:
        logq = torch.empty(B, gamma, K, K, dtype=torch.float32, device=cand_ids.device)
    _contig(logq, "logq")
    if out is None:
        out = tree_outputs(B, gamma, W, budget, cand_ids.device, with_mask)
    a, l = _host_f32(alpha, gamma), _host_f32(lam, gamma)
    st = lib().ubt_draft_tree(_ptr(phi), _ptr(psi), _ptr(gate), _dtype_code(phi), V, r, _ptr(anchor), _ptr(cand_ids),
                              _ptr(cand_logit), a, l, B, gamma, K, W, budget, float(zeta), _ptr(logq),
                              _ptr(out["n_nodes"]), _ptr(out["token"]), _ptr(out["parent"]), _ptr(out["depth"]),
                              _ptr(out["cand_rank"]), _ptr(out["score"]), _ptr(out.get("mask")), _stream(stream))
    _check("ubt_draft_tree", st)
    return {**out, "logq": logq}


def edge_scores(phi: torch.Tensor, psi: torch.Tensor, gate: torch.Tensor, anchor: torch.Tensor,
                cand_ids: torch.Tensor, cand_logprob: torch.Tensor, alpha, lam, out: dict | None = None,
                with_delta: bool = False, stream=None) -> dict:
    """``ubt_edge_scores``: unnormalised unigram-plus-bigram edge scores ``edge``
    ``[B, gamma, K, K]`` (and ``delta`` if asked) from ``topk``'s log-probabilities."""
    _need_gpu(phi, psi, gate, anchor, cand_ids, cand_logprob)
    for n, t in (("phi", phi), ("psi", psi), ("gate", gate), ("anchor", anchor), ("cand_ids", cand_ids),
                 ("cand_logprob", cand_logprob)):
        _contig(t, n)
    if not (phi.dtype == psi.dtype == gate.dtype):
        raise TypeError("phi, psi and gate must share one dtype")
    V, r = phi.shape
    B, gamma, K = cand_ids.shape
    dev = cand_ids.device
    if out is None:
        out = dict(delta=torch.empty(B, gamma, K, K, dtype=torch.float32, device=dev) if with_delta else None,
                   edge=torch.empty(B, gamma, K, K, dtype=torch.float32, device=dev))
    a, l = _host_f32(alpha, gamma), _host_f32(lam, gamma)
    st = lib().ubt_edge_scores(_ptr(phi), _ptr(psi), _ptr(gate), _dtype_code(phi), V, r, _ptr(anchor), _ptr(cand_ids),
                               _ptr(cand_logprob), a, l, B, gamma, K, _ptr(out.get("delta")), _ptr(out["edge"]),
                               _stream(stream))
    _check("ubt_edge_scores", st)
    return out


def build_tree_best_first(anchor: torch.Tensor, cand_ids: torch.Tensor, edge: torch.Tensor, budget: int,
                          zeta: float = 0.0, out: dict | None = None, with_mask: bool = True, stream=None) -> dict:
    """``ubt_build_tree_best_first``: the tree grown best-first under cumulative edge scores."""
    _need_gpu(anchor, cand_ids, edge)
    for n, t in (("anchor", anchor), ("cand_ids", cand_ids), ("edge", edge)):
        _contig(t, n)
    B, gamma, K = cand_ids.shape
    if out is None:
        out = tree_outputs(B, gamma, 1, budget, cand_ids.device, with_mask)
    st = lib().ubt_build_tree_best_first(_ptr(anchor), _ptr(cand_ids), _ptr(edge), B, gamma, K, budget, float(zeta),
                                         _ptr(out["n_nodes"]), _ptr(out["token"]), _ptr(out["parent"]),
                                         _ptr(out["depth"]), _ptr(out["cand_rank"]), _ptr(out["score"]),
                                         _ptr(out.get("mask")), _stream(stream))
    _check("ubt_build_tree_best_first", st)
    return out


def tree_mask(parent: torch.Tensor, n_nodes: torch.Tensor, out: torch.Tensor | None = None,
              stream=None) -> torch.Tensor:
    """Packed ancestor mask ``[B, N, ceil(N/32)]`` (int32 view of uint32 words)."""
    _need_gpu(parent, n_nodes)
    _contig(parent, "parent")
    B, N = parent.shape
    if out is None:
        out = torch.empty(B, N, (N + 31) // 32, dtype=torch.int32, device=parent.device)
    _check("ubt_tree_mask", lib().ubt_tree_mask(_ptr(parent), _ptr(n_nodes), B, N, _ptr(out), _stream(stream)))
    return out


def draft_step_workspace(B: int, gamma: int, V: int, K: int, dtype=torch.bfloat16, device="cuda") -> torch.Tensor:
    """A zero-filled workspace for :func:`draft_step` (uint8, 256-byte aligned).  Each
    call resets the counters it uses, so one workspace serves consecutive calls on one
    stream."""
    code = UBT_BF16 if dtype == torch.bfloat16 else UBT_F32
    n = lib().ubt_draft_step_workspace_bytes(B, gamma, V, K, code)
    if n == 0:
        raise ValueError("invalid shape for ubt_draft_step")
    ws = torch.zeros(n, dtype=torch.uint8, device=device)
    if ws.data_ptr() % 256:
        raise RuntimeError("workspace is not 256-byte aligned")
    return ws


class StepTimeout(RuntimeError):
    """A bounded wait inside a one-launch ``ubt_draft_step`` ran out of time."""


def draft_step_error(workspace: torch.Tensor) -> int:
    """The error word of a :func:`draft_step` workspace (its first 4 bytes; nonzero after
    a wait inside the launch timed out).  Reads device memory, so it synchronises with the
    workspace's device."""
    return int(workspace[:4].cpu().view(torch.int32)[0].item())


def draft_step(logits: torch.Tensor, phi: torch.Tensor, psi: torch.Tensor, gate: torch.Tensor, anchor: torch.Tensor,
               alpha, lam, K: int, W: int, budget: int, zeta: float = 0.0, workspace: torch.Tensor | None = None,
               cand: dict | None = None, logq: torch.Tensor | None = None, out: dict | None = None,
               with_mask: bool = True, stream=None) -> dict:
    """The whole draft step (``topk`` then ``draft_tree``) in one library call; returns the
    candidates, ``logq`` and the tree outputs."""
    _need_gpu(logits, phi, psi, gate, anchor)
    if logits.dim() != 3 or logits.stride(2) != 1:
        raise ValueError("logits must be [B, gamma, V] with unit stride along V")
    for n, t in (("phi", phi), ("psi", psi), ("gate", gate), ("anchor", anchor)):
        _contig(t, n)
    B, gamma, V = logits.shape
    r = phi.shape[1]
    dev = logits.device
    f32 = dict(dtype=torch.float32, device=dev)
    if cand is None:
        cand = dict(cand_ids=torch.empty(B, gamma, K, dtype=torch.int32, device=dev),
                    cand_logit=torch.empty(B, gamma, K, **f32), cand_logprob=torch.empty(B, gamma, K, **f32),
                    lse=torch.empty(B, gamma, **f32))
    if logq is None:
        logq = torch.empty(B, gamma, K, K, **f32)
    if out is None:
        out = tree_outputs(B, gamma, W, budget, dev, with_mask)
    if workspace is None:
        workspace = draft_step_workspace(B, gamma, V, K, logits.dtype, dev)
    a, l = _host_f32(alpha, gamma), _host_f32(lam, gamma)
    st = lib().ubt_draft_step(_ptr(logits), _dtype_code(logits), B, gamma, V, logits.stride(0), logits.stride(1), K,
                              _ptr(phi), _ptr(psi), _ptr(gate), _dtype_code(phi), r, _ptr(anchor), a, l, W, budget,
                              float(zeta), _ptr(cand["cand_ids"]), _ptr(cand["cand_logit"]),
                              _ptr(cand.get("cand_logprob")), _ptr(cand.get("lse")), _ptr(logq),
                              _ptr(out["n_nodes"]), _ptr(out["token"]), _ptr(out["parent"]), _ptr(out["depth"]),
                              _ptr(out["cand_rank"]), _ptr(out["score"]), _ptr(out.get("mask")), _ptr(workspace),
                              workspace.numel(), _stream(stream))
    _check("ubt_draft_step", st)
    return {**cand, "logq": logq, **out}


def draft_step_noalloc(logits: torch.Tensor, phi: torch.Tensor, psi: torch.Tensor, gate: torch.Tensor,
                       anchor: torch.Tensor, alpha, lam, K: int, W: int, budget: int, zeta: float = 0.0,
                       cand: dict | None = None, logq: torch.Tensor | None = None, out: dict | None = None,
                       with_mask: bool = True, stream=None) -> dict:
    """:func:`draft_step` through ``ubt_draft_step_noalloc``: no workspace argument; the
    library's static per-device array serves the one-launch kernel.  Outputs are allocated
    here unless given (pass them to allocate nothing)."""
    _need_gpu(logits, phi, psi, gate, anchor)
    if logits.dim() != 3 or logits.stride(2) != 1:
        raise ValueError("logits must be [B, gamma, V] with unit stride along V")
    for n, t in (("phi", phi), ("psi", psi), ("gate", gate), ("anchor", anchor)):
        _contig(t, n)
    B, gamma, V = logits.shape
    r = phi.shape[1]
    dev = logits.device
    f32 = dict(dtype=torch.float32, device=dev)
    if cand is None:
        cand = dict(cand_ids=torch.empty(B, gamma, K, dtype=torch.int32, device=dev),
                    cand_logit=torch.empty(B, gamma, K, **f32), cand_logprob=torch.empty(B, gamma, K, **f32),
                    lse=torch.empty(B, gamma, **f32))
    if logq is None:
        logq = torch.empty(B, gamma, K, K, **f32)
    if out is None:
        out = tree_outputs(B, gamma, W, budget, dev, with_mask)
    a, l = _host_f32(alpha, gamma), _host_f32(lam, gamma)
    st = lib().ubt_draft_step_noalloc(_ptr(logits), _dtype_code(logits), B, gamma, V, logits.stride(0),
                                      logits.stride(1), K, _ptr(phi), _ptr(psi), _ptr(gate), _dtype_code(phi), r,
                                      _ptr(anchor), a, l, W, budget, float(zeta), _ptr(cand["cand_ids"]),
                                      _ptr(cand["cand_logit"]), _ptr(cand.get("cand_logprob")), _ptr(cand.get("lse")),
                                      _ptr(logq), _ptr(out["n_nodes"]), _ptr(out["token"]), _ptr(out["parent"]),
                                      _ptr(out["depth"]), _ptr(out["cand_rank"]), _ptr(out["score"]),
                                      _ptr(out.get("mask")), _stream(stream))
    _check("ubt_draft_step_noalloc", st)
    return {**cand, "logq": logq, **out}


def tree_attention(q: torch.Tensor, k_cache: torch.Tensor | None, v_cache: torch.Tensor | None,
                   prefix_len: torch.Tensor, k_tree: torch.Tensor, v_tree: torch.Tensor, mask: torch.Tensor,
                   n_nodes: torch.Tensor, scale: float | None = None, out: torch.Tensor | None = None,
                   lse: torch.Tensor | None = None, out_dtype=torch.bfloat16, stream=None):
    """``ubt_tree_attention``: every tree node attends to the committed context and to
    its ancestors.  q ``[B, N, H, D]`` bf16; caches ``[B, P_max, H_kv, D]`` bf16 (or None
    with no context); k_tree / v_tree ``[B, N, H_kv, D]`` bf16; mask ``[B, N, words]``
    int32 (uint32 bits); prefix_len, n_nodes int32 ``[B]``.  Returns (out, lse)."""
    _need_gpu(q, k_cache, v_cache, prefix_len, k_tree, v_tree, mask, n_nodes)
    B, N, H, D = q.shape
    Hkv = k_tree.shape[2]
    Pmax = 0 if k_cache is None else k_cache.shape[1]
    for name, t in (("q", q), ("k_tree", k_tree), ("v_tree", v_tree), ("k_cache", k_cache), ("v_cache", v_cache)):
        if t is not None:
            _contig(t, name)
            if t.dtype != torch.bfloat16:
                raise TypeError(f"{name} must be bfloat16")
    if scale is None:
        scale = D ** -0.5
    if out is None:
        out = torch.empty(B, N, H, D, dtype=out_dtype, device=q.device)
    if lse is None:
        lse = torch.empty(B, N, H, dtype=torch.float32, device=q.device)
    st = lib().ubt_tree_attention(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(prefix_len), Pmax, _ptr(k_tree),
                                  _ptr(v_tree), _ptr(mask), _ptr(n_nodes), B, N, H, Hkv, D, float(scale), _ptr(out),
                                  _dtype_code(out), _ptr(lse), _stream(stream))
    _check("ubt_tree_attention", st)
    return out, lse


def verify_accept(token: torch.Tensor, parent: torch.Tensor, n_nodes: torch.Tensor, target: torch.Tensor,
                  out: dict | None = None, stream=None) -> dict:
    """``ubt_verify_accept``: the accepted path and the bonus token of each tree."""
    _need_gpu(token, parent, n_nodes, target)
    B, N = token.shape
    if out is None:
        i32 = dict(dtype=torch.int32, device=token.device)
        out = dict(accept_len=torch.empty(B, **i32), accept_nodes=torch.empty(B, N, **i32),
                   bonus=torch.empty(B, **i32))
    st = lib().ubt_verify_accept(_ptr(token), _ptr(parent), _ptr(n_nodes), _ptr(target), B, N,
                                 _ptr(out["accept_len"]), _ptr(out["accept_nodes"]), _ptr(out["bonus"]),
                                 _stream(stream))
    _check("ubt_verify_accept", st)
    return out


def commit_kv(k_tree: torch.Tensor, v_tree: torch.Tensor, accept_nodes: torch.Tensor, accept_len: torch.Tensor,
              prefix_len: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, stream=None) -> None:
    """``ubt_commit_kv``: appends the accepted path's key/value rows to the caches and
    advances ``prefix_len`` (in place)."""
    _need_gpu(k_tree, v_tree, accept_nodes, accept_len, prefix_len, k_cache, v_cache)
    B, N, Hkv, D = k_tree.shape
    st = lib().ubt_commit_kv(_ptr(k_tree), _ptr(v_tree), _ptr(accept_nodes), _ptr(accept_len), _ptr(prefix_len),
                             _ptr(k_cache), _ptr(v_cache), B, N, Hkv, D, k_cache.shape[1], _stream(stream))
    _check("ubt_commit_kv", st)


def tree_kl_loss(logits: torch.Tensor, cand: dict, target_logits: torch.Tensor, y_star: torch.Tensor,
                 anchor: torch.Tensor, phi: torch.Tensor, psi: torch.Tensor, gate: torch.Tensor, alpha, lam,
                 T_train: float = 1.0, beta: float = 0.1, with_grad: bool = True, out: dict | None = None,
                 stream=None) -> dict:
    """``ubt_tree_kl_loss``: the renormalised-KL objective per position and its gradients.
    ``cand`` holds ``ubt_topk``'s ``cand_ids``, ``cand_logit`` and ``lse`` for ``logits``;
    ``target_logits`` has the logits' shape and dtype (unit stride along V)."""
    _need_gpu(logits, target_logits, y_star, anchor, phi, psi, gate)
    B, gamma, V = logits.shape
    K = cand["cand_ids"].shape[2]
    r = phi.shape[1]
    if logits.stride(2) != 1 or target_logits.stride(2) != 1 or target_logits.shape != logits.shape:
        raise ValueError("logits and target_logits must be [B, gamma, V] with unit stride along V")
    if target_logits.dtype != logits.dtype:
        raise TypeError("target_logits must have the logits' dtype")
    a = (ctypes.c_float * gamma)(*[float(x) for x in alpha])
    l = (ctypes.c_float * gamma)(*[float(x) for x in lam])
    if out is None:
        f32 = dict(dtype=torch.float32, device=logits.device)
        out = dict(loss=torch.empty(B, gamma, **f32), kl=torch.empty(B, gamma, **f32),
                   ce=torch.empty(B, gamma, **f32), grad_s=torch.empty(B, gamma, K, **f32),
                   grad_logits=torch.empty(B, gamma, V, **f32) if with_grad else None)
    st = lib().ubt_tree_kl_loss(_ptr(logits), _dtype_code(logits), B, gamma, V, logits.stride(0), logits.stride(1),
                                _ptr(cand["lse"]), _ptr(cand["cand_ids"]), _ptr(cand["cand_logit"]), K,
                                _ptr(target_logits), target_logits.stride(0), target_logits.stride(1), _ptr(y_star),
                                _ptr(anchor), _ptr(phi), _ptr(psi), _ptr(gate), _dtype_code(phi), r, a, l,
                                float(T_train), float(beta), _ptr(out["loss"]), _ptr(out.get("kl")),
                                _ptr(out.get("ce")), _ptr(out.get("grad_s")), _ptr(out.get("grad_logits")),
                                _stream(stream))
    _check("ubt_tree_kl_loss", st)
    return out


class DraftStep:
    """One draft step (top-K -> selector -> tree + mask) with every buffer preallocated.

    ``run(logits)`` issues the library calls on the current stream and allocates nothing,
    so it can be captured into a HIP graph.  By default it is ``ubt_topk``, then the
    selector and the search through ``ubt_draft_tree``; ``one_call=True`` makes the whole
    step one ``ubt_draft_step`` call; ``fused=False``, ``with_delta`` or ``debug`` use the
    separate ``ubt_topk``, ``ubt_bigram_scores`` and ``ubt_build_tree`` calls."""

    def __init__(self, B: int, gamma: int, V: int, K: int, W: int, budget: int, phi: torch.Tensor,
                 psi: torch.Tensor, gate: torch.Tensor, anchor: torch.Tensor, alpha, lam, zeta: float = 0.0,
                 with_delta: bool = False, debug: bool = False, fused: bool = True, one_call: bool = False,
                 logit_dtype=torch.bfloat16):
        dev = phi.device
        self.shape = (B, gamma, V, K, W, budget)
        self.phi, self.psi, self.gate, self.anchor = phi, psi, gate, anchor
        self.alpha, self.lam, self.zeta = alpha, lam, zeta
        self.W, self.budget, self.K = W, budget, K
        f32 = dict(dtype=torch.float32, device=dev)
        self.cand = dict(cand_ids=torch.empty(B, gamma, K, dtype=torch.int32, device=dev),
                         cand_logit=torch.empty(B, gamma, K, **f32), cand_logprob=torch.empty(B, gamma, K, **f32),
                         lse=torch.empty(B, gamma, **f32))
        self.sel = dict(delta=torch.empty(B, gamma, K, K, **f32) if with_delta else None,
                        logq=torch.empty(B, gamma, K, K, **f32))
        self.tree = tree_outputs(B, gamma, W, budget, dev, True, debug)
        self.fused = fused and not with_delta and not debug
        self.one_call = one_call and self.fused
        self.workspace = draft_step_workspace(B, gamma, V, K, logit_dtype, dev) if self.one_call else None
        self.logit_dtype_code = UBT_BF16 if logit_dtype == torch.bfloat16 else UBT_F32

    def outputs(self) -> dict:
        """The step's output tensors (candidates, selector scores, tree)."""
        return {**self.cand, **self.sel, **self.tree}

    def check(self) -> None:
        """Synchronises the device and raises :class:`StepTimeout` if a bounded wait inside
        an earlier one-launch call ran out of time (the workspace's error word is set; the
        affected trees carry ``n_nodes == 0``).  The workspace is then zero-filled again, so
        later calls start clean.  Does nothing for the multi-launch paths."""
        if self.workspace is None:
            return
        torch.cuda.synchronize(self.workspace.device)
        if draft_step_error(self.workspace):
            self.workspace.zero_()
            torch.cuda.synchronize(self.workspace.device)
            raise StepTimeout("ubt_draft_step: a wait inside the launch timed out; outputs of that call are "
                              "unspecified (the workspace has been cleared)")

    def run(self, logits: torch.Tensor, stream=None) -> dict:
        if self.one_call:
            draft_step(logits, self.phi, self.psi, self.gate, self.anchor, self.alpha, self.lam, self.K, self.W,
                       self.budget, self.zeta, self.workspace, self.cand, self.sel["logq"], self.tree, stream=stream)
            return {**self.cand, **self.sel, **self.tree}
        topk(logits, self.K, self.cand, stream=stream)
        if self.fused:
            draft_tree(self.phi, self.psi, self.gate, self.anchor, self.cand["cand_ids"], self.cand["cand_logit"],
                       self.alpha, self.lam, self.W, self.budget, self.zeta, self.sel["logq"], self.tree,
                       stream=stream)
            return {**self.cand, **self.sel, **self.tree}
        bigram_scores(self.phi, self.psi, self.gate, self.anchor, self.cand["cand_ids"], self.cand["cand_logit"],
                      self.alpha, self.lam, self.sel, stream=stream)
        build_tree(self.anchor, self.cand["cand_ids"], self.sel["logq"], self.W, self.budget, self.zeta, self.tree,
                   stream=stream)
        return {**self.cand, **self.sel, **self.tree}


def bf16_tensor_from_bits(bits, device="cuda") -> torch.Tensor:
    """A bf16 tensor holding the given uint16 bit patterns (numpy array)."""
    import numpy as np

    a = np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)
    return torch.from_numpy(a).to(device).view(torch.bfloat16)
