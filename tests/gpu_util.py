"""Helpers for the GPU parity tests: move generator output to the device, run the HIP
path through the C ABI binding, and bring results back as numpy."""
from __future__ import annotations

import sys

import numpy as np
import torch

import paper_2609_39972_amd as ubt
import synth

DEV = torch.device("cuda:0")


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def dev_values(a: np.ndarray) -> torch.Tensor:
    """uint16 arrays are bf16 bit patterns; float32 arrays stay float32."""
    if a.dtype == np.uint16:
        return ubt.bf16_tensor_from_bits(a, DEV)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def dev_i32(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(DEV)


def to_np(out: dict) -> dict:
    res = {}
    for k, v in out.items():
        if v is None:
            continue
        a = v.detach().cpu().numpy()
        if k == "mask":
            a = a.view(np.uint32)
        res[k] = a
    return res


def run_pipeline(w: synth.Workload, d: dict, W: int | None = None, debug: bool = True, logits_t=None) -> dict:
    """The three library calls on workload `w` with generator inputs `d`."""
    W = w.W if W is None else W
    logits = dev_values(d["logits"]) if logits_t is None else logits_t
    step = ubt.DraftStep(w.B, w.gamma, w.V, w.K, W, w.budget, dev_values(d["phi"]), dev_values(d["psi"]),
                         dev_values(d["gate"]), dev_i32(d["anchor"]), d["alpha"], d["lam"], w.zeta,
                         with_delta=True, debug=debug)
    out = step.run(logits)
    torch.cuda.synchronize()
    return to_np(out)
