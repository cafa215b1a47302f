"""Builds ``libubt.so`` (gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libubt.so")
SOURCES = ["api.cpp", "topk.hip", "bigram.hip", "tree.hip", "step.hip", "bestfirst.hip", "lmhead.hip", "verify.hip", "loss.hip"]
ARCH = "gfx950"

FLAGS_COMPILE = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # Keep the compiler from forming packed fp32 instructions.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-result",
]


def sources() -> list[str]:
    return [os.path.join(CSRC, s) for s in SOURCES]


def _run(cmd: list[str]) -> str:
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}): {' '.join(cmd)}\n{err}")
    return err


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compiles every source to an object (in parallel, under ``_build/``), then links
    ``libubt.so``.  Always recompiles."""
    from concurrent.futures import ThreadPoolExecutor

    objdir = os.path.join(ROOT, "_build", "ubt")
    os.makedirs(objdir, exist_ok=True)
    tag = f".{os.getpid()}"
    objs, cmds = [], []
    for src in sources():
        obj = os.path.join(objdir, os.path.basename(src) + tag + ".o")
        objs.append(obj)
        cmds.append(["hipcc", *FLAGS_COMPILE, f"-I{INCLUDE}", f"-I{CSRC}", "-x", "hip", "-c", src, "-o", obj])
    if verbose:
        for c in cmds:
            print(" ".join(c), flush=True)
    n = jobs or max(1, min(len(cmds), os.cpu_count() or 1, 8))
    try:
        with ThreadPoolExecutor(n) as ex:
            for err in ex.map(_run, cmds):
                if err.strip() and verbose:
                    print(err)
        tmp = LIB + f".tmp{os.getpid()}"
        link = ["hipcc", f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
        if verbose:
            print(" ".join(link), flush=True)
        _run(link)
        os.replace(tmp, LIB)
    finally:
        for o in objs:
            if os.path.exists(o):
                os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
