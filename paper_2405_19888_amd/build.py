"""Build libparrot_attn.so in-tree with hipcc for gfx950.

Usage: python -m paper_2405_19888_amd.build   (or __graft_entry__.build()).
Each source compiles to an object under _build/ in parallel, then one shared
library is linked next to this file.  The library is always rebuilt.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(ROOT, "_build")
LIB_NAME = "libparrot_attn.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)

SOURCES = ["api.hip", "partials.hip", "prefill.hip", "merge.hip", "ceiling.hip",
           "context_store.cpp"]

# Packed fp32 arithmetic is disabled: the kernels write only scalar float code.
HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]


# Per-source flags.  The prefill kernel's arithmetic never depends on NaN
# semantics (masked logits are -inf by selection), so it lets the compiler drop
# the NaN-quieting of every max.
SOURCE_FLAGS = {"prefill.hip": ["-fno-honor-nans"]}


def _hipcc() -> str:
    env = os.environ.get("HIPCC")
    if env:
        return env
    for cand in ("/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines()
                    if "packed-fp32-ops" not in l and l.strip())
    if p.returncode != 0:
        raise RuntimeError(f"command failed ({p.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False, extra_flags=(), out_path: str = LIB_PATH,
          build_dir: str = BUILD) -> str:
    """Compile every source and link ``out_path``; ``extra_flags`` go to hipcc."""
    hipcc = _hipcc()
    os.makedirs(build_dir, exist_ok=True)
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        cmds.append([hipcc, *HIP_FLAGS, *SOURCE_FLAGS.get(src, []), *extra_flags, "-I", INCLUDE,
                     "-I", CSRC, "-c", os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as ex:
        for out in ex.map(_run, cmds):
            if verbose and out:
                print(out)
    tmp = out_path + ".tmp"
    _run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, out_path)
    if verbose:
        print(f"built {out_path}")
    return out_path


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
