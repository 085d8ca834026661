"""Build step of libscale.so: hipcc for gfx950, in-tree (the library ships next to this file)."""
from __future__ import annotations

import os
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
LIB_PATH = os.path.join(HERE, "libscale.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

KERNEL_SOURCES = ["rep_keys.hip", "select.hip", "select_tokens.hip", "sparse_attention.hip", "work_list.hip", "cluster.hip",
                  "static_select.hip"]
HOST_SOURCES = ["scale_api.cpp"]

# Packed fp32 VALU instructions are kept out of the generated code on purpose.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]

# Per-source flags. The attention kernel runs its items in a loop inside each persistent
# work-group; LLVM's machine loop-invariant code motion hoists the kernel's constants (LDS offsets,
# small integers, zero vectors) out of that loop into about ten VGPRs held for the whole kernel,
# which pushes the tile loop's prefetch registers into waits on their own loads.
SOURCE_FLAGS = {"sparse_attention.hip": ["-mllvm", "-disable-machine-licm"]}


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{msgs}")
    if verbose and msgs.strip():
        print(msgs)


def build(verbose: bool = False) -> str:
    """Compile every source (always recompiles) and link libscale.so."""
    with tempfile.TemporaryDirectory(prefix="scale_build_") as tmp:
        jobs = []
        for src in KERNEL_SOURCES + HOST_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            lang = ["-x", "hip"] if src.endswith(".cpp") else []
            jobs.append(([HIPCC, *HIP_FLAGS, *SOURCE_FLAGS.get(src, []), "-I", INCLUDE, "-c", *lang,
                          os.path.join(CSRC, src), "-o", obj], obj))
        with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
            list(ex.map(lambda j: _run(j[0], verbose), jobs))
        out = LIB_PATH + ".tmp"
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *[o for _, o in jobs], "-o", out], verbose)
        os.replace(out, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
