"""Build the HIP library libwm.so for gfx950 with hipcc (in-tree)."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCES = ["csrc/wm_api.hip", "csrc/wm_kernels.hip", "csrc/wm_text.hip"]
HOST_SOURCES = ["csrc/wm_pack.cpp"]      # plain C++ (the tests also build it alone)
LIB = os.path.join(HERE, "libwm.so")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # keep float code off the packed-fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # let the fully unrolled item streams of the rollout kernels unroll (their
    # register rings and operand arrays need compile-time indices)
    "-mllvm", "-pragma-unroll-threshold=1000000",
]


def build(verbose: bool = False) -> str:
    """Compile every HIP source (in parallel) and link libwm.so next to this
    file; returns its path."""
    from concurrent.futures import ThreadPoolExecutor
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    noise = "is not a recognized feature for this target"
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    cflags = [f for f in FLAGS if f != "-shared"]

    def compile_one(src):
        obj = os.path.join(objdir, os.path.basename(src) + ".o")
        if src in HOST_SOURCES:
            cmd = ["g++", "-std=c++17", "-O2", "-fPIC", "-c", os.path.join(HERE, src), "-o", obj]
        else:
            cmd = [hipcc, *cflags, "-c", os.path.join(HERE, src), "-o", obj]
        res = subprocess.run(cmd, capture_output=True, text=True)
        return obj, res

    srcs = SOURCES + HOST_SOURCES
    with ThreadPoolExecutor(max_workers=len(srcs)) as ex:
        results = list(ex.map(compile_one, srcs))
    objs = []
    for (obj, res), src in zip(results, srcs):
        err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
        if res.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src} ({res.returncode}):\n{err}")
        if verbose and err.strip():
            print(err, file=sys.stderr)
        objs.append(obj)
    tmp = LIB + ".tmp"
    res = subprocess.run([hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp],
                         capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed ({res.returncode}):\n{res.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
