"""Build libdels.so (gfx950) in-tree: hipcc compiles each source, then links a shared library.

Usage: python -m paper_2607_07409_amd.csrc.build   (or build() from the package entry point)
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
OBJ_DIR = os.path.join(ROOT, "_build", "dels")
LIB = os.path.join(PKG, "libdels.so")
SOURCES = ["api.cpp", "combine.hip", "draft.hip", "accept.hip", "prepare.hip", "draft_persistent.hip", "prior.hip",
           "noalloc.hip", "uncertainty.hip",
           # the persistent kernel's instantiations, one unit per rank size and decoding mode
           "persist_greedy_r128.hip", "persist_greedy_r256.hip", "persist_sampled_r128.hip",
           "persist_sampled_r256.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950", "-Wall", "-Wno-unused-function",
         # no packed fp32 arithmetic in any generated code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         # LDS atomics stay single instructions: the default rewrite into a scalar loop over the
         # active lanes costs about a microsecond per wave in the persistent kernel's key merge
         "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
         "-I", os.path.join(ROOT, "include")]


def _run(cmd):
    p = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (p.stdout + p.stderr).splitlines() if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        raise RuntimeError(f"command failed ({p.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False) -> str:
    os.makedirs(OBJ_DIR, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(OBJ_DIR, src + ".o")
        out = _run([HIPCC, *FLAGS, "-c", os.path.join(HERE, src), "-o", obj])
        if verbose and out.strip():
            print(out)
        return obj

    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
