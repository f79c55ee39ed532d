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
           "noalloc.hip", "uncertainty.hip", "peaks.hip",
           # the persistent kernel's instantiations, one unit per rank size and decoding mode
           "persist_greedy_r128.hip", "persist_greedy_r256.hip", "persist_sampled_r128.hip",
           "persist_sampled_r256.hip"]
# the test build libdels_stress.so recompiles the units that include the persistent kernel with
# DLS_STRESS_DELAYS (pauses before every hand-off publish) and reuses every other object
STRESS_LIB = os.path.join(PKG, "libdels_stress.so")
STRESS_UNITS = ["draft_persistent.hip", "persist_greedy_r128.hip", "persist_greedy_r256.hip",
                "persist_sampled_r128.hip", "persist_sampled_r256.hip"]
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


def build(verbose: bool = False, stress: bool = True) -> str:
    """Compile every source and link libdels.so; with `stress`, also the test build
    libdels_stress.so."""
    os.makedirs(os.path.join(OBJ_DIR, "stress"), exist_ok=True)

    def compile_one(job):
        src, extra, sub = job
        obj = os.path.join(OBJ_DIR, sub, src + ".o")
        out = _run([HIPCC, *FLAGS, *extra, "-c", os.path.join(HERE, src), "-o", obj])
        if verbose and out.strip():
            print(out)
        return obj

    jobs = [(src, [], "") for src in SOURCES]
    if stress:
        jobs += [(src, ["-DDLS_STRESS_DELAYS"], "stress") for src in STRESS_UNITS]
    with ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        objs = list(ex.map(compile_one, jobs))
    plain = objs[:len(SOURCES)]
    _link(plain, LIB)
    if stress:
        stressed = dict(zip(STRESS_UNITS, objs[len(SOURCES):]))
        _link([stressed.get(src, o) for src, o in zip(SOURCES, plain)], STRESS_LIB)
    return LIB


def _link(objs, lib):
    tmp = lib + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", "--offload-arch=gfx950", *objs, "-o", tmp])
    os.replace(tmp, lib)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
